"""Python binding of libvsa2 (the gfx950 routed sparse-attention library).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  The functions named vsa2_* mirror the C-ABI in include/vsa2.h one
to one and take raw device pointers (ints) and a hipStream_t (int); the
lower-case helpers below them take torch tensors, check dtypes/shapes,
allocate outputs and workspaces with torch (device memory only) and call the
C-ABI on torch's current stream.

The library must have been built (paper_2609_32882_amd/build.py): the first
call into it loads libvsa2.so and raises ImportError when it is missing;
there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvsa2.so")

VSA2_OK = 0
STATUS_NAMES = {0: "VSA2_OK", 1: "VSA2_ERR_NULL", 2: "VSA2_ERR_SHAPE", 3: "VSA2_ERR_DTYPE",
                4: "VSA2_ERR_SELECT", 5: "VSA2_ERR_CAPACITY", 6: "VSA2_ERR_ALIGN",
                7: "VSA2_ERR_WORKSPACE", 8: "VSA2_ERR_HIP", 9: "VSA2_ERR_UNSUPPORTED"}
VSA2_F32, VSA2_BF16 = 0, 1
VSA2_SEL_TOPK, VSA2_SEL_MASS, VSA2_SEL_SEQ_TOPK = 0, 1, 2

# Every symbol include/vsa2.h declares.
EXPORTS = ("vsa2_status_str", "vsa2_pool", "vsa2_route_capacity", "vsa2_route_workspace",
           "vsa2_route", "vsa2_attn_workspace", "vsa2_attn_fwd", "vsa2_attn_fwd_noalloc", "vsa2_attn_bwd",
           "vsa2_attn_bwd_prep", "vsa2_attn_bwd_dkdv", "vsa2_attn_bwd_dq",
           "vsa2_coarse_fwd", "vsa2_coarse_bwd", "vsa2_gate_merge", "vsa2_gate_merge_bwd",
           "vsa2_joint_capacity", "vsa2_joint_workspace", "vsa2_joint_lists", "vsa2_unpool_add",
           "vsa2_mfma_peak_probe", "vsa2_dq_atomic_probe")


class vsa2_problem(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("batch", "heads_q", "heads_kv", "head_dim", "T", "H", "W",
                 "Bt", "Bh", "Bw", "Rt", "Rh", "Rw", "dtype", "text_len")]


class vsa2_select(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("k", ctypes.c_int32), ("mass", ctypes.c_float),
                ("cap", ctypes.c_int32)]


class Vsa2Error(RuntimeError):
    def __init__(self, fn, status):
        super().__init__("%s failed: %s (%s)" % (fn, STATUS_NAMES.get(status, status),
                                                 _lib().vsa2_status_str(status).decode()))
        self.status = status


_L = None


def _lib():
    global _L
    if _L is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libvsa2.so is not built; run paper_2609_32882_amd/build.py "
                              "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        pp, ps = ctypes.POINTER(vsa2_problem), ctypes.POINTER(vsa2_select)
        L.vsa2_status_str.argtypes = [ctypes.c_int]
        L.vsa2_status_str.restype = ctypes.c_char_p
        L.vsa2_pool.argtypes = [pp, i32, P, i32, i32, i32, P, P]
        L.vsa2_route_capacity.argtypes = [pp, ps, ctypes.POINTER(i64)]
        L.vsa2_route_workspace.argtypes = [pp, ps, ctypes.POINTER(sz)]
        L.vsa2_route.argtypes = [pp, ps, P, P, P, P, i64, P, P, P, P, sz, P]
        L.vsa2_attn_workspace.argtypes = [pp, i32, ctypes.POINTER(sz)]
        L.vsa2_attn_fwd.argtypes = [pp, P, P, P, P, P, i64, P, P, P, P, sz, P]
        L.vsa2_attn_fwd_noalloc.argtypes = [pp, P, P, P, P, P, i64, P, P, P, P]
        L.vsa2_attn_bwd.argtypes = [pp, P, P, P, P, P, P, P, P, P, P, P, i64, P, P, P, P, sz, P]
        L.vsa2_attn_bwd_prep.argtypes = [pp, P, P, P, P, P, P, P, P, sz, P]
        L.vsa2_attn_bwd_dkdv.argtypes = [pp, P, P, P, P, P, P, i64, P, P, P, sz, P]
        L.vsa2_attn_bwd_dq.argtypes = [pp, P, P, P, P, P, P, i64, P, P, sz, P]
        L.vsa2_coarse_fwd.argtypes = [pp, P, P, P, P, P, P]
        L.vsa2_coarse_bwd.argtypes = [pp, P, P, P, P, P, P, P, P, sz, P]
        L.vsa2_gate_merge.argtypes = [pp, P, P, P, P, P]
        L.vsa2_gate_merge_bwd.argtypes = [pp, P, P, P, P, P, P]
        L.vsa2_unpool_add.argtypes = [pp, i32, P, i32, i32, i32, P, P]
        L.vsa2_joint_capacity.argtypes = [pp, ps, ctypes.POINTER(i64)]
        L.vsa2_joint_workspace.argtypes = [pp, ctypes.POINTER(sz)]
        L.vsa2_joint_lists.argtypes = [pp, P, P, i64, P, P, i64, P, P, P, sz, P]
        L.vsa2_mfma_peak_probe.argtypes = [i32, P, ctypes.POINTER(i64), P]
        L.vsa2_dq_atomic_probe.argtypes = [pp, P, P, i64, P, P]
        for n in EXPORTS[1:]:
            getattr(L, n).restype = ctypes.c_int
        _L = L
    return _L


def lib():
    """The loaded ctypes library (raises if libvsa2.so is missing)."""
    return _lib()


def _ref(x):
    return None if x is None else ctypes.byref(x)


def _check(fn, status):
    if status != VSA2_OK:
        raise Vsa2Error(fn, status)


# --------------------------------------------------------------------------
# C-ABI mirror (raw pointers)
# --------------------------------------------------------------------------

def vsa2_status_str(status: int) -> str:
    return _lib().vsa2_status_str(status).decode()


def vsa2_pool(p, heads, x, Pt, Ph, Pw, out, stream=0):
    return _lib().vsa2_pool(_ref(p), heads, x, Pt, Ph, Pw, out, stream)


def vsa2_route_capacity(p, s):
    n = ctypes.c_int64(0)
    st = _lib().vsa2_route_capacity(_ref(p), _ref(s), ctypes.byref(n))
    return st, n.value


def vsa2_route_workspace(p, s):
    n = ctypes.c_size_t(0)
    st = _lib().vsa2_route_workspace(_ref(p), _ref(s), ctypes.byref(n))
    return st, n.value


def vsa2_route(p, s, q_r, k_r, row_ptr, col_idx, col_cap, kv_ptr, kv_idx, block_scores, ws,
               ws_bytes, stream=0):
    return _lib().vsa2_route(_ref(p), _ref(s), q_r, k_r, row_ptr, col_idx, col_cap,
                             kv_ptr, kv_idx, block_scores, ws, ws_bytes, stream)


def vsa2_attn_workspace(p, pass_):
    n = ctypes.c_size_t(0)
    st = _lib().vsa2_attn_workspace(_ref(p), pass_, ctypes.byref(n))
    return st, n.value


def vsa2_attn_fwd(p, q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, ws, ws_bytes, stream=0):
    return _lib().vsa2_attn_fwd(_ref(p), q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, ws,
                                ws_bytes, stream)


def vsa2_attn_fwd_noalloc(p, q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, stream=0):
    return _lib().vsa2_attn_fwd_noalloc(_ref(p), q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, stream)


def vsa2_attn_bwd(p, q, k, v, o, lse, o_lo, dout, row_ptr, col_idx, kv_ptr, kv_idx, col_cap, dq,
                  dk, dv, ws, ws_bytes, stream=0):
    return _lib().vsa2_attn_bwd(_ref(p), q, k, v, o, lse, o_lo, dout, row_ptr, col_idx, kv_ptr,
                                kv_idx, col_cap, dq, dk, dv, ws, ws_bytes, stream)


def vsa2_attn_bwd_prep(p, q, k, v, o, lse, o_lo, dout, ws, ws_bytes, stream=0):
    return _lib().vsa2_attn_bwd_prep(_ref(p), q, k, v, o, lse, o_lo, dout, ws, ws_bytes, stream)


def vsa2_attn_bwd_dkdv(p, q, k, v, dout, kv_ptr, kv_idx, col_cap, dk, dv, ws, ws_bytes, stream=0):
    return _lib().vsa2_attn_bwd_dkdv(_ref(p), q, k, v, dout, kv_ptr, kv_idx, col_cap, dk, dv, ws,
                                     ws_bytes, stream)


def vsa2_attn_bwd_dq(p, q, k, v, dout, row_ptr, col_idx, col_cap, dq, ws, ws_bytes, stream=0):
    return _lib().vsa2_attn_bwd_dq(_ref(p), q, k, v, dout, row_ptr, col_idx, col_cap, dq, ws,
                                   ws_bytes, stream)


def vsa2_coarse_fwd(p, q_c, k_c, v_c, o_c, lse_c, stream=0):
    return _lib().vsa2_coarse_fwd(_ref(p), q_c, k_c, v_c, o_c, lse_c, stream)


def vsa2_coarse_bwd(p, q_c, k_c, v_c, do_c, dq_c, dk_c, dv_c, ws, ws_bytes, stream=0):
    return _lib().vsa2_coarse_bwd(_ref(p), q_c, k_c, v_c, do_c, dq_c, dk_c, dv_c, ws, ws_bytes, stream)


def vsa2_gate_merge(p, gate, o_c, o_f, out, stream=0):
    return _lib().vsa2_gate_merge(_ref(p), gate, o_c, o_f, out, stream)


def vsa2_gate_merge_bwd(p, gate, o_c, dout, do_c, dgate, stream=0):
    return _lib().vsa2_gate_merge_bwd(_ref(p), gate, o_c, dout, do_c, dgate, stream)


def vsa2_unpool_add(p, heads, dx_c, Pt, Ph, Pw, dx, stream=0):
    return _lib().vsa2_unpool_add(_ref(p), heads, dx_c, Pt, Ph, Pw, dx, stream)


def vsa2_dq_atomic_probe(p, kv_ptr, kv_idx, col_cap, acc, stream=0):
    return _lib().vsa2_dq_atomic_probe(_ref(p), kv_ptr, kv_idx, col_cap, acc, stream)


def vsa2_mfma_peak_probe(iters, sink, stream=0):
    """Launch the dense MFMA rate probe; returns (status, flops of the launch)."""
    f = ctypes.c_int64(0)
    st = _lib().vsa2_mfma_peak_probe(iters, sink, ctypes.byref(f), stream)
    return st, f.value


def vsa2_joint_capacity(p, s):
    n = ctypes.c_int64(0)
    st = _lib().vsa2_joint_capacity(_ref(p), _ref(s), ctypes.byref(n))
    return st, n.value


def vsa2_joint_workspace(p):
    n = ctypes.c_size_t(0)
    st = _lib().vsa2_joint_workspace(_ref(p), ctypes.byref(n))
    return st, n.value


def vsa2_joint_lists(p, row_ptr, col_idx, col_cap, j_row_ptr, j_col_idx, j_cap, j_kv_ptr, j_kv_idx, ws,
                     ws_bytes, stream=0):
    return _lib().vsa2_joint_lists(_ref(p), row_ptr, col_idx, col_cap, j_row_ptr, j_col_idx, j_cap,
                                   j_kv_ptr, j_kv_idx, ws, ws_bytes, stream)


# --------------------------------------------------------------------------
# torch-tensor helpers (device memory + streams only)
# --------------------------------------------------------------------------

def make_problem(batch, heads_q, heads_kv, head_dim, T, H, W, Bt=4, Bh=4, Bw=4, Rt=2, Rh=2, Rw=2,
                 dtype=VSA2_BF16, text_len=0) -> vsa2_problem:
    return vsa2_problem(batch, heads_q, heads_kv, head_dim, T, H, W, Bt, Bh, Bw, Rt, Rh, Rw, dtype,
                        text_len)


def problem_from(obj) -> vsa2_problem:
    """vsa2_problem from any object with the same field names."""
    if isinstance(obj, vsa2_problem):
        return obj
    return make_problem(obj.batch, obj.heads_q, obj.heads_kv, obj.head_dim, obj.T, obj.H, obj.W,
                        obj.Bt, obj.Bh, obj.Bw, obj.Rt, obj.Rh, obj.Rw, obj.dtype,
                        getattr(obj, "text_len", 0))


def select_from(obj) -> vsa2_select:
    if isinstance(obj, vsa2_select):
        return obj
    return vsa2_select(int(obj.mode), int(obj.k), float(obj.mass), int(obj.cap))


def _torch():
    import torch
    return torch


def _stream():
    return _torch().cuda.current_stream().cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


def _dims(p):
    B = p.Bt * p.Bh * p.Bw
    # an axis that is not a multiple of its cube size is padded up to one
    N = (-(-p.T // p.Bt)) * (-(-p.H // p.Bh)) * (-(-p.W // p.Bw))
    G = (p.Bt // p.Rt) * (p.Bh // p.Rh) * (p.Bw // p.Rw)
    return N, B, G


def _joint(p):
    """(blocks, tokens) of one (batch, head) sequence: the video cubes and
    then the text blocks (p.text_len > 0), padding included."""
    N, B, _ = _dims(p)
    Nj = N + (-(-p.text_len // B))
    return Nj, Nj * B


def _tdtype(p):
    torch = _torch()
    return torch.bfloat16 if p.dtype == VSA2_BF16 else torch.float32


def _expect(t, shape, dtype, name):
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous() or not t.is_cuda:
        raise ValueError("%s: expected contiguous %s %s on the GPU, got %s %s" %
                         (name, dtype, tuple(shape), t.dtype, tuple(t.shape)))


def pool(p, x, P, out=None):
    """MeanPool of x [batch, heads, L, D] over sub-cubes P = (Pt, Ph, Pw)
    (the video part of joint video + text sequences)."""
    p = problem_from(p)
    N, B, _ = _dims(p)
    Gp = (p.Bt // P[0]) * (p.Bh // P[1]) * (p.Bw // P[2])
    heads = x.shape[1]
    _expect(x, (p.batch, heads, _joint(p)[1], p.head_dim), _tdtype(p), "x")
    if out is None:
        out = _torch().empty((p.batch, heads, N * Gp, p.head_dim), dtype=x.dtype, device=x.device)
    _check("vsa2_pool", vsa2_pool(p, heads, x.data_ptr(), P[0], P[1], P[2], out.data_ptr(), _stream()))
    return out


def route(p, s, q_r, k_r, with_csc=True, with_scores=False):
    """Router + selection.  Returns dict(row_ptr, col_idx, kv_ptr, kv_idx,
    scores, col_cap); col_idx/kv_idx are sized to the capacity, the live
    prefix is row_ptr[-1]."""
    torch = _torch()
    p, s = problem_from(p), select_from(s)
    N, B, G = _dims(p)
    dev = q_r.device
    _expect(q_r, (p.batch, p.heads_q, N * G, p.head_dim), _tdtype(p), "q_r")
    _expect(k_r, (p.batch, p.heads_kv, N * G, p.head_dim), _tdtype(p), "k_r")
    st, cap = vsa2_route_capacity(p, s)
    _check("vsa2_route_capacity", st)
    st, wsb = vsa2_route_workspace(p, s)
    _check("vsa2_route_workspace", st)
    i32 = torch.int32
    row_ptr = torch.empty(p.batch * p.heads_q * N + 1, dtype=i32, device=dev)
    col_idx = torch.empty(max(cap, 1), dtype=i32, device=dev)
    kv_ptr = torch.empty(p.batch * p.heads_kv * N + 1, dtype=i32, device=dev) if with_csc else None
    kv_idx = torch.empty(max(cap, 1), dtype=i32, device=dev) if with_csc else None
    scores = torch.empty((p.batch, p.heads_q, N, N), dtype=torch.float32, device=dev) \
        if with_scores else None
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    _check("vsa2_route", vsa2_route(p, s, q_r.data_ptr(), k_r.data_ptr(), row_ptr.data_ptr(),
                                    col_idx.data_ptr(), cap, _ptr(kv_ptr), _ptr(kv_idx),
                                    _ptr(scores), ws.data_ptr(), wsb, _stream()))
    return dict(row_ptr=row_ptr, col_idx=col_idx, kv_ptr=kv_ptr, kv_idx=kv_idx, scores=scores,
                col_cap=cap, ws=ws)


def attn_fwd(p, q, k, v, row_ptr, col_idx, col_cap=None, o=None, lse=None, training=False,
             o_lo=None):
    """Returns (o, lse); with training=True (or an o_lo buffer given) also
    o_lo, the rounding remainder of O that attn_bwd needs: (o, lse, o_lo).
    With text tokens the tensors are joint sequences and the lists joint
    lists."""
    torch = _torch()
    p = problem_from(p)
    L = _joint(p)[1]
    dt = _tdtype(p)
    _expect(q, (p.batch, p.heads_q, L, p.head_dim), dt, "q")
    _expect(k, (p.batch, p.heads_kv, L, p.head_dim), dt, "k")
    _expect(v, (p.batch, p.heads_kv, L, p.head_dim), dt, "v")
    if o is None:
        o = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((p.batch, p.heads_q, L), dtype=torch.float32, device=q.device)
    cap = col_idx.numel() if col_cap is None else col_cap
    st, wsb = vsa2_attn_workspace(p, 0)
    _check("vsa2_attn_workspace", st)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    keep = training or o_lo is not None
    if keep and o_lo is None:
        o_lo = torch.empty_like(q)
    _check("vsa2_attn_fwd", vsa2_attn_fwd(p, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                          row_ptr.data_ptr(), col_idx.data_ptr(), cap,
                                          o.data_ptr(), lse.data_ptr(), _ptr(o_lo),
                                          ws.data_ptr(), wsb, _stream()))
    return (o, lse, o_lo) if keep else (o, lse)


def attn_bwd(p, q, k, v, o, lse, do, row_ptr, col_idx, kv_ptr, kv_idx, col_cap=None,
             dq=None, dk=None, dv=None, o_lo=None):
    """dQ, dK, dV.  o_lo is the forward's remainder (attn_fwd(..., training=True));
    the library requires it (without it the call fails with VSA2_ERR_NULL)."""
    torch = _torch()
    p = problem_from(p)
    L = _joint(p)[1]
    dt = _tdtype(p)
    for t, hh, nm in ((q, p.heads_q, "q"), (k, p.heads_kv, "k"), (v, p.heads_kv, "v"),
                      (o, p.heads_q, "o"), (do, p.heads_q, "do")):
        _expect(t, (p.batch, hh, L, p.head_dim), dt, nm)
    _expect(lse, (p.batch, p.heads_q, L), torch.float32, "lse")
    if o_lo is not None:
        _expect(o_lo, (p.batch, p.heads_q, L, p.head_dim), dt, "o_lo")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    cap = col_idx.numel() if col_cap is None else col_cap
    st, wsb = vsa2_attn_workspace(p, 1)
    _check("vsa2_attn_workspace", st)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    _check("vsa2_attn_bwd", vsa2_attn_bwd(p, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                          lse.data_ptr(), _ptr(o_lo), do.data_ptr(), row_ptr.data_ptr(),
                                          col_idx.data_ptr(), kv_ptr.data_ptr(), kv_idx.data_ptr(),
                                          cap, dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                          ws.data_ptr(), wsb, _stream()))
    return dq, dk, dv


def attn_bwd_staged(p, q, k, v, o, lse, do, row_ptr, col_idx, kv_ptr, kv_idx, col_cap=None,
                    dq=None, dk=None, dv=None, o_lo=None, marks=None):
    """The backward as its three C-ABI stages (prep, dK/dV, dQ) on the current
    stream; same results as attn_bwd.  `marks`, if given, is a list of four
    torch.cuda.Event recorded before the first stage and after each one."""
    torch = _torch()
    p = problem_from(p)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    cap = col_idx.numel() if col_cap is None else col_cap
    st, wsb = vsa2_attn_workspace(p, 1)
    _check("vsa2_attn_workspace", st)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    s = _stream()
    if marks:
        marks[0].record()
    _check("vsa2_attn_bwd_prep", vsa2_attn_bwd_prep(p, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                    o.data_ptr(), lse.data_ptr(), _ptr(o_lo),
                                                    do.data_ptr(), ws.data_ptr(), wsb, s))
    if marks:
        marks[1].record()
    _check("vsa2_attn_bwd_dkdv", vsa2_attn_bwd_dkdv(p, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                    do.data_ptr(), kv_ptr.data_ptr(),
                                                    kv_idx.data_ptr(), cap, dk.data_ptr(),
                                                    dv.data_ptr(), ws.data_ptr(), wsb, s))
    if marks:
        marks[2].record()
    _check("vsa2_attn_bwd_dq", vsa2_attn_bwd_dq(p, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                do.data_ptr(), row_ptr.data_ptr(), col_idx.data_ptr(),
                                                cap, dq.data_ptr(), ws.data_ptr(), wsb, s))
    if marks:
        marks[3].record()
    return dq, dk, dv


def coarse_fwd(p, q_c, k_c, v_c):
    """O_c_hat [b, Hq, N, D] and LSE [b, Hq, N] of the coarse branch."""
    torch = _torch()
    p = problem_from(p)
    N, _, _ = _dims(p)
    o_c = torch.empty((p.batch, p.heads_q, N, p.head_dim), dtype=q_c.dtype, device=q_c.device)
    lse = torch.empty((p.batch, p.heads_q, N), dtype=torch.float32, device=q_c.device)
    _check("vsa2_coarse_fwd", vsa2_coarse_fwd(p, q_c.data_ptr(), k_c.data_ptr(), v_c.data_ptr(),
                                              o_c.data_ptr(), lse.data_ptr(), _stream()))
    return o_c, lse


def coarse_bwd(p, q_c, k_c, v_c, do_c):
    """(dq_c, dk_c, dv_c) of the coarse branch for do_c."""
    torch = _torch()
    p = problem_from(p)
    st, wsb = vsa2_attn_workspace(p, 2)
    _check("vsa2_attn_workspace", st)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q_c.device)
    dq, dk, dv = torch.empty_like(q_c), torch.empty_like(k_c), torch.empty_like(v_c)
    _check("vsa2_coarse_bwd", vsa2_coarse_bwd(p, q_c.data_ptr(), k_c.data_ptr(), v_c.data_ptr(),
                                              do_c.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                              dv.data_ptr(), ws.data_ptr(), wsb, _stream()))
    return dq, dk, dv


def gate_merge(p, gate, o_c, o_f, out=None):
    """O = tanh(gate) * Repeat_B(o_c) + o_f."""
    torch = _torch()
    p = problem_from(p)
    out = torch.empty_like(o_f) if out is None else out
    _check("vsa2_gate_merge", vsa2_gate_merge(p, gate.data_ptr(), o_c.data_ptr(), o_f.data_ptr(),
                                              out.data_ptr(), _stream()))
    return out


def gate_merge_bwd(p, gate, o_c, dout):
    """(do_c, dgate) of the merge for dout."""
    torch = _torch()
    p = problem_from(p)
    do_c = torch.empty_like(o_c)
    dgate = torch.empty_like(gate)
    _check("vsa2_gate_merge_bwd", vsa2_gate_merge_bwd(p, gate.data_ptr(), o_c.data_ptr(),
                                                      dout.data_ptr(), do_c.data_ptr(),
                                                      dgate.data_ptr(), _stream()))
    return do_c, dgate


def joint_lists(p, r):
    """Joint video + text lists from the router's result r (route()).
    Returns dict(row_ptr, col_idx, kv_ptr, kv_idx, col_cap)."""
    torch = _torch()
    p = problem_from(p)
    Nj, _ = _joint(p)
    dev = r["row_ptr"].device
    cap = r["col_cap"] + p.batch * p.heads_q * (Nj - _dims(p)[0]) * (_dims(p)[0] + Nj)
    st, wsb = vsa2_joint_workspace(p)
    _check("vsa2_joint_workspace", st)
    i32 = torch.int32
    jrp = torch.empty(p.batch * p.heads_q * Nj + 1, dtype=i32, device=dev)
    jci = torch.empty(max(cap, 1), dtype=i32, device=dev)
    jkp = torch.empty(p.batch * p.heads_kv * Nj + 1, dtype=i32, device=dev)
    jki = torch.empty(max(cap, 1), dtype=i32, device=dev)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    _check("vsa2_joint_lists", vsa2_joint_lists(p, r["row_ptr"].data_ptr(), r["col_idx"].data_ptr(),
                                                r["col_cap"], jrp.data_ptr(), jci.data_ptr(), cap,
                                                jkp.data_ptr(), jki.data_ptr(), ws.data_ptr(), wsb, _stream()))
    return dict(row_ptr=jrp, col_idx=jci, kv_ptr=jkp, kv_idx=jki, col_cap=cap)


def unpool_add(p, dx_c, dx, P):
    """dx += MeanPool adjoint of dx_c over P = (Pt, Ph, Pw), in place."""
    p = problem_from(p)
    _check("vsa2_unpool_add", vsa2_unpool_add(p, dx.shape[1], dx_c.data_ptr(), P[0], P[1], P[2],
                                              dx.data_ptr(), _stream()))
    return dx
