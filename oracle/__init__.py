"""CPU oracle for the VSA2 routed sparse-attention path (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never loads it, and it shares no
code with the HIP kernels.  The arithmetic lives in vsa2_oracle.c (plain
loops in double); this module marshals numpy arrays and does the index-only
steps (CSR assembly, the CSR -> CSC transpose) with plain numpy.

Conventions: tensors are cube-major [batch, heads, L, D] float32 arrays that
hold exact input values (bf16 inputs widened).  Rows are numbered
(b*Hq + h)*N + n for query blocks and (b*Hkv + h)*N + n for key blocks.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vsa2_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

SEL_TOPK, SEL_MASS = 0, 1


def build(force: bool = False) -> str:
    """Compile vsa2_oracle.c with gcc into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, dbl = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.vo_round_bf16.argtypes = [P, P, i64]
        L.vo_pool.argtypes = [P, i64, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, P]
        L.vo_router_scores.argtypes = [P, P, i32, i32, i32, i64, i32, i32, P, i64, P, P, P, i32, i32,
                                       i32]
        L.vo_select_rows.argtypes = [P, i64, i32, i32, i32, dbl, i32, P, P]
        L.vo_select_seq.argtypes = [P, i64, i32, i32, P]
        L.vo_attn_fwd.argtypes = [P, P, P, i32, i32, i32, i64, i32, i32, P, P, P, i64, P, P, P]
        L.vo_attn_bwd_dq.argtypes = [P, P, P, P, i32, i32, i32, i64, i32, i32, P, P, P, i64, P, P]
        L.vo_attn_bwd_dkdv.argtypes = [P, P, P, P, i32, i32, i32, i64, i32, i32, P, P, P, i64,
                                       P, P, P]
        L.vo_coarse_fwd.argtypes = [P, P, P, i32, i32, i32, i32, i32, P, P]
        L.vo_coarse_bwd.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, P, P, P]
        L.vo_gate_merge.argtypes = [P, P, P, i64, i32, i32, i32, P]
        L.vo_gate_merge_bwd.argtypes = [P, P, P, i64, i32, i32, i32, P, P, P]
        L.vo_unpool_add.argtypes = [P, i64, i32, i32, i32, i32, i32, i32, i32, i32, i32, i32, P]
        for f in (L.vo_round_bf16, L.vo_pool, L.vo_router_scores, L.vo_select_rows,
                  L.vo_select_seq, L.vo_attn_fwd, L.vo_attn_bwd_dq, L.vo_attn_bwd_dkdv,
                  L.vo_coarse_fwd, L.vo_coarse_bwd, L.vo_gate_merge, L.vo_gate_merge_bwd,
                  L.vo_unpool_add):
            f.restype = None
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _geom(p):
    """{T, H, W, Bt, Bh, Bw, Lt}: the real grid, the cube (padded grids) and
    the number of text tokens joined to the video (0: none)."""
    return np.array([p.T, p.H, p.W, p.Bt, p.Bh, p.Bw, getattr(p, "text_len", 0)], np.int32)


def _video(x, p):
    """The video part [..., :L, :] of a joint [..., L_joint, D] tensor."""
    return np.ascontiguousarray(x[..., :p.L, :]) if x.shape[-2] != p.L else x


def threads() -> int:
    """Host threads the oracle's OpenMP loops use."""
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


# --------------------------------------------------------------------------
# Steps of the path
# --------------------------------------------------------------------------

def round_bf16(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, np.float32)
    lib().vo_round_bf16(_p(x), _p(out), x.size)
    return out


def pool(x, p, Pt: int, Ph: int, Pw: int) -> np.ndarray:
    """MeanPool over (Pt, Ph, Pw) sub-cubes of every cube (Eq. router_start
    with P = R; Eq. compress with P = B).  x: [b, h, L, D] -> [b, h, N*G, D]
    (of a joint video + text tensor, the video part is pooled)."""
    x = _f32(_video(x, p))
    nb, nh, L, D = x.shape
    G = (p.Bt // Pt) * (p.Bh // Ph) * (p.Bw // Pw)
    out = np.empty((nb, nh, p.N * G, D), np.float32)
    lib().vo_pool(_p(x), nb * nh, p.T, p.H, p.W, p.Bt, p.Bh, p.Bw, Pt, Ph, Pw, D,
                  int(p.dtype == 1), _p(out))
    return out


def router_scores(q_r, k_r, p, rows=None, with_lse: bool = False):
    """Block scores P_r (Eq. router_start .. router_end) for query-block rows
    (default: all).  Returns float64 [nrows, N] (and [nrows, G] LSE)."""
    q_r, k_r = _f32(q_r), _f32(k_r)
    nrow_all = p.batch * p.heads_q * p.N
    rows = np.arange(nrow_all, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, np.int64)
    out = np.empty((rows.size, p.N), np.float64)
    lse = np.empty((rows.size, p.G), np.float64)
    g = _geom(p)
    lib().vo_router_scores(_p(q_r), _p(k_r), p.batch, p.heads_q, p.heads_kv, p.N, p.G,
                           p.head_dim, _p(rows), rows.size, _p(out), _p(lse), _p(g), p.Rt, p.Rh, p.Rw)
    return (out, lse) if with_lse else out


def select_rows(scores, sel):
    """Per-query-block selection (top-k, or mass with cap) decided on the
    fp32-rounded scores ordered by (score desc, index asc).
    Returns (counts [nrows], lists: list of ascending int32 arrays)."""
    scores = np.ascontiguousarray(scores, np.float64)
    nrows, N = scores.shape
    counts = np.empty(nrows, np.int32)
    idx = np.empty((nrows, N), np.int32)
    lib().vo_select_rows(_p(scores), nrows, N, int(sel.mode), int(sel.k), float(sel.mass),
                         int(sel.cap), _p(counts), _p(idx))
    return counts, idx


def csr_from_selection(counts, idx):
    row_ptr = np.zeros(counts.size + 1, np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col_idx = np.concatenate([idx[r, :counts[r]] for r in range(counts.size)]) if counts.size else \
        np.zeros(0, np.int32)
    return row_ptr.astype(np.int32), col_idx.astype(np.int32)


def csr_to_csc(row_ptr, col_idx, p, N=None):
    """Transpose the query-block -> key-block lists into key-block ->
    (query head within the KV group, query block) lists, entries ordered by
    (hq_local, n_q) ascending, value hq_local*N + n_q.  N: blocks per
    sequence (default the video cubes; p.N_joint for joint lists)."""
    N = p.N if N is None else N
    grp = p.heads_q // p.heads_kv
    nrows = p.batch * p.heads_q * N
    mask = np.zeros((nrows, N), bool)
    counts = np.diff(row_ptr)
    rr = np.repeat(np.arange(nrows), counts)
    mask[rr, col_idx] = True
    # [b, Hkv, grp, Nq, Nk] -> [b, Hkv, Nk, grp, Nq]
    m = mask.reshape(p.batch, p.heads_kv, grp, N, N).transpose(0, 1, 4, 2, 3)
    m = m.reshape(p.batch * p.heads_kv * N, grp * N)
    kv_counts = m.sum(axis=1)
    kv_ptr = np.zeros(kv_counts.size + 1, np.int64)
    np.cumsum(kv_counts, out=kv_ptr[1:])
    _, cols = np.nonzero(m)
    return kv_ptr.astype(np.int32), cols.astype(np.int32)


def joint_lists(row_ptr, col_idx, p):
    """Block lists of the joint video + text attention (MMDiT; Eq.
    block_sparse extended with full video-to-text and text-to-video blocks,
    Sec. 2.2): a video query block keeps its routed video blocks and gains
    all M text blocks; a text query block takes every block.  Blocks are
    numbered 0..N-1 (video cubes), N..N+M-1 (text).  Returns the joint CSR
    (rows b*Hq*(N+M)) and CSC."""
    N, M = p.N, p.M
    Nj = N + M
    text = np.arange(N, Nj, dtype=np.int32)
    full = np.arange(Nj, dtype=np.int32)
    lists = []
    for bh in range(p.batch * p.heads_q):
        for n in range(N):
            r = bh * N + n
            lists.append(np.concatenate([col_idx[row_ptr[r]:row_ptr[r + 1]], text]))
        lists.extend([full] * M)
    counts = np.array([len(x) for x in lists], np.int64)
    rp = np.zeros(counts.size + 1, np.int64)
    np.cumsum(counts, out=rp[1:])
    ci = np.concatenate(lists).astype(np.int32)
    kp, ki = csr_to_csc(rp.astype(np.int32), ci, p, Nj)
    return rp.astype(np.int32), ci, kp, ki


def route(q, k, p, sel):
    """The whole router: pool (P = R), block scores, selection, CSR and CSC.
    Returns a dict with q_r, k_r, scores, row_ptr, col_idx, kv_ptr, kv_idx."""
    q_r = pool(q, p, p.Rt, p.Rh, p.Rw)
    k_r = pool(k, p, p.Rt, p.Rh, p.Rw)
    scores = router_scores(q_r, k_r, p)
    counts, idx = select_rows(scores, sel)
    row_ptr, col_idx = csr_from_selection(counts, idx)
    kv_ptr, kv_idx = csr_to_csc(row_ptr, col_idx, p)
    return dict(q_r=q_r, k_r=k_r, scores=scores, row_ptr=row_ptr, col_idx=col_idx,
                kv_ptr=kv_ptr, kv_idx=kv_idx)


def _nj(p):
    """Blocks of one (batch, head) sequence: video cubes plus text blocks."""
    return getattr(p, "N_joint", p.N)


def attn_fwd(q, k, v, p, row_ptr, col_idx, rows=None):
    """Block-sparse attention forward for query-block rows (default all).
    With text tokens (p.text_len > 0) q, k, v are joint [b, h, L_joint, D]
    sequences and the lists are joint lists (joint_lists).
    Returns O [nrows, B, D] float64 and LSE [nrows, B] float64."""
    q, k, v = _f32(q), _f32(k), _f32(v)
    nrow_all = p.batch * p.heads_q * _nj(p)
    rows = np.arange(nrow_all, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, np.int64)
    o = np.empty((rows.size, p.B, p.head_dim), np.float64)
    lse = np.empty((rows.size, p.B), np.float64)
    rp, ci = np.ascontiguousarray(row_ptr, np.int32), np.ascontiguousarray(col_idx, np.int32)
    g = _geom(p)
    lib().vo_attn_fwd(_p(q), _p(k), _p(v), p.batch, p.heads_q, p.heads_kv, _nj(p) * p.B, p.head_dim,
                      p.B, _p(rp), _p(ci), _p(rows), rows.size, _p(o), _p(lse), _p(g))
    return o, lse


def attn_bwd_dq(q, k, v, do, p, row_ptr, col_idx, rows=None):
    q, k, v, do = _f32(q), _f32(k), _f32(v), _f32(do)
    nrow_all = p.batch * p.heads_q * _nj(p)
    rows = np.arange(nrow_all, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, np.int64)
    dq = np.empty((rows.size, p.B, p.head_dim), np.float64)
    rp, ci = np.ascontiguousarray(row_ptr, np.int32), np.ascontiguousarray(col_idx, np.int32)
    g = _geom(p)
    lib().vo_attn_bwd_dq(_p(q), _p(k), _p(v), _p(do), p.batch, p.heads_q, p.heads_kv, _nj(p) * p.B,
                         p.head_dim, p.B, _p(rp), _p(ci), _p(rows), rows.size, _p(dq), _p(g))
    return dq


def attn_bwd_dkdv(q, k, v, do, p, row_ptr, col_idx, kv_rows=None):
    q, k, v, do = _f32(q), _f32(k), _f32(v), _f32(do)
    nkv_all = p.batch * p.heads_kv * _nj(p)
    kv_rows = np.arange(nkv_all, dtype=np.int64) if kv_rows is None else \
        np.ascontiguousarray(kv_rows, np.int64)
    dk = np.empty((kv_rows.size, p.B, p.head_dim), np.float64)
    dv = np.empty((kv_rows.size, p.B, p.head_dim), np.float64)
    rp, ci = np.ascontiguousarray(row_ptr, np.int32), np.ascontiguousarray(col_idx, np.int32)
    g = _geom(p)
    lib().vo_attn_bwd_dkdv(_p(q), _p(k), _p(v), _p(do), p.batch, p.heads_q, p.heads_kv, _nj(p) * p.B,
                           p.head_dim, p.B, _p(rp), _p(ci), _p(kv_rows), kv_rows.size,
                           _p(dk), _p(dv), _p(g))
    return dk, dv


def select_seq(scores_bh, N: int, k: int):
    """Sequence-level TopK_{NK} over each (batch, head)'s flattened N x N map.
    scores_bh: [nseq, N, N] float64 -> bool [nseq, N, N]."""
    s = np.ascontiguousarray(scores_bh, np.float64).reshape(-1, N * N)
    sel = np.empty(s.shape, np.uint8)
    lib().vo_select_seq(_p(s), s.shape[0], N, k, _p(sel))
    return sel.reshape(-1, N, N).astype(bool)


# --------------------------------------------------------------------------
# Coarse branch and gated merge (Sec. 2.2 "Coarse Branch", "Gated Merge")
# --------------------------------------------------------------------------


def coarse_fwd(qc, kc, vc, p):
    """Dense attention among the N cube means of each head (Eq. compress and
    the two equations after it).  qc [b, Hq, N, D], kc, vc [b, Hkv, N, D]
    (MeanPool_B outputs).  Returns O_c_hat [b, Hq, N, D] and the natural-log
    LSE [b, Hq, N], float64."""
    qc, kc, vc = _f32(qc), _f32(kc), _f32(vc)
    N, D = p.N, p.head_dim
    oc = np.empty((p.batch, p.heads_q, N, D), np.float64)
    lse = np.empty((p.batch, p.heads_q, N), np.float64)
    lib().vo_coarse_fwd(_p(qc), _p(kc), _p(vc), p.batch, p.heads_q, p.heads_kv, N, D, _p(oc), _p(lse))
    return oc, lse


def coarse_bwd(qc, kc, vc, doc, p):
    """Gradients (dqc, dkc, dvc) of coarse_fwd for the output gradient doc."""
    qc, kc, vc, doc = _f32(qc), _f32(kc), _f32(vc), _f32(doc)
    N, D = p.N, p.head_dim
    dqc = np.empty((p.batch, p.heads_q, N, D), np.float64)
    dkc = np.empty((p.batch, p.heads_kv, N, D), np.float64)
    dvc = np.empty((p.batch, p.heads_kv, N, D), np.float64)
    lib().vo_coarse_bwd(_p(qc), _p(kc), _p(vc), _p(doc), p.batch, p.heads_q, p.heads_kv, N, D,
                        _p(dqc), _p(dkc), _p(dvc))
    return dqc, dkc, dvc


def gate_merge(g, oc, of, p):
    """O = tanh(g) * Repeat_B(O_c_hat) + O_f (Eq. gate_linear, gated merge).
    g [b, Hq, L] gate pre-activations; oc [b, Hq, N, D]; of [b, Hq, L, D].
    Joint video + text sequences (L_joint tokens): the coarse branch covers
    the video tokens only, text tokens keep O_f."""
    g, oc, of = _f32(g), _f32(oc), _f32(of)
    out = of.astype(np.float64)
    gv, ofv = _f32(_video(g[..., None], p)[..., 0]), _video(of, p)
    ov = np.empty((p.batch, p.heads_q, p.L, p.head_dim), np.float64)
    lib().vo_gate_merge(_p(gv), _p(oc), _p(ofv), p.batch * p.heads_q, p.N, p.B, p.head_dim, _p(ov))
    out[..., :p.L, :] = ov
    return out


def gate_merge_bwd(g, oc, dout, p):
    """(d O_c_hat, d g) of gate_merge for dout; d O_f is dout itself."""
    g, oc, dout = _f32(g), _f32(oc), _f32(dout)
    Lg = g.shape[-1]
    g, dout = _f32(_video(g[..., None], p)[..., 0]), _video(dout, p)
    doc = np.empty((p.batch, p.heads_q, p.N, p.head_dim), np.float64)
    dg = np.zeros((p.batch, p.heads_q, Lg), np.float64)      # text tokens: no gate
    dgv = np.empty((p.batch, p.heads_q, p.L), np.float64)
    geom = _geom(p)
    lib().vo_gate_merge_bwd(_p(g), _p(oc), _p(dout), p.batch * p.heads_q, p.N, p.B, p.head_dim,
                            _p(doc), _p(dgv), _p(geom))
    dg[..., :p.L] = dgv
    return doc, dg


def unpool_add(dxc, dx, p, Pt: int, Ph: int, Pw: int):
    """dx += the adjoint of MeanPool over (Pt, Ph, Pw) applied to dxc.
    dxc [b, heads, N*Gp, D] and dx [b, heads, L, D], float64; dx is updated."""
    dxc = np.ascontiguousarray(dxc, np.float64)
    assert dx.dtype == np.float64 and dx.flags.c_contiguous
    nbh = dx.shape[0] * dx.shape[1]
    xv = _video(dx, p)                    # joint sequences: the video part
    lib().vo_unpool_add(_p(dxc), nbh, p.T, p.H, p.W, p.Bt, p.Bh, p.Bw, Pt, Ph, Pw, p.head_dim, _p(xv))
    if xv is not dx:
        dx[..., :p.L, :] = xv
    return dx
