"""CPU-side checks of the C-ABI library: it loads without a GPU, exports every
symbol include/vsa2.h declares, and rejects invalid arguments on the host
before touching the device (no compute call runs here)."""
import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vsa2.h")

vsa2 = pytest.importorskip("paper_2609_32882_amd")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vsa2_[a-z_0-9]+)\s*\(", src)))


def header_enum(name_prefix):
    src = open(HEADER).read()
    return {m.group(1): int(m.group(2)) for m in re.finditer(r"\b(%s[A-Z_0-9]*)\s*=\s*(\d+)" % name_prefix, src)}


def test_library_exports_every_declared_symbol():
    lib = vsa2.lib()
    decl = declared_functions()
    assert set(decl) == set(vsa2.EXPORTS), decl
    for name in decl:
        assert hasattr(lib, name), name


def test_status_codes_match_header():
    enum = header_enum("VSA2_ERR_")
    enum["VSA2_OK"] = 0
    assert {v: k for k, v in enum.items()} == vsa2.STATUS_NAMES
    for code in enum.values():
        assert vsa2.vsa2_status_str(code)


def test_problem_struct_layout_matches_header():
    src = open(HEADER).read()
    body = src[src.index("typedef struct {\n    int32_t batch;"):src.index("} vsa2_problem;")]
    fields = re.findall(r"int32_t\s+([^;]+);", body)
    names = [n.strip() for f in fields for n in f.split(",")]
    assert names == [f[0] for f in vsa2.vsa2_problem._fields_]
    assert ctypes.sizeof(vsa2.vsa2_problem) == 4 * len(names)
    assert ctypes.sizeof(vsa2.vsa2_select) == 16


def good():
    return vsa2.make_problem(1, 4, 2, 128, 8, 16, 16)


FAKE = 0x10000          # aligned, never dereferenced: every call below fails validation first
MISALIGNED = 0x10008


@pytest.mark.parametrize("mutate,expect", [
    (dict(dtype=7), "VSA2_ERR_DTYPE"),
    (dict(heads_q=3), "VSA2_ERR_SHAPE"),          # Hq % Hkv
    (dict(T=0), "VSA2_ERR_SHAPE"),                # empty grid
    (dict(Rt=3), "VSA2_ERR_SHAPE"),               # Bt % Rt
    (dict(batch=0), "VSA2_ERR_SHAPE"),
    (dict(head_dim=96), "VSA2_ERR_UNSUPPORTED"),
    (dict(Bw=8, W=16), "VSA2_ERR_UNSUPPORTED"),   # B = 128
])
def test_attn_fwd_rejects_bad_problem(mutate, expect):
    p = good()
    for k, v in mutate.items():
        setattr(p, k, v)
    st = vsa2.vsa2_attn_fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE, FAKE, None, FAKE, 1 << 40, None)
    assert vsa2.STATUS_NAMES[st] == expect


def test_grid_not_divisible_by_the_cube_is_padded_up():
    """T, H, W need not be multiples of the cube: the grid is padded up to
    whole cubes (N = ceil(T/Bt) ceil(H/Bh) ceil(W/Bw))."""
    sel = vsa2.vsa2_select(0, 5, 0.0, 0)
    for T, H, W, N in ((8, 16, 16, 32), (6, 16, 16, 32), (5, 13, 9, 2 * 4 * 3), (1, 1, 1, 1)):
        p = vsa2.make_problem(1, 4, 2, 128, T, H, W)
        st, n = vsa2.vsa2_route_capacity(p, sel)
        assert vsa2.STATUS_NAMES[st] == "VSA2_OK" and n == 4 * N * min(5, N), (T, H, W)


def test_joint_lists_checks():
    """Text tokens: the joint capacity adds the text blocks of the video rows
    and the full text rows; vsa2_joint_lists needs text, enough capacity
    and a workspace."""
    sel = vsa2.vsa2_select(0, 5, 0.0, 0)
    p = vsa2.make_problem(1, 4, 2, 128, 8, 16, 16, text_len=100)     # N = 32, M = 2
    st, cap = vsa2.vsa2_joint_capacity(p, sel)
    assert vsa2.STATUS_NAMES[st] == "VSA2_OK" and cap == 4 * 32 * 5 + 4 * (32 * 2 + 2 * 34)
    st, wsb = vsa2.vsa2_joint_workspace(p)
    assert vsa2.STATUS_NAMES[st] == "VSA2_OK" and wsb > 0
    call = lambda pp, jcap, ws, wsz: vsa2.STATUS_NAMES[vsa2.vsa2_joint_lists(
        pp, FAKE, FAKE, 4 * 32 * 5, FAKE, FAKE, jcap, FAKE, FAKE, ws, wsz, None)]
    assert call(vsa2.make_problem(1, 4, 2, 128, 8, 16, 16), cap, FAKE, wsb) == "VSA2_ERR_SHAPE"
    assert call(p, cap - 1, FAKE, wsb) == "VSA2_ERR_CAPACITY"
    assert call(p, cap, None, 0) == "VSA2_ERR_WORKSPACE"
    assert call(p, cap, FAKE, wsb - 1) == "VSA2_ERR_WORKSPACE"
    assert vsa2.STATUS_NAMES[vsa2.vsa2_joint_lists(p, None, FAKE, 1, FAKE, FAKE, cap, FAKE, FAKE, FAKE, wsb,
                                                   None)] == "VSA2_ERR_NULL"
    # the attention workspaces grow with the text blocks
    _, w0 = vsa2.vsa2_attn_workspace(vsa2.make_problem(1, 4, 2, 128, 8, 16, 16), 1)
    _, w1 = vsa2.vsa2_attn_workspace(p, 1)
    assert w1 > w0
    p.text_len = -1
    assert vsa2.STATUS_NAMES[vsa2.vsa2_joint_capacity(p, sel)[0]] == "VSA2_ERR_SHAPE"


def test_null_and_alignment_checks():
    p = good()
    assert vsa2.STATUS_NAMES[vsa2.vsa2_attn_fwd(p, None, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE, None,
                                                None, 0, None)] == "VSA2_ERR_NULL"
    assert vsa2.STATUS_NAMES[vsa2.vsa2_attn_fwd(p, MISALIGNED, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE,
                                                None, FAKE, 1 << 40, None)] == "VSA2_ERR_ALIGN"
    assert vsa2.STATUS_NAMES[vsa2.vsa2_attn_fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE,
                                                MISALIGNED, FAKE, 1 << 40, None)] == "VSA2_ERR_ALIGN"
    assert vsa2.STATUS_NAMES[vsa2.vsa2_pool(p, 4, FAKE, 2, 2, 2, MISALIGNED, None)] == "VSA2_ERR_ALIGN"
    assert vsa2.STATUS_NAMES[vsa2.vsa2_pool(p, 4, FAKE, 3, 2, 2, FAKE, None)] == "VSA2_ERR_SHAPE"
    assert vsa2.STATUS_NAMES[vsa2.vsa2_pool(None, 4, FAKE, 2, 2, 2, FAKE, None)] == "VSA2_ERR_NULL"
    # bwd needs a workspace for the per-query Delta, and the forward's o_lo
    st = vsa2.vsa2_attn_bwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1,
                            FAKE, FAKE, FAKE, None, 0, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_WORKSPACE"
    st = vsa2.vsa2_attn_bwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, 1,
                            FAKE, FAKE, FAKE, FAKE, 1 << 40, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_NULL"


def test_forward_needs_its_work_order_workspace():
    p = good()
    st, n = vsa2.vsa2_attn_workspace(p, 0)
    assert vsa2.STATUS_NAMES[st] == "VSA2_OK" and n >= 4 * p.batch * p.heads_q * 8 and n % 256 == 0
    st = vsa2.vsa2_attn_fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE, None, None, 0, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_WORKSPACE"
    st = vsa2.vsa2_attn_fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE, None, FAKE, n - 1, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_WORKSPACE"


def test_sequence_topk_rule_capacity_and_workspace():
    p = good()                                # N = 32 cubes, 4 query heads
    for k, want in ((5, 4 * 32 * 5), (40, 4 * 32 * 32)):
        st, n = vsa2.vsa2_route_capacity(p, vsa2.vsa2_select(2, k, 0.0, 0))
        assert vsa2.STATUS_NAMES[st] == "VSA2_OK" and n == want
    st0, w0 = vsa2.vsa2_route_workspace(p, vsa2.vsa2_select(0, 5, 0.0, 0))
    st2, w2 = vsa2.vsa2_route_workspace(p, vsa2.vsa2_select(2, 5, 0.0, 0))
    assert st0 == st2 == 0 and w2 > w0
    for bad in (vsa2.vsa2_select(2, 0, 0.0, 0), vsa2.vsa2_select(3, 5, 0.0, 0)):
        st, _ = vsa2.vsa2_route_capacity(p, bad)
        assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_SELECT"


def test_staged_backward_argument_checks():
    """The three backward stages validate like vsa2_attn_bwd, before any
    device work (fake pointers are never dereferenced)."""
    p = good()
    names = vsa2.STATUS_NAMES
    big = 1 << 40
    F5 = (FAKE,) * 5
    # prep(p, q, k, v, o, lse, o_lo, dout, ws, ws_bytes, stream)
    assert names[vsa2.vsa2_attn_bwd_prep(p, *F5, FAKE, FAKE, None, 0, None)] == "VSA2_ERR_WORKSPACE"
    assert names[vsa2.vsa2_attn_bwd_prep(p, *F5, None, FAKE, FAKE, big, None)] == "VSA2_ERR_NULL"
    assert names[vsa2.vsa2_attn_bwd_prep(p, None, *F5[1:], FAKE, FAKE, FAKE, big, None)] == "VSA2_ERR_NULL"
    assert names[vsa2.vsa2_attn_bwd_prep(p, *F5, MISALIGNED, FAKE, FAKE, big, None)] == "VSA2_ERR_ALIGN"
    assert names[vsa2.vsa2_attn_bwd_prep(p, FAKE, MISALIGNED, *F5[2:], FAKE, FAKE, FAKE, big,
                                         None)] == "VSA2_ERR_ALIGN"
    assert names[vsa2.vsa2_attn_bwd_prep(None, *F5, FAKE, FAKE, FAKE, big, None)] == "VSA2_ERR_NULL"
    # dkdv(p, q, k, v, dout, kv_ptr, kv_idx, col_cap, dk, dv, ws, ws_bytes, stream)
    assert names[vsa2.vsa2_attn_bwd_dkdv(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, None, FAKE, big,
                                         None)] == "VSA2_ERR_NULL"
    assert names[vsa2.vsa2_attn_bwd_dkdv(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, -1, FAKE, FAKE, FAKE, big,
                                         None)] == "VSA2_ERR_CAPACITY"
    assert names[vsa2.vsa2_attn_bwd_dkdv(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, MISALIGNED, FAKE,
                                         big, None)] == "VSA2_ERR_ALIGN"
    assert names[vsa2.vsa2_attn_bwd_dkdv(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE, FAKE, 0,
                                         None)] == "VSA2_ERR_WORKSPACE"
    # dq(p, q, k, v, dout, row_ptr, col_idx, col_cap, dq, ws, ws_bytes, stream)
    assert names[vsa2.vsa2_attn_bwd_dq(p, FAKE, FAKE, FAKE, FAKE, FAKE, None, 1, FAKE, FAKE, big,
                                       None)] == "VSA2_ERR_NULL"
    assert names[vsa2.vsa2_attn_bwd_dq(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, MISALIGNED, FAKE, big,
                                       None)] == "VSA2_ERR_ALIGN"
    assert names[vsa2.vsa2_attn_bwd_dq(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, None, 0,
                                       None)] == "VSA2_ERR_WORKSPACE"


def test_route_capacity_workspace_and_select_checks():
    p = good()
    N = (8 // 4) * (16 // 4) * (16 // 4)
    st, cap = vsa2.vsa2_route_capacity(p, vsa2.vsa2_select(0, 5, 0.0, 0))
    assert st == 0 and cap == 1 * 4 * N * 5
    st, cap = vsa2.vsa2_route_capacity(p, vsa2.vsa2_select(0, 10 ** 6, 0.0, 0))
    assert st == 0 and cap == 4 * N * N                     # k > N keeps every block
    st, cap = vsa2.vsa2_route_capacity(p, vsa2.vsa2_select(1, 0, 0.9, 7))
    assert st == 0 and cap == 4 * N * 7
    for bad in (vsa2.vsa2_select(0, 0, 0, 0), vsa2.vsa2_select(1, 0, 0.0, 5),
                vsa2.vsa2_select(1, 0, 1.5, 5), vsa2.vsa2_select(1, 0, 0.5, 0),
                vsa2.vsa2_select(9, 1, 0.5, 1)):
        assert vsa2.STATUS_NAMES[vsa2.vsa2_route_capacity(p, bad)[0]] == "VSA2_ERR_SELECT"
    s = vsa2.vsa2_select(0, 5, 0.0, 0)
    st, wsb = vsa2.vsa2_route_workspace(p, s)
    assert st == 0 and wsb >= 4 * N * N * 4
    # capacity below what the rule can emit
    st = vsa2.vsa2_route(p, s, FAKE, FAKE, FAKE, FAKE, 4 * N * 5 - 1, None, None, None, FAKE, wsb, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_CAPACITY"
    st = vsa2.vsa2_route(p, s, FAKE, FAKE, FAKE, FAKE, 4 * N * 5, None, None, None, FAKE, wsb - 1, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_WORKSPACE"
    st = vsa2.vsa2_route(p, s, FAKE, FAKE, FAKE, FAKE, 4 * N * 5, FAKE, None, None, FAKE, wsb, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_NULL"          # kv_ptr without kv_idx
    p16 = good()
    p16.Rt, p16.Rh, p16.Rw = 1, 1, 2                         # G = 32: not built
    st = vsa2.vsa2_route(p16, s, FAKE, FAKE, FAKE, FAKE, 10 ** 9, None, None, None, FAKE, 10 ** 12, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_UNSUPPORTED"


def test_product_path_has_no_oracle_or_fallback():
    """The binding and the library never reach the oracle or a CPU path."""
    pkg = os.path.join(ROOT, "paper_2609_32882_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                src = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in src.replace("oracle-free", ""), f


def test_mfma_peak_probe_checks():
    """The dense MFMA rate probe rejects a missing flops output, a missing
    sink when it would launch, and a negative round count, before any device
    work."""
    st, _ = vsa2.vsa2_mfma_peak_probe(-1, FAKE)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_SHAPE"
    st, _ = vsa2.vsa2_mfma_peak_probe(8, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_NULL"
    assert vsa2.STATUS_NAMES[vsa2.lib().vsa2_mfma_peak_probe(8, FAKE, None, None)] == "VSA2_ERR_NULL"


def test_missing_library_fails_loudly():
    """Without libvsa2.so the first call raises ImportError: there is no
    silent CPU path to fall back on."""
    code = ("import sys; sys.path.insert(0, %r)\n"
            "import paper_2609_32882_amd as v\n"
            "v.LIB_PATH = '/nonexistent/libvsa2.so'\n"
            "try:\n"
            "    v.lib()\n"
            "except ImportError as e:\n"
            "    print('raised', e)\n"
            "else:\n"
            "    print('loaded')\n") % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert out.stdout.startswith("raised") and "not built" in out.stdout


def test_router_rejects_more_than_4096_blocks():
    """N = 4096 cubes is the router's largest (tested on the GPU at that
    size); one more row of cubes is refused before any device work."""
    s = vsa2.vsa2_select(0, 8, 0.0, 0)
    from workload import Problem
    ok = vsa2.problem_from(Problem(1, 1, 1, 64, 64, 64, 64))          # N = 4096
    big = vsa2.problem_from(Problem(1, 1, 1, 64, 64, 64, 68))         # N = 16 x 16 x 17 = 4352
    st = vsa2.vsa2_route(big, s, FAKE, FAKE, FAKE, FAKE, 10 ** 9, None, None, None, FAKE, 10 ** 12, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_UNSUPPORTED"
    st = vsa2.vsa2_route(ok, s, FAKE, FAKE, FAKE, FAKE, 10 ** 9, None, None, None, FAKE, 0, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_WORKSPACE"                # past the size check

