"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test checks one oracle step against a closed form, an invariant the
paper's definitions imply, a special case that reduces to a textbook or
library routine (torch / numpy in float64), brute force, or a value the paper
prints.  Chosen so that a dropped term, wrong sign, wrong index or transposed
operand in the oracle fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from workload import BF16, F32, Problem, Selection, Workload, make_inputs, raster_to_cube_major, \
    round_bf16_f32

HERE = os.path.dirname(os.path.abspath(__file__))


def small(dtype=F32, T=4, H=8, W=8, Bt=2, Bh=4, Bw=4, Rt=1, Rh=2, Rw=2, hq=2, hkv=2, D=16):
    return Problem(1, hq, hkv, D, T, H, W, Bt, Bh, Bw, Rt, Rh, Rw, dtype)


def rand_qkv(p, seed=0, scale=1.0):
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((p.batch, p.heads_q, p.L, p.head_dim)) * scale).astype(np.float32)
    k = (rng.standard_normal((p.batch, p.heads_kv, p.L, p.head_dim)) * scale).astype(np.float32)
    v = rng.standard_normal((p.batch, p.heads_kv, p.L, p.head_dim)).astype(np.float32)
    do = rng.standard_normal((p.batch, p.heads_q, p.L, p.head_dim)).astype(np.float32)
    if p.dtype == BF16:
        q, k, v, do = (round_bf16_f32(t) for t in (q, k, v, do))
    return q, k, v, do


# ---------------------------------------------------------------- rounding

def test_bf16_rounding_ties_and_library():
    # ties round to even, exactly representable values stay, halfway above/below
    one = 1.0
    ulp = 2.0 ** -7
    cases = {
        one: one,
        one + ulp / 2: one,                    # tie -> even (1.0)
        one + 3 * ulp / 2: one + 2 * ulp,      # tie -> even (1 + 2 ulp)
        one + ulp / 2 + 2.0 ** -30: one + ulp,  # just above the tie
        -(one + ulp / 2): -one,
        2.0 ** -130: 2.0 ** -130,              # bf16 subnormal, exact
        3.0 * 2.0 ** -134: 2.0 ** -132,        # subnormal tie 1.5 ulp -> even (2 ulp)
    }
    got = oracle.round_bf16(np.array(list(cases.keys())))
    assert np.array_equal(got.astype(np.float64), np.array(list(cases.values())))
    # float32-exact values: torch's float -> bfloat16 conversion is RNE
    x = np.random.default_rng(1).standard_normal(20000).astype(np.float32) * 7
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(oracle.round_bf16(x.astype(np.float64)), ref)


# ---------------------------------------------------------------- pooling

@pytest.mark.parametrize("P", [(1, 2, 2), (2, 2, 2), (2, 4, 4), (1, 1, 1), (2, 1, 4)])
def test_pool_affine_ramp_closed_form(P):
    """Mean of an affine function over a sub-cube is its value at the centre."""
    p = small(T=4, H=8, W=12, Bt=2, Bh=4, Bw=4, D=3)
    Pt, Ph, Pw = P
    t, h, w = np.meshgrid(np.arange(p.T), np.arange(p.H), np.arange(p.W), indexing="ij")
    coef = np.array([[0.5, 2.0, -0.25], [1.0, -1.5, 0.125], [-2.0, 0.75, 4.0]])  # [D][t,h,w]
    off = np.array([1.0, -3.0, 0.5])
    x = np.stack([coef[d, 0] * t + coef[d, 1] * h + coef[d, 2] * w + off[d] for d in range(3)], -1)
    xr = raster_to_cube_major(x.reshape(1, 1, p.L, 3).astype(np.float32), p)
    out = oracle.pool(xr, p, Pt, Ph, Pw)
    Gt, Gh, Gw = p.Bt // Pt, p.Bh // Ph, p.Bw // Pw
    Nt, Nh, Nw = p.T // p.Bt, p.H // p.Bh, p.W // p.Bw
    exp = np.zeros_like(out)
    for nt in range(Nt):
        for nh in range(Nh):
            for nw in range(Nw):
                n = (nt * Nh + nh) * Nw + nw
                for gt in range(Gt):
                    for gh in range(Gh):
                        for gw in range(Gw):
                            g = (gt * Gh + gh) * Gw + gw
                            tc = nt * p.Bt + gt * Pt + (Pt - 1) / 2
                            hc = nh * p.Bh + gh * Ph + (Ph - 1) / 2
                            wc = nw * p.Bw + gw * Pw + (Pw - 1) / 2
                            exp[0, 0, n * Gt * Gh * Gw + g] = coef @ np.array([tc, hc, wc]) + off
    assert np.array_equal(out, exp)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_pool_matches_numpy_reshape_mean(dtype):
    p = small(dtype=dtype, T=4, H=8, W=8, D=8)
    x = np.random.default_rng(3).standard_normal((1, 2, p.L, p.head_dim)).astype(np.float32)
    if dtype == BF16:
        x = round_bf16_f32(x)
    out = oracle.pool(x, p, p.Rt, p.Rh, p.Rw)
    # raster grid, numpy mean over the pooling windows, then (n, g) order
    from workload import cube_major_to_raster
    xg = cube_major_to_raster(x, p).reshape(1, 2, p.T, p.H, p.W, p.head_dim).astype(np.float64)
    m = xg.reshape(1, 2, p.T // p.Rt, p.Rt, p.H // p.Rh, p.Rh, p.W // p.Rw, p.Rw, p.head_dim)
    m = m.mean(axis=(3, 5, 7))                       # [1,2,T/Rt,H/Rh,W/Rw,D]
    Gt, Gh, Gw = p.Bt // p.Rt, p.Bh // p.Rh, p.Bw // p.Rw
    m = m.reshape(1, 2, p.T // p.Bt, Gt, p.H // p.Bh, Gh, p.W // p.Bw, Gw, p.head_dim)
    m = m.transpose(0, 1, 2, 4, 6, 3, 5, 7, 8).reshape(1, 2, p.N * p.G, p.head_dim)
    # float64 -> dtype with one rounding (the bf16 rounding is pinned above)
    ref = m.astype(np.float32) if dtype == F32 else oracle.round_bf16(m)
    assert np.array_equal(out, ref)


# ---------------------------------------------------------------- router

def _softmax64(s):
    return torch.softmax(torch.from_numpy(s), dim=-1).numpy()


def test_router_R_equals_B_is_coarse_softmax():
    """G = 1: P_r is VSA's cube-level softmax(Q_c K_c^T / sqrt(D))."""
    p = small(T=4, H=8, W=8, Bt=2, Bh=4, Bw=4, Rt=2, Rh=4, Rw=4, D=16)
    q, k, _, _ = rand_qkv(p, 5)
    q_r, k_r = oracle.pool(q, p, p.Rt, p.Rh, p.Rw), oracle.pool(k, p, p.Rt, p.Rh, p.Rw)
    sc = oracle.router_scores(q_r, k_r, p).reshape(1, p.heads_q, p.N, p.N)
    qc = q.astype(np.float64).reshape(1, p.heads_q, p.N, p.B, p.head_dim).mean(3).astype(np.float32)
    kc = k.astype(np.float64).reshape(1, p.heads_kv, p.N, p.B, p.head_dim).mean(3).astype(np.float32)
    ref = _softmax64(np.einsum("bhid,bhjd->bhij", qc.astype(np.float64), kc.astype(np.float64))
                     / math.sqrt(p.head_dim))
    np.testing.assert_allclose(sc, ref, rtol=1e-12, atol=1e-15)


def test_router_R_one_is_block_mean_of_token_softmax():
    """R = 1 (G = B): P_r equals P_oracle = MeanPool_{BxB}(Softmax(QK^T/sqrt(D)))."""
    p = small(T=2, H=4, W=8, Bt=2, Bh=2, Bw=2, Rt=1, Rh=1, Rw=1, D=8)
    q, k, _, _ = rand_qkv(p, 6)
    q_r, k_r = oracle.pool(q, p, 1, 1, 1), oracle.pool(k, p, 1, 1, 1)
    assert np.array_equal(q_r, q) and np.array_equal(k_r, k)
    sc = oracle.router_scores(q_r, k_r, p).reshape(1, p.heads_q, p.N, p.N)
    P = _softmax64(np.einsum("bhid,bhjd->bhij", q.astype(np.float64), k.astype(np.float64))
                   / math.sqrt(p.head_dim))
    ref = P.reshape(1, p.heads_q, p.N, p.B, p.N, p.B).mean(axis=(3, 5))
    np.testing.assert_allclose(sc, ref, rtol=1e-12, atol=1e-16)


def test_router_rows_sum_to_inverse_G_and_nonnegative():
    p = small(T=4, H=8, W=8, D=16)
    q, k, _, _ = rand_qkv(p, 7, scale=2.0)
    q_r, k_r = oracle.pool(q, p, p.Rt, p.Rh, p.Rw), oracle.pool(k, p, p.Rt, p.Rh, p.Rw)
    sc, lse = oracle.router_scores(q_r, k_r, p, with_lse=True)
    assert (sc >= 0).all()
    np.testing.assert_allclose(sc.sum(1), 1.0 / p.G, rtol=1e-12)
    # LSE of the first pooled query, by torch
    s0 = q_r[0, 0, :1].astype(np.float64) @ k_r[0, 0].astype(np.float64).T / math.sqrt(p.head_dim)
    assert abs(lse[0, 0] - torch.logsumexp(torch.from_numpy(s0), -1).item()) < 1e-12


def test_router_gqa_head_mapping():
    """Query head h reads KV head h // (Hq/Hkv): same as MHA with K replicated."""
    p = small(hq=4, hkv=2, D=8)
    q, k, _, _ = rand_qkv(p, 8)
    q_r, k_r = oracle.pool(q, p, p.Rt, p.Rh, p.Rw), oracle.pool(k, p, p.Rt, p.Rh, p.Rw)
    sc = oracle.router_scores(q_r, k_r, p)
    pm = p.replace(heads_kv=4)
    sc2 = oracle.router_scores(q_r, np.repeat(k_r, 2, axis=1), pm)
    assert np.array_equal(sc, sc2)


def test_router_shared_means_pick_own_cube():
    """With Q and K of a head sharing cube means, each query block's own cube
    has the highest block score."""
    w = Workload("t", Problem(1, 2, 2, 64, 4, 8, 8, 2, 4, 4, 1, 2, 2, F32), Selection(0, 4), 77)
    x = make_inputs(w, shared_mean=True)
    r = oracle.route(x["q"], x["k"], w.problem, w.select)
    sc = r["scores"].reshape(2, w.problem.N, w.problem.N)
    assert (sc.argmax(-1) == np.arange(w.problem.N)).all()


# ---------------------------------------------------------------- selection

def test_topk_matches_lexsort_and_ties_take_lowest_index():
    rng = np.random.default_rng(9)
    s = rng.random((50, 37))
    s[3, [4, 9, 20]] = 0.99999          # exact ties at the top
    s[4, :] = 0.5                         # all tied
    counts, idx = oracle.select_rows(s, Selection(0, 5))
    assert (counts == 5).all()
    s32 = s.astype(np.float32)
    for r in range(50):
        order = np.lexsort((np.arange(37), -s32[r].astype(np.float64)))
        assert np.array_equal(idx[r, :5], np.sort(order[:5]))
        assert (idx[r, 5:] == -1).all()
    assert np.array_equal(idx[4, :5], np.arange(5))
    assert {4, 9, 20} <= set(idx[3, :5])
    c2, i2 = oracle.select_rows(s, Selection(0, 100))   # k > N keeps all
    assert (c2 == 37).all() and np.array_equal(i2[0], np.arange(37))


def test_topk_decides_in_fp32():
    """Scores equal after fp32 rounding tie, and the lower index wins."""
    a = np.float64(np.float32(0.3))
    s = np.array([[a, a + 1e-12, 0.1]])
    _, idx = oracle.select_rows(s, Selection(0, 1))
    assert idx[0, 0] == 0


@pytest.mark.parametrize("mass,cap", [(0.9, 1000), (0.5, 1000), (0.9, 3), (1.0, 1000)])
def test_mass_selection_invariants(mass, cap):
    rng = np.random.default_rng(10)
    s = rng.lognormal(0, 2, (40, 64))
    counts, idx = oracle.select_rows(s, Selection(1, 0, mass, cap))
    s32 = s.astype(np.float32).astype(np.float64)
    for r in range(40):
        c = counts[r]
        sel = idx[r, :c]
        order = np.lexsort((np.arange(64), -s32[r]))
        assert np.array_equal(np.sort(order[:c]), sel)
        total = s32[r].sum()
        cum = np.cumsum(s32[r][order])
        c_full = int(np.argmax(cum >= mass * total)) + 1 if (cum >= mass * total).any() else 64
        assert c == min(c_full, cap)
        if c < cap:
            assert s32[r][sel].sum() >= mass * total * (1 - 1e-15)
            if c > 1:
                assert cum[c - 2] < mass * total


def test_sequence_topk_matches_flat_sort():
    rng = np.random.default_rng(11)
    N, k = 12, 3
    s = rng.random((2, N, N))
    s[0, 0, :4] = 0.999                      # ties resolved by flat index
    sel = oracle.select_seq(s, N, k)
    assert sel.reshape(2, -1).sum(1).tolist() == [N * k, N * k]
    for b in range(2):
        flat = s[b].reshape(-1).astype(np.float32).astype(np.float64)
        order = np.lexsort((np.arange(N * N), -flat))[: N * k]
        ref = np.zeros(N * N, bool)
        ref[order] = True
        assert np.array_equal(sel[b].reshape(-1), ref)


def test_csc_is_transpose_of_csr():
    p = small(hq=4, hkv=2, D=8)
    rng = np.random.default_rng(12)
    counts = rng.integers(0, p.N + 1, p.batch * p.heads_q * p.N).astype(np.int32)
    lists = [np.sort(rng.choice(p.N, c, replace=False)).astype(np.int32) for c in counts]
    idx = np.full((counts.size, p.N), -1, np.int32)
    for r, l in enumerate(lists):
        idx[r, :l.size] = l
    rp, ci = oracle.csr_from_selection(counts, idx)
    kp, ki = oracle.csr_to_csc(rp, ci, p)
    grp = p.heads_q // p.heads_kv
    pairs = set()
    for hkv in range(p.heads_kv):
        for nk in range(p.N):
            row = hkv * p.N + nk
            ent = ki[kp[row]:kp[row + 1]]
            assert np.all(np.diff(ent) > 0)
            for e in ent:
                pairs.add((hkv * grp + e // p.N, e % p.N, nk))
    ref = {(r // p.N, r % p.N, c) for r in range(counts.size) for c in lists[r]}
    assert pairs == ref


# ---------------------------------------------------------------- attention

def _block_mask(p, row_ptr, col_idx):
    """Token-level boolean mask [b, Hq, L, L] of the selected block pairs."""
    M = np.zeros((p.batch * p.heads_q, p.N, p.N), bool)
    for r in range(p.batch * p.heads_q * p.N):
        M[r // p.N, r % p.N, col_idx[row_ptr[r]:row_ptr[r + 1]]] = True
    M = np.repeat(np.repeat(M, p.B, 1), p.B, 2)
    return M.reshape(p.batch, p.heads_q, p.L, p.L)


def _torch_ref(q, k, v, p, mask, do=None):
    grp = p.heads_q // p.heads_kv
    tq = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    tk = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    tv = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    kk = tk.repeat_interleave(grp, 1)
    vv = tv.repeat_interleave(grp, 1)
    o = torch.nn.functional.scaled_dot_product_attention(
        tq, kk, vv, attn_mask=None if mask is None else torch.from_numpy(mask))
    s = (tq @ kk.transpose(-1, -2)) / math.sqrt(p.head_dim)
    if mask is not None:
        s = s.masked_fill(~torch.from_numpy(mask), float("-inf"))
    lse = torch.logsumexp(s, -1)
    grads = None
    if do is not None:
        o.backward(torch.from_numpy(do.astype(np.float64)))
        grads = (tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy())
    return o.detach().numpy(), lse.detach().numpy(), grads


def _full_csr(p):
    nrows = p.batch * p.heads_q * p.N
    rp = (np.arange(nrows + 1) * p.N).astype(np.int32)
    ci = np.tile(np.arange(p.N), nrows).astype(np.int32)
    return rp, ci


def _random_csr(p, seed, kmin=1):
    rng = np.random.default_rng(seed)
    nrows = p.batch * p.heads_q * p.N
    counts = rng.integers(kmin, p.N + 1, nrows)
    lists = [np.sort(rng.choice(p.N, c, replace=False)) for c in counts]
    rp = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return rp, np.concatenate(lists).astype(np.int32)


def test_fwd_all_blocks_is_full_attention():
    p = small(T=2, H=8, W=8, Bt=2, Bh=2, Bw=4, D=16)
    q, k, v, _ = rand_qkv(p, 13)
    rp, ci = _full_csr(p)
    o, lse = oracle.attn_fwd(q, k, v, p, rp, ci)
    ref, lref, _ = _torch_ref(q, k, v, p, None)
    np.testing.assert_allclose(o.reshape(ref.shape), ref, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse.reshape(lref.shape), lref, rtol=1e-13)


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_fwd_sparse_equals_dense_masked_softmax(hq, hkv):
    """The gathered form equals Softmax(S + M) V with M = -inf off the
    selected blocks (the paper's masked attention, Sec. 2.1)."""
    p = small(T=2, H=8, W=8, Bt=2, Bh=2, Bw=4, hq=hq, hkv=hkv, D=16)
    q, k, v, _ = rand_qkv(p, 14)
    rp, ci = _random_csr(p, 15)
    o, lse = oracle.attn_fwd(q, k, v, p, rp, ci)
    ref, lref, _ = _torch_ref(q, k, v, p, _block_mask(p, rp, ci))
    np.testing.assert_allclose(o.reshape(ref.shape), ref, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse.reshape(lref.shape), lref, rtol=1e-12)


def test_fwd_special_values():
    p = small(T=2, H=8, W=8, Bt=2, Bh=2, Bw=4, D=8)
    q, k, v, _ = rand_qkv(p, 16)
    rp, ci = _random_csr(p, 17)
    vc = np.broadcast_to(np.arange(p.head_dim, dtype=np.float32), v.shape).copy()
    o, _ = oracle.attn_fwd(q, k, vc, p, rp, ci)
    np.testing.assert_allclose(o, np.broadcast_to(np.arange(p.head_dim), o.shape), atol=1e-12)
    o0, lse0 = oracle.attn_fwd(np.zeros_like(q), k, v, p, rp, ci)
    for r in range(p.batch * p.heads_q * p.N):
        sel = ci[rp[r]:rp[r + 1]]
        keys = np.concatenate([np.arange(s * p.B, s * p.B + p.B) for s in sel])
        h = (r // p.N) % p.heads_q
        np.testing.assert_allclose(o0[r], np.broadcast_to(v[0, h, keys].astype(np.float64).mean(0),
                                                          o0[r].shape), atol=1e-12)
        np.testing.assert_allclose(lse0[r], math.log(keys.size), rtol=1e-14)
    # empty selection: O = 0, LSE = -inf
    rp_e = np.zeros(p.batch * p.heads_q * p.N + 1, np.int32)
    oe, le = oracle.attn_fwd(q, k, v, p, rp_e, np.zeros(0, np.int32))
    assert (oe == 0).all() and np.isneginf(le).all()


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_bwd_matches_autograd_of_masked_attention(hq, hkv):
    p = small(T=2, H=8, W=8, Bt=2, Bh=2, Bw=4, hq=hq, hkv=hkv, D=16)
    q, k, v, do = rand_qkv(p, 18)
    rp, ci = _random_csr(p, 19)
    _, _, (gq, gk, gv) = _torch_ref(q, k, v, p, _block_mask(p, rp, ci), do)
    dq = oracle.attn_bwd_dq(q, k, v, do, p, rp, ci)
    dk, dv = oracle.attn_bwd_dkdv(q, k, v, do, p, rp, ci)
    np.testing.assert_allclose(dq.reshape(gq.shape), gq, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dk.reshape(gk.shape), gk, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv.reshape(gv.shape), gv, rtol=1e-10, atol=1e-12)


def test_bwd_finite_differences():
    """Central differences of L = sum(dO * O) with the block lists held fixed."""
    p = Problem(1, 2, 1, 8, 2, 4, 4, 2, 2, 2, 1, 1, 2, BF16)
    q, k, v, do = rand_qkv(p, 20)
    rp, ci = _random_csr(p, 21)
    dq = oracle.attn_bwd_dq(q, k, v, do, p, rp, ci).reshape(q.shape)
    dk, dv = oracle.attn_bwd_dkdv(q, k, v, do, p, rp, ci)
    dk, dv = dk.reshape(k.shape), dv.reshape(v.shape)

    def loss(qq, kk, vv):
        o, _ = oracle.attn_fwd(qq, kk, vv, p, rp, ci)
        return float((o.reshape(qq.shape) * do.astype(np.float64)).sum())

    h = 2.0 ** -10     # bf16 inputs +/- h stay exact in float32
    rng = np.random.default_rng(22)
    for name, t, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for flat in rng.choice(t.size, 12, replace=False):
            tp, tm = t.copy(), t.copy()
            tp.flat[flat] += np.float32(h)
            tm.flat[flat] -= np.float32(h)
            args_p = {"q": q, "k": k, "v": v, name: tp}
            args_m = {"q": q, "k": k, "v": v, name: tm}
            fd = (loss(args_p["q"], args_p["k"], args_p["v"]) -
                  loss(args_m["q"], args_m["k"], args_m["v"])) / (2 * h)
            assert abs(fd - g.flat[flat]) <= 1e-5 * max(1.0, abs(g).max()), (name, flat)


def test_bwd_sum_invariants():
    """Rows of P sum to 1: sum_j dV_j = sum_i dO_i; rows of dS sum to 0:
    sum_j dK_j = 0 (per head, MHA)."""
    p = small(T=2, H=8, W=8, Bt=2, Bh=2, Bw=4, D=16)
    q, k, v, do = rand_qkv(p, 23)
    rp, ci = _random_csr(p, 24)
    dk, dv = oracle.attn_bwd_dkdv(q, k, v, do, p, rp, ci)
    dk = dk.reshape(p.heads_kv, -1, p.head_dim)
    dv = dv.reshape(p.heads_kv, -1, p.head_dim)
    np.testing.assert_allclose(dv.sum(1), do[0].astype(np.float64).sum(1), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dk.sum(1), 0.0, atol=1e-10)


# ---------------------------------------------------------------- paper table

def test_appendix_b_sparsity_reproduces_table2():
    """Appendix B's model 1 - (1/R^2 + K*B/L) gives Table 2's sparsity column
    with block B = 128 tokens and router pool R = 8 tokens (token counts from
    the evaluation setup, Sec. 3)."""
    with open(os.path.join(HERE, "golden", "table2_sparsity.json")) as f:
        g = json.load(f)
    for row in g["rows"]:
        s = 1.0 - (1.0 / g["R"] ** 2 + row["topk"] * g["B"] / row["tokens"])
        assert round(s, 2) == row["sparsity"], row


def test_mass_threshold_reached_exactly():
    """The prefix stops at the first count whose sum reaches (>=) the
    threshold; dyadic scores make the sums exact."""
    s = np.array([[0.25, 0.5, 0.125, 0.125], [0.125, 0.125, 0.25, 0.5]])
    counts, idx = oracle.select_rows(s, Selection(1, 0, 0.75, 10))
    assert counts.tolist() == [2, 2]
    assert idx[0, :2].tolist() == [0, 1] and idx[1, :2].tolist() == [2, 3]
    counts, _ = oracle.select_rows(s, Selection(1, 0, 0.875, 10))
    assert counts.tolist() == [3, 3]


# ---------------------------------------------------------------- coarse branch, gated merge

def _torch_coarse(qc, kc, vc, doc=None):
    """Dense softmax attention over the cube means with torch in float64,
    KV heads repeated over their query-head group."""
    grp = qc.shape[1] // kc.shape[1]
    tq = torch.tensor(qc, dtype=torch.float64, requires_grad=doc is not None)
    tk = torch.tensor(kc, dtype=torch.float64, requires_grad=doc is not None)
    tv = torch.tensor(vc, dtype=torch.float64, requires_grad=doc is not None)
    kk = tk.repeat_interleave(grp, dim=1)
    vv = tv.repeat_interleave(grp, dim=1)
    s = tq @ kk.transpose(-1, -2) / math.sqrt(qc.shape[-1])
    o = torch.softmax(s, -1) @ vv
    lse = torch.logsumexp(s, -1)
    grads = None
    if doc is not None:
        (o * torch.tensor(doc, dtype=torch.float64)).sum().backward()
        grads = (tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy())
    return o.detach().numpy(), lse.detach().numpy(), grads


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_coarse_branch_matches_torch(hq, hkv):
    """Coarse branch (Sec. 2.2, Eq. compress ff.): forward and gradients
    against torch float64 softmax attention and autograd, GQA included."""
    p = small(T=4, H=8, W=12, Bt=2, Bh=2, Bw=2, hq=hq, hkv=hkv, D=16)   # N = 48 cubes
    rng = np.random.default_rng(40)
    qc = rng.standard_normal((1, hq, p.N, p.head_dim)).astype(np.float32)
    kc = rng.standard_normal((1, hkv, p.N, p.head_dim)).astype(np.float32)
    vc = rng.standard_normal((1, hkv, p.N, p.head_dim)).astype(np.float32)
    doc = rng.standard_normal((1, hq, p.N, p.head_dim)).astype(np.float32)
    oc, lse = oracle.coarse_fwd(qc, kc, vc, p)
    ref, lref, (gq, gk, gv) = _torch_coarse(qc, kc, vc, doc)
    np.testing.assert_allclose(oc, ref, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, lref, rtol=1e-13)
    dqc, dkc, dvc = oracle.coarse_bwd(qc, kc, vc, doc, p)
    np.testing.assert_allclose(dqc, gq, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dkc, gk, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dvc, gv, rtol=1e-10, atol=1e-12)


def test_gate_merge_matches_torch_autograd():
    """O = tanh(g) * Repeat_B(O_c_hat) + O_f and its gradients (d O_c_hat
    sums the gated output gradient over each cube's B tokens)."""
    p = small(T=2, H=8, W=8, Bt=2, Bh=2, Bw=4, hq=3, hkv=3, D=8)
    rng = np.random.default_rng(41)
    g = (rng.standard_normal((1, 3, p.L)) * 2).astype(np.float32)
    oc = rng.standard_normal((1, 3, p.N, p.head_dim)).astype(np.float32)
    of = rng.standard_normal((1, 3, p.L, p.head_dim)).astype(np.float32)
    dout = rng.standard_normal((1, 3, p.L, p.head_dim)).astype(np.float32)
    out = oracle.gate_merge(g, oc, of, p)
    tg = torch.tensor(g, dtype=torch.float64, requires_grad=True)
    toc = torch.tensor(oc, dtype=torch.float64, requires_grad=True)
    tof = torch.tensor(of, dtype=torch.float64, requires_grad=True)
    ref = torch.tanh(tg)[..., None] * toc.repeat_interleave(p.B, dim=2) + tof
    np.testing.assert_allclose(out, ref.detach().numpy(), rtol=1e-14, atol=1e-14)
    (ref * torch.tensor(dout, dtype=torch.float64)).sum().backward()
    doc, dg = oracle.gate_merge_bwd(g, oc, dout, p)
    np.testing.assert_allclose(doc, toc.grad.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(tof.grad.numpy(), dout)      # d O_f = dout
    # zero gate weights (the paper's initialisation) leave only O_f
    np.testing.assert_array_equal(oracle.gate_merge(np.zeros_like(g), oc, of, p), of.astype(np.float64))


@pytest.mark.parametrize("P", [(2, 2, 2), (1, 2, 4), (2, 4, 4)])
def test_unpool_is_the_adjoint_of_pool(P):
    """<MeanPool(x), y> = <x, Unpool(y)>, and MeanPool(Unpool(y)) = y / P."""
    p = small(T=4, H=8, W=8, Bt=2, Bh=4, Bw=4, hq=2, hkv=2, D=8)
    Pt, Ph, Pw = P
    Gp = (p.Bt // Pt) * (p.Bh // Ph) * (p.Bw // Pw)
    rng = np.random.default_rng(42)
    # values on a 2^-12 grid: every pooled mean is exact in float32
    x = (rng.integers(-4096, 4096, (1, 2, p.L, p.head_dim)) / 4096.0).astype(np.float32)
    y = rng.standard_normal((1, 2, p.N * Gp, p.head_dim))
    px = oracle.pool(x, p, Pt, Ph, Pw).astype(np.float64)
    ux = oracle.unpool_add(y, np.zeros((1, 2, p.L, p.head_dim)), p, Pt, Ph, Pw)
    np.testing.assert_allclose((px * y).sum(), (x.astype(np.float64) * ux).sum(), rtol=1e-12)
    ones = (rng.integers(-64, 64, y.shape) / 8.0)
    back = oracle.pool(oracle.unpool_add(ones, np.zeros((1, 2, p.L, p.head_dim)), p, Pt, Ph, Pw)
                       .astype(np.float32), p, Pt, Ph, Pw)
    np.testing.assert_array_equal(back.astype(np.float64), ones / (Pt * Ph * Pw))


@pytest.mark.parametrize("grid_thw,text_len", [((2, 4, 4), 0), ((3, 3, 4), 0), ((3, 3, 4), 11)])
def test_full_op_gradient_finite_differences(grid_thw, text_len):
    """The whole VSA2 attention op O = tanh(g) Repeat_B(Attn(Pool_B Q, Pool_B K,
    Pool_B V)) + BlockSparseAttn(Q, K, V; M): gradients composed from the
    oracle's steps (merge, coarse and fine backward, unpool) against central
    differences of sum(W * O) over the real tokens.  The 3 x 3 x 4 grid is
    padded to 4 x 4 x 4: the gradient of every padding token is 0.  With 11
    text tokens (two blocks of 8, the second padded) the fine branch is the
    joint attention and text tokens keep O_f."""
    T, H, W_ = grid_thw
    p = Problem(1, 2, 1, 8, T, H, W_, 2, 2, 2, 1, 1, 2, F32, text_len)    # cubes of B = 8
    rng = np.random.default_rng(43)
    grid = lambda shape: (rng.integers(-1024, 1024, shape) / 1024.0).astype(np.float32)
    Lj = p.L_joint
    q = grid((1, 2, Lj, p.head_dim))
    k = grid((1, 1, Lj, p.head_dim))
    v = grid((1, 1, Lj, p.head_dim))
    g = grid((1, 2, Lj))
    W = rng.standard_normal((1, 2, Lj, p.head_dim)).astype(np.float32).astype(np.float64)
    W *= p.token_real()[None, None, :, None]           # padding tokens are not outputs
    rp, ci = _random_csr(p, 44)
    if text_len:
        rp, ci, _, _ = oracle.joint_lists(rp, ci, p)
    Bt, Bh, Bw = p.Bt, p.Bh, p.Bw

    def forward(qq, kk, vv, gg):
        # float64 end to end (the oracle's merge takes float inputs, whose
        # rounding would swamp the differences; the merge itself is pinned
        # against torch above)
        of, _ = oracle.attn_fwd(qq, kk, vv, p, rp, ci)
        oc, _ = oracle.coarse_fwd(oracle.pool(qq, p, Bt, Bh, Bw), oracle.pool(kk, p, Bt, Bh, Bw),
                                  oracle.pool(vv, p, Bt, Bh, Bw), p)
        gate = np.tanh(gg[..., :p.L].astype(np.float64))[..., None]
        out = of.reshape(qq.shape).copy()
        out[..., :p.L, :] += gate * np.repeat(oc, p.B, axis=2)
        return out

    def loss(*a):
        return float((forward(*a) * W).sum())

    # analytic gradient, step by step
    oc, _ = oracle.coarse_fwd(oracle.pool(q, p, Bt, Bh, Bw), oracle.pool(k, p, Bt, Bh, Bw),
                              oracle.pool(v, p, Bt, Bh, Bw), p)
    doc, dg = oracle.gate_merge_bwd(g, oc, W, p)
    dqc, dkc, dvc = oracle.coarse_bwd(oracle.pool(q, p, Bt, Bh, Bw), oracle.pool(k, p, Bt, Bh, Bw),
                                      oracle.pool(v, p, Bt, Bh, Bw), doc, p)
    dq = oracle.attn_bwd_dq(q, k, v, W, p, rp, ci).reshape(q.shape)
    dk, dv = oracle.attn_bwd_dkdv(q, k, v, W, p, rp, ci)
    dk, dv = dk.reshape(k.shape).copy(), dv.reshape(v.shape).copy()
    oracle.unpool_add(dqc, dq, p, Bt, Bh, Bw)
    oracle.unpool_add(dkc, dk, p, Bt, Bh, Bw)
    oracle.unpool_add(dvc, dv, p, Bt, Bh, Bw)
    h = 2.0 ** -10
    if p.padded:
        real = p.token_real()
        for gr in (dq, dk, dv):
            assert (gr[:, :, ~real] == 0).all()
        assert (dg[:, :, ~real] == 0).all()
    for name, t, gr in (("q", q, dq), ("k", k, dk), ("v", v, dv), ("g", g, dg)):
        for flat in rng.choice(t.size, 12, replace=False):
            args = {"q": q, "k": k, "v": v, "g": g}
            tp, tm = t.copy(), t.copy()
            tp.flat[flat] += np.float32(h)
            tm.flat[flat] -= np.float32(h)
            lp = loss(*[tp if n == name else args[n] for n in ("q", "k", "v", "g")])
            lm = loss(*[tm if n == name else args[n] for n in ("q", "k", "v", "g")])
            fd = (lp - lm) / (2 * h)
            assert abs(fd - gr.flat[flat]) <= 2e-5 * max(1.0, abs(gr).max()), (name, flat, fd,
                                                                                gr.flat[flat])


# ---------------------------------------------------------------- padded grids
# A grid not divisible by the cube is padded up to whole cubes; padding
# tokens are masked out everywhere (Sec. 2.2, kernel implementation).

def padded(T=3, H=5, W=6, Bt=2, Bh=2, Bw=4, Rt=1, Rh=2, Rw=2, hq=2, hkv=2, D=8, dtype=F32):
    p = Problem(1, hq, hkv, D, T, H, W, Bt, Bh, Bw, Rt, Rh, Rw, dtype)
    assert p.padded
    return p


def _garbage_padding(x, p, seed):
    """x with its padding tokens overwritten by large random values."""
    y = x.copy()
    real = p.token_real()
    y[..., ~real, :] = np.random.default_rng(seed).standard_normal(y[..., ~real, :].shape) * 50
    return y.astype(x.dtype)


@pytest.mark.parametrize("P", [(1, 2, 2), (2, 2, 4), (1, 1, 1), (2, 1, 2)])
def test_padded_pool_is_nanmean_over_real_tokens(P):
    """Each pooled row is the mean of the sub-cube's tokens that lie in the
    real grid (numpy nanmean over a NaN-padded grid); an all-padding sub-cube
    pools to 0."""
    p = padded()
    Pt, Ph, Pw = P
    rng = np.random.default_rng(50)
    xr = rng.standard_normal((1, 2, p.T * p.H * p.W, p.head_dim)).astype(np.float32)
    x = raster_to_cube_major(xr, p)
    out = oracle.pool(_garbage_padding(x, p, 51), p, Pt, Ph, Pw)
    g = np.full((1, 2, p.Nt * p.Bt, p.Nh * p.Bh, p.Nw * p.Bw, p.head_dim), np.nan)
    g[:, :, :p.T, :p.H, :p.W] = xr.reshape(1, 2, p.T, p.H, p.W, p.head_dim)
    Gt, Gh, Gw = p.Bt // Pt, p.Bh // Ph, p.Bw // Pw
    m = g.reshape(1, 2, p.Nt, Gt, Pt, p.Nh, Gh, Ph, p.Nw, Gw, Pw, p.head_dim)
    with np.errstate(all="ignore"):
        import warnings
        with warnings.catch_warnings():
            warnings.simplefilter("ignore", RuntimeWarning)
            m = np.nanmean(m, axis=(4, 7, 10))
    m = np.nan_to_num(m, nan=0.0)
    m = m.transpose(0, 1, 2, 4, 6, 3, 5, 7, 8).reshape(1, 2, -1, p.head_dim)
    np.testing.assert_array_equal(out, m.astype(np.float32))
    if P == (1, 1, 1):
        assert (out[..., ~p.token_real(), :] == 0).all()


def test_padded_router_ignores_padding_and_keeps_row_mass():
    """Scores do not depend on what padding tokens hold, every row sums to
    1/G, and with R = B the router is the cube-level softmax over the means of
    each cube's real tokens."""
    p = padded()
    q, k, _, _ = rand_qkv(p, 52, scale=2.0)
    pool = lambda x: oracle.pool(x, p, p.Rt, p.Rh, p.Rw)
    sc = oracle.router_scores(pool(q), pool(k), p)
    sc2 = oracle.router_scores(pool(_garbage_padding(q, p, 53)), pool(_garbage_padding(k, p, 54)), p)
    np.testing.assert_array_equal(sc, sc2)
    assert (sc >= 0).all()
    np.testing.assert_allclose(sc.sum(1), 1.0 / p.G, rtol=1e-12)
    # R = B (G = 1)
    pc = padded(Rt=2, Rh=2, Rw=4)
    real = pc.token_real().reshape(pc.N, pc.B)
    cnt = real.sum(1)[:, None]

    def cube_means(x):
        xx = x.astype(np.float64).reshape(1, -1, pc.N, pc.B, pc.head_dim) * real[None, None, :, :, None]
        return (xx.sum(3) / cnt).astype(np.float32)

    s1 = oracle.router_scores(oracle.pool(q, pc, 2, 2, 4), oracle.pool(k, pc, 2, 2, 4), pc)
    qc, kc = cube_means(q).astype(np.float64), cube_means(k).astype(np.float64)
    ref = _softmax64(np.einsum("bhid,bhjd->bhij", qc, kc) / math.sqrt(pc.head_dim))
    np.testing.assert_allclose(s1.reshape(ref.shape), ref, rtol=1e-12, atol=1e-15)


def test_padded_router_R_one_is_block_mean_over_real_tokens():
    """R = 1: P_r[nq, nk] is the mean over the real query tokens of cube nq
    of the softmax mass (over real keys only) that falls on cube nk, over B."""
    p = padded(Rt=1, Rh=1, Rw=1)
    q, k, _, _ = rand_qkv(p, 55)
    sc = oracle.router_scores(oracle.pool(q, p, 1, 1, 1), oracle.pool(k, p, 1, 1, 1), p)
    real = p.token_real()
    s = torch.from_numpy(np.einsum("bhid,bhjd->bhij", q.astype(np.float64), k.astype(np.float64))
                         / math.sqrt(p.head_dim))
    s = s.masked_fill(~torch.from_numpy(real)[None, None, None, :], float("-inf"))
    P = torch.softmax(s, -1).numpy().reshape(1, p.heads_q, p.N, p.B, p.N, p.B)
    rq = real.reshape(p.N, p.B)
    ref = (P * rq[None, None, :, :, None, None]).sum(axis=(3, 5)) / (p.B * rq.sum(1))[None, None, :, None]
    np.testing.assert_allclose(sc.reshape(ref.shape), ref, rtol=1e-12, atol=1e-16)


def _padded_mask(p, rp, ci):
    real = p.token_real()
    return _block_mask(p, rp, ci) & real[None, None, None, :]


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_padded_attention_matches_masked_sdpa(hq, hkv):
    """Forward and backward on a padded grid equal torch's masked attention
    with the padding keys masked out, on the real queries; padding queries
    give O = 0, LSE = -inf and dQ = 0, padding keys dK = dV = 0, and nothing
    depends on the padding tokens' contents."""
    p = padded(hq=hq, hkv=hkv)
    q, k, v, do = rand_qkv(p, 56)
    real = p.token_real()
    rp, ci = _random_csr(p, 57)
    o, lse = oracle.attn_fwd(q, k, v, p, rp, ci)
    o, lse = o.reshape(q.shape), lse.reshape(q.shape[:3])
    do_real = do * real[None, None, :, None]
    ref, lref, (gq, gk, gv) = _torch_ref(q, k, v, p, _padded_mask(p, rp, ci), do_real)
    np.testing.assert_allclose(o[:, :, real], ref[:, :, real], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse[:, :, real], lref[:, :, real], rtol=1e-12)
    assert (o[:, :, ~real] == 0).all() and np.isneginf(lse[:, :, ~real]).all()
    dq = oracle.attn_bwd_dq(q, k, v, do, p, rp, ci).reshape(q.shape)
    dk, dv = oracle.attn_bwd_dkdv(q, k, v, do, p, rp, ci)
    np.testing.assert_allclose(dq[:, :, real], gq[:, :, real], rtol=1e-10, atol=1e-12)
    assert (dq[:, :, ~real] == 0).all()
    np.testing.assert_allclose(dk.reshape(gk.shape), gk, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv.reshape(gv.shape), gv, rtol=1e-10, atol=1e-12)
    assert (dk.reshape(k.shape)[:, :, ~real] == 0).all() and (dv.reshape(v.shape)[:, :, ~real] == 0).all()
    gq_, gk_, gv_, gdo = (_garbage_padding(t, p, 58 + i) for i, t in enumerate((q, k, v, do)))
    o2, _ = oracle.attn_fwd(gq_, gk_, gv_, p, rp, ci)
    dq2 = oracle.attn_bwd_dq(gq_, gk_, gv_, gdo, p, rp, ci).reshape(q.shape)
    dk2, dv2 = oracle.attn_bwd_dkdv(gq_, gk_, gv_, gdo, p, rp, ci)
    np.testing.assert_array_equal(o2.reshape(q.shape), o)
    np.testing.assert_array_equal(dq2, dq)
    np.testing.assert_array_equal(dk2, dk)
    np.testing.assert_array_equal(dv2, dv)


def test_padded_gate_merge_bwd_ignores_padding_outputs():
    """Padding tokens are not outputs: the merge backward equals autograd of
    the merge restricted to real tokens (dg = 0 on padding)."""
    p = padded(hq=3, hkv=3)
    real = p.token_real()
    rng = np.random.default_rng(62)
    g = (rng.standard_normal((1, 3, p.L)) * 2).astype(np.float32)
    oc = rng.standard_normal((1, 3, p.N, p.head_dim)).astype(np.float32)
    dout = rng.standard_normal((1, 3, p.L, p.head_dim)).astype(np.float32)
    tg = torch.tensor(g, dtype=torch.float64, requires_grad=True)
    toc = torch.tensor(oc, dtype=torch.float64, requires_grad=True)
    out = torch.tanh(tg)[..., None] * toc.repeat_interleave(p.B, dim=2)
    (out[:, :, torch.from_numpy(real)] * torch.tensor(dout[:, :, real], dtype=torch.float64)).sum().backward()
    doc, dg = oracle.gate_merge_bwd(g, oc, dout, p)
    np.testing.assert_allclose(doc, toc.grad.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-12, atol=1e-13)
    assert (dg[:, :, ~real] == 0).all()


@pytest.mark.parametrize("P", [(2, 2, 4), (1, 2, 2), (1, 1, 1)])
def test_padded_unpool_is_the_adjoint_of_pool(P):
    """<MeanPool(x), y> = <x, Unpool(y)> for the count-aware pool, padding
    tokens receive nothing, and MeanPool(Unpool(y)) = y / (real tokens of the
    sub-cube)."""
    p = padded()
    Pt, Ph, Pw = P
    Gt, Gh, Gw = p.Bt // Pt, p.Bh // Ph, p.Bw // Pw
    Gp = Gt * Gh * Gw
    rng = np.random.default_rng(63)
    x = (rng.integers(-4096, 4096, (1, 2, p.L, p.head_dim)) / 4096.0).astype(np.float32)
    y = rng.standard_normal((1, 2, p.N * Gp, p.head_dim))
    px = oracle.pool(x, p, Pt, Ph, Pw).astype(np.float64)
    ux = oracle.unpool_add(y, np.zeros((1, 2, p.L, p.head_dim)), p, Pt, Ph, Pw)
    real = p.token_real()
    assert (ux[:, :, ~real] == 0).all()
    np.testing.assert_allclose((px * y).sum(), (x.astype(np.float64) * ux).sum(), rtol=1e-12)
    # real tokens per sub-cube, counted from the token mask
    rc = real.reshape(p.N, Gt, Pt, Gh, Ph, Gw, Pw).sum(axis=(2, 4, 6)).reshape(p.N * Gp)
    yy = rng.integers(-64, 64, y.shape) / 8.0
    back = oracle.pool(oracle.unpool_add(yy, np.zeros((1, 2, p.L, p.head_dim)), p, Pt, Ph, Pw)
                       .astype(np.float32), p, Pt, Ph, Pw).astype(np.float64)
    nz = rc > 0
    np.testing.assert_allclose(back[:, :, nz], yy[:, :, nz] / rc[nz][:, None], rtol=1e-6)
    assert (back[:, :, ~nz] == 0).all()


# ---------------------------------------------------------------- text tokens
# MMDiT joint attention: Eq. block_sparse extended with full video-to-text
# and text-to-video blocks (Sec. 2.2).  One (batch, head) sequence is the
# cube-major video followed by the text tokens padded to whole blocks.

def _joint_mask(p, rp, ci):
    """Token-level boolean mask [b, Hq, L_joint, L_joint] of the joint
    attention, built from the video block lists and the text rule directly."""
    L, Lj = p.L, p.L_joint
    M = np.zeros((p.batch, p.heads_q, Lj, Lj), bool)
    M[:, :, :L, :L] = _block_mask(p, rp, ci)       # routed video blocks
    M[:, :, :L, L:] = True                         # video queries see all text
    M[:, :, L:, :] = True                          # text queries see everything
    return M & p.token_real()[None, None, None, :]  # padding keys masked


@pytest.mark.parametrize("grid,text_len,hq,hkv", [((3, 5, 6), 37, 2, 2), ((4, 8, 8), 16, 4, 2),
                                                  ((2, 4, 8), 5, 2, 1)])
def test_joint_text_attention_matches_masked_sdpa(grid, text_len, hq, hkv):
    """Joint video + text attention (forward and backward) equals torch's
    masked SDPA over the concatenated tokens with: routed blocks among video
    tokens, every text token for video queries, every token for text
    queries, padding keys masked; padding queries (video or text) give
    O = 0, LSE = -inf, no gradient."""
    T, H, W = grid
    p = Problem(1, hq, hkv, 8, T, H, W, 2, 2, 4, 1, 2, 2, F32, text_len)
    q, k, v, do = rand_qkv_joint(p, 70)
    rp, ci = _random_csr(p, 71)
    jrp, jci, jkp, jki = oracle.joint_lists(rp, ci, p)
    assert jrp.size == p.batch * hq * p.N_joint + 1
    real = p.token_real()
    o, lse = oracle.attn_fwd(q, k, v, p, jrp, jci)
    o, lse = o.reshape(q.shape), lse.reshape(q.shape[:3])
    ref, lref, (gq, gk, gv) = _torch_ref(q, k, v, p, _joint_mask(p, rp, ci), do * real[None, None, :, None])
    np.testing.assert_allclose(o[:, :, real], ref[:, :, real], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse[:, :, real], lref[:, :, real], rtol=1e-12)
    assert (o[:, :, ~real] == 0).all() and np.isneginf(lse[:, :, ~real]).all()
    dq = oracle.attn_bwd_dq(q, k, v, do, p, jrp, jci).reshape(q.shape)
    dk, dv = oracle.attn_bwd_dkdv(q, k, v, do, p, jrp, jci)
    np.testing.assert_allclose(dq[:, :, real], gq[:, :, real], rtol=1e-10, atol=1e-12)
    assert (dq[:, :, ~real] == 0).all()
    np.testing.assert_allclose(dk.reshape(gk.shape), gk, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv.reshape(gv.shape), gv, rtol=1e-10, atol=1e-12)
    # the transposed joint lists are the transpose of the joint CSR
    grp = hq // hkv
    Nj = p.N_joint
    for kr in range(p.batch * hkv * Nj):
        bkv, nk = divmod(kr, Nj)
        want = [hl * Nj + nq for hl in range(grp) for nq in range(Nj)
                if nk in jci[jrp[(bkv * grp + hl) * Nj + nq]:jrp[(bkv * grp + hl) * Nj + nq + 1]]]
        assert list(jki[jkp[kr]:jkp[kr + 1]]) == want


def test_joint_text_rows_are_full_attention_and_text_len_zero_is_video_only():
    """A text query block attends to every real token (textbook softmax
    attention over the whole sequence), and with no text the joint lists are
    the video lists."""
    p = Problem(1, 2, 2, 8, 2, 4, 8, 2, 2, 4, 1, 2, 2, F32, 20)
    q, k, v, _ = rand_qkv_joint(p, 72)
    rp, ci = _random_csr(p, 73)
    jrp, jci, _, _ = oracle.joint_lists(rp, ci, p)
    o, _ = oracle.attn_fwd(q, k, v, p, jrp, jci)
    o = o.reshape(q.shape)
    real = p.token_real()
    s = np.einsum("bhid,bhjd->bhij", q.astype(np.float64), k.astype(np.float64)) / math.sqrt(p.head_dim)
    s[..., ~real] = -np.inf
    P = _softmax64(s)
    full = P @ v.astype(np.float64)
    tq = np.arange(p.L, p.L_joint)[real[p.L:]]
    np.testing.assert_allclose(o[:, :, tq], full[:, :, tq], rtol=1e-12, atol=1e-13)
    p0 = p.replace(text_len=0)
    jrp0, jci0, jkp0, jki0 = oracle.joint_lists(rp, ci, p0)
    kp0, ki0 = oracle.csr_to_csc(rp, ci, p0)
    assert np.array_equal(jrp0, rp) and np.array_equal(jci0, ci)
    assert np.array_equal(jkp0, kp0) and np.array_equal(jki0, ki0)


def rand_qkv_joint(p, seed):
    """rand_qkv over the joint sequence with padding tokens zeroed."""
    rng = np.random.default_rng(seed)
    shp = lambda h: (p.batch, h, p.L_joint, p.head_dim)
    q = rng.standard_normal(shp(p.heads_q)).astype(np.float32)
    k = rng.standard_normal(shp(p.heads_kv)).astype(np.float32)
    v = rng.standard_normal(shp(p.heads_kv)).astype(np.float32)
    do = rng.standard_normal(shp(p.heads_q)).astype(np.float32)
    real = p.token_real()
    for t in (q, k, v, do):
        t[..., ~real, :] = 0.0
    return q, k, v, do
