"""GPU parity: the HIP path through the C-ABI against the CPU oracle on the
same seeded inputs, at sizes the oracle finishes in seconds (several tiles,
ragged router tiles, GQA, D = 64 and 128, fp32 and bf16, top-k and mass)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32882_amd as vsa2
from parity import assert_values, block_flags, check_seq_selection, compare_selection, to_dev, to_np
from workload import BF16, F32, Problem, Selection, Workload, WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def dtname(p):
    return "bf16" if p.dtype == BF16 else "f32"

CASES = {
    "tiny": WORKLOADS["tiny"],
    # N = 48 cubes, 384 pooled queries: one full and one ragged router tile
    "bf16-d128": Workload("bf16-d128", Problem(1, 2, 2, 128, 8, 16, 24), Selection(0, 12), 2001),
    "bf16-d64-gqa": Workload("bf16-d64-gqa", Problem(1, 4, 2, 64, 8, 16, 16), Selection(0, 6), 2002),
    "bf16-mass": Workload("bf16-mass", Problem(1, 2, 2, 128, 8, 16, 24), Selection(1, 0, 0.9, 20), 2003,
                          skewed=True),
    # k > N keeps every block: full attention; batch 2, 2 query heads on 1 KV head
    "bf16-full-b2": Workload("bf16-full-b2", Problem(2, 2, 1, 128, 4, 16, 16), Selection(0, 100), 2004),
    "f32-d128-mass": Workload("f32-d128-mass", Problem(1, 2, 1, 128, 4, 16, 16, dtype=F32),
                              Selection(1, 0, 0.5, 3), 2005, skewed=True),
    # router pool R = B (G = 1): the coarse cube-level router of VSA
    "bf16-router-R=B": Workload("bf16-router-R=B", Problem(1, 2, 2, 128, 8, 16, 24, Rt=4, Rh=4, Rw=4),
                                Selection(0, 12), 2006),
    # R = 2x2x4 (G = 4), GQA
    "bf16-router-G4": Workload("bf16-router-G4", Problem(1, 4, 2, 64, 8, 16, 16, Rt=2, Rh=2, Rw=4),
                               Selection(0, 6), 2007),
    # grids that are not multiples of the 4x4x4 cube, padded up to whole cubes
    # with the padding masked: cut along all three axes (N = 2*4*6 = 48) ...
    "bf16-padded": Workload("bf16-padded", Problem(1, 2, 2, 128, 7, 13, 22), Selection(0, 12), 2008),
    # ... GQA at D = 64 with mass selection on skewed inputs (N = 2*3*4) ...
    "f32-padded-gqa-mass": Workload("f32-padded-gqa-mass", Problem(1, 4, 2, 64, 5, 10, 15, dtype=F32),
                                    Selection(1, 0, 0.9, 12), 2009, skewed=True),
    # ... and one frame (T = 1 < Bt: 16 real tokens per cube, half of the
    # pooled sub-cubes empty), router pool 2x2x4 (G = 4), N = 5*5
    "bf16-padded-1frame-G4": Workload("bf16-padded-1frame-G4",
                                      Problem(1, 2, 2, 128, 1, 18, 20, Rt=2, Rh=2, Rw=4), Selection(0, 6), 2010),
}
PADDED = [name for name, w in CASES.items() if w.problem.padded]


@pytest.fixture(scope="module", params=list(CASES))
def case(request):
    w = CASES[request.param]
    p = w.problem
    print("\n[case %s] %s" % (w.name, p), flush=True)
    x = make_inputs(w, with_grad=True)
    ref = oracle.route(x["q"], x["k"], p, w.select)
    bf = p.dtype == BF16
    dev = {k: to_dev(v, bf) for k, v in x.items()}
    return w, x, ref, dev


def test_pool_matches_oracle(case):
    w, x, ref, dev = case
    p = w.problem
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    torch.cuda.synchronize()
    assert np.array_equal(to_np(q_r), ref["q_r"])
    assert np.array_equal(to_np(k_r), ref["k_r"])
    # coarse-branch pooling (P = B) of V as well
    v_c = vsa2.pool(p, dev["v"], (p.Bt, p.Bh, p.Bw))
    assert np.array_equal(to_np(v_c), oracle.pool(x["v"], p, p.Bt, p.Bh, p.Bw))


def test_route_matches_oracle(case):
    w, x, ref, dev = case
    p = w.problem
    bf = p.dtype == BF16
    r = vsa2.route(p, w.select, to_dev(ref["q_r"], bf), to_dev(ref["k_r"], bf), with_scores=True)
    torch.cuda.synchronize()
    sc = to_np(r["scores"]).reshape(-1, p.N)
    err = np.abs(sc - ref["scores"]) / (np.abs(ref["scores"]) + 1e-30)
    big = ref["scores"] > 1e-20
    print("scores: max rel err %.3e" % err[big].max())
    assert err[big].max() < 2e-5
    rp = r["row_ptr"].cpu().numpy()
    ci = r["col_idx"].cpu().numpy()
    assert rp[0] == 0 and (np.diff(rp) >= 0).all()
    nnz = int(rp[-1])
    for i in range(rp.size - 1):
        seg = ci[rp[i]:rp[i + 1]]
        assert (np.diff(seg) > 0).all() and (seg >= 0).all() and (seg < p.N).all()
    counts, idx = oracle.select_rows(ref["scores"], w.select)
    st = compare_selection(rp, ci, counts, idx, ref["scores"], mass_mode=w.select.mode == 1,
                           mass=w.select.mass)
    print("selection:", st)
    # the transposed lists are exact index work on the GPU's own CSR
    kp, ki = oracle.csr_to_csc(rp, ci[:nnz], p)
    assert np.array_equal(r["kv_ptr"].cpu().numpy(), kp)
    assert np.array_equal(r["kv_idx"].cpu().numpy()[:nnz], ki)


def test_fwd_matches_oracle(case):
    w, x, ref, dev = case
    p = w.problem
    rp = torch.from_numpy(ref["row_ptr"]).cuda()
    ci = torch.from_numpy(ref["col_idx"]).cuda()
    o, lse = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], rp, ci)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.attn_fwd(x["q"], x["k"], x["v"], p, ref["row_ptr"], ref["col_idx"])
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O", dtname(p))
    assert_values(to_np(lse).reshape(lse_ref.shape), lse_ref, "LSE", "f32", max_abs=1e-3, rel_l2=1e-5)


def test_end_to_end_path(case):
    """pool -> route -> fwd on the GPU, against the oracle's whole path."""
    w, x, ref, dev = case
    p = w.problem
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    r = vsa2.route(p, w.select, q_r, k_r)
    o, lse = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], r["row_ptr"], r["col_idx"])
    torch.cuda.synchronize()
    rp = r["row_ptr"].cpu().numpy()
    ci = r["col_idx"].cpu().numpy()[:rp[-1]]
    # the oracle forward on the GPU's own block lists (near-ties may differ)
    o_ref, _ = oracle.attn_fwd(x["q"], x["k"], x["v"], p, rp, ci)
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O (end to end)", dtname(p))


def test_fwd_deterministic_and_writes_everything(case):
    w, x, ref, dev = case
    p = w.problem
    rp = torch.from_numpy(ref["row_ptr"]).cuda()
    ci = torch.from_numpy(ref["col_idx"]).cuda()
    o1 = torch.full_like(dev["q"], float("nan"))
    l1 = torch.full((p.batch, p.heads_q, p.L), float("nan"), device="cuda")
    vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], rp, ci, o=o1, lse=l1)
    o2, l2 = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], rp, ci)
    torch.cuda.synchronize()
    assert not torch.isnan(o1).any() and not torch.isnan(l1).any()
    assert torch.equal(o1.view(torch.int16) if o1.dtype == torch.bfloat16 else o1.view(torch.int32),
                       o2.view(torch.int16) if o2.dtype == torch.bfloat16 else o2.view(torch.int32))
    assert torch.equal(l1, l2)


def test_fwd_empty_rows_and_malformed_entries():
    """Rows with no block give O = 0 and LSE = -inf; entries outside [0, N)
    are skipped."""
    w = CASES["bf16-d128"]
    p = w.problem
    x = make_inputs(w, with_grad=False)
    rng = np.random.default_rng(5)
    nrows = p.batch * p.heads_q * p.N
    counts = rng.integers(0, 5, nrows)
    counts[::7] = 0
    lists = [np.sort(rng.choice(p.N, c, replace=False)).astype(np.int32) for c in counts]
    rp = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    ci = np.concatenate(lists).astype(np.int32)
    bad = ci.copy()
    bad_pos = rng.choice(ci.size, 10, replace=False)
    bad[bad_pos] = np.where(np.arange(10) % 2 == 0, -3, p.N + 5)
    keep = np.ones(ci.size, bool)
    keep[bad_pos] = False
    rp_clean = np.concatenate([[0], np.cumsum([keep[rp[r]:rp[r + 1]].sum() for r in range(nrows)])]).astype(np.int32)
    o_ref, lse_ref = oracle.attn_fwd(x["q"], x["k"], x["v"], p, rp_clean, ci[keep])
    dq, dk, dv = (to_dev(x[t], True) for t in ("q", "k", "v"))
    o, lse = vsa2.attn_fwd(p, dq, dk, dv, torch.from_numpy(rp).cuda(), torch.from_numpy(bad).cuda())
    torch.cuda.synchronize()
    o_np, lse_np = to_np(o).reshape(o_ref.shape), to_np(lse).reshape(lse_ref.shape)
    empty = np.diff(rp_clean) == 0
    assert (o_np[empty] == 0).all() and np.isneginf(lse_np[empty]).all()
    assert_values(o_np, o_ref, "O (ragged rows)")
    assert np.allclose(lse_np[~empty], lse_ref[~empty], atol=1e-3)


def _bwd_inputs(case):
    """The forward of a training step (it keeps O's rounding remainder)."""
    w, x, ref, dev = case
    p = w.problem
    t = {k: torch.from_numpy(ref[k]).cuda() for k in ("row_ptr", "col_idx", "kv_ptr", "kv_idx")}
    o, lse, o_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], t["row_ptr"], t["col_idx"], training=True)
    return w, x, ref, dev, t, o, lse, o_lo


def test_bwd_matches_oracle(case):
    """Gradients against the oracle, element-wise and relative-L2, on every
    case (the skewed ones included: their large-magnitude blocks take the
    two-term products)."""
    w, x, ref, dev, t, o, lse, o_lo = _bwd_inputs(case)
    p = w.problem
    dq, dk, dv = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], t["row_ptr"],
                               t["col_idx"], t["kv_ptr"], t["kv_idx"], o_lo=o_lo)
    torch.cuda.synchronize()
    dq_ref = oracle.attn_bwd_dq(x["q"], x["k"], x["v"], x["do"], p, ref["row_ptr"], ref["col_idx"])
    dk_ref, dv_ref = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, ref["row_ptr"],
                                          ref["col_idx"])
    for name, got, want in (("dQ", dq, dq_ref), ("dK", dk, dk_ref), ("dV", dv, dv_ref)):
        assert_values(to_np(got).reshape(want.shape), want, name, dtname(p))


def test_bwd_staged_matches_whole_call(case):
    """prep + dK/dV + dQ as separate C-ABI calls give the same bits as
    vsa2_attn_bwd."""
    w, x, ref, dev, t, o, lse, o_lo = _bwd_inputs(case)
    p = w.problem
    args = (p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], t["row_ptr"], t["col_idx"],
            t["kv_ptr"], t["kv_idx"])
    a = vsa2.attn_bwd(*args, o_lo=o_lo)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    b = vsa2.attn_bwd_staged(*args, o_lo=o_lo, marks=marks)
    torch.cuda.synchronize()
    for x1, x2 in zip(a, b):
        iv = torch.int16 if x1.dtype == torch.bfloat16 else torch.int32
        assert torch.equal(x1.view(iv), x2.view(iv))
    assert all(marks[i].elapsed_time(marks[i + 1]) >= 0 for i in range(3))


def test_training_forward_remainder(case):
    """o + o_lo is the fp32 result: on query blocks with a large-magnitude
    value (every pair two-term) it matches the oracle's O to ~2^-16
    relative; elsewhere P enters P.V rounded to bf16 on the pairs of small
    blocks, so |o + o_lo - O| <= 2^-9 max|V| (sum_j p_j = 1) plus the fp32
    slack.  o itself meets the same bar as the inference forward's, which
    it equals bit for bit wherever no pair was two-term."""
    w, x, ref, dev = case
    p = w.problem
    rp = torch.from_numpy(ref["row_ptr"]).cuda()
    ci = torch.from_numpy(ref["col_idx"]).cuda()
    o1, _ = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], rp, ci)
    o2, _, o_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], rp, ci, training=True)
    torch.cuda.synchronize()
    o_ref, _ = oracle.attn_fwd(x["q"], x["k"], x["v"], p, ref["row_ptr"], ref["col_idx"])
    full = (to_np(o2).astype(np.float64) + to_np(o_lo)).reshape(o_ref.shape)
    scale = max(1.0, np.abs(o_ref).max())
    err = np.abs(full - o_ref).reshape(p.batch, p.heads_q, p.N, p.B, p.head_dim)
    if p.dtype == BF16:
        fq, fkv = block_flags(x, p)
        flagged = np.broadcast_to(fq[..., None, None], err.shape)
        vmax = np.abs(x["v"]).max()
        print("O + o_lo: max err %.3e on flagged query blocks (%d), %.3e elsewhere (bound %.3e)"
              % (err[flagged].max() if flagged.any() else 0.0, int(fq.sum()),
                 err[~flagged].max() if (~flagged).any() else 0.0, 2.0 ** -9 * vmax))
        if flagged.any():
            assert err[flagged].max() < 2e-5 * scale
        assert err.max() <= 2.0 ** -9 * vmax + 2e-5 * scale
    else:
        print("O + o_lo max rel err %.3e" % (err.max() / scale))
        assert err.max() < 1e-5 * scale
    assert_values(to_np(o2).reshape(o_ref.shape), o_ref, "O (training)", dtname(p))
    assert_values(to_np(o1).reshape(o_ref.shape), o_ref, "O (inference)", dtname(p))


def test_bwd_deterministic_sentinels_and_unselected_blocks(case):
    """Bitwise repeatable; every output element written (NaN sentinels);
    key blocks no query selected get dK = dV = 0."""
    w, x, ref, dev, t, o, lse, o_lo = _bwd_inputs(case)
    p = w.problem
    args = (p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], t["row_ptr"], t["col_idx"],
            t["kv_ptr"], t["kv_idx"])
    s = [torch.full_like(dev[k], float("nan")) for k in ("q", "k", "v")]
    vsa2.attn_bwd(*args, dq=s[0], dk=s[1], dv=s[2], o_lo=o_lo)
    r2 = vsa2.attn_bwd(*args, o_lo=o_lo)
    torch.cuda.synchronize()
    for a, b in zip(s, r2):
        assert not torch.isnan(a).any()
        iv = torch.int16 if a.dtype == torch.bfloat16 else torch.int32
        assert torch.equal(a.view(iv), b.view(iv))
    indeg = np.diff(ref["kv_ptr"])
    dk_np = to_np(s[1]).reshape(-1, p.B, p.head_dim)
    dv_np = to_np(s[2]).reshape(-1, p.B, p.head_dim)
    assert (dk_np[indeg == 0] == 0).all() and (dv_np[indeg == 0] == 0).all()


def test_block_flags_rule():
    """The large-magnitude flags the backward writes (index work, bit-exact):
    a block is flagged iff a real token holds a value above 7 in magnitude
    (7 itself is not), padding tokens never count, K and V flag their key
    block together, and the per-KV-group summary words say whether any block
    of the group is flagged (prep stage); the row byte of a query block
    holds its own flag (bit 0) and, in bit 1, whether its block list touches
    a flagged block, its own flag included, or one of its queries has
    |Delta| = |dO . (O + o_lo)| above 16, with one word per KV group saying
    whether any of the group's query blocks has bit 1 (dK/dV stage)."""
    a256 = lambda n: (n + 255) // 256 * 256
    for name in ("bf16-padded", "bf16-d64-gqa", "bf16-mass"):
        w = CASES[name]
        p = w.problem
        x = make_inputs(w, with_grad=True)
        real = p.token_real()
        tok = np.flatnonzero(real)
        x["q"][0, 0, tok[3], 5] = 7.0                 # exactly 7: not flagged
        x["q"][0, p.heads_q - 1, tok[-1], 2] = -7.03125  # just above (next bf16 value): flagged
        x["v"][0, 0, tok[200], 0] = 9.0               # V flags its key block
        if p.padded:                                   # padding never counts
            x["k"][0, 1, np.flatnonzero(~real)[0], 7] = 100.0
        fq, fkv = block_flags(x, p)
        # O (passed as o and as o_lo, so O + o_lo = 2 O): zero, except a
        # multiple of dO at a few real queries, far above (2.0) and far below
        # (0.02) the Delta threshold
        o_np = np.zeros_like(x["q"])
        for hh, t, c in ((0, tok[70], 2.0), (p.heads_q - 1, tok[len(tok) // 2], 2.0), (1, tok[5], 0.02)):
            o_np[0, hh, t] = x["do"][0, hh, t] * c
        dev = {k: to_dev(v, True) for k, v in x.items()}
        P = vsa2.problem_from(p)
        st, bwsb = vsa2.vsa2_attn_workspace(P, 1)
        assert st == 0
        bws = torch.zeros(bwsb, dtype=torch.uint8, device="cuda")
        o = to_dev(o_np, True)
        lse = torch.zeros(p.batch, p.heads_q, p.L, dtype=torch.float32, device="cuda")
        st = vsa2.vsa2_attn_bwd_prep(P, dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(),
                                     o.data_ptr(), lse.data_ptr(), o.data_ptr(), dev["do"].data_ptr(),
                                     bws.data_ptr(), bwsb, 0)
        assert st == 0
        ref = oracle.route(x["q"], x["k"], p, w.select)
        lists = {k: torch.from_numpy(ref[k]).cuda() for k in ("kv_ptr", "kv_idx")}
        dk, dv = torch.empty_like(dev["k"]), torch.empty_like(dev["v"])
        st = vsa2.vsa2_attn_bwd_dkdv(P, dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(),
                                     dev["do"].data_ptr(), lists["kv_ptr"].data_ptr(), lists["kv_idx"].data_ptr(),
                                     lists["kv_idx"].numel(), dk.data_ptr(), dv.data_ptr(), bws.data_ptr(), bwsb, 0)
        assert st == 0
        torch.cuda.synchronize()
        nq, nkv, groups = p.batch * p.heads_q * p.N, p.batch * p.heads_kv * p.N, p.batch * p.heads_kv
        off = a256(8 * nq * p.B) + a256(4 * nq) + a256(4 * nkv)
        raw = bws.cpu().numpy()
        got_q = raw[off:off + nq]
        got_kv = raw[off + a256(nq):off + a256(nq) + nkv]
        words = raw[off + a256(nq) + a256(nkv):][:8 * groups].view(np.int32)
        print("[flags %s] query blocks %d / %d, key blocks %d / %d" % (name, int(fq.sum()), nq, int(fkv.sum()),
                                                                       nkv))
        assert np.array_equal(got_q, fq.reshape(-1).astype(np.uint8))
        assert np.array_equal(got_kv, fkv.reshape(-1).astype(np.uint8))
        grp = p.heads_q // p.heads_kv
        any_q = fq.reshape(p.batch, p.heads_kv, grp * p.N).any(-1).reshape(-1)
        any_kv = fkv.reshape(groups, p.N).any(-1)
        assert np.array_equal(words[:groups], any_q.astype(np.int32))
        assert np.array_equal(words[groups:], any_kv.astype(np.int32))
        # row flags: own flag, or some block of the row's list flagged
        rp, ci = ref["row_ptr"], ref["col_idx"]
        fq_flat, fkv_flat = fq.reshape(-1), fkv.reshape(-1)
        rowf = np.zeros(nq, bool)
        for r in range(nq):
            bh = r // p.N
            kvbase = ((bh // p.heads_q) * p.heads_kv + (bh % p.heads_q) // grp) * p.N
            rowf[r] = fq_flat[r] or fkv_flat[kvbase + ci[rp[r]:rp[r + 1]]].any()
        ob = to_np(o).astype(np.float64)
        delta = (2 * ob * to_np(dev["do"]).astype(np.float64)).sum(-1)     # [b, h, L]
        assert np.all((np.abs(delta) > 40) | (np.abs(delta) < 8))          # far from the threshold
        dbig = (np.abs(delta) > 16).reshape(nq, p.B).any(-1)
        assert dbig.sum() == 2
        rowf |= dbig
        qoff = off + a256(nq) + a256(nkv) + a256(8 * groups)
        got_row = raw[qoff:qoff + nq]
        any_row = raw[qoff + a256(nq):][:4 * groups].view(np.int32)
        print("   row flags: %d / %d query blocks" % (int(rowf.sum()), nq))
        assert np.array_equal(got_row, (fq_flat.astype(np.uint8) | (2 * rowf).astype(np.uint8)))
        assert np.array_equal(any_row, rowf.reshape(p.batch, p.heads_kv, grp * p.N).any(-1).reshape(-1).astype(np.int32))
        assert fq.reshape(-1)[p.heads_q * p.N - 1] and fkv[0, 0, tok[200] // p.B]


def _fill_padding(t, p, seed):
    """Copy of t [batch, heads, L, D] with its padding tokens set to large
    random values."""
    real = torch.from_numpy(p.token_real()).cuda()
    g = torch.Generator(device="cuda").manual_seed(seed)
    noise = (torch.randn(t.shape, generator=g, device="cuda") * 40).to(t.dtype)
    return torch.where(real[None, None, :, None], t, noise)


@pytest.mark.parametrize("name", PADDED)
def test_padding_contents_do_not_matter(name):
    """Padding tokens are masked everywhere: with large random values in the
    padding of Q, K, V and dO, pooling, routing, the forward and the backward
    give the same bits on real tokens as with zero padding, and padding
    queries / keys get O = 0, LSE = -inf, dQ = dK = dV = 0."""
    w = CASES[name]
    p = w.problem
    print("\n[padding case %s] %s" % (name, p), flush=True)
    x = make_inputs(w, with_grad=True)
    bf = p.dtype == BF16
    clean = {k: to_dev(v, bf) for k, v in x.items()}
    dirty = {k: _fill_padding(v, p, i + 1) for i, (k, v) in enumerate(clean.items())}
    real = torch.from_numpy(p.token_real()).cuda()
    outs = []
    for d in (clean, dirty):
        R = (p.Rt, p.Rh, p.Rw)
        q_r, k_r = vsa2.pool(p, d["q"], R), vsa2.pool(p, d["k"], R)
        r = vsa2.route(p, w.select, q_r, k_r, with_scores=True)
        o, lse, o_lo = vsa2.attn_fwd(p, d["q"], d["k"], d["v"], r["row_ptr"], r["col_idx"], training=True)
        g = vsa2.attn_bwd(p, d["q"], d["k"], d["v"], o, lse, d["do"], r["row_ptr"], r["col_idx"],
                          r["kv_ptr"], r["kv_idx"], o_lo=o_lo)
        outs.append(dict(q_r=q_r, k_r=k_r, scores=r["scores"], rp=r["row_ptr"], ci=r["col_idx"], o=o, lse=lse,
                         o_lo=o_lo, dq=g[0], dk=g[1], dv=g[2]))
    torch.cuda.synchronize()
    a, b = outs
    bits = {torch.bfloat16: torch.int16, torch.float32: torch.int32, torch.int32: torch.int32}
    nnz = int(a["rp"][-1])
    a["ci"], b["ci"] = a["ci"][:nnz], b["ci"][:nnz]
    for k in ("q_r", "k_r", "scores", "rp", "ci", "o", "lse", "o_lo", "dq", "dk", "dv"):
        assert torch.equal(a[k].view(bits[a[k].dtype]), b[k].view(bits[b[k].dtype])), k
    pad = ~real
    assert (a["o"][:, :, pad] == 0).all() and torch.isneginf(a["lse"][:, :, pad]).all()
    assert (a["dq"][:, :, pad] == 0).all()
    assert (a["dk"][:, :, pad] == 0).all() and (a["dv"][:, :, pad] == 0).all()
    assert torch.isfinite(a["lse"][:, :, real]).all()


def test_bwd_unselected_blocks_are_zero_explicit():
    """A block list that leaves most key blocks unselected."""
    w = CASES["bf16-d128"]
    p = w.problem
    x = make_inputs(w, with_grad=True)
    nrows = p.batch * p.heads_q * p.N
    rp = (np.arange(nrows + 1) * 2).astype(np.int32)
    ci = np.tile(np.array([3, 17], np.int32), nrows)
    kp, ki = oracle.csr_to_csc(rp, ci, p)
    dev = {k: to_dev(v, True) for k, v in x.items()}
    tt = [torch.from_numpy(a).cuda() for a in (rp, ci, kp, ki)]
    o, lse, o_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], tt[0], tt[1], training=True)
    dq, dk, dv = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], *tt, o_lo=o_lo)
    torch.cuda.synchronize()
    dk_np = to_np(dk).reshape(p.heads_kv, p.N, p.B, p.head_dim)
    mask = np.ones(p.N, bool)
    mask[[3, 17]] = False
    assert (dk_np[:, mask] == 0).all() and (to_np(dv).reshape(dk_np.shape)[:, mask] == 0).all()
    dk_ref, dv_ref = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, rp, ci)
    assert_values(to_np(dk).reshape(dk_ref.shape), dk_ref, "dK (two blocks)")
    assert_values(to_np(dv).reshape(dv_ref.shape), dv_ref, "dV (two blocks)")


def _check_lpt_order(order, lengths, n_per_head):
    """order is a permutation of each segment where one of the 8 XCD ranges
    meets one head's rows, longest length class first (class = len * 32 //
    (max_len + 1) over the segment) and in row order inside a class."""
    n = lengths.size
    q, r = divmod(n, 8)
    cuts = sorted(set([x * q + min(x, r) for x in range(9)] + list(range(0, n + 1, n_per_head))))
    for beg, end in zip(cuts[:-1], cuts[1:]):
        if end <= beg:
            continue
        seg = order[beg:end].astype(np.int64)
        assert np.array_equal(np.sort(seg), np.arange(beg, end))
        ln = lengths[seg]
        cls = ln * 32 // (lengths[beg:end].max() + 1)
        assert (np.diff(cls) <= 0).all()
        same = np.diff(cls) == 0
        assert (np.diff(seg)[same] > 0).all()


def test_work_order_and_ragged_rows():
    """Rows of very different lengths (0 to N entries): the forward and the
    backward put each XCD's rows longest first in their workspaces, and the
    outputs still match the oracle (empty rows: O = 0, LSE = -inf)."""
    w = CASES["bf16-d128"]
    p = w.problem
    x = make_inputs(w, with_grad=True)
    rng = np.random.default_rng(11)
    nrows = p.batch * p.heads_q * p.N
    counts = rng.choice([0, 1, 2, 5, 17, p.N], size=nrows, p=[0.1, 0.2, 0.2, 0.2, 0.2, 0.1])
    rp = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    ci = np.concatenate([np.sort(rng.choice(p.N, c, replace=False)) for c in counts]).astype(np.int32)
    kp, ki = oracle.csr_to_csc(rp, ci, p)
    dev = {k: to_dev(v, True) for k, v in x.items()}
    t = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda()
         for k, v in (("rp", rp), ("ci", ci), ("kp", kp), ("ki", ki))}
    P = vsa2.problem_from(p)
    st, fws = vsa2.vsa2_attn_workspace(P, 0)
    assert st == 0
    ws = torch.full((fws // 4,), -7, dtype=torch.int32, device="cuda")
    o = torch.empty_like(dev["q"])
    o_lo = torch.empty_like(dev["q"])
    lse = torch.empty(p.batch, p.heads_q, p.L, dtype=torch.float32, device="cuda")
    st = vsa2.vsa2_attn_fwd(P, dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(),
                            t["rp"].data_ptr(), t["ci"].data_ptr(), t["ci"].numel(), o.data_ptr(),
                            lse.data_ptr(), o_lo.data_ptr(), ws.data_ptr(), fws, 0)
    assert st == 0
    dq, dk, dv = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], t["rp"], t["ci"],
                               t["kp"], t["ki"], o_lo=o_lo)
    torch.cuda.synchronize()
    _check_lpt_order(ws.cpu().numpy()[:nrows], np.diff(rp).astype(np.int64), p.N)
    # the backward's CSC order, read from a workspace of the staged call
    a256 = lambda n: (n + 255) // 256 * 256
    off = a256(8 * nrows * p.B) + a256(4 * nrows)
    nkv = p.batch * p.heads_kv * p.N
    bws = torch.empty(vsa2.vsa2_attn_workspace(P, 1)[1], dtype=torch.uint8, device="cuda")
    st = vsa2.vsa2_attn_bwd_prep(P, dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(), o.data_ptr(),
                                 lse.data_ptr(), o_lo.data_ptr(), dev["do"].data_ptr(), bws.data_ptr(),
                                 bws.numel(), 0)
    assert st == 0
    st = vsa2.vsa2_attn_bwd_dkdv(P, dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(),
                                 dev["do"].data_ptr(), t["kp"].data_ptr(), t["ki"].data_ptr(),
                                 t["ki"].numel(), torch.empty_like(dk).data_ptr(),
                                 torch.empty_like(dv).data_ptr(), bws.data_ptr(), bws.numel(), 0)
    assert st == 0
    torch.cuda.synchronize()
    kv_order = bws[off:off + 4 * nkv].view(torch.int32).cpu().numpy()
    _check_lpt_order(kv_order, np.diff(kp).astype(np.int64), p.N)
    o_ref, lse_ref = oracle.attn_fwd(x["q"], x["k"], x["v"], p, rp, ci)
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O (ragged rows)")
    empty = np.repeat(counts == 0, p.B)
    assert np.isneginf(lse.cpu().numpy().reshape(-1)[empty]).all()
    dq_ref = oracle.attn_bwd_dq(x["q"], x["k"], x["v"], x["do"], p, rp, ci)
    dk_ref, dv_ref = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, rp, ci)
    for name, got, want in (("dQ", dq, dq_ref), ("dK", dk, dk_ref), ("dV", dv, dv_ref)):
        assert_values(to_np(got).reshape(want.shape), want, name + " (ragged rows)")


@pytest.mark.parametrize("k", [3, 11])
def test_route_sequence_topk_matches_oracle(case, k):
    w, x, ref, dev = case
    p = w.problem
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    r = vsa2.route(p, Selection(2, k), q_r, k_r, with_scores=True)
    torch.cuda.synchronize()
    rp = r["row_ptr"].cpu().numpy()
    ci = r["col_idx"].cpu().numpy()
    check_seq_selection(p, k, rp, ci, ref["scores"], r["scores"].cpu().numpy())
    kp, ki = oracle.csr_to_csc(rp, ci[:rp[-1]], p)
    assert np.array_equal(r["kv_ptr"].cpu().numpy(), kp)
    assert np.array_equal(r["kv_idx"].cpu().numpy()[:rp[-1]], ki)


def test_route_sequence_topk_all_ties():
    """Zero pooled queries and keys make every block score equal: the rule
    keeps the first N*k pairs in flat order, i.e. rows 0 .. k-1 whole and
    nothing else; the forward then gives O = 0, LSE = -inf on the empty rows."""
    w = CASES["bf16-d128"]
    p = w.problem
    N = p.N
    k = 5
    z_q = torch.zeros(p.batch, p.heads_q, N * p.G, p.head_dim, dtype=torch.bfloat16, device="cuda")
    z_k = torch.zeros(p.batch, p.heads_kv, N * p.G, p.head_dim, dtype=torch.bfloat16, device="cuda")
    r = vsa2.route(p, Selection(2, k), z_q, z_k, with_scores=True)
    torch.cuda.synchronize()
    rp = r["row_ptr"].cpu().numpy()
    ci = r["col_idx"].cpu().numpy()
    sc = r["scores"].cpu().numpy()
    assert (sc == sc.reshape(-1)[0]).all()
    counts = np.diff(rp).reshape(-1, N)
    assert (counts[:, :k] == N).all() and (counts[:, k:] == 0).all()
    check_seq_selection(p, k, rp, ci, sc.astype(np.float64), sc)
    x = make_inputs(w, with_grad=False)
    d = {n: to_dev(x[n], True) for n in ("q", "k", "v")}
    o, lse = vsa2.attn_fwd(p, d["q"], d["k"], d["v"], r["row_ptr"], r["col_idx"])
    torch.cuda.synchronize()
    lse_np = lse.cpu().numpy().reshape(-1, N, p.B)
    assert np.isneginf(lse_np[:, k:]).all() and np.isfinite(lse_np[:, :k]).all()
    assert (to_np(o).reshape(-1, N, p.B, p.head_dim)[:, k:] == 0).all()
