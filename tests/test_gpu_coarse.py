"""GPU parity of the coarse branch, the gated merge and the MeanPool adjoint
(Sec. 2.2 "Coarse Branch", "Gated Merge") against the oracle, step by step
and as the whole VSA2 attention op (coarse + fine + merge, forward and
backward)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32882_amd as vsa2
from parity import assert_values, assert_values_bound, attn_fp32_logit_bounds, to_dev, to_np
from sweep_cases import CASES as SWEEP_CASES
from workload import BF16, F32, Problem, Selection, Workload, make_inputs

pytestmark = pytest.mark.gpu

CASES = {
    # N = 48 cubes: one ragged 64-row tile
    "bf16-d128-n48": Workload("c1", Problem(1, 2, 2, 128, 8, 16, 24), Selection(0, 12), 3001),
    # N = 96: a full tile and a ragged one; GQA
    "bf16-d64-gqa-n96": Workload("c2", Problem(1, 4, 2, 64, 8, 32, 24), Selection(0, 9), 3002),
    # a single cube
    "bf16-d128-n1": Workload("c3", Problem(1, 2, 1, 128, 4, 4, 4), Selection(0, 1), 3003),
    "f32-d64-n32": Workload("c4", Problem(1, 2, 2, 64, 8, 16, 16, dtype=F32), Selection(0, 8), 3004),
    # two batches, N = 130: three tiles, the last with 2 rows
    "bf16-d128-b2-n130": Workload("c5", Problem(2, 2, 2, 128, 8, 260, 4), Selection(0, 20), 3005,
                                  skewed=True),
    # grids padded up to whole cubes: cut along every axis (N = 48), and one
    # frame (T = 1) with GQA and a 2x2x4 router pool
    "bf16-d128-padded": Workload("c6", Problem(1, 2, 2, 128, 7, 13, 22), Selection(0, 12), 3006),
    "f32-d64-padded-1frame-gqa": Workload("c7", Problem(1, 4, 2, 64, 1, 18, 20, Rt=2, Rh=2, Rw=4, dtype=F32),
                                          Selection(0, 6), 3007),
}


# ten text-free configurations of the fine path's seeded random sweep
CASES.update({w.name: w for w in [c for c in SWEEP_CASES if c.problem.text_len == 0][:10]})


def dtname(p):
    return "bf16" if p.dtype == BF16 else "f32"


@pytest.fixture(scope="module", params=list(CASES))
def case(request):
    w = CASES[request.param]
    p = w.problem
    print("\n[coarse case %s] %s" % (request.param, p), flush=True)
    x = make_inputs(w, with_grad=True)
    bf = p.dtype == BF16
    dev = {k: to_dev(v, bf) for k, v in x.items()}
    rng = np.random.default_rng(w.seed)
    gate = (rng.standard_normal((p.batch, p.heads_q, p.L)) * 1.5).astype(np.float32)
    return w, x, dev, gate


def _pooled(p, dev):
    P = (p.Bt, p.Bh, p.Bw)
    return tuple(vsa2.pool(p, dev[n], P) for n in ("q", "k", "v"))


def test_coarse_forward_and_backward(case):
    w, x, dev, _ = case
    p = w.problem
    qc, kc, vc = _pooled(p, dev)
    oc, lse = vsa2.coarse_fwd(p, qc, kc, vc)
    rng = np.random.default_rng(5)
    doc_np = rng.standard_normal(tuple(oc.shape)).astype(np.float32)
    doc = to_dev(doc_np, p.dtype == BF16)
    dqc, dkc, dvc = vsa2.coarse_bwd(p, qc, kc, vc, doc)
    torch.cuda.synchronize()
    qn, kn, vn = (to_np(t) for t in (qc, kc, vc))
    oc_ref, lse_ref = oracle.coarse_fwd(qn, kn, vn, p)
    assert_values(to_np(oc), oc_ref, "O_c_hat", dtname(p))
    assert_values(lse.cpu().numpy(), lse_ref, "LSE_c", "f32", max_abs=1e-3, rel_l2=1e-5)
    # both sides take the same (rounded) dO_c_hat
    dq_ref, dk_ref, dv_ref = oracle.coarse_bwd(qn, kn, vn, to_np(doc), p)
    assert_values(to_np(dqc), dq_ref, "dQ_c", dtname(p))
    assert_values(to_np(dkc), dk_ref, "dK_c", dtname(p))
    assert_values(to_np(dvc), dv_ref, "dV_c", dtname(p))


def test_gate_merge_forward_and_backward(case):
    w, x, dev, gate = case
    p = w.problem
    bf = p.dtype == BF16
    rng = np.random.default_rng(6)
    oc_np = rng.standard_normal((p.batch, p.heads_q, p.N, p.head_dim)).astype(np.float32)
    oc = to_dev(oc_np, bf)
    g = torch.from_numpy(gate).cuda()
    out = vsa2.gate_merge(p, g, oc, dev["q"])
    doc, dg = vsa2.gate_merge_bwd(p, g, oc, dev["do"])
    torch.cuda.synchronize()
    ocv = to_np(oc)
    ref = oracle.gate_merge(gate, ocv, x["q"], p)
    assert_values(to_np(out), ref, "merged O", dtname(p))
    doc_ref, dg_ref = oracle.gate_merge_bwd(gate, ocv, x["do"], p)
    assert_values(to_np(doc), doc_ref, "dO_c_hat", dtname(p))
    assert_values(dg.cpu().numpy(), dg_ref, "dgate", "f32", max_abs=1e-3, rel_l2=1e-5)
    # zero gate pre-activations leave O_f untouched, bit for bit
    out0 = vsa2.gate_merge(p, torch.zeros_like(g), oc, dev["q"])
    torch.cuda.synchronize()
    iv = torch.int16 if bf else torch.int32
    assert torch.equal(out0.view(iv), dev["q"].view(iv))


@pytest.mark.parametrize("which", ["B", "R"])
def test_unpool_add(case, which):
    w, x, dev, _ = case
    p = w.problem
    P = (p.Bt, p.Bh, p.Bw) if which == "B" else (p.Rt, p.Rh, p.Rw)
    Gp = (p.Bt // P[0]) * (p.Bh // P[1]) * (p.Bw // P[2])
    rng = np.random.default_rng(7)
    dxc_np = rng.standard_normal((p.batch, p.heads_q, p.N * Gp, p.head_dim)).astype(np.float32)
    bf = p.dtype == BF16
    dxc = to_dev(dxc_np, bf)
    dx = dev["do"].clone()
    vsa2.unpool_add(p, dxc, dx, P)
    torch.cuda.synchronize()
    ref = oracle.unpool_add(to_np(dxc).astype(np.float64), x["do"].astype(np.float64).copy(), p, *P)
    assert_values(to_np(dx), ref, "dx + unpool(dx_c)", dtname(p))


def test_whole_op_forward_and_backward(case):
    """O = tanh(g) Repeat_B(Attn(Pool_B Q, Pool_B K, Pool_B V)) +
    BlockSparseAttn(Q, K, V; M), M from the fine router, and dQ, dK, dV, dg
    for a random dO: GPU step chain against the oracle's step chain."""
    w, x, dev, gate = case
    p = w.problem
    bf = p.dtype == BF16
    ref_route = oracle.route(x["q"], x["k"], p, w.select)
    rp, ci = ref_route["row_ptr"], ref_route["col_idx"]
    kp, ki = ref_route["kv_ptr"], ref_route["kv_idx"]
    t = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in
         (("rp", rp), ("ci", ci), ("kp", kp), ("ki", ki))}
    g = torch.from_numpy(gate).cuda()
    # forward
    qc, kc, vc = _pooled(p, dev)
    oc, lse_c = vsa2.coarse_fwd(p, qc, kc, vc)
    of, lse_f, of_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], t["rp"], t["ci"], training=True)
    o = vsa2.gate_merge(p, g, oc, of)
    # backward
    doc, dg = vsa2.gate_merge_bwd(p, g, oc, dev["do"])
    dqc, dkc, dvc = vsa2.coarse_bwd(p, qc, kc, vc, doc)
    dq, dk, dv = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], of, lse_f, dev["do"], t["rp"],
                               t["ci"], t["kp"], t["ki"], o_lo=of_lo)
    P = (p.Bt, p.Bh, p.Bw)
    vsa2.unpool_add(p, dqc, dq, P)
    vsa2.unpool_add(p, dkc, dk, P)
    vsa2.unpool_add(p, dvc, dv, P)
    torch.cuda.synchronize()

    # the oracle's chain
    qcr = oracle.pool(x["q"], p, *P)
    kcr = oracle.pool(x["k"], p, *P)
    vcr = oracle.pool(x["v"], p, *P)
    oc_r, _ = oracle.coarse_fwd(qcr, kcr, vcr, p)
    of_r, _ = oracle.attn_fwd(x["q"], x["k"], x["v"], p, rp, ci)
    o_r = oracle.gate_merge(gate, oc_r, of_r.reshape(x["q"].shape), p)
    # the merge reads O_c_hat and O_f as dtype outputs of the two branches:
    # their rounding is relative to |tanh(g) O_c_hat| + |O_f|, which can be
    # much larger than |O| when the two cancel (large-norm cube means)
    # The scores (and dP) of both branches are fp32 sums of D products; with
    # large-norm cube means (skewed: scores in the thousands) their rounding
    # alone moves the outputs by more than 2e-2.  Every element is held to
    # 2e-2 + its output rounding + the derived first-order bound of that
    # fp32 accumulation (tests/parity.py, attn_fp32_logit_bounds), per branch.
    doc_r, dg_r = oracle.gate_merge_bwd(gate, oc_r, x["do"], p)
    dqc_r, dkc_r, dvc_r = oracle.coarse_bwd(qcr, kcr, vcr, doc_r, p)
    D = p.head_dim
    sc = 1.0 / np.sqrt(D)
    grp = p.heads_q // p.heads_kv
    f64 = lambda a: np.asarray(a, np.float64)
    real = p.token_real()[:p.L]
    ebO, ebQ = np.zeros(x["q"].shape), np.zeros(x["q"].shape)
    ebK, ebV = np.zeros(x["k"].shape), np.zeros(x["v"].shape)
    for b in range(p.batch):
        for h in range(p.heads_q):
            hk = h // grp
            for n in range(p.N):
                r = (b * p.heads_q + h) * p.N + n
                sel = ci[rp[r]:rp[r + 1]]
                if sel.size == 0:
                    continue
                keys = (sel[:, None] * p.B + np.arange(p.B)[None, :]).reshape(-1)
                qs = slice(n * p.B, (n + 1) * p.B)
                e = attn_fp32_logit_bounds(f64(x["q"][b, h, qs]), f64(x["k"][b, hk, keys]), f64(x["v"][b, hk, keys]),
                                           f64(x["do"][b, h, qs]), sc, D, real[keys])
                ebO[b, h, qs] += e[0]
                ebQ[b, h, qs] += e[1]
                np.add.at(ebK[b, hk], keys, e[2])
                np.add.at(ebV[b, hk], keys, e[3])
    # the coarse branch's bounds, spread to the tokens of each cube (the
    # MeanPool adjoint divides by the cube's real-token count)
    cnt = real.reshape(p.N, p.B).sum(1).astype(np.float64)
    th_all = np.abs(np.tanh(gate.astype(np.float64)))
    ebOc = np.zeros(oc_r.shape)
    for b in range(p.batch):
        for h in range(p.heads_q):
            hk = h // grp
            e = attn_fp32_logit_bounds(f64(qcr[b, h]), f64(kcr[b, hk]), f64(vcr[b, hk]), f64(doc_r[b, h]), sc, D)
            ebOc[b, h] = e[0]
            ebO[b, h] += th_all[b, h][:, None] * np.repeat(e[0], p.B, axis=0)
            ebQ[b, h] += np.repeat(e[1] / cnt[:, None], p.B, axis=0)
            ebK[b, hk] += np.repeat(e[2] / cnt[:, None], p.B, axis=0)
            ebV[b, hk] += np.repeat(e[3] / cnt[:, None], p.B, axis=0)
    for eb in (ebO, ebQ, ebK, ebV):
        eb *= real[None, None, :, None]
    # three roundings to the dtype (u = 2^-8 for bf16): O_c_hat and O_f as
    # the branches' outputs, then the merged O
    th = th_all[..., None]
    scale = th * np.repeat(np.abs(oc_r), p.B, axis=2) + np.abs(of_r.reshape(x["q"].shape)) + np.abs(o_r)
    ulp = 2.0 ** -8 if bf else 2.0 ** -23
    err = np.abs(to_np(o).astype(np.float64) - o_r)
    bound = 2e-2 + ulp * scale + ebO
    print("O (whole op): max err %.3e, max err / bound %.3f (max fp32-score bound %.3e)" % (
        err.max(), (err / bound).max(), ebO.max()))
    assert (err <= bound).all()
    assert_values(to_np(o), o_r, "O (whole op, rel-L2)", dtname(p), max_abs=float("inf"))
    dq_r = oracle.attn_bwd_dq(x["q"], x["k"], x["v"], x["do"], p, rp, ci).reshape(x["q"].shape)
    dk_r, dv_r = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, rp, ci)
    dk_r, dv_r = dk_r.reshape(x["k"].shape).copy(), dv_r.reshape(x["v"].shape).copy()
    dq_r = dq_r.copy()
    # the fine gradients and the coarse ones spread to the tokens are each
    # rounded to the dtype before they are added (then the sum is rounded)
    parts = []
    for fine, coarse in ((dq_r, dqc_r), (dk_r, dkc_r), (dv_r, dvc_r)):
        spread = oracle.unpool_add(coarse, np.zeros(fine.shape), p, *P)
        parts.append(ulp * (np.abs(fine) + np.abs(spread)))
        oracle.unpool_add(coarse, fine, p, *P)
    for name, got, want, eb, rnd in (("dQ", dq, dq_r, ebQ, parts[0]), ("dK", dk, dk_r, ebK, parts[1]),
                                     ("dV", dv, dv_r, ebV, parts[2])):
        assert_values_bound(to_np(got), want, name + " (whole op)", dtname(p), eb + rnd)
    # dgate = (1 - tanh^2) dO . O_c_hat reads the bf16-rounded O_c_hat: its
    # error is bounded by the rounding (2^-9 relative per element, 2^-8 with
    # the bf16 dO product) of each term, i.e. relative to sum |dO| |O_c_hat|
    # rather than to the (cancelling) dot product itself
    th = np.tanh(gate.astype(np.float64))
    absdot = np.einsum("bhnte,bhne->bhnt",
                       np.abs(x["do"].astype(np.float64)).reshape(p.batch, p.heads_q, p.N, p.B, -1),
                       np.abs(oc_r)).reshape(dg_r.shape)
    # plus the fp32-score bound of O_c_hat (1 - tanh^2) sum |dO| e(O_c_hat)
    absdot_e = np.einsum("bhnte,bhne->bhnt",
                         np.abs(x["do"].astype(np.float64)).reshape(p.batch, p.heads_q, p.N, p.B, -1),
                         ebOc).reshape(dg_r.shape)
    bound = 2e-2 + (1.0 - th * th) * (2.0 ** -8 * absdot + absdot_e)
    err = np.abs(dg.cpu().numpy().astype(np.float64) - dg_r)
    print("dgate (whole op): max err %.3e, max err / bound %.3f" % (err.max(), (err / bound).max()))
    assert (err <= bound).all()
    assert_values(dg.cpu().numpy(), dg_r, "dgate (whole op)", "f32", max_abs=float("inf"), rel_l2=1e-2)


@pytest.mark.slow
def test_coarse_branch_fullsize_720p():
    """The coarse branch and the merge at the 720p shape (N = 1200 cubes,
    40 heads): two sampled heads against the oracle, every output written."""
    from workload import WORKLOADS
    w = WORKLOADS["720p"]
    p = w.problem
    x = make_inputs(w, with_grad=True)
    dev = {k: to_dev(v, True) for k, v in x.items()}
    P = (p.Bt, p.Bh, p.Bw)
    qc, kc, vc = (vsa2.pool(p, dev[n], P) for n in ("q", "k", "v"))
    oc, lse = vsa2.coarse_fwd(p, qc, kc, vc)
    rng = np.random.default_rng(8)
    gate = (rng.standard_normal((p.batch, p.heads_q, p.L)) * 1.5).astype(np.float32)
    g = torch.from_numpy(gate).cuda()
    o = vsa2.gate_merge(p, g, oc, dev["v"][:, :p.heads_q].contiguous())
    doc, dg = vsa2.gate_merge_bwd(p, g, oc, dev["do"])
    dqc, dkc, dvc = vsa2.coarse_bwd(p, qc, kc, vc, doc)
    torch.cuda.synchronize()
    for t in (oc, lse, o, doc, dg, dqc, dkc, dvc):
        assert torch.isfinite(t.float()).all()
    heads = [5, 33]
    sub = p.replace(heads_q=len(heads), heads_kv=len(heads))
    pick = lambda t: to_np(t[:, heads].contiguous())
    qn, kn, vn = pick(qc), pick(kc), pick(vc)
    oc_r, lse_r = oracle.coarse_fwd(qn, kn, vn, sub)
    assert_values(pick(oc), oc_r, "O_c_hat (720p, sampled heads)")
    assert_values(lse[:, heads].cpu().numpy(), lse_r, "LSE_c", "f32", max_abs=1e-3, rel_l2=1e-5)
    doc_n = pick(doc)
    dq_r, dk_r, dv_r = oracle.coarse_bwd(qn, kn, vn, doc_n, sub)
    assert_values(pick(dqc), dq_r, "dQ_c (720p, sampled heads)")
    assert_values(pick(dkc), dk_r, "dK_c (720p, sampled heads)")
    assert_values(pick(dvc), dv_r, "dV_c (720p, sampled heads)")
    gs = np.ascontiguousarray(gate[:, heads])
    doc_r, dg_r = oracle.gate_merge_bwd(gs, pick(oc), np.ascontiguousarray(x["do"][:, heads]), sub)
    assert_values(doc_n, doc_r, "dO_c_hat (720p, sampled heads)")
    assert_values(dg[:, heads].cpu().numpy(), dg_r, "dgate", "f32", max_abs=1e-3, rel_l2=1e-5)
    o_r = oracle.gate_merge(gs, pick(oc), np.ascontiguousarray(x["v"][:, heads]), sub)
    assert_values(pick(o), o_r, "merged O (720p, sampled heads)")
