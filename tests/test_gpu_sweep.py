"""Seeded sweep of small random configurations through the whole fine path
against the oracle: grids that are and are not multiples of the cube
(padding), batch 1-2, GQA groups 1-4, D = 64 / 128, bf16 / fp32, the four
router pools the kernels support (G = 1, 2, 4, 8), top-k (k up to past N)
and mass selection, joint text tokens, and skewed (log-normal norm) inputs.
Per configuration: pooling bit-exact, the router's selection against the
oracle's (near ties excused and counted), and the training forward and the
backward over the oracle's block lists (joint lists with text) at the
element-wise bars.  The configurations are drawn from a fixed seed, so the
set is the same on every run."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32882_amd as vsa2
from parity import assert_values, check_seq_selection, compare_selection, to_dev, to_np
from sweep_cases import CASES, REGRESSION
from workload import BF16, Selection, make_inputs

pytestmark = pytest.mark.gpu


def dtname(p):
    return "bf16" if p.dtype == BF16 else "f32"


@pytest.mark.parametrize("w", CASES + REGRESSION, ids=[w.name for w in CASES + REGRESSION])
def test_random_configuration_against_oracle(w):
    p = w.problem
    print("\n[%s] %s %s skewed=%s" % (w.name, p, w.select, w.skewed), flush=True)
    x = make_inputs(w, with_grad=True)
    bf = p.dtype == BF16
    dev = {k: to_dev(v, bf) for k, v in x.items()}
    ref = oracle.route(x["q"], x["k"], p, w.select)

    # pooling and the router
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    r = vsa2.route(p, w.select, q_r, k_r, with_scores=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(q_r), ref["q_r"]) and np.array_equal(to_np(k_r), ref["k_r"])
    sc = to_np(r["scores"]).reshape(-1, p.N)
    big = ref["scores"] > 1e-20
    assert (np.abs(sc - ref["scores"])[big] / ref["scores"][big]).max() < 2e-5
    rp = r["row_ptr"].cpu().numpy()
    ci = r["col_idx"].cpu().numpy()
    counts, idx = oracle.select_rows(ref["scores"], w.select)
    print("selection:", compare_selection(rp, ci, counts, idx, ref["scores"], mass_mode=w.select.mode == 1,
                                          mass=w.select.mass))
    nnz = int(rp[-1])
    kp, ki = oracle.csr_to_csc(rp, ci[:nnz], p)
    assert np.array_equal(r["kv_ptr"].cpu().numpy(), kp)
    assert np.array_equal(r["kv_idx"].cpu().numpy()[:nnz], ki)

    # attention over the oracle's lists (joint lists with text tokens)
    if p.text_len:
        lrp, lci, lkp, lki = oracle.joint_lists(ref["row_ptr"], ref["col_idx"], p)
    else:
        lrp, lci, lkp, lki = ref["row_ptr"], ref["col_idx"], ref["kv_ptr"], ref["kv_idx"]
    t = [torch.from_numpy(a).cuda() for a in (lrp, lci, lkp, lki)]
    o, lse, o_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], t[0], t[1], training=True)
    g = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], t[0], t[1], t[2], t[3], o_lo=o_lo)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.attn_fwd(x["q"], x["k"], x["v"], p, lrp, lci)
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O", dtname(p))
    fin = np.isfinite(lse_ref)
    lse_np = to_np(lse).reshape(lse_ref.shape)
    assert np.array_equal(np.isfinite(lse_np), fin)
    assert np.abs(lse_np[fin] - lse_ref[fin]).max() < 1e-3
    dq_ref = oracle.attn_bwd_dq(x["q"], x["k"], x["v"], x["do"], p, lrp, lci)
    dk_ref, dv_ref = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, lrp, lci)
    for name, got, want in (("dQ", g[0], dq_ref), ("dK", g[1], dk_ref), ("dV", g[2], dv_ref)):
        assert_values(to_np(got).reshape(want.shape), want, name, dtname(p))


SEQ_K = {w.name: int(np.random.default_rng(w.seed).integers(1, w.problem.N + 2)) for w in CASES}


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_random_configuration_sequence_rule(w):
    """The per-sequence rule (the N k best pairs of each (batch, head)'s
    N x N block-score map, k drawn per configuration, up to past N) on the
    same configurations: the selection bit for bit against the oracle's flat
    sort of the GPU's own scores and within the near-tie window of the
    oracle's, the transposed lists exact, and the forward over the GPU's
    lists (rows of 0 .. N blocks) against the oracle's."""
    p = w.problem
    k = SEQ_K[w.name]
    print("\n[%s seq k=%d] %s" % (w.name, k, p), flush=True)
    x = make_inputs(w, with_grad=False)
    bf = p.dtype == BF16
    dev = {n: to_dev(x[n], bf) for n in ("q", "k", "v")}
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    r = vsa2.route(p, Selection(2, k), q_r, k_r, with_scores=True)
    torch.cuda.synchronize()
    rp = r["row_ptr"].cpu().numpy()
    ci = r["col_idx"].cpu().numpy()
    ref_scores = oracle.router_scores(to_np(q_r), to_np(k_r), p)
    check_seq_selection(p, k, rp, ci, ref_scores, r["scores"].cpu().numpy())
    nnz = int(rp[-1])
    kp, ki = oracle.csr_to_csc(rp, ci[:nnz], p)
    assert np.array_equal(r["kv_ptr"].cpu().numpy(), kp)
    assert np.array_equal(r["kv_idx"].cpu().numpy()[:nnz], ki)
    if p.text_len:
        lrp, lci, _, _ = oracle.joint_lists(rp, ci[:nnz], p)
    else:
        lrp, lci = rp, ci[:nnz]
    o, lse = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], torch.from_numpy(lrp).cuda(), torch.from_numpy(lci).cuda())
    torch.cuda.synchronize()
    o_ref, _ = oracle.attn_fwd(x["q"], x["k"], x["v"], p, lrp, lci)
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O (sequence rule)", dtname(p))
