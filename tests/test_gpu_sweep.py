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
from parity import assert_values, compare_selection, to_dev, to_np
from workload import BF16, F32, Problem, Selection, Workload, make_inputs

pytestmark = pytest.mark.gpu

N_CASES = 24
POOLS = [(2, 2, 2), (4, 4, 4), (2, 2, 4), (2, 4, 4)]     # G = 8, 1, 4, 2


def _draw(i, rng):
    heads_kv = int(rng.integers(1, 3))
    grp = int(rng.choice([1, 2, 4]))
    if heads_kv * grp > 4:
        grp = 2
    D = int(rng.choice([64, 128]))
    dtype = F32 if rng.random() < 0.2 else BF16
    T, H, W = int(rng.integers(1, 10)), int(rng.integers(4, 21)), int(rng.integers(4, 25))
    Rt, Rh, Rw = POOLS[int(rng.integers(0, len(POOLS)))]
    text = int(rng.integers(1, 141)) if rng.random() < 0.3 else 0
    p = Problem(int(rng.integers(1, 3)), heads_kv * grp, heads_kv, D, T, H, W, Rt=Rt, Rh=Rh, Rw=Rw,
                dtype=dtype, text_len=text)
    if rng.random() < 0.6:
        sel = Selection(0, int(rng.integers(1, p.N + 4)))
    else:
        sel = Selection(1, 0, float(rng.choice([0.5, 0.9, 0.99])), int(rng.integers(1, p.N + 1)))
    return Workload("sweep%02d" % i, p, sel, 9100 + i, skewed=bool(rng.random() < 0.3))


def _cases():
    rng = np.random.default_rng(9000)
    return [_draw(i, rng) for i in range(N_CASES)]


CASES = _cases()

# Skewed configurations drawn by the same generator from another seed, where
# two-term dS only on the pairs that touch a flagged block, and a softmax
# denominator summed from the unrounded probabilities, left dQ or dK above
# the bar (errors 1.0-2.1x the 2e-2 bar, rel-L2 up to 1.35e-2): rows whose
# other blocks are flagged (their large Delta makes every dS of the row
# large), and single-block rows with a peaked softmax (P's rounding in O
# reaches every dS of the row through Delta).
REGRESSION = [
    Workload("peaked-top1", Problem(1, 4, 2, 64, 1, 5, 13, Rt=4, Rh=4, Rw=4), Selection(0, 1), 3100, skewed=True),
    Workload("mixed-rows-mass", Problem(1, 4, 2, 128, 5, 11, 14, Rt=2, Rh=2, Rw=4), Selection(1, 0, 0.5, 14), 3107,
             skewed=True),
    Workload("peaked-cap1", Problem(1, 4, 1, 128, 3, 19, 8, Rt=4, Rh=4, Rw=4), Selection(1, 0, 0.99, 1), 3110,
             skewed=True),
    Workload("mixed-rows-b2", Problem(2, 4, 2, 64, 6, 10, 12), Selection(0, 16), 3112, skewed=True),
    Workload("mixed-rows-cap5", Problem(2, 4, 2, 128, 2, 14, 5, Rt=4, Rh=4, Rw=4), Selection(1, 0, 0.9, 5), 3115,
             skewed=True),
    # a query block with values up to 7.06 in a row with no flagged block
    # and a peaked softmax (cap 2): over the bar with the magnitude threshold
    # at 8 even under the rules above
    Workload("near-threshold-cap2", Problem(1, 4, 2, 64, 9, 10, 11, Rt=4, Rh=4, Rw=4), Selection(1, 0, 0.9, 2), 3326,
             skewed=True),
]


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
