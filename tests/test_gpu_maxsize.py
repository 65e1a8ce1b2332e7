"""GPU parity at the router's maximum block count: N = 4096 cubes per head
(grid 64 x 64 x 64, 262,144 tokens), the largest N the router and the
selection accept (each lane of a selection wave then holds 64 scores).  The
oracle recomputes sampled router rows and query / key blocks; the CSR and
CSC are checked whole.  (A larger grid is rejected on the host: test_abi.)"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32882_amd as vsa2
from parity import assert_values, compare_selection, to_dev, to_np
from workload import Problem, Selection, Workload, make_inputs

pytestmark = pytest.mark.gpu

MAXN = {
    "topk": Workload("max-topk", Problem(1, 2, 1, 64, 64, 64, 64), Selection(0, 17), 8001),
    "mass": Workload("max-mass", Problem(1, 1, 1, 64, 64, 64, 64), Selection(1, 0, 0.5, 40), 8002, skewed=True),
    "seq": Workload("max-seq", Problem(1, 1, 1, 64, 64, 64, 64), Selection(2, 9), 8003),
}


@pytest.mark.parametrize("name", list(MAXN))
def test_router_and_attention_at_the_largest_block_count(name):
    w = MAXN[name]
    p = w.problem
    assert p.N == 4096
    print("\n[max N %s] %s %s" % (name, p, w.select), flush=True)
    x = make_inputs(w, with_grad=True)
    dev = {k: to_dev(v, True) for k, v in x.items()}
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    r = vsa2.route(p, w.select, q_r, k_r, with_scores=True)
    o, lse, o_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], r["row_ptr"], r["col_idx"], training=True)
    g = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], r["row_ptr"], r["col_idx"],
                      r["kv_ptr"], r["kv_idx"], o_lo=o_lo)
    torch.cuda.synchronize()
    qr_ref = oracle.pool(x["q"], p, p.Rt, p.Rh, p.Rw)
    kr_ref = oracle.pool(x["k"], p, p.Rt, p.Rh, p.Rw)
    assert np.array_equal(to_np(q_r), qr_ref) and np.array_equal(to_np(k_r), kr_ref)
    rp = r["row_ptr"].cpu().numpy()
    nnz = int(rp[-1])
    ci = r["col_idx"].cpu().numpy()[:nnz]
    nrows = p.batch * p.heads_q * p.N
    counts = np.diff(rp)
    if w.select.mode == 0:
        assert (counts == w.select.k).all()
    elif w.select.mode == 1:
        assert counts.min() >= 1 and counts.max() <= w.select.cap
    else:
        assert (counts.reshape(-1, p.N).sum(1) == p.N * w.select.k).all()
    kp, ki = oracle.csr_to_csc(rp, ci, p)
    assert np.array_equal(r["kv_ptr"].cpu().numpy(), kp)
    assert np.array_equal(r["kv_idx"].cpu().numpy()[:nnz], ki)
    rng = np.random.default_rng(3)
    rows = np.sort(np.concatenate([rng.choice(nrows, 12, replace=False), [0, nrows - 1]])).astype(np.int64)
    ref = oracle.router_scores(qr_ref, kr_ref, p, rows)
    got = to_np(r["scores"]).reshape(-1, p.N)[rows]
    big = ref > 1e-20
    print("router scores: max rel err %.3e" % (np.abs(got - ref) / np.abs(ref))[big].max())
    assert (np.abs(got - ref) / np.abs(ref))[big].max() < 2e-5
    if w.select.mode != 2:
        sc, idx = oracle.select_rows(ref, w.select)
        sub_ptr = np.concatenate([[0], np.cumsum(counts[rows])])
        sub_idx = np.concatenate([ci[rp[i]:rp[i + 1]] for i in rows])
        print("selection:", compare_selection(sub_ptr, sub_idx, sc, idx, ref, mass_mode=w.select.mode == 1,
                                              mass=w.select.mass))
    o_ref, _ = oracle.attn_fwd(x["q"], x["k"], x["v"], p, rp, ci, rows)
    assert_values(to_np(o).reshape(-1, p.B, p.head_dim)[rows], o_ref, "O (sampled rows)")
    dq_ref = oracle.attn_bwd_dq(x["q"], x["k"], x["v"], x["do"], p, rp, ci, rows)
    assert_values(to_np(g[0]).reshape(-1, p.B, p.head_dim)[rows], dq_ref, "dQ (sampled rows)")
    kvrows = np.sort(np.concatenate([rng.choice(p.batch * p.heads_kv * p.N, 10, replace=False),
                                     [int(np.argmax(np.diff(kp)))]])).astype(np.int64)
    dk_ref, dv_ref = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, rp, ci, kvrows)
    assert_values(to_np(g[1]).reshape(-1, p.B, p.head_dim)[kvrows], dk_ref, "dK (sampled blocks)")
    assert_values(to_np(g[2]).reshape(-1, p.B, p.head_dim)[kvrows], dv_ref, "dV (sampled blocks)")

