"""How well a router's block selection recovers the oracle router's.

The paper's oracle router P_oracle is the token-level softmax of each query
over all keys, summed over the keys of each block and averaged over the
queries of each query block (Sec. 2.2, "Router"); it is the fine router with
pooling R = 1 token.  For sampled query blocks this compares the top-k
blocks of a router with pooling R (the fine router R = 2x2x2, VSA's coarse
router R = B) against the top-k of P_oracle:
  recall   |TopK(P_R) & TopK(P_oracle)| / k
  capture  sum of P_oracle over TopK(P_R) / sum of P_oracle over TopK(P_oracle)
(capture <= 1, with equality when R selects P_oracle's top-k mass).
Everything is computed with the CPU oracle (test infrastructure).

  python tests/router_recall.py [workload] [rows] [k] [sigma]   prints the table
  (sigma > 0 adds per-2x2x2-sub-cube offsets to Q and K, intra-cube structure
  that a cube-level router cannot see)
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import oracle  # noqa: E402
from workload import Selection, WORKLOADS, make_inputs  # noqa: E402


def scores_for_pool(x, p, pool, rows):
    """Block scores of the router with pooling `pool` = (Rt, Rh, Rw)."""
    pr = p.replace(Rt=pool[0], Rh=pool[1], Rw=pool[2])
    q_r = oracle.pool(x["q"], pr, *pool)
    k_r = oracle.pool(x["k"], pr, *pool)
    return oracle.router_scores(q_r, k_r, pr, rows)


def recall_stats(scores, s_oracle, k):
    """(mean recall, min recall, mean capture, min capture) of the top-k of
    `scores` against the top-k of `s_oracle` (rows of both, same order)."""
    sel = Selection(0, k)
    ca, ia = oracle.select_rows(scores, sel)
    cb, ib = oracle.select_rows(s_oracle, sel)
    rec, cap = [], []
    for r in range(scores.shape[0]):
        a, b = ia[r, :ca[r]], ib[r, :cb[r]]
        rec.append(np.intersect1d(a, b).size / float(b.size))
        cap.append(s_oracle[r, a].sum() / s_oracle[r, b].sum())
    rec, cap = np.array(rec), np.array(cap)
    return float(rec.mean()), float(rec.min()), float(cap.mean()), float(cap.min())


def add_subcube_structure(x, p, sigma, seed=11):
    """Intra-cube structure for the comparison: every 2x2x2 sub-cube of every
    cube gets an offset drawn N(0, sigma^2) per element, shared by its 8
    tokens (Q and K independently), on top of the cube mean + token noise of
    the workload recipe; values stay float32 (both routers read the same
    values)."""
    bt, bh, bw = np.meshgrid(np.arange(p.Bt), np.arange(p.Bh), np.arange(p.Bw), indexing="ij")
    sub = (((bt // 2) * (p.Bh // 2) + bh // 2) * (p.Bw // 2) + bw // 2).reshape(-1)   # token beta -> sub-cube
    nsub = (p.Bt // 2) * (p.Bh // 2) * (p.Bw // 2)
    rng = np.random.default_rng(seed)
    out = dict(x)
    for t in ("q", "k"):
        a = x[t].copy()
        b, h, L, D = a.shape
        nu = rng.standard_normal((b, h, p.N, nsub, D)).astype(np.float32) * np.float32(sigma)
        a[:, :, :p.N * p.B] += nu[:, :, :, sub, :].reshape(b, h, p.N * p.B, D)
        out[t] = a
    return out


def recall_table(w, nrows, k, seed=7, pools=None, subcube_sigma=0.0):
    p = w.problem
    x = make_inputs(w, with_grad=False)
    if subcube_sigma > 0:
        x = add_subcube_structure(x, p, subcube_sigma)
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(p.batch * p.heads_q * p.N, nrows, replace=False)).astype(np.int64)
    t0 = time.time()
    s_or = scores_for_pool(x, p, (1, 1, 1), rows)
    t_or = time.time() - t0
    pools = pools or [(2, 2, 2), (p.Bt, p.Bh, p.Bw)]
    out = {"rows": int(nrows), "k": int(k), "oracle_s": t_or, "routers": {}}
    for pool in [(1, 1, 1)] + list(pools):
        s = s_or if pool == (1, 1, 1) else scores_for_pool(x, p, pool, rows)
        out["routers"]["x".join(map(str, pool))] = recall_stats(s, s_or, k)
    return out


if __name__ == "__main__":
    name = sys.argv[1] if len(sys.argv) > 1 else "720p"
    nrows = int(sys.argv[2]) if len(sys.argv) > 2 else 32
    k = int(sys.argv[3]) if len(sys.argv) > 3 else WORKLOADS[name].select.k
    sigma = float(sys.argv[4]) if len(sys.argv) > 4 else 0.0
    t = recall_table(WORKLOADS[name], nrows, k, subcube_sigma=sigma)
    print("workload %s%s, %d sampled query blocks, top-%d (P_oracle rows took %.1f s)" % (
        name, (" + sub-cube offsets sigma %g" % sigma) if sigma else "", t["rows"], t["k"], t["oracle_s"]))
    print("| router pool R | recall mean | recall min | capture mean | capture min |")
    print("|---|---|---|---|---|")
    for r, (rm, rmin, cm, cmin) in t["routers"].items():
        print("| %s | %.3f | %.3f | %.4f | %.4f |" % (r, rm, rmin, cm, cmin))
