"""Comparison helpers for the GPU parity tests (HIP path vs the CPU oracle)."""
from __future__ import annotations

import numpy as np

import oracle

# Parity bar for outputs and gradients (bf16 inputs, fp32 accumulation):
# |got - ref| <= MAX_ABS + ulp_rel * |ref| element-wise, and relative L2 error
# <= REL_L2.  The ulp_rel term is the output dtype's own rounding (outputs are
# stored in the input dtype, the oracle's are exact): one bf16 ulp relative is
# 2^-8, so a flat 2e-2 alone would fail on correctly rounded values above 5.
MAX_ABS = 2e-2
REL_L2 = 1e-2
ULP_REL = {"bf16": 2.0 ** -8, "f32": 2.0 ** -23}
# a router index mismatch is excused when the oracle scores of the blocks
# involved sit within NEAR_TIE_REL * tau of the row's boundary score tau
# (fp32 near-ties): the GPU's scores are asserted within 2e-5 relative of the
# oracle's, so two scores closer than twice that can swap places; excused
# rows are counted, and also under the tighter 1e-6 * tau reading
NEAR_TIE_REL = 4e-5


# bf16 attention: a 64-token block of Q, or of K and V together, is
# "large-magnitude" when a real token holds a value above this; block pairs
# that touch such a block take two-term (hi + lo) P and dS operands
BIG_VALUE = 7.0


def block_flags(x, p):
    """(query-block flags [b, Hq, Nj], key-block flags [b, Hkv, Nj]) of the
    rule above (Nj blocks of the joint sequence: video cubes, then text
    blocks), from the host copies of the (dtype-rounded) inputs; padding
    tokens do not count."""
    real = p.token_real()

    def amax(t):
        a = np.abs(np.asarray(t, np.float64)) * real[None, None, :, None]
        return a.reshape(t.shape[0], t.shape[1], p.N_joint, p.B * t.shape[3]).max(-1)

    fq = amax(x["q"]) > BIG_VALUE
    fkv = np.maximum(amax(x["k"]), amax(x["v"])) > BIG_VALUE
    return fq, fkv


def to_dev(x: np.ndarray, dtype_bf16: bool):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    if dtype_bf16:
        t = t.to(torch.bfloat16)
    return t.cuda()


def to_np(t) -> np.ndarray:
    return t.float().cpu().numpy()


def value_errors(got, ref, ulp_rel=0.0):
    """(max |got-ref|, max excess over the element-wise bound's ulp term,
    relative L2 error)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    # infinities (LSE = -inf of a query without keys: empty rows, padding
    # queries) must match exactly; the rest is compared numerically
    inf = np.isinf(ref) | ~np.isfinite(got)
    if inf.any():
        assert np.array_equal(got[inf], ref[inf]), "infinite / NaN entries differ"
        got, ref = got[~inf], ref[~inf]
    diff = np.abs(got - ref)
    max_abs = float(diff.max()) if diff.size else 0.0
    scaled = float((diff - ulp_rel * np.abs(ref)).max()) if diff.size else 0.0
    den = float(np.sqrt((ref ** 2).sum()))
    rel_l2 = float(np.sqrt((diff ** 2).sum()) / den) if den > 0 else float(np.sqrt((diff ** 2).sum()))
    return max_abs, scaled, rel_l2


def assert_values(got, ref, name, dtype="bf16", max_abs=MAX_ABS, rel_l2=REL_L2):
    a, sc, r = value_errors(got, ref, ULP_REL[dtype])
    print("%s: max_abs=%.3e (beyond output rounding %.3e) rel_l2=%.3e" % (name, a, sc, r))
    assert sc <= max_abs and r <= rel_l2, "%s: max_abs=%.3e beyond-rounding=%.3e rel_l2=%.3e" % (
        name, a, sc, r)
    return a, r


def compare_selection(gpu_ptr, gpu_idx, ora_counts, ora_idx, ora_scores, rows=None,
                      mass_mode=False, mass=0.9, gap=NEAR_TIE_REL):
    """Check the GPU's CSR rows against the oracle's selection.

    Indices must match exactly, except where the disagreeing blocks' oracle
    scores (fp32-rounded, the decision precision) lie within `gap` * tau of
    the row's boundary score tau; in mass mode the counts may also differ by
    one when the boundary prefix sum is within `gap`-relative of the
    threshold.
    Returns a dict of counters (rows compared, rows excused, relative-gap
    statistics)."""
    gpu_ptr = np.asarray(gpu_ptr, np.int64)
    gpu_idx = np.asarray(gpu_idx)
    nrows = ora_counts.shape[0]
    rows = np.arange(nrows) if rows is None else np.asarray(rows)
    stats = dict(rows=int(len(rows)), exact=0, excused=0, excused_rel_1e6=0, max_rel_gap=0.0)
    for i, r in enumerate(rows):
        g = np.sort(gpu_idx[gpu_ptr[r]:gpu_ptr[r + 1]])
        c = int(ora_counts[i])
        o = ora_idx[i, :c]
        if np.array_equal(g, o):
            stats["exact"] += 1
            continue
        s32 = ora_scores[i].astype(np.float32).astype(np.float64)
        order = np.lexsort((np.arange(s32.size), -s32))
        tau = s32[order[c - 1]] if c > 0 else 0.0
        diff = np.setxor1d(g, o)
        gaps = np.abs(s32[diff] - tau)
        ok_gap = bool((gaps <= gap * tau).all())
        if mass_mode and g.size != o.size:
            total = s32.sum()
            cum = np.cumsum(s32[order])
            thr = mass * total
            near = abs(cum[c - 1] - thr) <= gap * max(thr, 1e-30) or \
                (c >= 2 and abs(cum[c - 2] - thr) <= gap * max(thr, 1e-30))
            ok_gap = ok_gap and abs(g.size - o.size) <= 1 and near
        assert ok_gap, "row %d: gpu %s vs oracle %s (gaps %s, tau %.9g)" % (
            r, g[:16], o[:16], gaps[:8], tau)
        stats["excused"] += 1
        rel = float((gaps / max(tau, 1e-30)).max())
        stats["max_rel_gap"] = max(stats["max_rel_gap"], rel)
        if rel <= 1e-6:
            stats["excused_rel_1e6"] += 1
    return stats


def attn_fp32_logit_bounds(q, k, v, do, scale, D, kmask=None):
    """First-order worst-case effect of fp32 accumulation in the score and
    dP products on softmax attention of m queries over n keys (all float64
    host arrays: q, do [m, D]; k, v [n, D]).  A D-term dot product of exact
    products accumulated in fp32 is off by at most gamma * sum |terms|,
    gamma = (D + 3) 2^-24 (n u / (1 - n u) with the scaling and the
    exponent's multiply-add), so every score of query l is off by at most
    d_l = gamma max_j sum_d |q_ld k_jd| scale, P_lj by 2 d_l P_lj (the
    normaliser moves with the scores), and the outputs by
      O:  sum_j |dP_lj| |v_j|
      dS: |dP_lj| |dP_lj - Delta_l| + P_lj (gamma sum_d |dO_ld v_jd| + |dDelta_l|)
      dQ: sum_j |ddS_lj| |k_j| scale,  dK: sum_l |ddS_lj| |q_l| scale,
      dV: sum_l |dP_lj| |dO_l|.
    kmask (bool [n]) leaves keys out of the softmax (padding).
    Returns the element-wise bounds (eO, edQ, edK, edV)."""
    gam = (D + 3) * 2.0 ** -24
    A = (np.abs(q) @ np.abs(k).T) * scale
    S = (q @ k.T) * scale
    if kmask is not None:
        S = np.where(kmask[None, :], S, -np.inf)
        A = np.where(kmask[None, :], A, 0.0)
    P = np.exp(S - S.max(1, keepdims=True))
    P /= P.sum(1, keepdims=True)
    dl = gam * A.max(1, keepdims=True)
    eP = 2.0 * dl * P
    eO = eP @ np.abs(v)
    dPv = do @ v.T
    Delta = (P * dPv).sum(1, keepdims=True)
    eDelta = (np.abs(do) * eO).sum(1, keepdims=True)
    edS = eP * np.abs(dPv - Delta) + P * (gam * (np.abs(do) @ np.abs(v).T) + eDelta)
    return eO, edS @ np.abs(k) * scale, edS.T @ np.abs(q) * scale, eP.T @ np.abs(do)


def assert_values_bound(got, ref, name, dtype, extra):
    """assert_values with the element-wise bound widened by a derived
    per-element term `extra` (same shape as ref)."""
    got = np.asarray(got, np.float64).reshape(ref.shape)
    ref = np.asarray(ref, np.float64)
    diff = np.abs(got - ref) - ULP_REL[dtype] * np.abs(ref)
    ratio = float((diff / (MAX_ABS + extra)).max())
    den = float(np.sqrt((ref ** 2).sum()))
    rel = float(np.sqrt(((got - ref) ** 2).sum()) / den) if den > 0 else 0.0
    print("%s: max (err - ulp) / (2e-2 + derived bound) = %.3f, max derived bound %.3e, rel_l2=%.3e" % (
        name, ratio, float(np.max(extra)), rel))
    assert ratio <= 1.0 and rel <= REL_L2, (name, ratio, rel)


def check_seq_selection(p, k, rp, ci, ref_scores, exact_scores=None):
    """GPU per-sequence top-(N k) lists against the oracle's flat sort.
    With exact_scores (the GPU's own fp32 scores) the oracle must reproduce
    the selection bit for bit; against the oracle's fp64 scores a pair may
    differ only if its score lies within 1e-6 (relative) of its sequence's
    threshold."""
    N = p.N
    nseq = p.batch * p.heads_q
    keep = min(N * k, N * N)
    got = np.zeros((nseq * N, N), bool)
    counts = np.diff(rp)
    assert (counts >= 0).all() and (counts <= N).all()
    for r in range(nseq * N):
        c = ci[rp[r]:rp[r + 1]]
        assert (np.diff(c) > 0).all() and (c >= 0).all() and (c < N).all()
        got[r, c] = True
    got = got.reshape(nseq, N, N)
    assert (got.reshape(nseq, -1).sum(1) == keep).all()
    if exact_scores is not None:
        want = oracle.select_seq(exact_scores.reshape(nseq, N, N).astype(np.float64), N, k)
        assert np.array_equal(got, want)
    want = oracle.select_seq(ref_scores.reshape(nseq, N, N), N, k)
    sc32 = ref_scores.reshape(nseq, N * N).astype(np.float32).astype(np.float64)
    excused = 0
    for sq in range(nseq):
        diff = got[sq].reshape(-1) != want[sq].reshape(-1)
        if diff.any():
            tau = np.sort(sc32[sq])[::-1][keep - 1]
            assert (np.abs(sc32[sq][diff] - tau) <= 1e-6 * tau).all()
            excused += int(diff.sum())
    print("sequence top-k: %d sequences, %d pairs each, %d near-tie differences" % (nseq, keep, excused))
