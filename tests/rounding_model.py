"""A CPU model of the attention kernels' bf16 roundings, used to study their
precision rules on large-norm inputs (test infrastructure; it shares no
code with the HIP path).

Everything is computed in fp64 except the roundings the kernels apply:
- forward: P rounded to bf16 before the P.V product (hi + lo, i.e. about 16
  bits, on a two-term pair: with p_row_rule every pair of a row that touches
  a flagged block, else the pairs that touch one); O divided by the sum of
  the rounded P
  (rounded_sum=True) or of the unrounded P; O stored as o + o_lo (two bf16
  terms), which Delta = dO . O reads;
- backward: dS = P (dP - Delta) rounded to bf16 (hi + lo on a two-term
  pair) before the dS.K (dQ) and dS^T.Q (dK) products, with P the exact
  softmax (the kernels recompute it in fp32 from the LSE);
- outputs rounded to bf16.
A block is flagged when a real token holds a value above `tau`.  A pair is
two-term for dS when its query block or its key block (K or V) is flagged,
and on every pair of the row when row_rule=True and the row touches a
flagged block, or when one of the row's queries has |Delta| above
delta_tau.  fp32 accumulation
is not modelled (its error is far below these roundings on the inputs
studied).

model_errors returns, for dQ and dK, the largest element error beyond the
output rounding as a share of the 2e-2 bar, and the relative L2 error."""
import numpy as np

import oracle
from workload import make_inputs, round_bf16_f32

BAR = 2e-2


def _bf(a):
    return round_bf16_f32(np.asarray(a, np.float32)).astype(np.float64)


def _two(a):
    hi = _bf(a)
    return hi + _bf(a - hi)


def block_flags(x, p, tau):
    real = p.token_real()

    def amax(t):
        a = np.abs(t) * real[None, None, :, None]
        return a.reshape(t.shape[0], t.shape[1], p.N_joint, p.B * t.shape[-1]).max(-1)

    return amax(x["q"]) > tau, (amax(x["k"]) > tau) | (amax(x["v"]) > tau)


def model_errors(w, tau=7.0, row_rule=True, rounded_sum=True, p_row_rule=True, delta_tau=16.0):
    """(dQ max share, dK max share, dQ rel-L2, dK rel-L2) of the modelled
    kernels on workload w (bf16, no text tokens)."""
    p = w.problem
    assert p.text_len == 0
    x = make_inputs(w, with_grad=True, threads=1)
    ref = oracle.route(x["q"], x["k"], p, w.select)
    rp, ci = ref["row_ptr"], ref["col_idx"]
    real = p.token_real()
    D, B, N = p.head_dim, p.B, p.N
    sc = 1.0 / np.sqrt(D)
    grp = p.heads_q // p.heads_kv
    fq, fkv = block_flags(x, p, tau)
    dq_ex = np.zeros((p.batch, p.heads_q, p.L, D))
    dq_md = np.zeros_like(dq_ex)
    dk_ex = np.zeros((p.batch, p.heads_kv, p.L, D))
    dk_md = np.zeros_like(dk_ex)
    for b in range(p.batch):
        Q, K, V, dO = (x[t][b].astype(np.float64) for t in ("q", "k", "v", "do"))
        for h in range(p.heads_q):
            hk = h // grp
            for n in range(N):
                r = (b * p.heads_q + h) * N + n
                sel = ci[rp[r]:rp[r + 1]]
                if sel.size == 0:
                    continue
                keys = (sel[:, None] * B + np.arange(B)[None, :]).reshape(-1)
                qs = slice(n * B, (n + 1) * B)
                q, k, v, do = Q[h, qs], K[hk, keys], V[hk, keys], dO[h, qs]
                s = (q @ k.T) * sc
                s[:, ~real[keys]] = -np.inf
                pu = np.exp(s - s.max(1, keepdims=True))
                P = pu / pu.sum(1, keepdims=True)
                dP = do @ v.T
                qreal = real[qs]
                d_ex = P * (dP - (do * (P @ v)).sum(1, keepdims=True))
                d_ex[~qreal] = 0
                dq_ex[b, h, qs] = d_ex @ k * sc
                dk_ex[b, hk, keys] += d_ex.T @ q * sc
                pair = np.array([fq[b, h, n] or fkv[b, hk, c] for c in sel])
                row = row_rule and pair.any()
                # forward: O from the rounded P, divided by either sum
                O = np.zeros((B, D))
                lr = np.zeros((B, 1))
                two_p = pair | pair.any() if p_row_rule else pair
                for j, two in enumerate(two_p):
                    pj = pu[:, j * B:(j + 1) * B]
                    pr = _two(pj) if two else _bf(pj)
                    O += pr @ v[j * B:(j + 1) * B]
                    lr += pr.sum(1, keepdims=True)
                O /= lr if rounded_sum else pu.sum(1, keepdims=True)
                delta = (do * _two(O)).sum(1, keepdims=True)
                if delta_tau is not None and qreal.any() and np.abs(delta[qreal]).max() > delta_tau:
                    row = True
                dS = P * (dP - delta)
                dS[~qreal] = 0
                acc = np.zeros((B, D))
                for j, two in enumerate(pair):
                    dj = dS[:, j * B:(j + 1) * B]
                    dr = _two(dj) if (two or row) else _bf(dj)
                    acc += dr @ k[j * B:(j + 1) * B]
                    dk_md[b, hk, keys[j * B:(j + 1) * B]] += dr.T @ q * sc
                dq_md[b, h, qs] = acc * sc

    def share(got, ex):
        return float((np.abs(_bf(got) - ex) - 2.0 ** -8 * np.abs(ex)).max() / BAR)

    def rel(got, ex):
        return float(np.linalg.norm(_bf(got) - ex) / max(np.linalg.norm(ex), 1e-30))

    return share(dq_md, dq_ex), share(dk_md, dk_ex), rel(dq_md, dq_ex), rel(dk_md, dk_ex)
