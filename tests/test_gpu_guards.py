"""Guard canaries: every output and workspace buffer of every C-ABI call is
placed between two guard regions filled with a byte pattern; after the calls
the guards must hold the pattern unchanged (no write before the start or past
the end of any buffer), and the outputs must match the same calls made on
plain tensors bit for bit.  Cases: a padded grid (the masked kernel
variants), GQA with mass selection on skewed inputs (large-magnitude blocks),
fp32, and joint video + text sequences."""
import numpy as np
import pytest
import torch

import paper_2609_32882_amd as vsa2
from parity import to_dev
from workload import BF16, F32, Problem, Selection, Workload, make_inputs

pytestmark = pytest.mark.gpu

HEAD = 256          # guard before each buffer (keeps 256-byte alignment)
TAIL = 8192         # guard after it
PATTERN = 0xA5

CASES = {
    "bf16-padded": Workload("g1", Problem(1, 2, 2, 128, 7, 13, 22), Selection(0, 12), 7001),
    "bf16-d64-gqa-mass-skewed": Workload("g2", Problem(1, 4, 2, 64, 8, 16, 16), Selection(1, 0, 0.9, 12), 7002,
                                         skewed=True),
    "f32-d128": Workload("g3", Problem(1, 2, 1, 128, 4, 16, 16, dtype=F32), Selection(0, 5), 7003),
    "bf16-text100": Workload("g4", Problem(1, 2, 2, 128, 8, 16, 24, text_len=100), Selection(0, 12), 7004),
}


class Guarded:
    """nbytes of device memory at .ptr with pattern-filled guards around it."""

    def __init__(self, nbytes):
        self.n = int(nbytes)
        self.buf = torch.full((HEAD + max(self.n, 1) + TAIL,), PATTERN, dtype=torch.uint8, device="cuda")
        self.ptr = self.buf.data_ptr() + HEAD

    def data(self, dtype, shape):
        return self.buf[HEAD:HEAD + self.n].view(dtype).view(shape)

    def intact(self):
        return bool((self.buf[:HEAD] == PATTERN).all()) and bool((self.buf[HEAD + self.n:] == PATTERN).all())


def _ok(name, st):
    assert st == 0, "%s -> %s" % (name, vsa2.STATUS_NAMES.get(st, st))


@pytest.mark.parametrize("name", list(CASES))
def test_no_write_outside_any_buffer(name):
    w = CASES[name]
    p = w.problem
    print("\n[guards %s] %s" % (name, p), flush=True)
    P = vsa2.problem_from(p)
    S = vsa2.select_from(w.select)
    bf = p.dtype == BF16
    E = 2 if bf else 4
    tdt = torch.bfloat16 if bf else torch.float32
    x = make_inputs(w, with_grad=True)
    dev = {k: to_dev(v, bf) for k, v in x.items()}
    b, Hq, Hkv, D, N, G = p.batch, p.heads_q, p.heads_kv, p.head_dim, p.N, p.G
    Nj, Lj = p.N_joint, p.L_joint
    guards = {}

    def g(key, nbytes):
        guards[key] = Guarded(nbytes)
        return guards[key]

    # pooling for the router and for the coarse branch
    q_r = g("q_r", b * Hq * N * G * D * E)
    k_r = g("k_r", b * Hkv * N * G * D * E)
    _ok("pool", vsa2.vsa2_pool(P, Hq, dev["q"].data_ptr(), p.Rt, p.Rh, p.Rw, q_r.ptr, 0))
    _ok("pool", vsa2.vsa2_pool(P, Hkv, dev["k"].data_ptr(), p.Rt, p.Rh, p.Rw, k_r.ptr, 0))
    # router, selection, CSR and CSC
    st, cap = vsa2.vsa2_route_capacity(P, S)
    _ok("route_capacity", st)
    st, rws = vsa2.vsa2_route_workspace(P, S)
    _ok("route_workspace", st)
    rp = g("row_ptr", 4 * (b * Hq * N + 1))
    ci = g("col_idx", 4 * cap)
    kp = g("kv_ptr", 4 * (b * Hkv * N + 1))
    ki = g("kv_idx", 4 * cap)
    sc = g("scores", 4 * b * Hq * N * N)
    rwsb = g("route_ws", rws)
    _ok("route", vsa2.vsa2_route(P, S, q_r.ptr, k_r.ptr, rp.ptr, ci.ptr, cap, kp.ptr, ki.ptr, sc.ptr, rwsb.ptr,
                                 rws, 0))
    a_rp, a_ci, a_kp, a_ki, a_cap = rp, ci, kp, ki, cap
    if p.text_len:
        st, jcap = vsa2.vsa2_joint_capacity(P, S)
        _ok("joint_capacity", st)
        st, jws = vsa2.vsa2_joint_workspace(P)
        _ok("joint_workspace", st)
        a_rp, a_ci = g("j_row_ptr", 4 * (b * Hq * Nj + 1)), g("j_col_idx", 4 * jcap)
        a_kp, a_ki = g("j_kv_ptr", 4 * (b * Hkv * Nj + 1)), g("j_kv_idx", 4 * jcap)
        jw = g("joint_ws", jws)
        _ok("joint_lists", vsa2.vsa2_joint_lists(P, rp.ptr, ci.ptr, cap, a_rp.ptr, a_ci.ptr, jcap, a_kp.ptr,
                                                 a_ki.ptr, jw.ptr, jws, 0))
        a_cap = jcap
    # forward (training: with O's remainder) and the three backward stages
    o = g("o", b * Hq * Lj * D * E)
    lse = g("lse", 4 * b * Hq * Lj)
    o_lo = g("o_lo", b * Hq * Lj * D * E)
    st, fws = vsa2.vsa2_attn_workspace(P, 0)
    _ok("attn_workspace", st)
    fw = g("fwd_ws", fws)
    q, k, v, do = (dev[n].data_ptr() for n in ("q", "k", "v", "do"))
    _ok("attn_fwd", vsa2.vsa2_attn_fwd(P, q, k, v, a_rp.ptr, a_ci.ptr, a_cap, o.ptr, lse.ptr, o_lo.ptr, fw.ptr,
                                       fws, 0))
    st, bws = vsa2.vsa2_attn_workspace(P, 1)
    _ok("attn_workspace", st)
    bw = g("bwd_ws", bws)
    dq = g("dq", b * Hq * Lj * D * E)
    dk = g("dk", b * Hkv * Lj * D * E)
    dv = g("dv", b * Hkv * Lj * D * E)
    _ok("bwd_prep", vsa2.vsa2_attn_bwd_prep(P, q, k, v, o.ptr, lse.ptr, o_lo.ptr, do, bw.ptr, bws, 0))
    _ok("bwd_dkdv", vsa2.vsa2_attn_bwd_dkdv(P, q, k, v, do, a_kp.ptr, a_ki.ptr, a_cap, dk.ptr, dv.ptr, bw.ptr,
                                            bws, 0))
    _ok("bwd_dq", vsa2.vsa2_attn_bwd_dq(P, q, k, v, do, a_rp.ptr, a_ci.ptr, a_cap, dq.ptr, bw.ptr, bws, 0))
    # the whole backward in one call, into guarded outputs of its own
    bw2 = g("bwd_ws2", bws)
    dq2, dk2, dv2 = g("dq2", b * Hq * Lj * D * E), g("dk2", b * Hkv * Lj * D * E), g("dv2", b * Hkv * Lj * D * E)
    _ok("attn_bwd", vsa2.vsa2_attn_bwd(P, q, k, v, o.ptr, lse.ptr, o_lo.ptr, do, a_rp.ptr, a_ci.ptr, a_kp.ptr,
                                       a_ki.ptr, a_cap, dq2.ptr, dk2.ptr, dv2.ptr, bw2.ptr, bws, 0))
    # coarse branch, gated merge and the MeanPool adjoint
    Bp = (p.Bt, p.Bh, p.Bw)
    qc, kc, vc = g("q_c", b * Hq * N * D * E), g("k_c", b * Hkv * N * D * E), g("v_c", b * Hkv * N * D * E)
    _ok("pool_c", vsa2.vsa2_pool(P, Hq, q, *Bp, qc.ptr, 0))
    _ok("pool_c", vsa2.vsa2_pool(P, Hkv, k, *Bp, kc.ptr, 0))
    _ok("pool_c", vsa2.vsa2_pool(P, Hkv, v, *Bp, vc.ptr, 0))
    oc, lsec = g("o_c", b * Hq * N * D * E), g("lse_c", 4 * b * Hq * N)
    _ok("coarse_fwd", vsa2.vsa2_coarse_fwd(P, qc.ptr, kc.ptr, vc.ptr, oc.ptr, lsec.ptr, 0))
    gate = torch.from_numpy(np.random.default_rng(3).standard_normal((b, Hq, Lj)).astype(np.float32)).cuda()
    out = g("merged", b * Hq * Lj * D * E)
    _ok("gate_merge", vsa2.vsa2_gate_merge(P, gate.data_ptr(), oc.ptr, o.ptr, out.ptr, 0))
    doc, dg = g("do_c", b * Hq * N * D * E), g("dgate", 4 * b * Hq * Lj)
    _ok("gate_merge_bwd", vsa2.vsa2_gate_merge_bwd(P, gate.data_ptr(), oc.ptr, do, doc.ptr, dg.ptr, 0))
    st, cws = vsa2.vsa2_attn_workspace(P, 2)
    _ok("attn_workspace", st)
    cw = g("coarse_ws", cws)
    dqc, dkc, dvc = g("dq_c", b * Hq * N * D * E), g("dk_c", b * Hkv * N * D * E), g("dv_c", b * Hkv * N * D * E)
    _ok("coarse_bwd", vsa2.vsa2_coarse_bwd(P, qc.ptr, kc.ptr, vc.ptr, doc.ptr, dqc.ptr, dkc.ptr, dvc.ptr, cw.ptr,
                                           cws, 0))
    _ok("unpool_add", vsa2.vsa2_unpool_add(P, Hq, dqc.ptr, *Bp, dq.ptr, 0))
    torch.cuda.synchronize()
    bad = [key for key, gd in guards.items() if not gd.intact()]
    assert not bad, "writes outside buffers: %s" % bad

    # the outputs equal those of the same calls on plain tensors
    r = vsa2.route(p, w.select, q_r.data(tdt, (b, Hq, N * G, D)), k_r.data(tdt, (b, Hkv, N * G, D)),
                   with_scores=True)
    nnz = int(r["row_ptr"][-1])
    assert torch.equal(rp.data(torch.int32, (-1,)), r["row_ptr"])
    assert torch.equal(ci.data(torch.int32, (-1,))[:nnz], r["col_idx"][:nnz])
    assert torch.equal(kp.data(torch.int32, (-1,)), r["kv_ptr"])
    lists = r if not p.text_len else vsa2.joint_lists(p, r)
    o2, lse2, lo2 = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], lists["row_ptr"], lists["col_idx"],
                                  training=True)
    g2 = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o2, lse2, dev["do"], lists["row_ptr"], lists["col_idx"],
                       lists["kv_ptr"], lists["kv_idx"], o_lo=lo2)
    torch.cuda.synchronize()
    iv = torch.int16 if bf else torch.int32
    shp_q, shp_k = (b, Hq, Lj, D), (b, Hkv, Lj, D)
    for got, want in ((o.data(tdt, shp_q), o2), (o_lo.data(tdt, shp_q), lo2), (dq2.data(tdt, shp_q), g2[0]),
                      (dk.data(tdt, shp_k), g2[1]), (dv.data(tdt, shp_k), g2[2]), (dk2.data(tdt, shp_k), g2[1]),
                      (dv2.data(tdt, shp_k), g2[2])):
        assert torch.equal(got.view(iv), want.view(iv))
    assert torch.equal(lse.data(torch.float32, (b, Hq, Lj)), lse2)
