"""GPU parity of the joint video + text attention (MMDiT: Eq. block_sparse
extended with full video-to-text and text-to-video blocks, Sec. 2.2)
against the oracle: the joint block lists, pooling of joint sequences, the
forward and backward over joint lists, and the coarse branch with the
gated merge on joint sequences."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32882_amd as vsa2
from parity import assert_values, to_dev, to_np
from workload import BF16, F32, Problem, Selection, Workload, make_inputs

pytestmark = pytest.mark.gpu

CASES = {
    # N = 48 cubes, 100 text tokens (two blocks, the second cut)
    "bf16-d128-text100": Workload("t1", Problem(1, 2, 2, 128, 8, 16, 24, text_len=100), Selection(0, 12), 4001),
    # padded grid, GQA, one full text block, mass selection
    "f32-d64-padded-gqa-text64": Workload("t2", Problem(1, 4, 2, 64, 5, 10, 15, dtype=F32, text_len=64),
                                          Selection(1, 0, 0.9, 12), 4002, skewed=True),
    # eight text blocks (512 tokens) against 16 cubes, batch 2
    "bf16-d128-b2-text512": Workload("t3", Problem(2, 2, 1, 128, 4, 16, 16, text_len=512), Selection(0, 6), 4003),
}


def dtname(p):
    return "bf16" if p.dtype == BF16 else "f32"


@pytest.fixture(scope="module", params=list(CASES))
def case(request):
    w = CASES[request.param]
    p = w.problem
    print("\n[text case %s] %s" % (request.param, p), flush=True)
    x = make_inputs(w, with_grad=True)
    ref = oracle.route(x["q"], x["k"], p, w.select)
    jrp, jci, jkp, jki = oracle.joint_lists(ref["row_ptr"], ref["col_idx"], p)
    ref.update(jrp=jrp, jci=jci, jkp=jkp, jki=jki)
    bf = p.dtype == BF16
    dev = {k: to_dev(v, bf) for k, v in x.items()}
    return w, x, ref, dev


def _gpu_joint_lists(p, rp, ci):
    r = dict(row_ptr=torch.from_numpy(rp).cuda(), col_idx=torch.from_numpy(ci).cuda(), col_cap=ci.size)
    return vsa2.joint_lists(p, r)


def test_joint_lists_exact(case):
    """The expansion of the video lists is exact index work."""
    w, x, ref, dev = case
    p = w.problem
    j = _gpu_joint_lists(p, ref["row_ptr"], ref["col_idx"])
    torch.cuda.synchronize()
    rp = j["row_ptr"].cpu().numpy()
    nnz = int(rp[-1])
    assert np.array_equal(rp, ref["jrp"])
    assert np.array_equal(j["col_idx"].cpu().numpy()[:nnz], ref["jci"])
    assert np.array_equal(j["kv_ptr"].cpu().numpy(), ref["jkp"])
    assert np.array_equal(j["kv_idx"].cpu().numpy()[:nnz], ref["jki"])


def test_pool_reads_the_video_part(case):
    w, x, ref, dev = case
    p = w.problem
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    v_c = vsa2.pool(p, dev["v"], (p.Bt, p.Bh, p.Bw))
    torch.cuda.synchronize()
    assert np.array_equal(to_np(q_r), ref["q_r"])
    assert np.array_equal(to_np(v_c), oracle.pool(x["v"], p, p.Bt, p.Bh, p.Bw))


def test_joint_forward_and_backward(case):
    w, x, ref, dev = case
    p = w.problem
    t = {k: torch.from_numpy(ref[k]).cuda() for k in ("jrp", "jci", "jkp", "jki")}
    o, lse, o_lo = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], t["jrp"], t["jci"], training=True)
    g = vsa2.attn_bwd(p, dev["q"], dev["k"], dev["v"], o, lse, dev["do"], t["jrp"], t["jci"], t["jkp"],
                      t["jki"], o_lo=o_lo)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.attn_fwd(x["q"], x["k"], x["v"], p, ref["jrp"], ref["jci"])
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O (joint)", dtname(p))
    assert_values(lse.cpu().numpy().reshape(lse_ref.shape), lse_ref, "LSE (joint)", "f32", max_abs=1e-3,
                  rel_l2=1e-5)
    dq_ref = oracle.attn_bwd_dq(x["q"], x["k"], x["v"], x["do"], p, ref["jrp"], ref["jci"])
    dk_ref, dv_ref = oracle.attn_bwd_dkdv(x["q"], x["k"], x["v"], x["do"], p, ref["jrp"], ref["jci"])
    for name, got, want in (("dQ", g[0], dq_ref), ("dK", g[1], dk_ref), ("dV", g[2], dv_ref)):
        assert_values(to_np(got).reshape(want.shape), want, name + " (joint)", dtname(p))
    real = torch.from_numpy(p.token_real()).cuda()
    assert (o[:, :, ~real] == 0).all() and torch.isneginf(lse[:, :, ~real]).all()
    assert (g[0][:, :, ~real] == 0).all() and (g[1][:, :, ~real] == 0).all() and (g[2][:, :, ~real] == 0).all()


def test_end_to_end_joint_path(case):
    """pool -> route -> joint lists -> forward on the GPU, against the oracle
    forward on the GPU's own lists (router near-ties may differ)."""
    w, x, ref, dev = case
    p = w.problem
    q_r = vsa2.pool(p, dev["q"], (p.Rt, p.Rh, p.Rw))
    k_r = vsa2.pool(p, dev["k"], (p.Rt, p.Rh, p.Rw))
    r = vsa2.route(p, w.select, q_r, k_r, with_csc=False)
    j = vsa2.joint_lists(p, r)
    o, _ = vsa2.attn_fwd(p, dev["q"], dev["k"], dev["v"], j["row_ptr"], j["col_idx"])
    torch.cuda.synchronize()
    rp = j["row_ptr"].cpu().numpy()
    ci = j["col_idx"].cpu().numpy()[:rp[-1]]
    o_ref, _ = oracle.attn_fwd(x["q"], x["k"], x["v"], p, rp, ci)
    assert_values(to_np(o).reshape(o_ref.shape), o_ref, "O (joint, end to end)", dtname(p))


def test_joint_repeatable_and_padding_free(case):
    """Bitwise repeatable, every output written (NaN sentinels), and the
    same bits with large random values in every padding token."""
    w, x, ref, dev = case
    p = w.problem
    t = {k: torch.from_numpy(ref[k]).cuda() for k in ("jrp", "jci", "jkp", "jki")}
    real = torch.from_numpy(p.token_real()).cuda()
    gen = torch.Generator(device="cuda").manual_seed(5)
    dirty = {k: torch.where(real[None, None, :, None], v,
                            (torch.randn(v.shape, generator=gen, device="cuda") * 40).to(v.dtype))
             for k, v in dev.items()}
    outs = []
    for d, sentinel in ((dev, False), (dev, True), (dirty, False)):
        o = torch.full_like(d["q"], float("nan")) if sentinel else None
        lse = torch.full((p.batch, p.heads_q, p.L_joint), float("nan"), device="cuda") if sentinel else None
        lo = torch.full_like(d["q"], float("nan")) if sentinel else None
        o, lse, lo = vsa2.attn_fwd(p, d["q"], d["k"], d["v"], t["jrp"], t["jci"], o=o, lse=lse, o_lo=lo,
                                   training=True)
        sent = [torch.full_like(d[n], float("nan")) for n in ("q", "k", "v")] if sentinel else [None] * 3
        g = vsa2.attn_bwd(p, d["q"], d["k"], d["v"], o, lse, d["do"], t["jrp"], t["jci"], t["jkp"], t["jki"],
                          dq=sent[0], dk=sent[1], dv=sent[2], o_lo=lo)
        outs.append((o, lse, lo) + tuple(g))
    torch.cuda.synchronize()
    bits = {torch.bfloat16: torch.int16, torch.float32: torch.int32}
    for other in outs[1:]:
        for a, b in zip(outs[0], other):
            assert not torch.isnan(b).any()
            assert torch.equal(a.view(bits[a.dtype]), b.view(bits[b.dtype]))


def test_gate_merge_and_unpool_on_joint_sequences(case):
    """The coarse branch covers the video tokens: text tokens keep O_f and
    get dgate = 0; the MeanPool adjoint updates the video part only."""
    w, x, ref, dev = case
    p = w.problem
    bf = p.dtype == BF16
    rng = np.random.default_rng(9)
    gate = (rng.standard_normal((p.batch, p.heads_q, p.L_joint)) * 1.5).astype(np.float32)
    oc_np = rng.standard_normal((p.batch, p.heads_q, p.N, p.head_dim)).astype(np.float32)
    oc = to_dev(oc_np, bf)
    g = torch.from_numpy(gate).cuda()
    out = vsa2.gate_merge(p, g, oc, dev["q"])
    doc, dg = vsa2.gate_merge_bwd(p, g, oc, dev["do"])
    P = (p.Bt, p.Bh, p.Bw)
    dxc_np = rng.standard_normal((p.batch, p.heads_q, p.N, p.head_dim)).astype(np.float32)
    dxc = to_dev(dxc_np, bf)
    dx = dev["do"].clone()
    vsa2.unpool_add(p, dxc, dx, P)
    torch.cuda.synchronize()
    ocv = to_np(oc)
    assert_values(to_np(out), oracle.gate_merge(gate, ocv, x["q"], p), "merged O (joint)", dtname(p))
    iv = torch.int16 if bf else torch.int32
    assert torch.equal(out[:, :, p.L:].view(iv), dev["q"][:, :, p.L:].view(iv))
    doc_ref, dg_ref = oracle.gate_merge_bwd(gate, ocv, x["do"], p)
    assert_values(to_np(doc), doc_ref, "dO_c_hat (joint)", dtname(p))
    assert_values(dg.cpu().numpy(), dg_ref, "dgate (joint)", "f32", max_abs=1e-3, rel_l2=1e-5)
    assert (dg[:, :, p.L:] == 0).all()
    ref_dx = oracle.unpool_add(to_np(dxc).astype(np.float64), x["do"].astype(np.float64).copy(), p, *P)
    assert_values(to_np(dx), ref_dx, "dx + unpool (joint)", dtname(p))
    assert torch.equal(dx[:, :, p.L:].view(iv), dev["do"][:, :, p.L:].view(iv))
