"""The allocation-free forward (vsa2_attn_fwd_noalloc, workspace in the
library's fixed per-GPU array) against vsa2_attn_fwd with a caller
workspace: the same bits for O, LSE and O's remainder, on two calls in a
row, the second with a smaller problem; captured in a HIP graph and
replayed with other calls in between; and the size limit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32882_amd as vsa2
from parity import to_dev
from workload import Problem, Selection, Workload, make_inputs

# a skewed (large-magnitude) case so that the block flags in the array matter,
# then a smaller one with GQA and a padded grid
CASES = [Workload("na1", Problem(1, 4, 2, 128, 8, 16, 24), Selection(1, 0, 0.9, 20), 5001, skewed=True),
         Workload("na2", Problem(1, 2, 1, 64, 5, 10, 15), Selection(0, 4), 5002)]


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _run(w):
    p = w.problem
    x = make_inputs(w, with_grad=False)
    ref = oracle.route(x["q"], x["k"], p, w.select)
    dev = {n: to_dev(x[n], True) for n in ("q", "k", "v")}
    rp = torch.from_numpy(ref["row_ptr"]).cuda()
    ci = torch.from_numpy(ref["col_idx"]).cuda()
    P = vsa2.problem_from(p)
    outs = []
    for noalloc in (False, True):
        o = torch.full_like(dev["q"], float("nan"))
        o_lo = torch.full_like(dev["q"], float("nan"))
        lse = torch.full((p.batch, p.heads_q, p.L), float("nan"), device="cuda")
        args = (P, dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(), rp.data_ptr(), ci.data_ptr(),
                ci.numel(), o.data_ptr(), lse.data_ptr(), o_lo.data_ptr())
        if noalloc:
            st = vsa2.vsa2_attn_fwd_noalloc(*args, 0)
        else:
            st_, wsb = vsa2.vsa2_attn_workspace(P, 0)
            assert st_ == 0
            ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
            st = vsa2.vsa2_attn_fwd(*args, ws.data_ptr(), wsb, 0)
        assert st == 0, vsa2.STATUS_NAMES.get(st, st)
        outs.append((o, lse, o_lo))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert not torch.isnan(b).any()
        assert torch.equal(_bits(a), _bits(b))


@pytest.mark.gpu
def test_noalloc_forward_matches_workspace_forward_twice():
    print("\n[no-alloc forward] %s then %s" % (CASES[0].problem, CASES[1].problem), flush=True)
    _run(CASES[0])
    _run(CASES[1])      # smaller: the array still holds the first call's larger contents


@pytest.mark.gpu
def test_noalloc_forward_in_a_hip_graph():
    """The call captured in a HIP graph (it allocates nothing, so it can be):
    three replays, each after eager work that refills the outputs with NaN
    and runs the allocation-free forward of another problem (which rewrites
    the library's array), give the eager call's bits every time."""
    w, w2 = CASES
    p, p2 = w.problem, w2.problem
    print("\n[no-alloc forward in a graph] %s" % p, flush=True)

    def setup(w):
        p = w.problem
        x = make_inputs(w, with_grad=False)
        ref = oracle.route(x["q"], x["k"], p, w.select)
        dev = {n: to_dev(x[n], True) for n in ("q", "k", "v")}
        dev["rp"] = torch.from_numpy(ref["row_ptr"]).cuda()
        dev["ci"] = torch.from_numpy(ref["col_idx"]).cuda()
        dev["o"] = torch.full_like(dev["q"], float("nan"))
        dev["o_lo"] = torch.full_like(dev["q"], float("nan"))
        dev["lse"] = torch.full((p.batch, p.heads_q, p.L), float("nan"), device="cuda")
        return dev

    def call(P, d, stream):
        return vsa2.vsa2_attn_fwd_noalloc(P, d["q"].data_ptr(), d["k"].data_ptr(), d["v"].data_ptr(),
                                          d["rp"].data_ptr(), d["ci"].data_ptr(), d["ci"].numel(), d["o"].data_ptr(),
                                          d["lse"].data_ptr(), d["o_lo"].data_ptr(), stream)

    P, P2 = vsa2.problem_from(p), vsa2.problem_from(p2)
    d, d2 = setup(w), setup(w2)
    assert call(P, d, torch.cuda.current_stream().cuda_stream) == 0        # eager reference
    torch.cuda.synchronize()
    want = [t.clone() for t in (d["o"], d["lse"], d["o_lo"])]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st = call(P, d, torch.cuda.current_stream().cuda_stream)
    assert st == 0
    for rep in range(3):
        for t in (d["o"], d["lse"], d["o_lo"]):
            t.fill_(float("nan"))
        assert call(P2, d2, torch.cuda.current_stream().cuda_stream) == 0
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(want, (d["o"], d["lse"], d["o_lo"])):
            assert torch.equal(_bits(a), _bits(b)), "replay %d" % rep


def test_noalloc_forward_rejects_problems_beyond_its_array():
    """Checked on the host before any device work (fake pointers)."""
    fake = 1 << 20
    big = vsa2.problem_from(Problem(1, 64, 64, 128, 64, 256, 256))   # 64 heads x 65,536 cubes
    st = vsa2.vsa2_attn_fwd_noalloc(big, fake, fake, fake, fake, fake, 1, fake, fake, None, 0)
    assert vsa2.STATUS_NAMES[st] == "VSA2_ERR_WORKSPACE"
