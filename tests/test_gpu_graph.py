"""Replays of captured HIP graphs of the attention calls.  The persistent
attention kernels reset their row-queue counters with a small kernel (not a
memset), so a captured launch sequence must give the eager result on every
replay.  Each graph is replayed several times with the program's own eager
work and synchronisations in between, and every replay is compared bit for
bit with the eager call."""
import numpy as np
import pytest

import synth
from _pipeline import Run, log

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


W = {
    "ragged_bf16_d128": synth.Workload("ragged_bf16_d128", 1, 2, 128, "bf16", 4, 13, 37, 128,
                                       0.25, 4.0, 0.6, seed=78, tile_h=8, tile_w=16),
    "ragged_bf16_d64": synth.Workload("ragged_bf16_d64", 2, 2, 64, "bf16", 3, 11, 29, 128,
                                      0.1, 8.0, 0.95, seed=79, tile_h=8, tile_w=16),
}


@pytest.mark.parametrize("name,layout", [(n, "packed") for n in W] + [("ragged_bf16_d128", "tiles")])
def test_graph_replays_match_eager(name, layout):
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    run = Run(W[name], radius_override=40, block_layout=layout)   # partial lists
    outs = {k: torch.empty_like(run.O_sp) for k in ("sp", "d", "tok", "ent_o")}
    lse = {k: torch.empty_like(run.lse_sp) for k in ("sp", "d", "tok")}
    H = torch.empty_like(run.H)

    def calls():
        tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, run.cnt, run.cols, None, outs["sp"], lse["sp"])
        tra.tra_dense_attention(run.plan, run.q, run.k, run.v, outs["d"], lse["d"])
        tra.tra_token_attention(run.plan, run.q, run.k, run.v, run.rad, run.cnt, run.cols, None,
                                outs["tok"], lse["tok"])
        tra.tra_entropy(run.plan, run.q, run.k, run.v, outs["ent_o"], H)

    calls()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in list(outs.items()) + [("lse_" + k, v) for k, v in lse.items()] + [("H", H)]}

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        calls()                                    # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    scratch = torch.zeros(1 << 20, device=run.q.device)
    for rep in range(4):
        for v in list(outs.values()) + list(lse.values()) + [H]:
            v.fill_(float("nan"))                  # eager work between replays
        scratch.add_(1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = {k: v for k, v in list(outs.items()) + [("lse_" + k, v) for k, v in lse.items()] + [("H", H)]}
        for k in eager:
            assert torch.equal(got[k], eager[k]), (rep, k)
        log(f"{name} ({layout}): replay {rep} equals the eager calls")
