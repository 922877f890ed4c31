"""Caller-owned workspaces.  The plan holds only tables that no call writes, so
one plan serves calls on several streams at once, each stream with its own
workspace; a caller may also pass a workspace of its own.  Sizes, alignment
and NULL workspaces are checked before anything is launched."""
import ctypes

import pytest

import synth
from _pipeline import Run, log, torch_inputs

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


W = synth.Workload("ws_bf16", 1, 3, 128, "bf16", 4, 13, 37, 128, 0.25, 4.0, 0.6, seed=91,
                   tile_h=8, tile_w=16)


def _calls(tra, plan, run, qkv, out):
    q, k, v = qkv
    tra.tra_sparse_attention(plan, q, k, v, run.cnt, run.cols, run.order, out["sp"], out["lse"])
    tra.tra_dense_attention(plan, q, k, v, out["d"])
    tra.tra_entropy(plan, q, k, v, out["ent_o"], out["H"])
    tra.tra_token_attention(plan, q, k, v, run.rad, run.cnt, run.cols, None, out["tok"])


def test_plan_shared_by_two_streams():
    """Two input sets on one plan, issued on two streams at once (each call
    sequence repeated so that the streams overlap), give bit for bit the
    results of the same calls run one after the other."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    run = Run(W, radius_override=40)                      # partial lists, a ragged last block
    sets = [(run.q, run.k, run.v), torch_inputs(W, *synth.generate(W.replace(seed=92)))]

    def outs():
        return {"sp": torch.empty_like(run.q), "lse": torch.empty_like(run.lse_sp),
                "d": torch.empty_like(run.q), "ent_o": torch.empty_like(run.q),
                "H": torch.empty_like(run.H), "tok": torch.empty_like(run.q)}

    ref = [outs(), outs()]
    for i in range(2):
        _calls(tra, run.plan, run, sets[i], ref[i])
    torch.cuda.synchronize()
    got = [outs(), outs()]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for _ in range(4):
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                _calls(tra, run.plan, run, sets[i], got[i])
    torch.cuda.synchronize()
    assert len(run.plan._ws) >= 3                          # default stream + the two side streams
    for i in range(2):
        for k in ref[i]:
            assert torch.equal(got[i][k], ref[i][k]), (i, k)
    assert not torch.equal(ref[0]["sp"], ref[1]["sp"])
    log("one plan on two concurrent streams: every output equals the sequential calls")


def test_explicit_workspace_and_checks():
    """A caller's workspace of exactly tra_workspace_size bytes gives the same
    output; a smaller, misaligned or NULL one is refused with
    TRA_ERR_INVALID_ARG and the output is left untouched."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    run = Run(W, radius_override=40)
    plan = run.plan
    need = tra.tra_workspace_size(plan, tra.TRA_CALL_SPARSE)
    assert need >= 2 * W.batch * W.heads * plan.n_blocks * 128 * W.head_dim * 2
    for c in (tra.TRA_CALL_ENTROPY, tra.TRA_CALL_TOKEN, tra.TRA_CALL_DENSE, tra.TRA_CALL_BLOCK_MASK):
        assert 0 < tra.tra_workspace_size(plan, c) <= need
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    o = torch.empty_like(run.q)
    tra.tra_sparse_attention(plan, run.q, run.k, run.v, run.cnt, run.cols, None, o, workspace=ws[:need])
    torch.cuda.synchronize()
    assert torch.equal(o, run.O_sp)

    o.fill_(7.0)
    for bad, why in ((ws[:need - 256], "holds"), (ws[1:need + 1], "aligned")):
        with pytest.raises(tra.TraError) as e:
            tra.tra_sparse_attention(plan, run.q, run.k, run.v, run.cnt, run.cols, None, o, workspace=bad)
        assert e.value.status == 1 and why in str(e.value)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    st = tra.lib().tra_sparse_attention(plan.handle, p(run.q), p(run.k), p(run.v), p(run.cnt), p(run.cols),
                                        None, p(o), None, None, 0, None)
    assert st == 1 and b"workspace is NULL" in tra.lib().tra_last_error()
    # the mask call needs a workspace only for the order
    mask, cnt, cols = torch.empty_like(run.mask), torch.empty_like(run.cnt), torch.empty_like(run.cols)
    st = tra.lib().tra_build_block_mask(plan.handle, p(run.rad), p(mask), p(cnt), p(cols), None, None, 0, None)
    assert st == 0, tra.lib().tra_last_error()
    torch.cuda.synchronize()
    assert torch.equal(cnt, run.cnt) and torch.equal(cols, run.cols) and torch.equal(mask, run.mask)
    order = torch.empty_like(run.order)
    st = tra.lib().tra_build_block_mask(plan.handle, p(run.rad), p(mask), p(cnt), p(cols), p(order), None, 0,
                                        None)
    assert st == 1 and b"workspace is NULL" in tra.lib().tra_last_error()
    torch.cuda.synchronize()
    assert bool((o == 7.0).all())                           # nothing was launched
    log(f"workspace of {need} bytes accepted; smaller, misaligned and NULL ones refused")


def test_fp32_plan_workspace_sizes():
    """fp32 plans need a workspace only for the mask call's row order."""
    _gpu()
    import paper_2608_02504_amd as tra
    plan = tra.Plan(tra.Config.from_workload(synth.workload("tiny")))
    sizes = {c: tra.tra_workspace_size(plan, c) for c in range(5)}
    assert sizes[tra.TRA_CALL_BLOCK_MASK] > 0
    assert all(sizes[c] == 0 for c in sizes if c != tra.TRA_CALL_BLOCK_MASK), sizes
    with pytest.raises(tra.TraError):
        tra.tra_workspace_size(plan, 5)
