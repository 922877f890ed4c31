"""Kernel timing hook of the C ABI (tra_kernel_timing / tra_kernel_times):
only the chosen kind of call is recorded, at most n of them, each a positive
time no longer than the whole call measured around it on the same stream."""
import pytest

import synth
from _pipeline import Run, log

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_kernel_timing_records_the_chosen_calls():
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    w = synth.Workload("timing_bf16", 1, 2, 128, "bf16", 4, 13, 37, 128, 0.25, 4.0, 0.6, seed=93,
                       tile_h=8, tile_w=16)
    run = Run(w, radius_override=40)
    o = torch.empty_like(run.q)
    H = torch.empty_like(run.H)
    call_ms = []
    tra.tra_kernel_timing(tra.TRA_CALL_SPARSE, 3)
    for i in range(4):                      # the fourth sparse call is past n
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, run.cnt, run.cols, None, o)
        b.record()
        tra.tra_entropy(run.plan, run.q, run.k, None, None, H)   # another kind: not recorded
        torch.cuda.synchronize()
        call_ms.append(a.elapsed_time(b))
    times = tra.tra_kernel_times(8)
    assert len(times) == 3, times
    for k, c in zip(times, call_ms):
        assert 0.0 < k <= c, (k, c)
    assert torch.equal(o, run.O_sp)          # timing changes nothing in the result
    tra.tra_kernel_timing(tra.TRA_CALL_SPARSE, 0)
    assert tra.tra_kernel_times(8) == []
    tra.tra_kernel_timing(tra.TRA_CALL_DENSE, 2)
    tra.tra_dense_attention(run.plan, run.q, run.k, run.v, o)
    assert len(tra.tra_kernel_times(2)) == 1
    tra.tra_kernel_timing(tra.TRA_CALL_DENSE, 0)
    log(f"kernel times {[round(t, 4) for t in times]} ms within calls {[round(c, 4) for c in call_ms]} ms")
