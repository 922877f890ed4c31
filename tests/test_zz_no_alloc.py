"""The entry point that allocates nothing, tra_build_block_mask_noalloc,
against tra_build_block_mask through the C ABI: on the same radii both give
the same mask, lists and heaviest-first order bit for bit, on two calls in a
row with the second on a smaller plan (the library's scratch array then still
holds the first call's workspace), with and without an order; sizes beyond
the scratch array are refused before anything is launched."""
import ctypes

import numpy as np
import pytest

import synth
from _pipeline import log

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _radii(tra, w, shift):
    """The workload's entropies lowered by `shift` nats, through the budget
    stage: partial masks with unequal row lengths."""
    import torch
    q_np, k_np, _ = synth.generate(w)
    conv = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    q, k = conv(q_np), conv(k_np)
    plan = tra.Plan(tra.Config.from_workload(w))
    B, Ha, N, _ = q.shape
    H = torch.empty(B, Ha, N, device="cuda")
    rad = torch.empty(B, Ha, N, dtype=torch.int32, device="cuda")
    tra.tra_entropy(plan, q, k, None, None, H)
    H.sub_(shift)
    tra.tra_budget_radius(plan, H, None, rad)
    return plan, rad


def _outputs(plan, rad, with_order):
    import torch
    B, Ha = rad.shape[:2]
    NB = plan.n_blocks
    return (torch.full((B, Ha, NB, NB), 7, dtype=torch.uint8, device="cuda"),
            torch.full((B, Ha, NB), -7, dtype=torch.int32, device="cuda"),
            torch.full((B, Ha, NB, NB), -7, dtype=torch.int32, device="cuda"),
            torch.full((plan.rows,), -7, dtype=torch.int32, device="cuda") if with_order else None)


@pytest.mark.parametrize("with_order", [True, False])
def test_noalloc_mask_matches_allocating_call(with_order):
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    big = synth.workload("wan13b_480p")
    small = synth.Workload("noalloc_small", 1, 2, 128, "bf16", 4, 13, 37, 128, 0.25, 4.0, 0.6,
                           seed=78, tile_h=8, tile_w=16)
    for w, shift in ((big, 1.7), (small, 1.0)):   # the second call on a smaller input
        plan, rad = _radii(tra, w, shift)
        ref = _outputs(plan, rad, with_order)
        got = _outputs(plan, rad, with_order)
        tra.tra_build_block_mask(plan, rad, *ref)
        tra.tra_build_block_mask_noalloc(plan, rad, *got)
        torch.cuda.synchronize()
        for a, b_, name in zip(ref, got, ("mask", "cnt", "cols", "order")):
            if a is not None:
                assert torch.equal(a, b_), f"{w.name}: {name} differs"
        cnt = ref[1].reshape(-1)
        assert 0 < int(cnt.min()) < int(cnt.max())          # unequal rows: a non-trivial order
        log(f"{w.name}: rows {plan.rows}, row lengths {int(cnt.min())}..{int(cnt.max())}, order {with_order}: equal")


def test_noalloc_refuses_sizes_beyond_the_scratch():
    """(NB + 1) * ceil(rows / 256) above 2^20: 4,076 blocks per head and 17
    heads need 4,077 * 271 ints; refused with TRA_ERR_UNSUPPORTED before any
    launch (the buffers are never touched); without an order the same plan is
    accepted by the size check."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    w = synth.Workload("noalloc_limit", 1, 17, 64, "bf16", 63, 90, 92, 128, 0.25, 4.0, 0.6,
                       tile_h=8, tile_w=16)
    plan = tra.Plan(tra.Config.from_workload(w))
    assert plan.n_blocks == 4076 and plan.rows == 17 * 4076
    buf = torch.zeros(64, dtype=torch.int32, device="cuda")
    p = ctypes.c_void_p(buf.data_ptr())
    st = tra.lib().tra_build_block_mask_noalloc(plan.handle, p, p, p, p, p, None)
    assert st == 2, st                                   # TRA_ERR_UNSUPPORTED
    assert b"scratch" in tra.lib().tra_last_error()
