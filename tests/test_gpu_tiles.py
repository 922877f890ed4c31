"""GPU parity of tile-aligned padded blocks (TRA_BLOCKS_TILES): every video
block is one tile of one frame, a tile clipped by the frame edge padded, text
tokens in blocks of their own.  Against the oracle's padded order: budgets,
radii, masks and lists bit-exact; block-sparse and token-level outputs within
2e-2 max-abs; entropy and dense outputs (layout-independent calls) as for the
packed layout."""
import math

import numpy as np
import pytest

import oracle as O
import synth
from _pipeline import (TOL_O_BF16, TOL_O_FP32, OracleTables, Run, check_head, check_lists, log,
                       retained_fraction, sample_blocks)

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


W = {
    # 13 x 37 frames with 8 x 16 tiles: clipped tiles of 80, 40 and 25 tokens
    "ragged_bf16_d128": synth.Workload("ragged_bf16_d128", 1, 2, 128, "bf16", 4, 13, 37, 128,
                                       0.25, 4.0, 0.6, seed=78, tile_h=8, tile_w=16),
    "ragged_bf16_d64": synth.Workload("ragged_bf16_d64", 2, 2, 64, "bf16", 3, 11, 29, 128,
                                      0.1, 8.0, 0.95, seed=79, tile_h=8, tile_w=16),
    # 5 x 9 frames: one clipped tile of 45 tokens per frame
    "small_frames_bf16": synth.Workload("small_frames_bf16", 1, 2, 64, "bf16", 7, 5, 9, 128,
                                        0.25, 4.0, 0.6, seed=83, tile_h=8, tile_w=16),
    # 30 x 52 frames (the 480p grid) over 5 frames: 96-, 32- and 24-token tiles,
    # rows long enough to be computed in merged pieces
    "split_bf16": synth.Workload("split_bf16", 1, 2, 128, "bf16", 5, 30, 52, 128,
                                 0.25, 4.0, 0.6, seed=88, tile_h=8, tile_w=16),
}
W["joint_bf16_d128"] = W["ragged_bf16_d128"].replace(name="joint_bf16_d128", text_tokens=77)
W["joint_bf16_d64"] = W["ragged_bf16_d64"].replace(name="joint_bf16_d64", text_tokens=200)
# fp32 plans (the correctness path): 8 x 16 tiles over 7 x 19 frames (clipped
# tiles of 112, 56 and 21 tokens), and 8 x 8 tiles with b = 64 over 9 x 11
W["ragged_fp32_d128"] = synth.Workload("ragged_fp32_d128", 1, 2, 128, "fp32", 3, 7, 19, 128,
                                       0.25, 4.0, 0.6, seed=77, tile_h=8, tile_w=16)
W["fp32_b64_d64_text"] = synth.Workload("fp32_b64_d64_text", 1, 2, 64, "fp32", 2, 9, 11, 64,
                                        0.25, 4.0, 0.6, seed=82, tile_h=8, tile_w=8, text_tokens=50)


def _tol(w):
    return TOL_O_BF16 if w.dtype == "bf16" else TOL_O_FP32


def _full(run, tabs, report):
    w = run.w
    for b in range(w.batch):
        for h in range(w.heads):
            check_head(run, tabs, b, h, np.arange(tabs.n_blocks), _tol(w), report)
    check_lists(run)
    assert report["near_integer_budgets"] == 0


@pytest.mark.parametrize("name", list(W))
@pytest.mark.parametrize("rule", ["vote", "union"])
@pytest.mark.parametrize("radius", [None, 40])
def test_tiles_full_parity(name, rule, radius):
    """Every stage on every block of every head: the workload's own entropies,
    and a forced radius of 40 (partial masks, partially covered clipped tiles)."""
    _gpu()
    w = W[name]
    run = Run(w, rule=rule, radius_override=radius, block_layout="tiles")
    tabs = OracleTables(w, block_layout="tiles")
    assert run.plan.n_blocks == tabs.n_blocks
    report = {}
    _full(run, tabs, report)
    log(f"{name} tiles {rule} radius {radius}: NB {tabs.n_blocks} rho={retained_fraction(run, tabs):.4f} {report}")


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "joint_bf16_d128", "small_frames_bf16",
                                  "ragged_fp32_d128", "fp32_b64_d64_text"])
@pytest.mark.parametrize("radius", [0, 3, 40])
@pytest.mark.parametrize("distance", ["2d", "1d"])
def test_tiles_token_attention(name, radius, distance):
    """Token-level attention on tile-aligned blocks against the oracle's
    token_attention_rows over the padded order (union lists, so Eq. 16 over all
    keys), with the 2-D distance and the 1-D ablation."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    w = W[name]
    run = Run(w, rule="union", radius_override=radius, block_layout="tiles", distance=distance)
    tabs = OracleTables(w, block_layout="tiles")
    o = torch.empty_like(run.q)
    lse = torch.empty_like(run.lse_sp)
    tra.tra_token_attention(run.plan, run.q, run.k, run.v, run.rad, run.cnt, run.cols, run.order, o, lse)
    torch.cuda.synchronize()
    worst = 0.0
    for b in range(w.batch):
        for h in range(w.heads):
            q, k, v = (synth.to_f64(a[b, h], w.dtype) for a in (run.q_np, run.k_np, run.v_np))
            M = run.mask[b, h].cpu().numpy().astype(bool)
            rows, o_ref, lse_ref = O.token_attention_rows(
                q, k, v, tabs.perm, w.block, list(range(tabs.n_blocks)), M, run.rad[b, h].cpu().numpy(),
                tabs.F, tabs.H, tabs.W, w.gamma, distance=distance, return_lse=True)
            err = np.abs(o[b, h].double().cpu().numpy()[rows] - o_ref).max()
            assert err <= _tol(w), f"token attention max-abs {err:.3e} (b={b}, h={h})"
            lse_gpu = lse[b, h].double().cpu().numpy()[rows]
            assert np.abs(lse_gpu - lse_ref).max() <= 1e-4 + 1e-5 * np.abs(lse_ref).max(), "token lse"
            worst = max(worst, float(err))
    log(f"{name} tiles token {distance} radius {radius}: max-abs {worst:.2e}")


def test_tiles_equal_packed_when_tiles_divide_the_frame():
    """16 x 32 frames with 8 x 16 tiles: no padding, the two layouts are the
    same order, so masks, lists and every output agree bit for bit."""
    _gpu()
    import torch
    w = synth.Workload("aligned_bf16", 1, 2, 128, "bf16", 5, 16, 32, 128, 0.25, 4.0, 0.6, seed=80,
                       tile_h=8, tile_w=16)
    a = Run(w, radius_override=40)
    t = Run(w, radius_override=40, block_layout="tiles")
    for name in ("mask", "cnt", "cols", "order", "O_sp", "lse_sp", "O_d", "H", "O_ent"):
        assert torch.equal(getattr(a, name), getattr(t, name)), name


def test_tiles_720p_sampled():
    """The 720p grid (21 x 45 x 80, 40 heads) on tile-aligned blocks (630 per
    head, 105 of them clipped to 80 tokens) with a uniform budget of 7,997 keys:
    32 sampled query blocks of every fourth head (and the last) against the
    oracle: budgets, radii, mask rows and block-sparse outputs."""
    _gpu()
    w = synth.workload("wan14b_720p")
    run = Run(w, block_layout="tiles", entropy_override=math.log(7997 / 0.9))
    tabs = OracleTables(w, block_layout="tiles")
    assert tabs.n_blocks == 630
    blocks = sample_blocks(w, 32, seed=7, nb=tabs.n_blocks)
    report = {}
    for h in list(range(0, w.heads, 4)) + [w.heads - 1]:
        check_head(run, tabs, 0, h, blocks[(0, h)], TOL_O_BF16, report, dense=False)
    assert report["near_integer_budgets"] == 0
    log(f"wan14b_720p tiles: rho={retained_fraction(run, tabs):.4f} {report}")
