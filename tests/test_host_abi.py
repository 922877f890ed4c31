"""CPU tests of the C ABI: the library loads, exports every declared symbol,
its host-side tables agree with the oracle's independent ones, and bad
arguments come back as status codes (no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2608_02504_amd as tra
import synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "tra.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tra_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = tra.lib()
    declared = _declared_functions()
    assert set(declared) == set(tra.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(L, name), name
    assert "gfx950" in tra.tra_version()


@pytest.mark.parametrize("name", ["tiny", "wan13b_480p", "wan14b_720p", "hunyuan_720p",
                                  "hunyuan_joint_720p", "tiny_text"])
def test_host_tables_match_oracle(name):
    w = synth.workload("tiny").replace(text_tokens=77) if name == "tiny_text" else synth.workload(name)
    cfg = tra.Config.from_workload(w)
    perm, thr, thr1, blocks, ncap = tra.tra_plan_host_tables(cfg)
    N = w.n_video
    assert ncap == O.n_cap(w.height, w.width)
    assert np.array_equal(perm, O.joint_order(
        O.tile_major_order(w.frames, w.height, w.width, w.tile_h, w.tile_w), w.text_tokens))
    assert np.array_equal(thr, O.threshold_table(ncap, w.frames, w.gamma))
    assert np.array_equal(thr1, O.threshold_table_1d(ncap, w.frames, w.gamma))
    f, x, y = O.grid_coords(w.frames, w.height, w.width)
    for u, (lo, hi) in enumerate(O.block_bounds(w.n_tokens, w.block)):
        r = perm[lo:hi]
        rv, n_text = r[r < N], int((r >= N).sum())
        if len(rv):
            want = [f[rv].min(), f[rv].max(), x[rv].min(), x[rv].max(), y[rv].min(), y[rv].max(),
                    len(rv), rv.min(), rv.max(), n_text]
        else:
            want = [w.frames, -1, w.height, -1, w.width, -1, 0, N, -1, n_text]
        assert list(blocks[u]) == want, u


@pytest.mark.parametrize("name", ["wan13b_480p", "wan14b_720p", "hunyuan_joint_720p", "ragged_text"])
def test_tile_aligned_host_tables_match_oracle(name):
    """Tile-aligned padded blocks: the plan's order equals the oracle's padded
    order (-1 at padding), and every block's info is that of its own tokens."""
    w = (synth.Workload("ragged_text", 1, 2, 128, "bf16", 3, 11, 29, 128, 0.25, 4.0, 0.6,
                        tile_h=8, tile_w=16, text_tokens=130) if name == "ragged_text" else synth.workload(name))
    cfg = tra.Config.from_workload(w, block_layout="tiles")
    perm, thr, thr1, blocks, ncap = tra.tra_plan_host_tables(cfg)
    want = O.tile_aligned_order(w.frames, w.height, w.width, w.tile_h, w.tile_w, w.block,
                                text_tokens=w.text_tokens)
    assert np.array_equal(perm, want)
    assert cfg.n_blocks == len(want) // w.block == blocks.shape[0]
    N = w.n_video
    f, x, y = O.grid_coords(w.frames, w.height, w.width)
    for u in range(cfg.n_blocks):
        r = O.block_tokens(want, w.block, u)
        rv, n_text = r[r < N], int((r >= N).sum())
        if len(rv):
            exp = [f[rv].min(), f[rv].max(), x[rv].min(), x[rv].max(), y[rv].min(), y[rv].max(),
                   len(rv), rv.min(), rv.max(), n_text]
        else:
            exp = [w.frames, -1, w.height, -1, w.width, -1, 0, N, -1, n_text]
        assert list(blocks[u]) == exp, u


def test_tiny_layout_sizes():
    cfg = tra.Config.from_workload(synth.workload("wan14b_720p"))
    assert cfg.n_tokens == 75600 and cfg.n_blocks == 591
    cfg_t = tra.Config.from_workload(synth.workload("wan14b_720p"), block_layout="tiles")
    assert cfg_t.n_blocks == 21 * 6 * 5 == 630 and cfg_t.n_positions == 630 * 128
    cfg3 = tra.Config.from_workload(synth.workload("hunyuan_720p"))
    assert cfg3.n_tokens == 118800 and cfg3.n_blocks == 929
    assert cfg3.n_tokens - (cfg3.n_blocks - 1) * 128 == 16
    cfg4 = tra.Config.from_workload(synth.workload("hunyuan_joint_720p"))
    assert cfg4.n_video == 118800 and cfg4.n_tokens == 119056 and cfg4.n_blocks == 931


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=96), 2), (dict(block=32), 2), (dict(block=64), 2),   # bf16 needs block 128
    (dict(frames=0), 1), (dict(frames=65), 2), (dict(height=2000), 2),
    (dict(tau=1.0), 1), (dict(tau=0.0), 1), (dict(gamma=-0.1), 1),
    (dict(gamma=float("nan")), 1), (dict(tile_h=0), 1), (dict(dtype="fp16"), 1),
    (dict(rule="maj"), 1), (dict(batch=0), 1), (dict(budget="gamma"), 1),
    (dict(distance="3d"), 1), (dict(text_tokens=-1), 1),
    (dict(text_tokens=4096 * 128), 2),   # more than 4096 blocks
    (dict(block_layout="tiles", tile_h=8, tile_w=8), 1),           # a tile must hold one block
    (dict(block_layout="diag"), 1),
])
def test_invalid_configs_rejected(change, status):
    base = dict(batch=1, heads=2, frames=3, height=8, width=16, head_dim=128)
    base.update(change)
    cfg = tra.Config(**base)
    with pytest.raises(tra.TraError) as ei:
        tra.tra_plan_host_tables(cfg)
    assert ei.value.status == status


def test_fp32_block64_accepted_host_side():
    cfg = tra.Config(batch=1, heads=1, frames=2, height=8, width=8, head_dim=64, block=64,
                     tile_h=8, tile_w=8, dtype="fp32")
    perm, thr, thr1, blocks, ncap = tra.tra_plan_host_tables(cfg)
    assert ncap == 98 and thr.shape == (99, 2) and thr1.shape == (99, 2) and blocks.shape == (2, 10)


def test_null_arguments_are_errors_not_crashes():
    L = tra.lib()
    assert L.tra_plan_host_tables(None, None, None, None, None, None) == 1
    assert L.tra_plan_create(None, None) == 1
    assert L.tra_workspace_size(None, 0, None) == 1
    assert L.tra_entropy(None, None, None, None, None, None, None, 0, None) == 1
    assert L.tra_budget_radius(None, None, None, None, None) == 1
    assert L.tra_build_block_mask(None, None, None, None, None, None, None, 0, None) == 1
    assert L.tra_build_block_mask_noalloc(None, None, None, None, None, None, None) == 1
    assert L.tra_sparse_attention(None, None, None, None, None, None, None, None, None, None, 0, None) == 1
    assert L.tra_token_attention(None, None, None, None, None, None, None, None, None, None, None, 0,
                                 None) == 1
    assert L.tra_dense_attention(None, None, None, None, None, None, None, 0, None) == 1
    assert L.tra_kernel_times(None, 0, None) == 1
    assert b"NULL" in L.tra_last_error()
    assert L.tra_kernel_timing(tra.TRA_CALL_BLOCK_MASK, 1) == 1   # not an attention call
    assert L.tra_kernel_timing(tra.TRA_CALL_SPARSE, -1) == 1
    assert L.tra_kernel_timing(tra.TRA_CALL_SPARSE, 5000) == 1
    assert L.tra_kernel_timing(tra.TRA_CALL_SPARSE, 0) == 0      # stopping needs no device
    assert tra.tra_kernel_times(4) == []
    assert L.tra_plan_destroy(None) == 0
    assert L.tra_last_error() == b""


def test_plan_create_without_gpu_reports_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    cfg = tra.Config.from_workload(synth.workload("tiny"))
    with pytest.raises(tra.TraError) as ei:
        tra.Plan(cfg)
    assert ei.value.status in (2, 3)
