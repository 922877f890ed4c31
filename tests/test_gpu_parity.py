"""GPU parity of every stage of the path against the CPU oracle, through the
C ABI.  Bars: radii, budgets, masks and lists bit-exact; entropy within
max(1e-3 |H|, 1e-4) nats; attention outputs within 2e-2 max-abs (bf16 I/O) or
1e-5 (fp32 I/O)."""
import math
import os

import numpy as np
import pytest

import oracle as O
import synth
from _pipeline import (TOL_H_ABS, TOL_H_REL, TOL_O_BF16, TOL_O_FP32, OracleTables, Run, check_head, check_lists,
                       dense_reference, log, retained_fraction, sample_blocks, to_np_f64)

pytestmark = pytest.mark.gpu

BLOCKS_PER_HEAD = int(os.environ.get("TRA_TEST_BLOCKS", "32"))


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# Small workloads the oracle checks completely: several tiles, ragged tails.
SMALL = {
    "tiny": synth.workload("tiny"),
    "tiny_union": synth.workload("tiny"),
    "ragged_fp32_d128_b128": synth.Workload("ragged_fp32_d128_b128", 1, 2, 128, "fp32", 3, 7, 19, 128,
                                            0.25, 4.0, 0.6, seed=77, tile_h=8, tile_w=16),
    "ragged_bf16_d128": synth.Workload("ragged_bf16_d128", 1, 2, 128, "bf16", 4, 13, 37, 128,
                                       0.25, 4.0, 0.6, seed=78, tile_h=8, tile_w=16),
    "ragged_bf16_d64": synth.Workload("ragged_bf16_d64", 2, 2, 64, "bf16", 3, 11, 29, 128,
                                      0.1, 8.0, 0.95, seed=79, tile_h=8, tile_w=16),
    "aligned_bf16": synth.Workload("aligned_bf16", 1, 2, 128, "bf16", 5, 16, 32, 128,
                                   0.25, 4.0, 0.6, seed=80, tile_h=8, tile_w=16),
    "single_token": synth.Workload("single_token", 1, 1, 128, "bf16", 1, 1, 1, 128,
                                   0.25, 4.0, 0.6, seed=81, tile_h=8, tile_w=16),
    "fp32_b64_d128": synth.Workload("fp32_b64_d128", 1, 1, 128, "fp32", 2, 9, 11, 64,
                                    0.25, 4.0, 0.6, seed=82, tile_h=8, tile_w=8),
    # 45-token frames: each 128-token block spans three or four frames, which the
    # mask builder's two-frame packed pair test does not cover
    "small_frames_bf16": synth.Workload("small_frames_bf16", 1, 2, 64, "bf16", 7, 5, 9, 128,
                                        0.25, 4.0, 0.6, seed=83, tile_h=8, tile_w=16),
    # the largest frame count a plan accepts (64): per-query thresholds for 64
    # frame distances, blocks spanning four 32-token frames
    "max_frames_bf16": synth.Workload("max_frames_bf16", 1, 1, 128, "bf16", 64, 4, 8, 128,
                                      0.25, 4.0, 0.6, seed=85, tile_h=8, tile_w=16),
    # a single frame: only the frame distance 0 exists
    "one_frame_bf16": synth.Workload("one_frame_bf16", 1, 2, 128, "bf16", 1, 30, 52, 128,
                                     0.25, 4.0, 0.6, seed=86, tile_h=8, tile_w=16),
    # 61 blocks per head and a small total: block-sparse rows longer than 48
    # blocks are computed in merged pieces
    "split_bf16": synth.Workload("split_bf16", 1, 2, 128, "bf16", 5, 30, 52, 128,
                                 0.25, 4.0, 0.6, seed=88, tile_h=8, tile_w=16),
}

# 90 x 160 frames: n_cap = 89^2 + 159^2 = 33,202, beyond the range of the mask
# builder's 16-bit packed distances, so every pair takes the 32-bit test.
WIDE = synth.Workload("wide_frame_bf16", 1, 1, 64, "bf16", 2, 90, 160, 128,
                      0.25, 4.0, 0.6, seed=84, tile_h=8, tile_w=16)

# Close to the largest block count a plan accepts (4,096 per head): 63 frames of
# 90 x 92 = 521,640 tokens, 4,076 blocks, the last one ragged (40 tokens).
MAXB = synth.Workload("max_blocks_bf16", 1, 1, 64, "bf16", 63, 90, 92, 128,
                      0.25, 4.0, 0.6, seed=87, tile_h=8, tile_w=16)


@pytest.mark.parametrize("name", list(SMALL))
def test_small_full_parity(name):
    _gpu()
    w = SMALL[name]
    rule = "union" if name.endswith("union") else "vote"
    run = Run(w, rule=rule)
    tabs = OracleTables(w)
    tol = TOL_O_BF16 if w.dtype == "bf16" else TOL_O_FP32
    report = {}
    for b in range(w.batch):
        for h in range(w.heads):
            check_head(run, tabs, b, h, np.arange(w.n_blocks), tol, report)
    check_lists(run)
    log(f"{name}: rho={retained_fraction(run):.4f} {report}")
    assert report["near_integer_budgets"] == 0


# Joint text-video workloads: video grid + text tokens (ragged and aligned video
# lengths, so the mixed video/text block and a pure text block both occur).
JOINT = {
    "joint_bf16_d128": SMALL["ragged_bf16_d128"].replace(name="joint_bf16_d128", text_tokens=77),
    "joint_bf16_d64": SMALL["ragged_bf16_d64"].replace(name="joint_bf16_d64", text_tokens=200),
    "joint_aligned_bf16": SMALL["aligned_bf16"].replace(name="joint_aligned_bf16", text_tokens=128),
    "joint_fp32_tiny": synth.workload("tiny").replace(name="joint_fp32_tiny", text_tokens=40),
}


def _full_check(run, report):
    w = run.w
    tabs = OracleTables(w)
    tol = TOL_O_BF16 if w.dtype == "bf16" else TOL_O_FP32
    for b in range(w.batch):
        for h in range(w.heads):
            check_head(run, tabs, b, h, np.arange(w.n_blocks), tol, report)
    check_lists(run)
    assert report["near_integer_budgets"] == 0


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "fp32_b64_d128"])
def test_lognormal_budget_parity(name):
    """App. A.2 lognormal mapping: budgets (fp64 on both sides, ties at an integer
    allowed one apart), radii, masks and outputs against the oracle."""
    _gpu()
    run = Run(SMALL[name], budget="lognormal")
    report = {}
    _full_check(run, report)
    log(f"{name} lognormal: rho={retained_fraction(run):.4f} {report}")


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "fp32_b64_d128"])
@pytest.mark.parametrize("rule", ["vote", "union"])
def test_sequence_distance_parity(name, rule):
    """Sequence-distance ablation (App. C.1): masks bit-exact, outputs within
    tolerance, against the oracle's 1-D test."""
    _gpu()
    run = Run(SMALL[name], rule=rule, distance="1d")
    report = {}
    _full_check(run, report)
    log(f"{name} 1d {rule}: rho={retained_fraction(run):.4f} {report}")


@pytest.mark.parametrize("name", list(JOINT))
def test_joint_text_video_parity(name):
    """Joint text-video attention (Sec. 3.2): entropy over all S keys, text
    tokens FULL, text blocks dense as rows and columns, outputs against the
    oracle over the joint sequence."""
    _gpu()
    w = JOINT[name]
    run = Run(w)
    report = {}
    _full_check(run, report)
    mask = run.mask.cpu().numpy().astype(bool)
    first_text = w.n_video // w.block
    assert mask[:, :, first_text:, :].all() and mask[:, :, :, first_text:].all()
    log(f"{name}: rho={retained_fraction(run):.4f} {report}")


@pytest.mark.parametrize("name", ["joint_bf16_d128", "joint_fp32_tiny"])
def test_joint_zero_radius(name):
    """Video radii 0: the video part of the mask is block diagonal (vote), the
    text part dense; every video query still sees every text key."""
    _gpu()
    w = JOINT[name]
    run = Run(w, radius_override=0)
    mask = run.mask.cpu().numpy().astype(bool)
    first_text = w.n_video // w.block
    vid = mask[:, :, :first_text, :first_text]
    assert np.array_equal(vid, np.broadcast_to(np.eye(first_text, dtype=bool), vid.shape))
    assert mask[:, :, first_text:, :].all() and mask[:, :, :, first_text:].all()
    check_lists(run)


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "fp32_b64_d128",
                                  "joint_bf16_d128", "small_frames_bf16", "max_frames_bf16",
                                  "one_frame_bf16"])
@pytest.mark.parametrize("radius", [3, 40, 250])
@pytest.mark.parametrize("rule,distance", [("vote", "2d"), ("union", "2d"), ("vote", "1d")])
def test_mid_radius_masks_exact(name, radius, rule, distance):
    """Radii where most block pairs are partially covered (the key-by-key path
    of the mask builder): every mask row and list equals the oracle's Alg. 1.
    (250 exceeds the tiny grid's n_cap = 98, where it must act as FULL.)"""
    _gpu()
    w = JOINT.get(name) or SMALL[name]
    run = Run(w, rule=rule, distance=distance, radius_override=radius)
    tabs = OracleTables(w)
    n_full = run.rad.cpu().numpy()
    # a radius above n_cap is documented to act as FULL
    n_full = np.where(n_full > tabs.ncap, O.RADIUS_FULL, n_full)
    mask = run.mask.cpu().numpy().astype(bool)
    for b in range(w.batch):
        for h in range(w.heads):
            M_ref = O.block_mask_rows(n_full[b, h], tabs.perm, w.block, tabs.F, tabs.H, tabs.W,
                                      w.gamma, list(range(w.n_blocks)), rule=rule, distance=distance)
            assert np.array_equal(mask[b, h], M_ref), (b, h, np.nonzero((mask[b, h] != M_ref).any(1))[0][:5])
    check_lists(run)


@pytest.mark.parametrize("budget", [1500, 6000])
def test_wide_frame_sampled(budget):
    """Every stage on sampled query blocks of the 90 x 160 grid, with one constant
    entropy ln(budget / tau) for every token: the radius bisection runs over
    [0, 33,202] and the block masks are partial."""
    _gpu()
    w = WIDE
    tabs = OracleTables(w)
    assert tabs.ncap >= 32767
    run = Run(w, with_order=False, entropy_override=float(np.log(budget / w.tau)))
    report = {}
    for (b, h), blocks in sample_blocks(w, 16, seed=5).items():
        check_head(run, tabs, b, h, blocks, TOL_O_BF16, report)
    check_lists(run)
    rho = retained_fraction(run)
    log(f"{w.name} budget {budget}: rho={rho:.4f} {report}")
    assert 0.0 < rho < 0.9


@pytest.mark.slow
def test_max_blocks_sampled():
    """Every stage on sampled query blocks (the ragged last among them) of a
    4,076-block sequence, with a uniform budget of 20,000 keys (partial masks)
    and the heaviest-first row order: block lists, the row-order histogram and
    the sparse kernel's staged list at nearly their largest."""
    _gpu()
    w = MAXB
    assert w.n_blocks == 4076 and w.n_tokens % w.block == 40
    tabs = OracleTables(w)
    run = Run(w, entropy_override=float(np.log(20000 / w.tau)))
    report = {}
    for (b, h), blocks in sample_blocks(w, 4, seed=9).items():
        check_head(run, tabs, b, h, blocks, TOL_O_BF16, report)
    check_lists(run)
    rho = retained_fraction(run)
    log(f"{w.name}: rho={rho:.4f} {report}")
    assert 0.0 < rho < 0.9


def test_wide_frame_mask_exact():
    """A partially covering radius (n = 2,000) on the 90 x 160 grid: every mask
    row equals the oracle's Alg. 1."""
    _gpu()
    w = WIDE
    run = Run(w, radius_override=2000)
    tabs = OracleTables(w)
    n_full = run.rad.cpu().numpy()
    mask = run.mask.cpu().numpy().astype(bool)
    M_ref = O.block_mask_rows(n_full[0, 0], tabs.perm, w.block, tabs.F, tabs.H, tabs.W, w.gamma,
                              list(range(w.n_blocks)))
    assert np.array_equal(mask[0, 0], M_ref), np.nonzero((mask[0, 0] != M_ref).any(1))[0][:5]
    assert 0.05 < M_ref.mean() < 0.95
    check_lists(run)


def test_single_token_closed_form():
    """N = 1: the only key has p = 1, so H = 0, o = v, radius 0, mask [[1]]."""
    _gpu()
    run = Run(SMALL["single_token"])
    assert abs(float(run.H[0, 0, 0])) < 1e-6
    assert int(run.rad[0, 0, 0]) == 0 and int(run.cnt[0, 0, 0]) == 1
    assert np.array_equal(run.np("O_sp")[0, 0], synth.to_f64(run.v_np[0, 0], "bf16"))
    assert np.array_equal(run.np("O_d")[0, 0], synth.to_f64(run.v_np[0, 0], "bf16"))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_entropy_closed_forms(dtype):
    """Uniform scores -> H = log N; one dominant key -> H = 0 (Eq. 2 bounds)."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    w = synth.Workload("cf", 1, 2, 128, dtype, 2, 12, 20, 128, 0.25, 4.0, 0.6, tile_h=8, tile_w=16)
    cfg = tra.Config.from_workload(w)
    plan = tra.Plan(cfg)
    N, d = w.n_tokens, 128
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    q = torch.randn(1, 2, N, d, generator=torch.Generator().manual_seed(0)).to(tdt).cuda()
    k = torch.zeros(1, 2, N, d, dtype=tdt, device="cuda")
    k[:, :, :] = torch.randn(d, generator=torch.Generator().manual_seed(1)).to(tdt).cuda()
    k[:, 1] = 0.0
    q[:, 1] = 0.0
    q[:, 1, :, 0] = 1.0
    k[:, 1, 123, 0] = 64.0 * math.sqrt(d)    # key 123 leads every other score by 64
    H = torch.empty(1, 2, N, device="cuda")
    tra.tra_entropy(plan, q, k, None, None, H)
    torch.cuda.synchronize()
    Hn = H.cpu().numpy()
    assert np.abs(Hn[0, 0] - math.log(N)).max() < 1e-4 * math.log(N)
    assert np.abs(Hn[0, 1]).max() < 1e-4


def test_scores_jumping_in_late_tiles():
    """Scores that rise block by block along the tile-major order (0, 5, 15,
    35 nats plus a small spread): after the first tile the entropy and token
    kernels take weights against the reference without a tile max, accept the
    +5 nat tile (weights up to 2^7.2) and redo the +15 and +35 nat tiles from
    their max (weights past 2^20).  Entropy-only, fused entropy + output,
    dense and token-level (full radius, every block listed) results against
    the oracle (Eq. 2, Eq. 1)."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    w = synth.Workload("jumps", 1, 2, 128, "bf16", 2, 12, 20, 128, 0.25, 4.0, 0.6, tile_h=8, tile_w=16)
    plan = tra.Plan(tra.Config.from_workload(w))
    N, d = w.n_tokens, w.head_dim
    perm = O.tile_major_order(w.frames, w.height, w.width, w.tile_h, w.tile_w)
    rng = np.random.default_rng(5)
    level = np.array([0.0, 5.0, 15.0, 35.0])[np.arange(N) // 128]   # by tile-major position
    q = np.zeros((2, N, d), np.float32)
    k = rng.standard_normal((2, N, d)).astype(np.float32) * 0.5
    v = rng.standard_normal((2, N, d)).astype(np.float32)
    q[:, :, 0] = 1.0
    q[1, :, 0] = rng.uniform(0.5, 1.0, N)                 # per-query temperature on head 1
    k[:, perm, 0] = (level + 0.3 * rng.uniform(0, 1, N)) * math.sqrt(d)
    qb, kb, vb = (synth.bf16_bits_from_f32(a) for a in (q, k, v))
    dev = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).reshape(1, 2, N, d).cuda()
    qt, kt, vt = dev(qb), dev(kb), dev(vb)
    H = torch.empty(1, 2, N, device="cuda")
    Hf = torch.empty_like(H)
    Of, Od, Ot = (torch.empty_like(qt) for _ in range(3))
    tra.tra_entropy(plan, qt, kt, None, None, H)
    tra.tra_entropy(plan, qt, kt, vt, Of, Hf)
    tra.tra_dense_attention(plan, qt, kt, vt, Od)
    NB = plan.n_blocks
    rad = torch.full((1, 2, N), tra.TRA_RADIUS_FULL, dtype=torch.int32, device="cuda")
    cnt = torch.full((1, 2, NB), NB, dtype=torch.int32, device="cuda")
    cols = torch.arange(NB, dtype=torch.int32, device="cuda").repeat(1, 2, NB, 1)
    tra.tra_token_attention(plan, qt, kt, vt, rad, cnt, cols, None, Ot)
    torch.cuda.synchronize()
    for h in range(2):
        q64, k64, v64 = (synth.to_f64(a[h], "bf16") for a in (qb, kb, vb))
        H_ref, O_ref, _ = dense_reference(q64, k64, v64, np.arange(N))
        tol = np.maximum(TOL_H_REL * np.abs(H_ref), TOL_H_ABS)
        for name, got in (("entropy", H), ("fused entropy", Hf)):
            dH = np.abs(got[0, h].double().cpu().numpy() - H_ref)
            assert (dH <= tol).all(), f"{name} head {h}: max |dH| {dH.max():.3e}"
        for name, got in (("fused output", Of), ("dense", Od), ("token-level", Ot)):
            err = np.abs(got[0, h].double().cpu().numpy() - O_ref).max()
            assert err <= TOL_O_BF16, f"{name} head {h}: max-abs {err:.3e}"
        log(f"score jumps head {h}: H in [{H_ref.min():.3f}, {H_ref.max():.3f}] nats, all within the bars")


def _close_to_rounding(a, b):
    """Equal up to rounding: a row computed in merged pieces takes each piece's
    probabilities in bf16 relative to that piece's own running max, so they
    round differently from an unsplit pass, and the bf16 outputs can then
    differ by a few steps (1.6e-2 seen at |o| ~ 1).  Both sides are within the
    2e-2 parity bar of the exact values (checked against the oracle elsewhere),
    so they are compared at that bar."""
    return (a.float() - b.float()).abs().max().item() <= TOL_O_BF16


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "split_bf16"])
def test_full_radius_sparse_equals_dense_bitwise(name):
    """All radii FULL -> every block retained -> the sparse kernel walks the
    same key blocks in the same order as the dense one: bitwise equal while
    no row is split (lists of at most 48 blocks never are); a split row
    (split_bf16: 61 blocks) is merged from pieces and agrees to rounding."""
    _gpu()
    w = SMALL[name]
    run = Run(w, radius_override=2 ** 31 - 1)
    assert run.mask.all()
    import torch
    if w.dtype == "fp32" or w.n_blocks <= 48:
        assert torch.equal(run.O_sp, run.O_d)
        assert torch.equal(run.lse_sp, run.lse_d)
    else:
        log(f"{name}: split sparse vs dense max |do| {(run.O_sp.float() - run.O_d.float()).abs().max().item():.3e}")
        assert _close_to_rounding(run.O_sp, run.O_d)
        assert (run.lse_sp - run.lse_d).abs().max().item() <= 1e-5 * run.lse_d.abs().max().item() + 1e-6
    # the fused warm-up output of the entropy pass is dense attention too, up
    # to rounding (its kernel splits the key blocks over two wave groups)
    assert (run.O_ent.float() - run.O_d.float()).abs().max().item() <= 2e-2


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "tiny"])
def test_zero_radius_is_block_diagonal(name):
    """All radii 0 -> (vote) only the diagonal block survives -> block-diagonal
    attention, i.e. textbook attention inside each block."""
    _gpu()
    w = SMALL[name]
    run = Run(w, radius_override=0)
    m = run.mask.cpu().numpy()
    eye = np.broadcast_to(np.eye(w.n_blocks, dtype=np.uint8), m.shape)
    assert np.array_equal(m, eye)
    tabs = OracleTables(w)
    tol = TOL_O_BF16 if w.dtype == "bf16" else TOL_O_FP32
    perm = tabs.perm
    for h in range(w.heads):
        q, k, v = (synth.to_f64(a[0, h], w.dtype) for a in (run.q_np, run.k_np, run.v_np))
        O_gpu = run.np("O_sp")[0, h]
        for u in range(w.n_blocks):
            idx = perm[u * w.block:min((u + 1) * w.block, w.n_tokens)]
            want = O.dense_attention(q[idx], k[idx], v[idx])
            assert np.abs(O_gpu[idx] - want).max() <= tol


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "split_bf16"])
def test_out_of_range_column_ids_are_skipped(name):
    """Key-block ids outside [0, NB) in a list are skipped: padding every list
    with -1 and NB entries (between and around the valid ids) leaves o and lse
    equal to the call with the clean list -- bitwise where no row is split
    (48 blocks or fewer), else to rounding (the longer padded lists are cut
    into different pieces)."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    w = SMALL[name]
    run = Run(w)
    NB = run.plan.n_blocks
    cnt, cols = run.cnt.cpu().numpy(), run.cols.cpu().numpy()
    cnt2 = np.zeros_like(cnt)
    cols2 = np.full_like(cols, -1)
    rng = np.random.default_rng(7)
    padded = 0
    for idx in np.ndindex(cnt.shape):
        valid = cols[idx][:cnt[idx]].tolist()
        out = []
        for c in valid:
            out += [-1, NB][:rng.integers(0, 3)]  # 0, 1 or 2 invalid ids first
            out.append(c)
        out = (out + [NB, -5])[:NB]  # a list holds at most NB entries
        kept = [c for c in out if 0 <= c < NB]
        padded += len(out) - len(kept)
        cnt2[idx], cols2[idx][:len(out)] = len(out), out
        cnt[idx], cols[idx][:len(kept)] = len(kept), kept
    assert padded > 0
    dev = run.q.device
    ref_o, ref_l = torch.empty_like(run.O_sp), torch.empty_like(run.lse_sp)
    got_o, got_l = torch.empty_like(run.O_sp), torch.empty_like(run.lse_sp)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, t(cnt), t(cols), None, ref_o, ref_l)
    tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, t(cnt2), t(cols2), None, got_o, got_l)
    torch.cuda.synchronize()
    if w.dtype == "fp32" or NB <= 48:
        assert torch.equal(got_o, ref_o)
        assert torch.equal(got_l, ref_l)
        return
    # split rows: both calls against the oracle's Eq. 16 over the clean lists
    tabs = OracleTables(w)
    tol = TOL_O_BF16
    diff = (got_o.float() - ref_o.float()).abs()
    log(f"{name}: padded vs clean max |do| {diff.max().item():.3e}, "
        f"max |dlse| {(got_l - ref_l).abs().max().item():.3e}")
    for b in range(w.batch):
        for h in range(w.heads):
            q, k, v = (synth.to_f64(a[b, h], w.dtype) for a in (run.q_np, run.k_np, run.v_np))
            M = np.zeros((NB, NB), dtype=bool)
            for u in range(NB):
                M[u, cols[b, h, u, :cnt[b, h, u]]] = True
            rows, o_ref, l_ref = O.masked_attention_rows(q, k, v, tabs.perm, w.block, list(range(NB)), M,
                                                         return_lse=True)
            for name_, oo, ll in (("clean", ref_o, ref_l), ("padded", got_o, got_l)):
                err = np.abs(to_np_f64(oo[b, h])[rows] - o_ref).max()
                assert err <= tol, f"{name_} lists: output max-abs {err:.3e} (b={b}, h={h})"
                lerr = np.abs(ll[b, h].double().cpu().numpy()[rows] - l_ref).max()
                assert lerr <= 1e-4 + 1e-5 * np.abs(l_ref).max(), f"{name_} lists: lse {lerr:.3e}"


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "split_bf16"])
def test_row_schedule_does_not_change_results(name):
    """Rows are independent: the schedule (per-XCD row queues without an
    order, the heaviest-first order, a random permutation, an order with
    out-of-range entries that are skipped) changes only which workgroup
    computes a row, and each result is bitwise the same; repeated calls start
    from freshly reset row queues."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    run = Run(SMALL[name])
    rows = run.plan.rows
    dev = run.q.device
    rng = np.random.default_rng(11)
    perm = rng.permutation(rows).astype(np.int32)
    padded = np.insert(perm, rng.integers(0, rows, 5), [-1, rows, -3, rows + 7, -1]).astype(np.int32)[:rows]
    kept = set(int(r) for r in padded if 0 <= r < rows)
    orders = [None, run.order, torch.from_numpy(perm).to(dev), None]
    outs = []
    for od in orders:
        o, l = torch.empty_like(run.O_sp), torch.empty_like(run.lse_sp)
        tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, run.cnt, run.cols, od, o, l)
        torch.cuda.synchronize()
        outs.append((o, l))
    for o, l in outs:
        assert torch.equal(o, outs[0][0]) and torch.equal(l, outs[0][1])
    # rows missing from the order (entries out of range) are not computed
    o = torch.full_like(run.O_sp, 7.0)
    tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, run.cnt, run.cols,
                             torch.from_numpy(padded).to(dev), o, None)
    torch.cuda.synchronize()
    NB = run.plan.n_blocks
    perm_tok = OracleTables(run.w).perm
    S = o.shape[2]
    blk = np.arange(S) // run.w.block                    # tile-major position -> block
    for r in range(rows):
        bh, u = divmod(r, NB)
        b, h = divmod(bh, o.shape[1])
        toks = perm_tok[(blk == u)]
        got = o[b, h, toks]
        if r in kept:
            assert torch.equal(got, outs[0][0][b, h, toks]), r
        else:
            assert bool((got == 7.0).all()), r


@pytest.mark.parametrize("name", ["ragged_bf16_d128", "ragged_bf16_d64", "tiny", "split_bf16"])
def test_empty_rows_give_zero_output(name):
    """A row whose list is empty (cnt = 0, or only out-of-range ids) has no key
    to attend to: its queries get o = 0 and lse = -inf, as the header states;
    every other row is bitwise the normal call's."""
    _gpu()
    import torch
    import paper_2608_02504_amd as tra
    run = Run(SMALL[name])
    NB = run.plan.n_blocks
    rows = run.plan.rows
    cnt, cols = run.cnt.cpu().numpy().copy(), run.cols.cpu().numpy().copy()
    flat_c, flat_l = cnt.reshape(-1), cols.reshape(rows, NB)
    empty = np.arange(0, rows, 3)
    flat_c[empty[::2]] = 0
    flat_l[empty[1::2], :] = -1            # non-zero count, but no valid id
    dev = run.q.device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    o, l = torch.empty_like(run.O_sp), torch.empty_like(run.lse_sp)
    tra.tra_sparse_attention(run.plan, run.q, run.k, run.v, t(cnt), t(cols), None, o, l)
    torch.cuda.synchronize()
    perm_tok = OracleTables(run.w).perm
    S = o.shape[2]
    blk = np.arange(S) // run.w.block
    for r in range(rows):
        bh, u = divmod(r, NB)
        b, h = divmod(bh, o.shape[1])
        toks = perm_tok[blk == u]
        if r in set(empty.tolist()):
            assert bool((o[b, h, toks] == 0).all()), r
            assert bool(torch.isneginf(l[b, h, toks]).all()), r
        else:
            assert torch.equal(o[b, h, toks], run.O_sp[b, h, toks]), r
            assert torch.equal(l[b, h, toks], run.lse_sp[b, h, toks]), r
    # the token-level call (same lists) follows the same rule
    ot, lt = torch.empty_like(o), torch.empty_like(l)
    tra.tra_token_attention(run.plan, run.q, run.k, run.v, run.rad, t(cnt), t(cols), None, ot, lt)
    torch.cuda.synchronize()
    for r in empty.tolist():
        bh, u = divmod(r, NB)
        b, h = divmod(bh, o.shape[1])
        toks = perm_tok[blk == u]
        assert bool((ot[b, h, toks] == 0).all()) and bool(torch.isneginf(lt[b, h, toks]).all()), r


def test_determinism_bitwise():
    _gpu()
    import torch
    w = SMALL["ragged_bf16_d64"]
    inputs = synth.generate(w)
    a, b = Run(w, inputs=inputs), Run(w, inputs=inputs)
    for name in ("H", "H_only", "O_ent", "budget", "rad", "mask", "cnt", "cols", "order", "O_sp",
                 "lse_sp", "O_d", "lse_d"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name


# ---------------------------------------------------------------- large shapes
# The model-shaped workloads are run once on the GPU (every head) and checked
# against the oracle on a seeded sample of 32 query blocks (4,096 rows, the
# ragged last block among them) of EVERY head, a few heads per test so that each
# test's host-side check stays well under a minute.  One large run is kept
# alive at a time.
HEAD_GROUP = 5
_RUNS = {}


def _cached_run(key, make):
    if key not in _RUNS:
        import gc

        import torch
        _RUNS.clear()
        gc.collect()
        torch.cuda.empty_cache()
        _RUNS[key] = make()
    return _RUNS[key]


# name -> (workload, Run options, check the entropy-side stages?)
#   wan14b_720p:      as the benchmark times it (no row order)
#   wan14b_720p_u15:  one constant entropy ln(7997 / tau) for every token (a
#                     uniform budget of 7,997 keys) keeps ~15 % of the blocks,
#                     no row order; its inputs, entropy and dense-side kernels
#                     are those of wan14b_720p, so only budget, radius, mask and
#                     sparse output are checked again
LARGE = {
    "wan13b_480p": ("wan13b_480p", {}, True),
    "wan14b_720p": ("wan14b_720p", {"with_order": False}, True),
    "wan14b_720p_u15": ("wan14b_720p", {"with_order": False,
                                        "entropy_override": float(np.log(7997 / 0.9))}, False),
    "hunyuan_720p": ("hunyuan_720p", {}, True),
    "hunyuan_joint_720p": ("hunyuan_joint_720p", {}, True),
}
LARGE_CASES = [(name, h0) for name, (wname, _, _) in LARGE.items()
               for h0 in range(0, synth.workload(wname).heads, HEAD_GROUP)]


@pytest.mark.slow
@pytest.mark.parametrize("name,h0", LARGE_CASES, ids=[f"{n}-heads{h}" for n, h in LARGE_CASES])
def test_large_sampled(name, h0):
    _gpu()
    wname, kw, dense = LARGE[name]
    w = synth.workload(wname)
    run = _cached_run(name, lambda: Run(w, **kw))
    tabs = OracleTables(w)
    if h0 == 0:
        check_lists(run)
    samples = sample_blocks(w, BLOCKS_PER_HEAD, seed=2024)
    report = {}
    for h in range(h0, min(h0 + HEAD_GROUP, w.heads)):
        for b in range(w.batch):
            check_head(run, tabs, b, h, samples[(b, h)], TOL_O_BF16, report, dense=dense)
            log(f"{name}: batch {b} head {h} checked")
    rho = retained_fraction(run)
    log(f"{name} heads {h0}..{min(h0 + HEAD_GROUP, w.heads) - 1}: rho={rho:.4f} {report}")
    assert report["near_integer_budgets"] == 0
    if name == "wan14b_720p_u15":
        assert 0.12 < rho < 0.18, rho
    if w.text_tokens:
        mask = run.mask.cpu().numpy().astype(bool)
        first_text = w.n_video // w.block
        assert mask[:, :, first_text:, :].all() and mask[:, :, :, first_text:].all()
