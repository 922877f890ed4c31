"""Shared helpers for the GPU tests: run the library's path on a workload and
compute the oracle's answer on sampled query blocks."""
from __future__ import annotations

import math
import sys
import time

import numpy as np

import oracle as O
import paper_2608_02504_amd as tra
import synth

TOL_O_BF16 = 2e-2      # max-abs on attention outputs, bf16 I/O
TOL_O_FP32 = 1e-5      # max-abs on attention outputs, fp32 I/O
TOL_H_REL = 1e-3       # entropy: |dH| <= max(1e-3 |H|, 1e-4) nats
TOL_H_ABS = 1e-4


def log(msg):
    sys.stdout.write(f"[tra-test {time.strftime('%H:%M:%S')}] {msg}\n")
    sys.stdout.flush()


def torch_inputs(w, q, k, v, device="cuda"):
    import torch
    if w.dtype == "bf16":
        conv = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    else:
        conv = lambda a: torch.from_numpy(a).to(device)
    return conv(q), conv(k), conv(v)


def to_np_f64(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


class Run:
    """All stage outputs of one pass of the path on the GPU."""

    def __init__(self, w, rule="vote", with_order=True, inputs=None, radius_override=None,
                 budget="uniform", distance="2d", entropy_override=None, block_layout="packed"):
        import torch
        self.w = w
        self.radius_override = radius_override
        self.cfg = tra.Config.from_workload(w, rule=rule, budget=budget, distance=distance,
                                            block_layout=block_layout)
        self.plan = tra.Plan(self.cfg)
        log(f"workload {w.name} S={w.n_tokens} (text {w.text_tokens}) heads={w.heads} d={w.head_dim} "
            f"{w.dtype} rule={rule} budget={budget} distance={distance}")
        if inputs is None:
            inputs = synth.generate(w)
        self.q_np, self.k_np, self.v_np = inputs
        q, k, v = torch_inputs(w, *inputs)
        B, Ha, N, d = q.shape
        NB = self.plan.n_blocks
        dev = q.device
        f32, i32 = torch.float32, torch.int32
        self.H = torch.empty(B, Ha, N, dtype=f32, device=dev)
        self.H_only = torch.empty_like(self.H)
        self.O_ent = torch.empty_like(q)
        self.budget = torch.empty(B, Ha, N, dtype=i32, device=dev)
        self.rad = torch.empty(B, Ha, N, dtype=i32, device=dev)
        self.mask = torch.empty(B, Ha, NB, NB, dtype=torch.uint8, device=dev)
        self.cnt = torch.empty(B, Ha, NB, dtype=i32, device=dev)
        self.cols = torch.empty(B, Ha, NB, NB, dtype=i32, device=dev)
        self.order = torch.empty(B * Ha * NB, dtype=i32, device=dev) if with_order else None
        self.O_sp = torch.empty_like(q)
        self.lse_sp = torch.empty(B, Ha, N, dtype=f32, device=dev)
        self.O_d = torch.empty_like(q)
        self.lse_d = torch.empty(B, Ha, N, dtype=f32, device=dev)

        tra.tra_entropy(self.plan, q, k, v, self.O_ent, self.H)
        tra.tra_entropy(self.plan, q, k, None, None, self.H_only)
        # entropy_override: one constant entropy for every token feeds the budget
        # and radius stage (a uniform budget, as in the paper's ablation), so
        # the mask keeps a chosen fraction of the blocks
        self.H_budget = self.H
        if entropy_override is not None:
            self.H_budget = torch.full_like(self.H, float(entropy_override))
        tra.tra_budget_radius(self.plan, self.H_budget, self.budget, self.rad)
        if radius_override is not None:
            self.rad[:, :, :w.n_video] = int(radius_override)
        tra.tra_build_block_mask(self.plan, self.rad, self.mask, self.cnt, self.cols, self.order)
        tra.tra_sparse_attention(self.plan, q, k, v, self.cnt, self.cols, self.order, self.O_sp,
                                 self.lse_sp)
        tra.tra_dense_attention(self.plan, q, k, v, self.O_d, self.lse_d)
        torch.cuda.synchronize()
        self.q, self.k, self.v = q, k, v
        log(f"workload {w.name}: GPU path done")

    def np(self, name):
        t = getattr(self, name)
        if t.dtype.is_floating_point:
            return to_np_f64(t)
        return t.cpu().numpy()


def sample_blocks(w, n_blocks_per_head: int, seed: int, nb=None):
    """Seeded query blocks per (batch, head); always includes the last block
    (the ragged one of a packed layout).  nb: blocks per head (default the
    packed layout's)."""
    rng = np.random.default_rng(seed)
    nb = w.n_blocks if nb is None else nb
    out = {}
    for b in range(w.batch):
        for h in range(w.heads):
            if n_blocks_per_head >= nb:
                sel = np.arange(nb)
            else:
                sel = np.unique(np.concatenate([rng.choice(nb - 1, n_blocks_per_head - 1, replace=False),
                                                [nb - 1]]))
            out[(b, h)] = sel
    return out


class OracleTables:
    def __init__(self, w, block_layout="packed"):
        self.F, self.H, self.W = w.frames, w.height, w.width
        self.ncap = O.n_cap(w.height, w.width)
        self.thr = O.threshold_table(self.ncap, w.frames, w.gamma)
        self.disk = O.disk_count_table(w.height, w.width, self.ncap)
        if block_layout == "tiles":
            self.perm = O.tile_aligned_order(w.frames, w.height, w.width, w.tile_h, w.tile_w, w.block,
                                             text_tokens=w.text_tokens)
        else:
            self.perm = O.joint_order(O.tile_major_order(w.frames, w.height, w.width, w.tile_h, w.tile_w),
                                      w.text_tokens)
        self.n_blocks = -(-len(self.perm) // w.block)
        self.sizes = O.block_sizes(self.perm, w.block)
        self.f, self.x, self.y = O.grid_coords(w.frames, w.height, w.width)


def dense_reference(q, k, v, rows):
    """The oracle's entropy (Eq. 2), dense output (Eq. 1) and log-partition for
    the query rows `rows` (raster indices), evaluated 128 rows at a time so that
    the fp64 score matrices stay small."""
    import torch
    vt = torch.as_tensor(v)
    H, Od, L = [], [], []
    for c0 in range(0, len(rows), 128):
        s = O.scores(q[rows[c0:c0 + 128]], k)
        p = O.softmax_rows(s)
        H.append(O.entropy_from_probs(p))
        Od.append((p @ vt).numpy())
        L.append(torch.logsumexp(s, dim=1).numpy())
    return np.concatenate(H), np.concatenate(Od), np.concatenate(L)


def check_head(run: Run, tabs: OracleTables, b: int, h: int, blocks, tol_o: float, report: dict,
               dense: bool = True):
    """Compare every stage for the sampled query blocks of one (batch, head).

    dense=False leaves out the entropy, fused-output and dense-output checks
    (for a second run whose inputs and entropy-side kernels are those of a run
    already checked with dense=True); budget, radius, mask and sparse output
    are always checked."""
    w = run.w
    N, bs = w.n_tokens, w.block
    perm = tabs.perm
    q = synth.to_f64(run.q_np[b, h], w.dtype)
    k = synth.to_f64(run.k_np[b, h], w.dtype)
    v = synth.to_f64(run.v_np[b, h], w.dtype)
    rows = np.concatenate([O.block_tokens(perm, bs, u) for u in blocks])

    O_ref = lse_ref = None
    if dense:
        # entropy and dense output (Eq. 1, Eq. 2)
        H_ref, O_ref, lse_ref = dense_reference(q, k, v, rows)
        H_gpu = run.H[b, h].double().cpu().numpy()[rows]
        dH = np.abs(H_gpu - H_ref)
        assert (dH <= np.maximum(TOL_H_REL * np.abs(H_ref), TOL_H_ABS)).all(), \
            f"entropy: max |dH| {dH.max():.3e} at H={H_ref[dH.argmax()]:.4f}"
        # the entropy-only call (no output) is its own kernel: same bar on its own
        H_only = run.H_only[b, h].double().cpu().numpy()[rows]
        dHo = np.abs(H_only - H_ref)
        assert (dHo <= np.maximum(TOL_H_REL * np.abs(H_ref), TOL_H_ABS)).all(), \
            f"entropy-only: max |dH| {dHo.max():.3e} at H={H_ref[dHo.argmax()]:.4f}"
        # the warm-up output fused with the entropy pass (Alg. 2 with O)
        O_e = to_np_f64(run.O_ent[b, h])[rows]
        erre = np.abs(O_e - O_ref).max()
        assert erre <= tol_o, f"fused entropy+output max-abs {erre:.3e}"
        O_d = to_np_f64(run.O_d[b, h])[rows]
        errd = np.abs(O_d - O_ref).max()
        assert errd <= tol_o, f"dense output max-abs {errd:.3e}"
        lse_d = run.lse_d[b, h].double().cpu().numpy()[rows]
        assert np.abs(lse_d - lse_ref).max() <= 1e-4 + 1e-5 * np.abs(lse_ref).max(), "dense lse"
        report["max_dH"] = max(report.get("max_dH", 0.0), float(dH.max()))
        report["max_err_dense"] = max(report.get("max_err_dense", 0.0), float(errd))
        report["max_err_fused"] = max(report.get("max_err_fused", 0.0), float(erre))

    # budget and radius from the GPU's fp32 entropy (Eqs. 8, 13, 14, or the
    # lognormal mapping of App. A.2): bit-exact for video tokens; text tokens
    # carry budget S and the FULL radius.  The radius is the oracle's from the
    # oracle's own budget; only where tau e^H (or S Phibar) lies within rounding
    # of an integer may the two budgets differ by one, and there the GPU radius
    # must be the oracle's radius of the GPU's budget.
    Nv = w.n_video
    video = rows < Nv
    kh_gpu = run.budget[b, h].cpu().numpy()[rows]
    n_gpu = run.rad[b, h].cpu().numpy()[rows]
    assert (kh_gpu[~video] == N).all() and (n_gpu[~video] == O.RADIUS_FULL).all(), "text budget/radius"
    Hv, rv = run.H_budget[b, h].double().cpu().numpy()[rows][video], rows[video]
    if run.cfg.budget == "lognormal":
        khat_ref = O.token_budget_lognormal(Hv, w.tau, N)
        sigma = np.sqrt(2.0 * np.maximum(0.0, math.log(N) - Hv))
        t = N * O.normal_tail(sigma - O.normal_quantile(w.tau))
        tol = 1e-9  # the device's erfc and the host's differ in the last bits
    else:
        khat_ref = O.token_budget(Hv, w.tau, N)
        t = w.tau * np.exp(Hv)
        tol = 1e-12
    near = np.abs(t - np.round(t)) <= tol * np.maximum(t, 1.0)
    report["near_integer_budgets"] = report.get("near_integer_budgets", 0) + int(near.sum())
    khv = kh_gpu[video]
    assert np.array_equal(khv[~near], khat_ref[~near]), "budget mismatch"
    assert (np.abs(khv[near] - khat_ref[near]) <= 1).all(), "budget mismatch at an integer boundary"
    fv, xv, yv = tabs.f[rv], tabs.x[rv], tabs.y[rv]
    nv_gpu = n_gpu[video]
    if run.radius_override is not None:
        # the radii the test wrote over the budget stage's output
        assert (nv_gpu == int(run.radius_override)).all(), "forced radius"
    else:
        n_ref = O.select_radius(khat_ref, fv, xv, yv, tabs.F, tabs.thr, tabs.disk)
        assert np.array_equal(nv_gpu[~near], n_ref[~near]), \
            f"radius mismatch at {np.nonzero((nv_gpu != n_ref) & ~near)[0][:5]}"
        if near.any():
            n_alt = O.select_radius(khv[near], fv[near], xv[near], yv[near], tabs.F, tabs.thr, tabs.disk)
            assert np.array_equal(nv_gpu[near], n_alt), "radius mismatch at an integer budget boundary"

    # block mask rows (Alg. 1) from the GPU radii: bit-exact
    n_full = run.rad[b, h].cpu().numpy()
    M_ref = O.block_mask_rows(n_full, perm, bs, tabs.F, tabs.H, tabs.W, w.gamma, list(blocks),
                              rule=run.cfg.rule, distance=run.cfg.distance)
    M_gpu = run.mask[b, h].cpu().numpy()[blocks].astype(bool)
    assert np.array_equal(M_gpu, M_ref), f"mask mismatch in blocks {np.nonzero((M_gpu != M_ref).any(1))[0][:5]}"

    # block-sparse attention (Eq. 16 at block granularity).  A query block whose
    # mask row keeps every key block attends to every key, where Eq. 16 is Eq. 1
    # (an oracle pin checks that identity), so the dense reference serves there.
    full_row = M_ref.all(axis=1)
    if O_ref is not None and full_row.any():
        O_ms, lse_ms = O_ref.copy(), lse_ref.copy()
        part = [u for u, f in zip(blocks, full_row) if not f]
        if part:
            r2, Op, Lp = O.masked_attention_rows(q, k, v, perm, bs, part, M_ref[~full_row], return_lse=True)
            pos = {int(r): i for i, r in enumerate(rows)}
            idx = np.array([pos[int(r)] for r in r2])
            O_ms[idx], lse_ms[idx] = Op, Lp
    else:
        r2, O_ms, lse_ms = O.masked_attention_rows(q, k, v, perm, bs, list(blocks), M_ref, return_lse=True)
        assert np.array_equal(r2, rows)
    O_s = to_np_f64(run.O_sp[b, h])[rows]
    errs = np.abs(O_s - O_ms).max()
    assert errs <= tol_o, f"sparse output max-abs {errs:.3e}"
    lse_s = run.lse_sp[b, h].double().cpu().numpy()[rows]
    assert np.abs(lse_s - lse_ms).max() <= 1e-4 + 1e-5 * np.abs(lse_ms).max(), "sparse lse"
    report["max_err_sparse"] = max(report.get("max_err_sparse", 0.0), float(errs))
    return M_ref


def check_lists(run: Run):
    """cnt / cols / order agree with the mask for every row (integer, exact)."""
    mask = run.mask.cpu().numpy().astype(bool)
    cnt = run.cnt.cpu().numpy()
    cols = run.cols.cpu().numpy()
    B, Ha, NB, _ = mask.shape
    m2 = mask.reshape(-1, NB)
    c2 = cols.reshape(-1, NB)
    n2 = cnt.reshape(-1)
    assert np.array_equal(n2, m2.sum(axis=1))
    for r in range(m2.shape[0]):
        nz = np.nonzero(m2[r])[0]
        assert np.array_equal(c2[r, :n2[r]], nz)
        assert (c2[r, n2[r]:] == -1).all()
    if run.order is not None:
        order = run.order.cpu().numpy()
        assert np.array_equal(np.sort(order), np.arange(m2.shape[0]))
        w = n2[order]
        assert (np.diff(w) <= 0).all()
        ties = np.diff(w) == 0
        assert (np.diff(order)[ties] > 0).all()
    # diagonal always retained
    idx = np.arange(NB)
    assert mask[:, :, idx, idx].all()


def retained_fraction(run: Run, tabs=None):
    sizes = tabs.sizes if tabs is not None else None
    return O.retained_fraction(run.mask.cpu().numpy().astype(bool), run.w.n_tokens, run.w.block, sizes=sizes)
