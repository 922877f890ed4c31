"""Plain CPU fp64 oracle of the Token Radius Attention (TRA) hot path.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import or run this module.  The GPU library never calls
it, and it shares no code, table or helper with the library: every quantity
here is recomputed from the paper's definitions.

Precision: all floating-point work is fp64 (numpy, and torch CPU ops in
float64 for the large matrix products, softmax and exponentials).  Integer
geometry is numpy int64.

Conventions
-----------
* Raster token index i = (f*H + x)*W + y on an F x H x W latent grid
  (Sec. 2.1: a token carries a coordinate (f, x, y)).
* Tensors per head are (N, d) in raster order.
* "FULL" radius (the full-support candidate radius of Sec. 3.2) is returned as
  ``RADIUS_FULL`` (2**31 - 1), matching the library's sentinel value, and is
  treated as an infinite radius.

Readings of the paper this oracle takes where the paper is silent are listed in
the design notes; each function below names the passage it follows.
"""
from __future__ import annotations

import math
from statistics import NormalDist

import numpy as np
import torch
from scipy.special import erfc

RADIUS_FULL = 2 ** 31 - 1
PAD = -1  # an empty position of a padded block layout

__all__ = [
    "RADIUS_FULL", "PAD", "grid_coords", "tile_major_order", "tile_aligned_order",
    "block_tokens", "block_sizes", "block_bounds",
    "scores", "softmax_rows", "dense_attention", "entropy_from_probs",
    "entropy_from_scores", "token_budget", "n_cap", "threshold_table",
    "within_radius", "grid_count_bruteforce", "disk_count_table", "grid_count",
    "select_radius", "select_radius_linear", "token_mask_rows",
    "block_mask_rows", "masked_attention_rows", "retained_fraction",
    "top_tau_support", "analytic_radius", "token_budget_lognormal",
    "lognormal_top_mass", "normal_quantile", "normal_tail", "threshold_table_1d",
    "within_radius_1d", "joint_order", "token_attention_rows",
]


# ============================================================ geometry, layout
def grid_coords(F: int, H: int, W: int):
    """(f, x, y) of every raster token (Sec. 2.1)."""
    i = np.arange(F * H * W, dtype=np.int64)
    return i // (H * W), (i // W) % H, i % W


def tile_major_order(F: int, H: int, W: int, tile_h: int, tile_w: int) -> np.ndarray:
    """Tile-major token order (Sec. 3.3, "Flash Radius Mask Kernel"; App. C.1,
    "Kernel execution").

    Each H x W frame is cut into tile_h x tile_w tiles (edge tiles clipped, not
    padded); tokens are listed frame by frame, tile row by tile row, tile by
    tile, and row-major inside a tile.  Returns perm with perm[p] = raster index
    of the token at tile-major position p.
    """
    frame = []
    for ty in range(0, H, tile_h):
        for tx in range(0, W, tile_w):
            for x in range(ty, min(H, ty + tile_h)):
                for y in range(tx, min(W, tx + tile_w)):
                    frame.append(x * W + y)
    frame = np.asarray(frame, dtype=np.int64)
    return np.concatenate([f * H * W + frame for f in range(F)])


def joint_order(perm_video, text_tokens: int) -> np.ndarray:
    """Sequence order of joint text-video attention (Sec. 3.2): the video tokens
    in tile-major order, then the text tokens (indices N .. N+T-1) unchanged."""
    perm_video = np.asarray(perm_video, dtype=np.int64)
    n = perm_video.shape[0]
    return np.concatenate([perm_video, np.arange(n, n + text_tokens, dtype=np.int64)])


def tile_aligned_order(F: int, H: int, W: int, tile_h: int, tile_w: int, b: int,
                       text_tokens: int = 0) -> np.ndarray:
    """Tile-aligned padded blocks: the tile-major order of Sec. 3.3 with every
    block holding exactly one tile_h x tile_w tile of one frame (tile_h *
    tile_w = b).  App. D names the work a retained block does on keys outside
    a query's radius as the method's main limitation; a block that is one
    spatial tile has the smallest footprint a block of b tokens can have.

    Frames in order, tiles in tile-row-major order inside a frame, tokens
    row-major inside a tile; a tile clipped by the frame edge fills the first
    positions of its block and the rest of the block is padding (PAD).  Text
    tokens N .. N+T-1 follow in blocks of b, the last one padded.  Returns perm
    of length NB * b: perm[p] = token index at position p, or PAD.
    """
    if tile_h * tile_w != b:
        raise ValueError("a tile must hold exactly one block")
    out = []
    for f in range(F):
        for x0 in range(0, H, tile_h):
            for y0 in range(0, W, tile_w):
                blk = [(f * H + x) * W + y for x in range(x0, min(H, x0 + tile_h))
                       for y in range(y0, min(W, y0 + tile_w))]
                out += blk + [PAD] * (b - len(blk))
    N = F * H * W
    for s0 in range(0, text_tokens, b):
        blk = list(range(N + s0, N + min(text_tokens, s0 + b)))
        out += blk + [PAD] * (b - len(blk))
    return np.asarray(out, dtype=np.int64)


def block_tokens(perm, b: int, u: int) -> np.ndarray:
    """Tokens of block u: positions [u*b, (u+1)*b) of the sequence order
    (App. C: blocks of b consecutive positions), padding dropped."""
    r = np.asarray(perm[u * b:(u + 1) * b], dtype=np.int64)
    return r[r >= 0]


def block_sizes(perm, b: int) -> np.ndarray:
    """Number of tokens in each block of the sequence order (padding excluded)."""
    perm = np.asarray(perm, dtype=np.int64)
    nb = -(-perm.shape[0] // b)
    return np.array([len(block_tokens(perm, b, u)) for u in range(nb)], dtype=np.int64)


def block_bounds(N: int, b: int):
    """Block u holds tile-major positions [u*b, min((u+1)*b, N)) (App. C:
    B = ceil(S/b) blocks of b tokens)."""
    nb = -(-N // b)
    return [(u * b, min((u + 1) * b, N)) for u in range(nb)]


# ===================================================== attention and entropy
def _t(x):
    return torch.as_tensor(np.asarray(x, dtype=np.float64))


def scores(q, k):
    """s_ij = q_i . k_j / sqrt(d) (Sec. 2.1, Eq. 1), fp64."""
    q, k = _t(q), _t(k)
    return (q @ k.T) / math.sqrt(q.shape[1])


def softmax_rows(s):
    """p_ij = exp(s_ij) / sum_n exp(s_in) (Eq. 1); entries at -inf get 0."""
    s = _t(s) if not isinstance(s, torch.Tensor) else s
    m = s.max(dim=1, keepdim=True).values
    e = torch.exp(s - m)
    return e / e.sum(dim=1, keepdim=True)


def dense_attention(q, k, v, return_probs=False):
    """o_i = sum_j p_ij v_j (Eq. 1).  q: (R, d) rows, k, v: (N, d)."""
    p = softmax_rows(scores(q, k))
    o = p @ _t(v)
    return (o.numpy(), p) if return_probs else o.numpy()


def entropy_from_probs(p) -> np.ndarray:
    """H_i = -sum_j p_ij log p_ij in nats, with 0 log 0 = 0 (Sec. 2.2, Eq. 2)."""
    p = p if isinstance(p, torch.Tensor) else _t(p)
    safe = torch.where(p > 0, p, torch.ones_like(p))
    return (-(p * torch.log(safe)).sum(dim=1)).numpy()


def entropy_from_scores(q, k):
    """H_i = log Z_i - sum_j p_ij s_ij over whole rows (the identity behind the
    fused entropy kernel, App. C.2), fp64: log Z by logsumexp, p by softmax."""
    s = scores(q, k)
    p = softmax_rows(s)
    return (torch.logsumexp(s, dim=1) - (p * s).sum(dim=1)).numpy()


# ====================================================== entropy -> budget
def token_budget(H, tau: float, N: int) -> np.ndarray:
    """K_hat = ceil(tau * exp(H)) (Sec. 3.1, Eq. 8; App. C.1,
    Eq. implementation-budget-radius), in fp64, clamped to the key count
    range [1, N] (N the number of keys of the row; a budget outside it has no
    meaning)."""
    H = np.asarray(H, dtype=np.float64)
    k = np.ceil(tau * np.exp(H))
    return np.clip(k, 1, N).astype(np.int64)


def normal_quantile(p: float) -> float:
    """Phi^{-1}(p) of the standard normal (library routine, fp64)."""
    return NormalDist().inv_cdf(p)


def normal_tail(z):
    """Phibar(z) = 1 - Phi(z) = erfc(z / sqrt 2) / 2 (fp64)."""
    return 0.5 * erfc(np.asarray(z, dtype=np.float64) / math.sqrt(2.0))


def lognormal_top_mass(q, sigma):
    """L_LN(q) = Phibar(Phi^{-1}(1 - q) - sigma): the expected share of the total
    held by the largest fraction q of Lognormal(mu, sigma^2) samples (App. A.2,
    "Entropy-identified Lognormal mapping")."""
    q = np.asarray(q, dtype=np.float64)
    zq = np.vectorize(lambda a: NormalDist().inv_cdf(a))(1.0 - q)
    return normal_tail(zq - np.asarray(sigma, dtype=np.float64))


def token_budget_lognormal(H, tau: float, S: int) -> np.ndarray:
    """Lognormal entropy-to-budget mapping (App. A.2): the weights of a row of S
    keys are modelled as Lognormal(mu, sigma^2); entropy fixes
    sigma = sqrt(2 (log S - H)) (H = log S - sigma^2 / 2), and the retained
    fraction solving L_LN(q) = tau is B = Phibar(sigma - Phi^{-1}(tau)).  The key
    budget is ceil(S * B) in fp64, clamped to [1, S] (H above log S, possible
    only by rounding, is taken as log S)."""
    H = np.asarray(H, dtype=np.float64)
    sigma = np.sqrt(2.0 * np.maximum(0.0, math.log(S) - H))
    k = np.ceil(S * normal_tail(sigma - normal_quantile(tau)))
    return np.clip(k, 1, S).astype(np.int64)


# ====================================================== budget -> radius
def n_cap(H: int, W: int) -> int:
    """Largest squared in-frame distance (H-1)^2 + (W-1)^2: beyond it a disk
    covers its whole frame, so candidate squared radii stop there."""
    return (H - 1) ** 2 + (W - 1) ** 2


def threshold_table(ncap: int, F: int, gamma: float) -> np.ndarray:
    """thr[n, delta] = floor(n * exp(-2 gamma delta)), n in [0, ncap], delta in [0, F).

    For a squared base radius n (r = sqrt n) and an integer squared spatial
    distance D, the test d_s <= r phi(delta) of Eq. 15 with phi = exp(-gamma
    delta) (Eq. 10) is D <= n exp(-2 gamma delta), i.e. D <= thr[n, delta]."""
    n = np.arange(ncap + 1, dtype=np.float64)[:, None]
    delta = np.arange(F, dtype=np.float64)[None, :]
    return np.floor(n * np.exp(-2.0 * gamma * delta)).astype(np.int64)


def within_radius(D, n, delta, gamma: float):
    """Eq. 15 literally, in fp64: sqrt(D) <= sqrt(n) * exp(-gamma * delta),
    with the FULL radius treated as infinite (keeps every key)."""
    D = np.asarray(D, dtype=np.float64)
    n = np.asarray(n)
    r = np.where(n == RADIUS_FULL, np.inf, np.sqrt(n.astype(np.float64)))
    with np.errstate(invalid="ignore"):
        rho = r * np.exp(-gamma * np.asarray(delta, dtype=np.float64))
    return np.sqrt(D) <= rho


def threshold_table_1d(ncap: int, F: int, gamma: float) -> np.ndarray:
    """thr1[n, delta] = floor(((pi/2) n) exp(-gamma delta)): the sequence-distance
    ablation (App. C.1, Eq. area-matched-1d) replaces d_s by |i - j| and the
    radius by rho_1D = (pi/2) rho_2D^2 = (pi/2) n, so an integer distance passes
    iff |i - j| <= thr1[n, delta]."""
    n = np.arange(ncap + 1, dtype=np.float64)[:, None]
    delta = np.arange(F, dtype=np.float64)[None, :]
    return np.floor((math.pi / 2.0 * n) * np.exp(-gamma * delta)).astype(np.int64)


def within_radius_1d(dr, n, delta, gamma: float):
    """The 1-D test literally, in fp64: |dr| <= (pi/2) n exp(-gamma delta), the
    FULL radius infinite."""
    n = np.asarray(n)
    r = np.where(n == RADIUS_FULL, np.inf, (math.pi / 2.0) * n.astype(np.float64))
    with np.errstate(invalid="ignore"):
        rho = r * np.exp(-gamma * np.asarray(delta, dtype=np.float64))
    return np.abs(np.asarray(dr, dtype=np.float64)) <= rho


def grid_count_bruteforce(i: int, n: int, F: int, H: int, W: int, gamma: float) -> int:
    """C_i^grid(r) of Sec. 3.2, Eq. 13, by checking every key j against Eq. 15."""
    f, x, y = grid_coords(F, H, W)
    D = (x - x[i]) ** 2 + (y - y[i]) ** 2
    return int(within_radius(D, n, np.abs(f - f[i]), gamma).sum())


def disk_count_table(H: int, W: int, tmax: int) -> np.ndarray:
    """disk[x, y, T] = #{(x', y') in the H x W frame : (x-x')^2 + (y-y')^2 <= T},
    T in [0, tmax].  The per-frame lattice count of Eq. 13."""
    xs, ys = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    xs, ys = xs.ravel(), ys.ravel()
    out = np.empty((H, W, tmax + 1), dtype=np.int64)
    for x in range(H):
        for y in range(W):
            D = (xs - x) ** 2 + (ys - y) ** 2
            out[x, y] = np.cumsum(np.bincount(D, minlength=tmax + 1)[: tmax + 1])
    return out


def grid_count(f, x, y, n, F: int, thr: np.ndarray, disk: np.ndarray) -> np.ndarray:
    """C_i^grid for arrays of queries (f, x, y) and squared radii n (Eq. 13):
    sum over frames t of the lattice points of frame t inside the disk of
    squared radius thr[n, |t - f|].  n == FULL counts every key."""
    f, x, y, n = (np.asarray(a, dtype=np.int64) for a in (f, x, y, n))
    H, W, T1 = disk.shape
    full = n == RADIUS_FULL
    nn = np.where(full, 0, n)
    total = np.zeros(f.shape, dtype=np.int64)
    for t in range(F):
        T = np.minimum(thr[nn, np.abs(t - f)], T1 - 1)
        total += disk[x, y, T]
    return np.where(full, F * H * W, total)


def select_radius_linear(khat: int, i: int, F: int, H: int, W: int, gamma: float) -> int:
    """r_i = min{r in R : C_i^grid(r) >= K_hat} (Sec. 3.2, Eq. 14) by scanning
    every candidate squared radius n = 0, 1, ..., n_cap in order, counting by
    brute force; the full-support radius if none reaches K_hat."""
    for n in range(n_cap(H, W) + 1):
        if grid_count_bruteforce(i, n, F, H, W, gamma) >= khat:
            return n
    return RADIUS_FULL


def select_radius(khat, f, x, y, F: int, thr: np.ndarray, disk: np.ndarray) -> np.ndarray:
    """Eq. 14 for arrays of queries: the smallest n in [0, n_cap] with
    C_i^grid(n) >= K_hat, else FULL.  C_i^grid is non-decreasing in n (a larger
    disk contains a smaller one), so the minimum is found by bisection."""
    khat = np.asarray(khat, dtype=np.int64)
    ncap = thr.shape[0] - 1
    lo = np.zeros(khat.shape, dtype=np.int64)
    hi = np.full(khat.shape, ncap, dtype=np.int64)
    ok_at_cap = grid_count(f, x, y, hi, F, thr, disk) >= khat
    while True:
        active = lo < hi
        if not active.any():
            break
        mid = (lo + hi) // 2
        ge = grid_count(f, x, y, mid, F, thr, disk) >= khat
        hi = np.where(active & ge, mid, hi)
        lo = np.where(active & ~ge, mid + 1, lo)
    return np.where(ok_at_cap, lo, RADIUS_FULL)


def analytic_radius(khat, f, F: int, gamma: float) -> np.ndarray:
    """Continuous initialisation r~ = sqrt(K_hat / (pi * sum_t phi^2)) of
    Sec. 3.2, Eq. 12 (boundaries and lattice effects ignored)."""
    t = np.arange(F)[None, :]
    s = np.exp(-2.0 * gamma * np.abs(t - np.asarray(f)[:, None])).sum(axis=1)
    return np.sqrt(np.asarray(khat, dtype=np.float64) / (math.pi * s))


# ====================================================== radius -> masks
def token_mask_rows(rows, n_rows, F: int, H: int, W: int, gamma: float, keys=None,
                    distance: str = "2d"):
    """M_ij for video query rows ``rows`` (raster indices) with squared radii
    ``n_rows`` against keys ``keys`` (token indices, default all video tokens).
    Video keys: M_ij = [d_s(i, j) <= r_i phi(|f_j - f_i|)] (Sec. 3.2, Eq. 15), or
    for distance "1d" the sequence-distance ablation |i - j| <= (pi/2) n_i
    phi(|f_j - f_i|) (App. C.1).  Text keys (index >= F*H*W) are always visible
    (Sec. 3.2: all text keys remain visible).  Returns a bool torch tensor."""
    N = F * H * W
    f, x, y = grid_coords(F, H, W)
    rows = np.asarray(rows, dtype=np.int64)
    keys = np.arange(N) if keys is None else np.asarray(keys, dtype=np.int64)
    text = keys >= N
    kv = np.where(text, 0, keys)
    fr, xr, yr = (torch.as_tensor(a[rows])[:, None] for a in (f, x, y))
    fk, xk, yk = (torch.as_tensor(a[kv])[None, :] for a in (f, x, y))
    delta = (fr - fk).abs().to(torch.float64)
    n = torch.as_tensor(np.asarray(n_rows, dtype=np.int64))
    full = (n == RADIUS_FULL)[:, None]
    if distance == "2d":
        D = ((xr - xk) ** 2 + (yr - yk) ** 2).to(torch.float64)
        r = torch.where(n == RADIUS_FULL, torch.tensor(math.inf, dtype=torch.float64),
                        torch.sqrt(n.to(torch.float64)))[:, None]
        m = torch.sqrt(D) <= r * torch.exp(-gamma * delta)
    elif distance == "1d":
        dr = (torch.as_tensor(rows)[:, None] - torch.as_tensor(kv)[None, :]).abs().to(torch.float64)
        r = torch.where(n == RADIUS_FULL, torch.tensor(math.inf, dtype=torch.float64),
                        (math.pi / 2.0) * n.to(torch.float64))[:, None]
        m = dr <= r * torch.exp(-gamma * delta)
    else:
        raise ValueError(distance)
    return (m | full) | torch.as_tensor(text)[None, :]


def block_mask_rows(n_raster, perm, b: int, F: int, H: int, W: int, gamma: float,
                    blocks, rule: str = "vote", distance: str = "2d"):
    """Block-mask rows M[u, :] of Alg. 1 (App. C.1) for the query blocks
    ``blocks``, from per-token squared radii ``n_raster`` (token order).

    ``perm`` is the sequence order (tile-major video tokens, then any text
    tokens, with PAD at empty positions of a padded layout); blocks are b
    consecutive positions of it.  For a video query block
    u and a video key block v, every valid key column j of v gets the count c_j
    of valid queries i of u with M_ij = 1 (Eq. 15, or the 1-D test).
    C = {j : c_j > 0}, C_hi = {j : c_j > n_u / 3}.
    vote:  retained iff |C| > 0 and 10 |C_hi| > 6 |C|   (Alg. 1);
    union: retained iff |C| > 0.
    The diagonal block (u, u) is always retained (every query keeps its own key).
    Joint text-video attention (Alg. 1, u >= B_v or v >= B_v): a block holding
    any text token is retained in every row, and its own row retains every
    block (reading: a block mixing the last video tokens with the first text
    tokens counts as a text block, so every text key stays visible).
    n_u is the number of valid queries of u (padding is neither a query nor a
    key); the high-coverage test is written 3 c_j > n_u.  Returns a bool array
    (len(blocks), NB).
    """
    perm = np.asarray(perm, dtype=np.int64)
    P = perm.shape[0]
    N = F * H * W
    nb = -(-P // b)
    members = [block_tokens(perm, b, v) for v in range(nb)]
    text_block = np.array([bool((m >= N).any()) for m in members])
    valid = np.nonzero(perm >= 0)[0]
    keys = perm[valid]
    out = np.zeros((len(blocks), nb), dtype=bool)
    for r, u in enumerate(blocks):
        if text_block[u]:
            out[r] = True
            continue
        rows = members[u]
        n_u = len(rows)
        M = token_mask_rows(rows, np.asarray(n_raster)[rows], F, H, W, gamma, keys=keys,
                            distance=distance)
        c = np.zeros(nb * b, dtype=np.int64)           # per key column, by position
        c[valid] = M.sum(dim=0).numpy()
        c = c.reshape(nb, b)
        nonempty = (c > 0).sum(axis=1)
        high = (3 * c > n_u).sum(axis=1)
        if rule == "vote":
            keep = (nonempty > 0) & (10 * high > 6 * nonempty)
        elif rule == "union":
            keep = nonempty > 0
        else:
            raise ValueError(rule)
        keep[u] = True
        keep[text_block] = True
        out[r] = keep
    return out


def masked_attention_rows(q, k, v, perm, b: int, blocks, mask_rows, return_lse=False):
    """TRA attention (Sec. 3.2, Eq. 16) at block granularity: a query of block u
    attends, with one softmax, to every key of every key block v with
    M[u, v] = 1, and to no other key.

    q, k, v: (N, d) raster order; blocks are positions of ``perm`` as in
    block_mask_rows (padding dropped).  Returns the output rows of the queries
    in ``blocks`` as (rows, O)."""
    perm = np.asarray(perm, dtype=np.int64)
    qt, kt, vt = _t(q), _t(k), _t(v)
    alpha = 1.0 / math.sqrt(qt.shape[1])
    rows_out, o_out, lse_out = [], [], []
    for r, u in enumerate(blocks):
        rows = block_tokens(perm, b, u)
        keys = np.concatenate([block_tokens(perm, b, v) for v in np.nonzero(mask_rows[r])[0]])
        s = alpha * (qt[rows] @ kt[keys].T)
        m = s.max(dim=1, keepdim=True).values
        e = torch.exp(s - m)
        z = e.sum(dim=1, keepdim=True)
        o_out.append(((e / z) @ vt[keys]).numpy())
        lse_out.append((m + torch.log(z))[:, 0].numpy())
        rows_out.append(rows)
    rows_out = np.concatenate(rows_out)
    if return_lse:
        return rows_out, np.concatenate(o_out), np.concatenate(lse_out)
    return rows_out, np.concatenate(o_out)


def token_attention_rows(q, k, v, perm, b: int, blocks, mask_rows, n_tok, F: int, H: int, W: int,
                         gamma: float, distance: str = "2d", return_lse=False):
    """TRA attention at token level (Sec. 3.2, Eq. 16 with the bias B(M) of
    Eq. tra_attention_final) inside the retained blocks: a query i of block u
    attends, with one softmax, to the keys j of the key blocks v with
    M[u, v] = 1 for which M_ij = 1 (Eq. 15, or the 1-D test; text keys always,
    text queries to every such key), and to no other key.  With block rows from
    the union rule every covered key lies in a retained block, so this is Eq. 16
    over all keys.  n_tok: per-token squared radii (token order).

    q, k, v: (S, d) token order.  Returns (rows, O) [and lse] for the queries of
    ``blocks``."""
    perm = np.asarray(perm, dtype=np.int64)
    N = F * H * W
    qt, kt, vt = _t(q), _t(k), _t(v)
    alpha = 1.0 / math.sqrt(qt.shape[1])
    n_tok = np.asarray(n_tok)
    rows_out, o_out, lse_out = [], [], []
    for r, u in enumerate(blocks):
        rows = block_tokens(perm, b, u)
        keys = np.concatenate([block_tokens(perm, b, v) for v in np.nonzero(mask_rows[r])[0]])
        video = rows < N
        M = torch.ones(len(rows), len(keys), dtype=torch.bool)
        if video.any():
            M[torch.as_tensor(video)] = token_mask_rows(rows[video], n_tok[rows[video]], F, H, W, gamma,
                                                        keys=keys, distance=distance)
        s = alpha * (qt[rows] @ kt[keys].T)
        s = torch.where(M, s, torch.tensor(-math.inf, dtype=torch.float64))
        m = s.max(dim=1, keepdim=True).values
        e = torch.exp(s - m)
        z = e.sum(dim=1, keepdim=True)
        o_out.append(((e / z) @ vt[keys]).numpy())
        lse_out.append((m + torch.log(z))[:, 0].numpy())
        rows_out.append(rows)
    rows_out = np.concatenate(rows_out)
    if return_lse:
        return rows_out, np.concatenate(o_out), np.concatenate(lse_out)
    return rows_out, np.concatenate(o_out)


def retained_fraction(mask, N: int, b: int, sizes=None) -> float:
    """Fraction of query-key interactions inside retained blocks,
    sum over retained (u, v) of n_u n_v, over (heads * N^2).  mask: (..., NB, NB).
    sizes: tokens per block (block_sizes); default b per block with the last
    one ragged (a packed order of N tokens)."""
    mask = np.asarray(mask, dtype=bool)
    nb = mask.shape[-1]
    if sizes is not None:
        n = np.asarray(sizes, dtype=np.int64)
    else:
        n = np.full(nb, b, dtype=np.int64)
        n[-1] = N - (nb - 1) * b
    per = np.einsum("...uv,u,v->...", mask.astype(np.int64), n, n)
    return float(np.sum(per) / (np.prod(mask.shape[:-2]) * N * N))


# ====================================================== diagnostics
def top_tau_support(p, tau: float) -> np.ndarray:
    """Oracle support size K_i^tau = min{k : top-k probability mass >= tau}
    (Sec. 3.1, Eq. 4).  A diagnostic: it needs the whole sorted row."""
    p = p.numpy() if isinstance(p, torch.Tensor) else np.asarray(p, dtype=np.float64)
    cs = np.cumsum(-np.sort(-p, axis=1), axis=1)
    return (cs < tau).sum(axis=1) + 1
