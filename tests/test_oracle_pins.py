"""Pins of the CPU oracle against closed forms, invariants, hand-derived
fixtures and brute force -- never against a retyping of its own formulas.

Each test names the property of the paper or of mathematics that fixes the
expected value.
"""
import math
import os

import numpy as np
import pytest

import oracle as O
import synth

RNG = np.random.default_rng(12345)


def _read_golden(golden_dir, name):
    rows = []
    with open(os.path.join(golden_dir, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(t) for t in line.split()])
    return rows


# ------------------------------------------------------------------ attention
def test_two_key_closed_form():
    """d = 1, q = 1, keys ln 3 and 0: p = (3/4, 1/4) exactly, so
    o = 3/4 v1 + 1/4 v2 and H = ln 4 - (3/4) ln 3 (Eq. 1, Eq. 2)."""
    q = np.array([[1.0]])
    k = np.array([[math.log(3.0)], [0.0]])
    v = np.array([[2.0, -1.0], [6.0, 3.0]])
    o, p = O.dense_attention(q, k, v, return_probs=True)
    assert np.allclose(p.numpy(), [[0.75, 0.25]], atol=1e-15)
    assert np.allclose(o, [[3.0, 0.0]], atol=1e-14)
    H = O.entropy_from_probs(p)
    assert abs(H[0] - (math.log(4) - 0.75 * math.log(3))) < 1e-14
    H2 = O.entropy_from_scores(q, k)
    assert abs(H2[0] - (math.log(4) - 0.75 * math.log(3))) < 1e-14


@pytest.mark.parametrize("N", [7, 256, 1000])
def test_uniform_scores_give_log_n(N):
    """All keys equal -> every p_ij = 1/N -> H = log N, the upper bound of Eq. 2,
    and o = the mean of v."""
    d = 16
    q = RNG.standard_normal((5, d))
    k = np.tile(RNG.standard_normal((1, d)), (N, 1))
    v = RNG.standard_normal((N, 3))
    o, p = O.dense_attention(q, k, v, return_probs=True)
    H = O.entropy_from_probs(p)
    assert np.allclose(H, math.log(N), atol=1e-12)
    assert np.allclose(o, v.mean(axis=0), atol=1e-12)
    H2 = O.entropy_from_scores(q, k)
    assert np.allclose(H2, math.log(N), atol=1e-12)


def test_one_hot_scores_give_zero_entropy():
    """One key ahead of all others by a score margin of 40: H < N e^-40 * 41,
    which is ~0 (the lower bound of Eq. 2), and o = that key's value."""
    N, d = 256, 4
    k = np.zeros((N, d))
    k[17, 0] = 40.0 * math.sqrt(d)
    q = np.array([[1.0, 0.0, 0.0, 0.0]])
    v = RNG.standard_normal((N, 2))
    o, p = O.dense_attention(q, k, v, return_probs=True)
    H = O.entropy_from_probs(p)
    assert 0.0 <= H[0] < N * math.exp(-40) * 41
    assert np.allclose(o[0], v[17], atol=1e-12)
    H2 = O.entropy_from_scores(q, k)
    assert abs(H2[0]) < 1e-9


@pytest.mark.parametrize("m", [3, 37, 151])
def test_m_equal_keys_give_log_m(m):
    """m keys share the top score and the rest trail by 30: the distribution is
    uniform on m keys up to ~N e^-30, so H = log m (Eq. 6, m = exp(H)) and the
    budget is ceil(0.9 m) (Eq. 8)."""
    N, d = 400, 8
    k = np.zeros((N, d))
    top = RNG.choice(N, m, replace=False)
    k[top, 0] = 30.0 * math.sqrt(d)
    q = np.eye(d)[:1]
    _, p = O.dense_attention(q, k, np.zeros((N, 1)), return_probs=True)
    H = O.entropy_from_probs(p)
    assert abs(H[0] - math.log(m)) < N * math.exp(-30) * 31 + 1e-12
    assert O.token_budget(H, 0.9, N)[0] == math.ceil(0.9 * m)


def test_lognormal_scores_entropy():
    """i.i.d. N(0, sigma^2) scores: E[e^s] = e^{sigma^2/2} and
    E[s e^s] / E[e^s] = sigma^2, so H -> log N - sigma^2 / 2 for large N (the
    lognormal case of the distributional analysis, App. A.2).  Statistical,
    tolerance ~5 standard errors."""
    N, d, sigma = 200_000, 4, 1.0
    k = RNG.standard_normal((N, d))
    q = np.array([[sigma * math.sqrt(d), 0.0, 0.0, 0.0]])
    _, p = O.dense_attention(q, k, np.zeros((N, 1)), return_probs=True)
    H = O.entropy_from_probs(p)[0]
    assert abs(H - (math.log(N) - sigma ** 2 / 2)) < 0.02


def test_entropy_bounds_and_two_forms_agree():
    """0 <= H <= log N (Eq. 2), and the direct -sum p log p agrees with the
    identity H = log Z - sum_j p_j s_j (App. C.2) to 1e-12."""
    w = synth.workload("tiny")
    q, k, v = synth.generate(w)
    q, k, v = (synth.to_f64(a[0, 1], w.dtype) for a in (q, k, v))
    o, p = O.dense_attention(q, k, v, return_probs=True)
    H = O.entropy_from_probs(p)
    assert (H >= 0).all() and (H <= math.log(256) + 1e-12).all()
    H2 = O.entropy_from_scores(q, k)
    assert np.abs(H2 - H).max() < 1e-12


def test_attention_key_permutation_invariance():
    """Permuting keys and values together leaves o_i unchanged (Eq. 1 sums over
    all keys)."""
    q = RNG.standard_normal((9, 8))
    k = RNG.standard_normal((50, 8))
    v = RNG.standard_normal((50, 5))
    pi = RNG.permutation(50)
    assert np.allclose(O.dense_attention(q, k, v), O.dense_attention(q, k[pi], v[pi]),
                       atol=1e-13)


def test_top_tau_support_uniform():
    """Uniform mass on m keys: the smallest top-k set reaching tau has
    ceil(tau m) keys (Eq. 4), matching the entropy budget (Eq. 8)."""
    for m in (5, 23, 200):
        p = np.zeros((1, 400))
        p[0, :m] = 1.0 / m
        assert O.top_tau_support(p, 0.9)[0] == math.ceil(0.9 * m - 1e-9)


# ------------------------------------------------------------------ budget
def test_budget_clamps_and_monotone():
    H = np.linspace(-5, 15, 2001)
    kh = O.token_budget(H, 0.9, 5000)
    assert kh.min() == 1 and kh.max() == 5000
    assert (np.diff(kh) >= 0).all()


# ------------------------------------------------------------------ layout
def test_tile_order_golden(golden_dir):
    want = np.array(_read_golden(golden_dir, "tile_order_F2_H3_W5_tile2x2.txt")[0], dtype=np.int64)
    assert (O.tile_major_order(2, 3, 5, 2, 2) == want).all()


@pytest.mark.parametrize("grid,tile", [((4, 8, 8), (8, 8)), ((21, 30, 52), (8, 16)),
                                       ((3, 45, 80), (8, 16))])
def test_tile_order_is_bijection(grid, tile):
    F, H, W = grid
    perm = O.tile_major_order(F, H, W, *tile)
    assert np.array_equal(np.sort(perm), np.arange(F * H * W))


def test_tiny_tile_order_is_identity():
    """An 8 x 8 frame with 8 x 8 tiles is one tile, so tile-major = raster."""
    assert np.array_equal(O.tile_major_order(4, 8, 8, 8, 8), np.arange(256))


def test_full_tiles_are_contiguous_runs():
    """Every full tile occupies tile_h*tile_w consecutive positions whose
    coordinates span exactly the tile (Sec. 3.3: neighbouring tokens become
    contiguous in the sequence)."""
    F, H, W = 2, 16, 32
    perm = O.tile_major_order(F, H, W, 8, 16)
    f, x, y = O.grid_coords(F, H, W)
    for s in range(0, F * H * W, 128):
        r = perm[s:s + 128]
        assert len(set(f[r])) == 1
        assert x[r].max() - x[r].min() == 7 and y[r].max() - y[r].min() == 15


# ------------------------------------------------- tile-aligned padded blocks
def test_tile_aligned_order_golden(golden_dir):
    want = np.array(_read_golden(golden_dir, "tile_aligned_order_F2_H3_W5_tile2x2_b4_T3.txt")[0],
                    dtype=np.int64)
    assert np.array_equal(O.tile_aligned_order(2, 3, 5, 2, 2, 4, text_tokens=3), want)


@pytest.mark.parametrize("grid,tile,T", [((21, 30, 52), (8, 16), 0), ((3, 45, 80), (8, 16), 0),
                                         ((2, 5, 9), (2, 4), 5), ((3, 11, 29), (8, 16), 130)])
def test_tile_aligned_blocks_are_single_tiles(grid, tile, T):
    """Every token appears exactly once; every video block lies in one frame and
    one tile (its coordinates inside [x0, x0 + tile_h) x [y0, y0 + tile_w) of
    one tile origin); tokens fill a prefix of the block; a text block holds
    only text tokens; the block count is F * ceil(H/th) * ceil(W/tw) + ceil(T/b)."""
    F, H, W = grid
    th, tw = tile
    b = th * tw
    N = F * H * W
    perm = O.tile_aligned_order(F, H, W, th, tw, b, text_tokens=T)
    nb = perm.shape[0] // b
    assert perm.shape[0] % b == 0
    assert nb == F * (-(-H // th)) * (-(-W // tw)) + (-(-T // b))
    valid = perm[perm >= 0]
    assert np.array_equal(np.sort(valid), np.arange(N + T))
    f, x, y = O.grid_coords(F, H, W)
    for u in range(nb):
        blk = perm[u * b:(u + 1) * b]
        n = int((blk >= 0).sum())
        assert n > 0 and (blk[:n] >= 0).all() and (blk[n:] == O.PAD).all()
        r = blk[:n]
        if (r >= N).any():
            assert (r >= N).all()
            continue
        assert len(set(f[r])) == 1
        assert len(set(x[r] // th)) == 1 and len(set(y[r] // tw)) == 1
    assert np.array_equal(O.block_sizes(perm, b), [(perm[u * b:(u + 1) * b] >= 0).sum() for u in range(nb)])


def test_tile_aligned_equals_tile_major_when_tiles_divide_the_frame():
    """With tiles dividing the frame exactly there is no padding and the two
    orders coincide."""
    assert np.array_equal(O.tile_aligned_order(3, 16, 32, 8, 16, 128), O.tile_major_order(3, 16, 32, 8, 16))
    assert np.array_equal(O.tile_aligned_order(4, 8, 8, 8, 8, 64), np.arange(256))


def _brute_block_mask(n_raster, members, F, H, W, gamma, rule):
    """Alg. 1 by loops over explicit token lists: c_j counts the queries i of u
    with sqrt((x_i-x_j)^2 + (y_i-y_j)^2) <= sqrt(n_i) exp(-gamma |f_i - f_j|)."""
    nb = len(members)
    out = np.zeros((nb, nb), dtype=bool)
    for u in range(nb):
        for v in range(nb):
            c = []
            for j in members[v]:
                fj, xj, yj = j // (H * W), (j // W) % H, j % W
                cnt = 0
                for i in members[u]:
                    fi, xi, yi = i // (H * W), (i // W) % H, i % W
                    if math.sqrt((xi - xj) ** 2 + (yi - yj) ** 2) <= \
                            math.sqrt(n_raster[i]) * math.exp(-gamma * abs(fi - fj)):
                        cnt += 1
                c.append(cnt)
            C = sum(1 for cj in c if cj > 0)
            Chi = sum(1 for cj in c if 3 * cj > len(members[u]))
            out[u, v] = (C > 0 and (10 * Chi > 6 * C if rule == "vote" else True)) or u == v
    return out


@pytest.mark.parametrize("rule", ["vote", "union"])
def test_block_mask_on_padded_blocks_matches_brute_force(rule):
    """Tile-aligned blocks with clipped edge tiles (2 x 5 x 6 grid, 2 x 4
    tiles, b = 8: blocks of 8, 4, 8, 4 and 2 tokens per frame): the oracle's
    mask equals Alg. 1 evaluated by loops over each block's token list, with
    padding neither a query nor a key."""
    F, H, W, th, tw, gamma = 2, 5, 6, 2, 4, 0.6
    perm = O.tile_aligned_order(F, H, W, th, tw, th * tw)
    nb = perm.shape[0] // 8
    members = [O.block_tokens(perm, 8, u) for u in range(nb)]
    assert sorted(len(m) for m in members[:6]) == [2, 4, 4, 4, 8, 8]
    rng = np.random.default_rng(5)
    n = rng.integers(0, 12, size=F * H * W)
    got = O.block_mask_rows(n, perm, 8, F, H, W, gamma, range(nb), rule=rule)
    assert np.array_equal(got, _brute_block_mask(n, members, F, H, W, gamma, rule))
    assert 0 < got.sum() < nb * nb


def test_masked_attention_on_padded_blocks():
    """Padded blocks: a full mask gives dense attention over every token; the
    identity mask gives attention restricted to each tile's own tokens."""
    w = synth.workload("tiny")
    q, k, v = (synth.to_f64(a[0, 0], w.dtype) for a in synth.generate(w))
    perm = O.tile_aligned_order(4, 8, 8, 3, 8, 24)           # 8 rows = 3 + 3 + 2: partial tiles
    nb = perm.shape[0] // 24
    rows, o = O.masked_attention_rows(q, k, v, perm, 24, range(nb), np.ones((nb, nb), bool))
    assert np.array_equal(np.sort(rows), np.arange(256))
    assert np.abs(o - O.dense_attention(q[rows], k, v)).max() < 1e-12
    rows, o = O.masked_attention_rows(q, k, v, perm, 24, [2, 5], np.eye(nb, dtype=bool)[[2, 5]])
    at = 0
    for u in (2, 5):
        idx = O.block_tokens(perm, 24, u)
        want = O.dense_attention(q[idx], k[idx], v[idx])
        assert np.abs(o[at:at + len(idx)] - want).max() < 1e-12
        at += len(idx)


def test_retained_fraction_with_block_sizes():
    sizes = np.array([8, 4, 2])
    eye = np.eye(3, dtype=bool)[None]
    assert abs(O.retained_fraction(eye, 14, 8, sizes=sizes) - (64 + 16 + 4) / 196) < 1e-15


# ------------------------------------------------------------------ radius
def test_threshold_golden(golden_dir):
    for gamma, n, *want in _read_golden(golden_dir, "thresholds.txt"):
        thr = O.threshold_table(int(n), 4, gamma)
        assert list(thr[int(n)]) == [int(t) for t in want], (gamma, n)


@pytest.mark.parametrize("name", ["tiny", "wan13b_480p", "wan14b_720p", "hunyuan_720p"])
def test_threshold_equals_literal_mask_test(name):
    """The integer test D <= thr[n][delta] equals the literal fp64 test of
    Eq. 15 at the boundary for every candidate n and every temporal distance of
    the grid: D = thr passes and D = thr + 1 fails.  This also shows that no
    n * exp(-2 gamma delta) sits within rounding of an integer for these grids."""
    w = synth.workload(name)
    nc = O.n_cap(w.height, w.width)
    thr = O.threshold_table(nc, w.frames, w.gamma)
    n = np.arange(nc + 1)[:, None].repeat(w.frames, 1)
    delta = np.arange(w.frames)[None, :].repeat(nc + 1, 0)
    assert O.within_radius(thr, n, delta, w.gamma).all()
    assert not O.within_radius(thr + 1, n, delta, w.gamma).any()
    assert (thr[:, 0] == np.arange(nc + 1)).all()
    assert (np.diff(thr, axis=1) <= 0).all() and (np.diff(thr, axis=0) >= 0).all()


def test_gauss_circle_golden(golden_dir):
    want = np.array(_read_golden(golden_dir, "gauss_circle.txt")[0], dtype=np.int64)
    disk = O.disk_count_table(21, 21, 16)
    assert (disk[10, 10] == want).all()
    # a corner point sees one quadrant: T=1 -> (0,0),(1,0),(0,1)
    assert disk[0, 0, 0] == 1 and disk[0, 0, 1] == 3 and disk[0, 0, 2] == 4


def test_grid_count_matches_bruteforce_tiny():
    """C_i^grid(n) (Eq. 13) by the per-frame disk table equals brute force over
    all keys with the literal test of Eq. 15, for every query and every
    candidate radius of the tiny grid, plus FULL."""
    F, H, W, gamma = 4, 8, 8, 0.6
    nc = O.n_cap(H, W)
    thr = O.threshold_table(nc, F, gamma)
    disk = O.disk_count_table(H, W, nc)
    f, x, y = O.grid_coords(F, H, W)
    for n in list(range(nc + 1)) + [O.RADIUS_FULL]:
        fast = O.grid_count(f, x, y, np.full(256, n), F, thr, disk)
        for i in range(0, 256, 5):
            assert fast[i] == O.grid_count_bruteforce(i, n, F, H, W, gamma), (i, n)


def test_grid_count_matches_bruteforce_sampled_large():
    F, H, W, gamma = 5, 45, 80, 0.95
    nc = O.n_cap(H, W)
    thr = O.threshold_table(nc, F, gamma)
    disk = O.disk_count_table(H, W, nc)
    f, x, y = O.grid_coords(F, H, W)
    for _ in range(60):
        i = int(RNG.integers(F * H * W))
        n = int(RNG.integers(nc + 1))
        got = O.grid_count(f[i:i + 1], x[i:i + 1], y[i:i + 1], np.array([n]), F, thr, disk)[0]
        assert got == O.grid_count_bruteforce(i, n, F, H, W, gamma)


def test_count_special_values():
    """C_i(0) = F (only the query's own pixel in every frame); C_i(FULL) = N."""
    F, H, W = 5, 9, 11
    nc = O.n_cap(H, W)
    thr = O.threshold_table(nc, F, 0.6)
    disk = O.disk_count_table(H, W, nc)
    f, x, y = O.grid_coords(F, H, W)
    assert (O.grid_count(f, x, y, np.zeros_like(f), F, thr, disk) == F).all()
    assert (O.grid_count(f, x, y, np.full_like(f, O.RADIUS_FULL), F, thr, disk) == F * H * W).all()


def test_select_radius_matches_linear_scan_tiny():
    """Eq. 14 by bisection equals a plain scan over all candidate radii with
    brute-force counts, on every query of the tiny grid at several budgets."""
    F, H, W, gamma = 4, 8, 8, 0.6
    nc = O.n_cap(H, W)
    thr = O.threshold_table(nc, F, gamma)
    disk = O.disk_count_table(H, W, nc)
    f, x, y = O.grid_coords(F, H, W)
    for khat in (1, 4, 5, 13, 40, 100, 200, 255, 256):
        got = O.select_radius(np.full(256, khat), f, x, y, F, thr, disk)
        for i in range(0, 256, 9):
            assert got[i] == O.select_radius_linear(khat, i, F, H, W, gamma), (i, khat)


def test_select_radius_monotone_in_budget():
    F, H, W = 6, 30, 52
    nc = O.n_cap(H, W)
    thr = O.threshold_table(nc, F, 0.6)
    disk = O.disk_count_table(H, W, nc)
    f, x, y = O.grid_coords(F, H, W)
    idx = RNG.choice(F * H * W, 40, replace=False)
    prev = np.zeros(40, dtype=np.int64)
    for khat in np.unique(np.geomspace(1, F * H * W, 60).astype(int)):
        n = O.select_radius(np.full(40, khat), f[idx], x[idx], y[idx], F, thr, disk)
        nn = np.where(n == O.RADIUS_FULL, nc + 1, n)
        assert (nn >= prev).all()
        prev = nn


def test_selected_radius_near_analytic_interior():
    """Sanity only: for small budgets far from every border the lattice radius
    sqrt(n) is within 1.5 lattice steps of the continuous radius of Eq. 12."""
    F, H, W, gamma = 21, 45, 80, 0.6
    nc = O.n_cap(H, W)
    thr = O.threshold_table(nc, F, gamma)
    disk = O.disk_count_table(H, W, nc)
    f = np.array([10]); x = np.array([22]); y = np.array([40])
    for khat in (50, 200, 800, 2000):
        n = O.select_radius(np.array([khat]), f, x, y, F, thr, disk)[0]
        r = O.analytic_radius(np.array([khat]), f, F, gamma)[0]
        assert abs(math.sqrt(n) - r) < 1.5, (khat, n, r)


# ------------------------------------------------------------------ block mask
def _line_grid_mask(nq, rule):
    """F=1, H=1, W=8, b=4 (tiles 1x4): block 0 = y 0..3, block 1 = y 4..7.
    D = (y_i - y_j)^2.  Returns M[0, :] for radii nq of block-0 queries."""
    n = np.zeros(8, dtype=np.int64)
    n[:4] = nq
    perm = O.tile_major_order(1, 1, 8, 1, 4)
    return O.block_mask_rows(n, perm, 4, 1, 1, 8, 0.6, [0], rule=rule)[0]


def test_vote_hand_cases():
    """Hand-derived columns counts for (u=0, v=1), n_u = 4 (Alg. 1):
    * queries y=2, y=3 with n=4: y=3 covers keys 4,5 and y=2 covers key 4, so
      c = (2,1,0,0), C = {4,5}, C_hi = {c > 4/3} = {4}; 10*1 > 6*2 fails -> drop;
      union keeps it.
    * y=2 with n=9 instead: covers 4 and 5, c = (2,2,0,0): 10*2 > 6*2 -> keep.
    * only y=3 with n=1: c = (1,0,0,0), C_hi empty -> drop; union keeps.
    * all n=0: no key of block 1 is hit -> drop under both rules."""
    assert list(_line_grid_mask([0, 0, 4, 4], "vote")) == [True, False]
    assert list(_line_grid_mask([0, 0, 4, 4], "union")) == [True, True]
    assert list(_line_grid_mask([0, 0, 9, 4], "vote")) == [True, True]
    assert list(_line_grid_mask([0, 0, 0, 1], "vote")) == [True, False]
    assert list(_line_grid_mask([0, 0, 0, 1], "union")) == [True, True]
    assert list(_line_grid_mask([0, 0, 0, 0], "union")) == [True, False]


def test_vote_partial_block_threshold():
    """Partial last block: with n_u valid queries the high-coverage test is
    3 c_j > n_u.  Grid W=6, b=4: block 1 holds y=4,5 (n_u=2).  Query y=4 with
    FULL radius hits every key once: c_j = 1 and 3*1 > 2, so block 1 -> block 0
    is retained under the vote."""
    n = np.zeros(6, dtype=np.int64)
    n[4] = O.RADIUS_FULL
    perm = O.tile_major_order(1, 1, 6, 1, 4)
    m = O.block_mask_rows(n, perm, 4, 1, 1, 6, 0.6, [1], rule="vote")[0]
    assert list(m) == [True, True]


@pytest.mark.parametrize("name", ["tiny", "wan13b_480p"])
def test_full_radius_gives_all_ones_and_zero_radius_identity(name):
    w = synth.workload(name)
    F, H, W, b = w.frames, w.height, w.width, w.block
    N = F * H * W
    perm = O.tile_major_order(F, H, W, w.tile_h, w.tile_w)
    nb = -(-N // b)
    blocks = list(range(0, nb, max(1, nb // 6))) + [nb - 1]
    full = O.block_mask_rows(np.full(N, O.RADIUS_FULL), perm, b, F, H, W, w.gamma, blocks)
    assert full.all()
    zero = O.block_mask_rows(np.zeros(N, dtype=np.int64), perm, b, F, H, W, w.gamma, blocks)
    eye = np.zeros_like(zero)
    for r, u in enumerate(blocks):
        eye[r, u] = True
    assert (zero == eye).all()


def test_union_contains_vote():
    w = synth.workload("tiny")
    F, H, W = w.frames, w.height, w.width
    n = RNG.integers(0, 40, size=256)
    perm = O.tile_major_order(F, H, W, 8, 8)
    vote = O.block_mask_rows(n, perm, 64, F, H, W, w.gamma, range(4), "vote")
    union = O.block_mask_rows(n, perm, 64, F, H, W, w.gamma, range(4), "union")
    assert (union >= vote).all()


def test_retained_fraction_closed_forms():
    N, b = 300, 128                    # blocks 128, 128, 44
    assert O.retained_fraction(np.ones((2, 3, 3)), N, b) == 1.0
    eye = np.eye(3, dtype=bool)[None]
    assert abs(O.retained_fraction(eye, N, b) - (128 ** 2 * 2 + 44 ** 2) / N ** 2) < 1e-15


# ------------------------------------------------------------------ masked attention
def test_masked_attention_full_mask_is_dense():
    w = synth.workload("tiny")
    q, k, v = (synth.to_f64(a[0, 0], w.dtype) for a in synth.generate(w))
    perm = O.tile_major_order(4, 8, 8, 8, 8)
    rows, o = O.masked_attention_rows(q, k, v, perm, 64, [0, 2], np.ones((2, 4), bool))
    assert np.abs(o - O.dense_attention(q[rows], k, v)).max() < 1e-12


def test_masked_attention_identity_is_block_diagonal():
    """Identity block mask: each query block attends only to its own block,
    i.e. textbook attention restricted to that block's keys."""
    w = synth.workload("tiny")
    q, k, v = (synth.to_f64(a[0, 1], w.dtype) for a in synth.generate(w))
    perm = O.tile_major_order(4, 8, 8, 8, 8)
    rows, o = O.masked_attention_rows(q, k, v, perm, 64, [1, 3], np.eye(4, dtype=bool)[[1, 3]])
    for r, u in enumerate([1, 3]):
        idx = perm[u * 64:(u + 1) * 64]
        want = O.dense_attention(q[idx], k[idx], v[idx])
        assert np.abs(o[r * 64:(r + 1) * 64] - want).max() < 1e-12


def test_masked_attention_lse_is_log_partition():
    """lse_i = log sum_j exp(s_ij) over retained keys; with a full mask it is the
    dense log-partition."""
    w = synth.workload("tiny")
    q, k, v = (synth.to_f64(a[0, 0], w.dtype) for a in synth.generate(w))
    perm = np.arange(256)
    rows, _, lse = O.masked_attention_rows(q, k, v, perm, 64, [0], np.ones((1, 4), bool),
                                           return_lse=True)
    s = q[rows] @ k.T / 8.0
    assert np.abs(lse - np.log(np.exp(s).sum(axis=1))).max() < 1e-12


# ------------------------------------------------------- lognormal budget (App. A.2)
@pytest.mark.parametrize("S", [256, 32760, 75600, 119056])
def test_lognormal_budget_at_max_entropy_is_tau_s(S):
    """At H = log S the fitted sigma is 0 (equal weights), Phibar(-Phi^{-1}(tau))
    = tau, so the lognormal budget is ceil(tau S): the uniform mapping's value."""
    H = math.log(S)
    assert int(O.token_budget_lognormal(H, 0.9, S)) == math.ceil(0.9 * S)
    # the uniform form evaluates tau * exp(log S) in fp64, which can land just
    # above an integer tau S (S = 75600: 68040.00000000006)
    uni = int(O.token_budget(H, 0.9, S))
    tau_s = 0.9 * S
    assert uni == math.ceil(tau_s) or (tau_s == round(tau_s) and uni == tau_s + 1)


def test_lognormal_budget_inverts_top_mass():
    """B = Phibar(sigma - Phi^{-1}(tau)) solves L_LN(B) = tau (App. A.2): with
    Phi^{-1}(1 - B) = sigma - Phi^{-1}(tau), L_LN(B) = Phibar(-Phi^{-1}(tau))."""
    z = O.normal_quantile(0.9)
    for sigma in (0.0, 0.3, 1.0, 2.5, 4.0):
        q = float(O.normal_tail(sigma - z))
        assert abs(float(O.lognormal_top_mass(q, sigma)) - 0.9) < 1e-12


def test_normal_quantile_and_tail_special_values():
    assert O.normal_quantile(0.5) == 0.0
    assert abs(float(O.normal_tail(0.0)) - 0.5) < 1e-16
    assert abs(float(O.normal_tail(1.959963984540054)) - 0.025) < 1e-15
    for p in (0.1, 0.5, 0.9, 0.99):
        assert abs(float(O.normal_tail(-O.normal_quantile(p))) - p) < 1e-14


@pytest.mark.parametrize("sigma", [0.5, 1.0, 1.5])
def test_lognormal_mapping_on_lognormal_weights(sigma):
    """On weights that ARE lognormal the derivation is exact in the large-sample
    limit: H = log n - sigma^2 / 2 recovers sigma, and the budget is the number
    of largest weights holding tau of the mass (checked on 400k seeded draws,
    tolerances from the sampling error)."""
    rng = np.random.default_rng(7)
    n = 400_000
    x = np.exp(rng.normal(0.3, sigma, size=n))
    p = x / x.sum()
    H = float(-(p * np.log(p)).sum())
    assert abs(math.sqrt(2.0 * (math.log(n) - H)) - sigma) < 0.015 * sigma
    k = int(O.token_budget_lognormal(H, 0.9, n))
    ps = np.sort(p)[::-1]
    assert abs(float(ps[:k].sum()) - 0.9) < 0.004
    true_k = int(np.searchsorted(np.cumsum(ps), 0.9) + 1)
    assert abs(k / true_k - 1.0) < 0.015


def test_lognormal_budget_monotone_and_clamped():
    S = 75600
    H = np.linspace(-5.0, math.log(S) + 1.0, 400)
    k = O.token_budget_lognormal(H, 0.9, S)
    assert np.all(np.diff(k) >= 0)
    assert k.min() >= 1 and k.max() == math.ceil(0.9 * S)


# ------------------------------------------------ sequence-distance ablation (App. C.1)
def test_threshold_1d_first_column_and_literal_test():
    """thr1[n, 0] = floor((pi/2) n); and |dr| <= thr1[n, delta] is the literal
    fp64 test |dr| <= (pi/2) n exp(-gamma delta) for every integer distance."""
    ncap, F, gamma = 200, 5, 0.6
    t1 = O.threshold_table_1d(ncap, F, gamma)
    assert np.array_equal(t1[:, 0], np.floor(np.arange(ncap + 1) * (math.pi / 2)).astype(np.int64))
    dr = np.arange(0, 400)
    for n in range(ncap + 1):
        for d in range(F):
            lit = O.within_radius_1d(dr, n, d, gamma)
            assert np.array_equal(lit, dr <= t1[n, d]), (n, d)


def test_token_mask_1d_brute_force_tiny():
    """token_mask_rows(distance="1d") against a loop over raster indices."""
    F, H, W, gamma = 3, 4, 5, 0.6
    N = F * H * W
    rng = np.random.default_rng(3)
    rows = rng.choice(N, 10, replace=False)
    n = rng.integers(0, 40, 10)
    n[0] = O.RADIUS_FULL
    M = O.token_mask_rows(rows, n, F, H, W, gamma, distance="1d").numpy()
    for a, (i, ni) in enumerate(zip(rows, n)):
        for j in range(N):
            fi, fj = i // (H * W), j // (H * W)
            want = ni == O.RADIUS_FULL or abs(i - j) <= (math.pi / 2) * ni * math.exp(-gamma * abs(fi - fj))
            assert M[a, j] == want


# -------------------------------------------------------- joint text-video (Sec. 3.2)
def test_joint_text_keys_visible_and_text_blocks_dense():
    """Text keys stay visible to every query; a block holding text is kept in
    every row and its own row keeps every block (Alg. 1)."""
    F, H, W, gamma, b, T = 2, 8, 8, 0.6, 64, 40
    N = F * H * W
    perm = O.joint_order(O.tile_major_order(F, H, W, 8, 8), T)
    S = N + T
    n = np.zeros(S, dtype=np.int64)
    M = O.token_mask_rows(np.arange(N), n[:N], F, H, W, gamma, keys=perm)
    assert M[:, N:].all()
    assert M[:, :N].sum() == N * F                 # radius 0: its own (x, y) in every frame
    nb = -(-S // b)
    mask = O.block_mask_rows(n, perm, b, F, H, W, gamma, range(nb))
    video_blocks = N // b
    assert mask[video_blocks:].all()               # text rows dense
    assert mask[:, video_blocks:].all()            # text columns kept
    assert np.array_equal(mask[:video_blocks, :video_blocks], np.eye(video_blocks, dtype=bool))


def test_joint_mixed_block_counts_as_text():
    """N not a multiple of b: the block holding the last video tokens and the
    first text tokens is a text block (dense row and column)."""
    F, H, W, gamma, b, T = 1, 5, 13, 0.6, 64, 10      # N = 65: block 1 = 1 video + 10 text
    N = F * H * W
    perm = O.joint_order(O.tile_major_order(F, H, W, 8, 8), T)
    n = np.zeros(N + T, dtype=np.int64)
    mask = O.block_mask_rows(n, perm, b, F, H, W, gamma, range(2))
    assert mask.all()


def test_joint_without_text_is_video_only():
    w = synth.workload("tiny")
    perm = O.tile_major_order(w.frames, w.height, w.width, w.tile_h, w.tile_w)
    rng = np.random.default_rng(5)
    n = rng.integers(0, 60, w.n_video)
    a = O.block_mask_rows(n, perm, w.block, w.frames, w.height, w.width, w.gamma, range(4))
    b = O.block_mask_rows(n, O.joint_order(perm, 0), w.block, w.frames, w.height, w.width,
                          w.gamma, range(4))
    assert np.array_equal(a, b)


def test_joint_all_blocks_kept_is_dense_over_s():
    """Every block retained: TRA attention over the joint sequence is dense
    attention over all S keys (Eq. 16 with M = 1)."""
    rng = np.random.default_rng(11)
    F, H, W, b, T, d = 1, 8, 8, 64, 20, 16
    N, S = F * H * W, F * H * W + T
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    perm = O.joint_order(O.tile_major_order(F, H, W, 8, 8), T)
    nb = -(-S // b)
    rows, o = O.masked_attention_rows(q, k, v, perm, b, range(nb), np.ones((nb, nb), dtype=bool))
    want = O.dense_attention(q[rows], k, v)
    assert np.allclose(o, want, atol=1e-12)


# ------------------------------------------------ token-level attention (Eq. 16)
def _rand_qkv(S, d, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((S, d)) for _ in range(3))


def test_token_attention_full_radius_is_block_attention():
    """FULL radii keep every key of a retained block: token level = block level."""
    F, H, W, b, d = 3, 8, 8, 64, 16
    S = F * H * W
    q, k, v = _rand_qkv(S, d, 21)
    perm = O.tile_major_order(F, H, W, 8, 8)
    nb = S // b
    rng = np.random.default_rng(2)
    mask = rng.random((nb, nb)) < 0.5
    np.fill_diagonal(mask, True)
    n = np.full(S, O.RADIUS_FULL)
    r1, o1 = O.token_attention_rows(q, k, v, perm, b, range(nb), mask, n, F, H, W, 0.6)
    r2, o2 = O.masked_attention_rows(q, k, v, perm, b, range(nb), mask)
    assert np.array_equal(r1, r2) and np.allclose(o1, o2, atol=1e-13)


@pytest.mark.parametrize("distance", ["2d", "1d"])
def test_token_attention_on_union_lists_is_eq16_over_all_keys(distance):
    """Union-rule block rows contain every covered key, so token-level attention
    on them equals a softmax over {j : M_ij = 1} taken over ALL keys."""
    F, H, W, b, d, gamma = 3, 8, 16, 64, 16, 0.6
    S = F * H * W
    q, k, v = _rand_qkv(S, d, 23)
    perm = O.tile_major_order(F, H, W, 8, 8)
    rng = np.random.default_rng(4)
    n = rng.integers(0, 60, S)
    nb = S // b
    mask = O.block_mask_rows(n, perm, b, F, H, W, gamma, range(nb), rule="union", distance=distance)
    rows, o = O.token_attention_rows(q, k, v, perm, b, range(nb), mask, n, F, H, W, gamma, distance)
    M = O.token_mask_rows(rows, n[rows], F, H, W, gamma, distance=distance).numpy()
    s = (q[rows] @ k.T) / math.sqrt(d)
    s = np.where(M, s, -np.inf)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    assert np.allclose(o, p @ v, atol=1e-12)


def test_token_attention_radius_zero_closed_form():
    """Radius 0: query i sees exactly the keys at its own (x, y) in every frame
    (thresholds are 0 for every delta), i.e. a softmax over F keys."""
    F, H, W, b, d = 4, 8, 8, 64, 8
    S = F * H * W
    q, k, v = _rand_qkv(S, d, 25)
    perm = O.tile_major_order(F, H, W, 8, 8)
    nb = S // b
    n = np.zeros(S, dtype=np.int64)
    rows, o = O.token_attention_rows(q, k, v, perm, b, range(nb), np.ones((nb, nb), bool), n, F, H, W, 0.6)
    for a, i in enumerate(rows[:40]):
        same = np.arange(F) * H * W + i % (H * W)
        s = q[i] @ k[same].T / math.sqrt(d)
        p = np.exp(s - s.max())
        p /= p.sum()
        assert np.allclose(o[a], p @ v[same], atol=1e-12)


def test_token_attention_joint_text_keys_visible():
    """Joint sequence: text queries attend to every retained key, video queries
    additionally to every text key."""
    F, H, W, b, d, T = 2, 8, 8, 64, 8, 30
    N, S = F * H * W, F * H * W + T
    q, k, v = _rand_qkv(S, d, 27)
    perm = O.joint_order(O.tile_major_order(F, H, W, 8, 8), T)
    nb = -(-S // b)
    n = np.concatenate([np.zeros(N, dtype=np.int64), np.full(T, O.RADIUS_FULL)])
    rows, o = O.token_attention_rows(q, k, v, perm, b, range(nb), np.ones((nb, nb), bool), n, F, H, W, 0.6)
    for a, i in enumerate(rows):
        if i >= N:
            keys = np.arange(S)
        else:
            keys = np.concatenate([np.arange(F) * H * W + i % (H * W), np.arange(N, S)])
        s = q[i] @ k[keys].T / math.sqrt(d)
        p = np.exp(s - s.max())
        p /= p.sum()
        assert np.allclose(o[a], p @ v[keys], atol=1e-12)
