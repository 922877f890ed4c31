"""What tile-aligned padded blocks change in the method's own terms, computed
by the oracle on the 480p grid (21 x 30 x 52, 8 x 16 tiles, b = 128) with one
uniform budget of 3,000 keys for every query (the paper's w/o Budget Mapping
ablation) and the vote of Alg. 1.

App. D names the work a retained block does on keys outside a query's radius
as the block-granular method's main limitation.  For each layout the test
counts executed token pairs (every query of a retained block with every key
of it), useful pairs (pairs inside retained blocks that the token mask of
Eq. 15 keeps) and all pairs the token mask keeps.  Packed blocks straddle
tiles and frames (3,120-token frames are not a multiple of 128), so their
boxes are larger than one tile; tile-aligned blocks keep each block inside one
tile of one frame.  At equal radii the tile-aligned layout executes fewer pairs
and more of them are useful, and the retained blocks cover more of the token
mask."""
import numpy as np

import oracle as O

F, H, W, TH, TW, B, GAMMA, KHAT = 21, 30, 52, 8, 16, 128, 0.6, 3000


def _radii():
    ncap = O.n_cap(H, W)
    thr = O.threshold_table(ncap, F, GAMMA)
    disk = O.disk_count_table(H, W, ncap)
    f, x, y = O.grid_coords(F, H, W)
    return O.select_radius(np.full(F * H * W, KHAT), f, x, y, F, thr, disk)


def _stats(perm, n):
    nb = len(perm) // B if len(perm) % B == 0 else -(-len(perm) // B)
    keep = O.block_mask_rows(n, perm, B, F, H, W, GAMMA, range(nb))
    sizes = O.block_sizes(perm, B)
    block_of = np.empty(F * H * W, dtype=np.int64)
    for u in range(nb):
        block_of[O.block_tokens(perm, B, u)] = u
    keys = np.arange(F * H * W)
    executed = useful = covered = 0
    for u in range(nb):
        rows = O.block_tokens(perm, B, u)
        M = O.token_mask_rows(rows, n[rows], F, H, W, GAMMA, keys=keys).numpy()
        per_key = M.sum(axis=0)
        covered += int(per_key.sum())
        useful += int(per_key[keep[u][block_of]].sum())
        executed += int(len(rows) * sizes[keep[u]].sum())
    return executed, useful, covered


def test_tile_aligned_blocks_cut_in_block_waste():
    n = _radii()
    packed = O.tile_major_order(F, H, W, TH, TW)
    tiles = O.tile_aligned_order(F, H, W, TH, TW, B)
    ep, up, cp = _stats(packed, n)
    et, ut, ct = _stats(tiles, n)
    assert cp == ct                                       # the token mask does not depend on the layout
    N2 = float(F * H * W) ** 2
    print(f"packed: executed {ep / N2:.4f} of N^2, useful/executed {up / ep:.4f}, covered kept {up / cp:.4f}")
    print(f"tiles:  executed {et / N2:.4f} of N^2, useful/executed {ut / et:.4f}, covered kept {ut / ct:.4f}")
    assert et < ep
    assert ut / et > up / ep + 0.05
    assert ut > up
