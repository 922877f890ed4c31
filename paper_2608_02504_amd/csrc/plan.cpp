// Shape tables of a TRA plan, built on the host in integer / fp64 arithmetic.
//
//  * tile-major order of Sec. 3.3 ("Flash Radius Mask Kernel") and App. C.1
//    ("Kernel execution"): frames in order, each frame cut into
//    tile_h x tile_w tiles (edge tiles clipped), tiles in row-major tile
//    order, tokens row-major inside a tile;
//  * squared-radius thresholds: for squared base radius n (r = sqrt n) and
//    temporal distance delta, the test d_s <= r * phi(delta) of Eq. 15 with
//    phi(delta) = exp(-gamma delta) (Eq. 10) holds for an integer squared
//    distance D iff D <= floor(n * exp(-2 gamma delta));
//  * the sequence-distance ablation (App. C.1, Eq. area-matched-1d): the 1-D
//    radius is (pi/2) r^2 = (pi/2) n and the test |i - j| <= (pi/2) n phi(delta)
//    holds for an integer distance iff |i - j| <= floor((pi/2) n exp(-gamma delta));
//  * per-block bounding boxes used to skip block pairs (App. C.1, "Kernel
//    execution": a bounding-box test rejects pairs with no valid
//    interaction);
//  * text tokens of joint text-video attention (Sec. 3.2) follow the video
//    tokens in the sequence and keep their order;
//  * block layouts: packed (block u = positions [u b, (u+1) b) of the order)
//    or tile-aligned padded blocks (one tile of one frame per block, a clipped
//    edge tile padded; App. D's in-block redundancy is smallest when a block's
//    spatial footprint is).
#include <algorithm>
#include <cmath>

#include "tra_internal.h"

namespace tra {

tra_status validate_config(const tra_config* cfg, std::string* why) {
  if (!cfg) { *why = "config is NULL"; return TRA_ERR_INVALID_ARG; }
  const tra_config& c = *cfg;
  if (c.batch < 1 || c.heads < 1) { *why = "batch and heads must be >= 1"; return TRA_ERR_INVALID_ARG; }
  if (c.frames < 1 || c.height < 1 || c.width < 1) { *why = "frames, height and width must be >= 1"; return TRA_ERR_INVALID_ARG; }
  if (c.frames > kMaxFrames) { *why = "frames > 64 is not supported"; return TRA_ERR_UNSUPPORTED; }
  if (c.height > 1023 || c.width > 1023) { *why = "height and width must be <= 1023"; return TRA_ERR_UNSUPPORTED; }
  if (c.tile_h < 1 || c.tile_w < 1) { *why = "tile_h and tile_w must be >= 1"; return TRA_ERR_INVALID_ARG; }
  if (c.budget_map != TRA_BUDGET_UNIFORM && c.budget_map != TRA_BUDGET_LOGNORMAL) { *why = "unknown budget mapping"; return TRA_ERR_INVALID_ARG; }
  if (c.distance != TRA_DIST_2D && c.distance != TRA_DIST_1D) { *why = "unknown distance"; return TRA_ERR_INVALID_ARG; }
  if (c.text_tokens < 0) { *why = "text_tokens must be >= 0"; return TRA_ERR_INVALID_ARG; }
  if (c.dtype != TRA_BF16 && c.dtype != TRA_FP32) { *why = "unknown dtype"; return TRA_ERR_INVALID_ARG; }
  if (c.rule != TRA_MASK_VOTE && c.rule != TRA_MASK_UNION) { *why = "unknown mask rule"; return TRA_ERR_INVALID_ARG; }
  if (!(c.tau > 0.0 && c.tau < 1.0)) { *why = "tau must be in (0, 1)"; return TRA_ERR_INVALID_ARG; }
  if (!(c.gamma >= 0.0) || !std::isfinite(c.gamma)) { *why = "gamma must be finite and >= 0"; return TRA_ERR_INVALID_ARG; }
  if (c.head_dim != 64 && c.head_dim != 128) { *why = "head_dim must be 64 or 128"; return TRA_ERR_UNSUPPORTED; }
  if (c.block != 64 && c.block != 128) { *why = "block must be 64 or 128"; return TRA_ERR_UNSUPPORTED; }
  if (c.dtype == TRA_BF16 && c.block != 128) { *why = "bf16 needs block 128"; return TRA_ERR_UNSUPPORTED; }
  if (c.block_layout != TRA_BLOCKS_PACKED && c.block_layout != TRA_BLOCKS_TILES) { *why = "unknown block layout"; return TRA_ERR_INVALID_ARG; }
  if (c.block_layout == TRA_BLOCKS_TILES) {
    if ((int64_t)c.tile_h * c.tile_w != c.block) { *why = "tile-aligned blocks need tile_h * tile_w == block"; return TRA_ERR_INVALID_ARG; }
  }
  const int64_t n = (int64_t)c.frames * c.height * c.width + c.text_tokens;
  const int64_t nb = c.block_layout == TRA_BLOCKS_TILES
                         ? (int64_t)c.frames * ((c.height + c.tile_h - 1) / c.tile_h) *
                                   ((c.width + c.tile_w - 1) / c.tile_w) +
                               (c.text_tokens + c.block - 1) / c.block
                         : (n + c.block - 1) / c.block;
  if (nb > kMaxBlocks) { *why = "more than 4096 blocks per head"; return TRA_ERR_UNSUPPORTED; }
  const int64_t rows = (int64_t)c.batch * c.heads * nb;
  if (rows * nb >= (int64_t)1 << 31 || (int64_t)c.batch * c.heads * nb * c.block >= (int64_t)1 << 31) {
    *why = "batch * heads * tokens too large for 32-bit indexing";
    return TRA_ERR_UNSUPPORTED;
  }
  return TRA_OK;
}

uint16_t f16_bits_of_int(int v) {
  if (v == 0) return 0;
  const uint16_t sign = v < 0 ? 0x8000 : 0;
  unsigned a = (unsigned)(v < 0 ? -v : v);  // 1 .. 2048
  int e = 0;
  while ((a >> (e + 1)) != 0) ++e;           // a = 1.m x 2^e, e <= 11
  const unsigned mant = ((a << 10) >> e) & 0x3FF;
  return (uint16_t)(sign | ((unsigned)(e + 15) << 10) | mant);
}

double normal_quantile(double p) {
  // Phi(x) = erfc(-x / sqrt 2) / 2 is increasing; bisect until the bracket
  // stops shrinking in fp64.
  double lo = -40.0, hi = 40.0;
  for (int it = 0; it < 200; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (mid == lo || mid == hi) break;
    if (0.5 * std::erfc(-mid / std::sqrt(2.0)) < p) lo = mid;
    else hi = mid;
  }
  return 0.5 * (lo + hi);
}

void build_host_tables(const tra_config& c, HostTables* t, bool with_perm_coord,
                       bool with_thr, bool with_thr1, bool with_blocks, bool with_kinfo) {
  const int F = c.frames, H = c.height, W = c.width, b = c.block;
  const bool tiles = c.block_layout == TRA_BLOCKS_TILES;
  t->N = F * H * W;
  t->S = t->N + c.text_tokens;
  const int tiles_h = (H + c.tile_h - 1) / c.tile_h, tiles_w = (W + c.tile_w - 1) / c.tile_w;
  t->NB = tiles ? F * tiles_h * tiles_w + (c.text_tokens + b - 1) / b : (t->S + b - 1) / b;
  t->P = tiles ? t->NB * b : t->S;
  t->n_cap = (H - 1) * (H - 1) + (W - 1) * (W - 1);

  std::vector<int32_t> perm;
  if (with_perm_coord || with_blocks || with_kinfo) {
    // One frame's tile-major order, then offset per frame; text tokens last.
    std::vector<int32_t> frame;
    frame.reserve((size_t)H * W);
    for (int ty = 0; ty < H; ty += c.tile_h)
      for (int tx = 0; tx < W; tx += c.tile_w)
        for (int x = ty; x < std::min(H, ty + c.tile_h); ++x)
          for (int y = tx; y < std::min(W, tx + c.tile_w); ++y) frame.push_back(x * W + y);
    std::vector<int32_t> packed(t->S);
    for (int f = 0; f < F; ++f)
      for (int p = 0; p < H * W; ++p) packed[(size_t)f * H * W + p] = f * H * W + frame[p];
    for (int p = t->N; p < t->S; ++p) packed[p] = p;
    if (tiles) {
      // one block per tile: the tile's tokens (row-major) then padding
      perm.assign((size_t)t->P, -1);
      size_t at = 0;
      for (int f = 0; f < F; ++f)
        for (int ty = 0; ty < H; ty += c.tile_h)
          for (int tx = 0; tx < W; tx += c.tile_w) {
            size_t j = at;
            for (int x = ty; x < std::min(H, ty + c.tile_h); ++x)
              for (int y = tx; y < std::min(W, tx + c.tile_w); ++y) perm[j++] = (f * H + x) * W + y;
            at += b;
          }
      for (int s0 = 0; s0 < c.text_tokens; s0 += b, at += b)
        for (int j = 0; j < b && s0 + j < c.text_tokens; ++j) perm[at + j] = t->N + s0 + j;
      if (with_perm_coord) t->perm_attn = std::move(packed);
    } else {
      perm = std::move(packed);
    }
  }
  if (with_perm_coord) {
    t->coord.assign(t->P, 0);
    for (int p = 0; p < t->P; ++p) {
      const int i = perm[p];
      if (i >= 0 && i < t->N) t->coord[p] = pack_coord(i / (H * W), (i / W) % H, i % W);
    }
  }
  if (with_thr) {
    t->thr.resize((size_t)(t->n_cap + 1) * F);
    for (int n = 0; n <= t->n_cap; ++n)
      for (int d = 0; d < F; ++d) {
        // n * exp(-2 gamma delta), floored.  delta = 0 gives n exactly.
        const double e = std::exp(-2.0 * c.gamma * (double)d);
        t->thr[(size_t)n * F + d] = d == 0 ? n : (int32_t)std::floor((double)n * e);
      }
  }
  if (with_thr1) {
    t->thr1.resize((size_t)(t->n_cap + 1) * F);
    const double half_pi = 1.5707963267948966;  // pi / 2
    for (int n = 0; n <= t->n_cap; ++n)
      for (int d = 0; d < F; ++d) {
        // ((pi/2) n) exp(-gamma delta), floored
        const double e = std::exp(-c.gamma * (double)d);
        t->thr1[(size_t)n * F + d] = (int32_t)std::floor((half_pi * (double)n) * e);
      }
  }
  if (with_blocks) {
    // Every block's tokens fill its first positions: video tokens first, then
    // text tokens (only the packed layout mixes the two, in one block).
    t->blocks.assign((size_t)t->NB * kBlockInfo, 0);
    for (int u = 0; u < t->NB; ++u) {
      int fmin = F, fmax = -1, xmin = H, xmax = -1, ymin = W, ymax = -1;
      int rmin = t->N, rmax = -1, n_video = 0, n_text = 0;
      const int lo = u * b, hi = std::min(t->P, lo + b);
      for (int p = lo; p < hi; ++p) {
        const int i = perm[p];
        if (i < 0) continue;
        if (i >= t->N) {
          ++n_text;
          continue;
        }
        ++n_video;
        const int f = i / (H * W), x = (i / W) % H, y = i % W;
        fmin = std::min(fmin, f); fmax = std::max(fmax, f);
        xmin = std::min(xmin, x); xmax = std::max(xmax, x);
        ymin = std::min(ymin, y); ymax = std::max(ymax, y);
        rmin = std::min(rmin, i); rmax = std::max(rmax, i);
      }
      int32_t* o = &t->blocks[(size_t)u * kBlockInfo];
      o[0] = fmin; o[1] = fmax; o[2] = xmin; o[3] = xmax; o[4] = ymin; o[5] = ymax;
      o[6] = n_video; o[7] = rmin; o[8] = rmax; o[9] = n_text;
    }
  }
  if (with_kinfo) {
    // key side of the token mask: one word per key of every block (and one
    // zero block after the last, so a 1 KB copy of the last block stays in
    // bounds).  2-D: x | y << 16, 1-D: the raster index; plus a flag bit
    // (bit 15 for 2-D, bit 30 for 1-D) when the key lies in the block's second
    // frame (a packed block of at most H*W tokens spans at most two; a tile
    // block one), and bit 31 for a text key.  Padding stays 0 (masked apart by
    // the block's token count).
    const bool one_d = c.distance == TRA_DIST_1D;
    t->kinfo.assign((size_t)(t->NB + 1) * kKeyInfo, 0);
    for (int u = 0; u < t->NB; ++u) {
      const int first = u * b < t->P ? perm[(size_t)u * b] : -1;
      const int f0 = first >= 0 && first < t->N ? first / (H * W) : 0;
      for (int j = 0; j < b; ++j) {
        const int p = u * b + j;
        const int i = p < t->P ? perm[p] : -1;
        uint32_t word = 0;
        if (i >= 0 && i < t->N) {
          const bool second = i / (H * W) != f0;
          word = one_d ? (uint32_t)i | (second ? 1u << 30 : 0u)
                       : (uint32_t)((i / W) % H) | ((uint32_t)(i % W) << 16) | (second ? 1u << 15 : 0u);
        } else if (i >= t->N) {
          word = 1u << 31;
        }
        t->kinfo[(size_t)u * kKeyInfo + j] = (int32_t)word;
      }
    }
    if (!one_d) {
      // key side of the token mask as a matrix product (Eq. 15): with the
      // squared radius thresholds T_lo, T_hi of a query i for the block's
      // first and second frame, A = T - (x_i^2 + y_i^2) split as 2048 h + l
      // (0 <= l < 2048) and the key's x^2 + y^2 as 2048 hj + lj, the query
      // vector a_i = (h_lo, l_lo, h_hi, l_hi, 2048, 1, 2 x_i, 2 y_i) and the key
      // vector b_j = (2048, 1, 0, 0, -hj, -lj, x_j, y_j) (first frame; (0, 0,
      // 2048, 1, ...) in the second) give a_i . b_j = T - (x_i - x_j)^2 -
      // (y_i - y_j)^2, so the key is covered iff it is >= 0.  Every entry is an
      // integer of magnitude <= 2048, exact in f16, and every partial sum stays
      // below 2^24, exact in fp32.  A text key is (0, 0, 0, 0, 0, 1, 0, 0)
      // (a . b = 1, always covered); padding is 0.
      t->kfeat.assign((size_t)t->NB * b * kKeyFeat, 0);
      for (int u = 0; u < t->NB; ++u) {
        const int first = u * b < t->P ? perm[(size_t)u * b] : -1;
        const int f0 = first >= 0 && first < t->N ? first / (H * W) : 0;
        for (int j = 0; j < b; ++j) {
          const int p = u * b + j;
          const int i = p < t->P ? perm[p] : -1;
          int v[kKeyFeat] = {0, 0, 0, 0, 0, 0, 0, 0};
          if (i >= 0 && i < t->N) {
            const int x = (i / W) % H, y = i % W, sq = x * x + y * y;
            const int o = i / (H * W) != f0 ? 2 : 0;
            v[o] = 2048;
            v[o + 1] = 1;
            v[4] = -(sq >> 11);
            v[5] = -(sq & 2047);
            v[6] = x;
            v[7] = y;
          } else if (i >= t->N) {
            v[5] = 1;
          }
          // stored half-major, [u][k / 4][j][k % 4]: a wave's lane half h reads
          // components 4h..4h+3 of 32 keys as 32 consecutive 8-byte words
          for (int k = 0; k < kKeyFeat; ++k)
            t->kfeat[(((size_t)u * 2 + k / 4) * b + j) * 4 + k % 4] = f16_bits_of_int(v[k]);
        }
      }
    }
  }
  if (with_perm_coord) t->perm = std::move(perm);
}

}  // namespace tra
