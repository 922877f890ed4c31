// Host-side check of the plan's table builder (plan.cpp), built by the CPU
// test suite with AddressSanitizer and UndefinedBehaviorSanitizer: every
// workload shape and a set of edge shapes (text tokens, 1-D distance, block
// 64, a single token, clipped tiles) are validated and built, and the tables'
// invariants checked; invalid configurations must be rejected.  Exit status 0
// and no sanitizer report mean pass.
#include <cmath>
#include <cstdio>
#include <string>
#include <vector>

#include "tra_internal.h"

namespace {

int failures = 0;

// Value of an f16 bit pattern (normal numbers and zero).
double f16_value(uint16_t h) {
  const int e = (h >> 10) & 31, m = h & 1023;
  if (e == 0 && m == 0) return (h & 0x8000) ? -0.0 : 0.0;
  const double v = std::ldexp(1.0 + m / 1024.0, e - 15);
  return (h & 0x8000) ? -v : v;
}

void expect(bool ok, const char* what, int cfg) {
  if (!ok) {
    std::printf("FAIL config %d: %s\n", cfg, what);
    ++failures;
  }
}

tra_config make(int F, int H, int W, int d, int b, int th, int tw, int text, int dtype, int dist) {
  tra_config c{};
  c.batch = 1; c.heads = 2; c.frames = F; c.height = H; c.width = W; c.head_dim = d; c.block = b;
  c.tile_h = th; c.tile_w = tw; c.dtype = dtype; c.rule = TRA_MASK_VOTE; c.budget_map = TRA_BUDGET_UNIFORM;
  c.distance = dist; c.text_tokens = text; c.tau = 0.9f; c.gamma = 0.6f;
  return c;
}

}  // namespace

int main() {
  const std::vector<tra_config> good = {
      make(4, 8, 8, 64, 64, 8, 8, 0, TRA_FP32, TRA_DIST_2D),          // tiny
      make(21, 30, 52, 128, 128, 8, 16, 0, TRA_BF16, TRA_DIST_2D),    // 480p
      make(21, 45, 80, 128, 128, 8, 16, 0, TRA_BF16, TRA_DIST_2D),    // 720p
      make(33, 45, 80, 128, 128, 8, 16, 256, TRA_BF16, TRA_DIST_2D),  // joint, 129 frames
      make(3, 11, 29, 64, 128, 8, 16, 0, TRA_BF16, TRA_DIST_1D),      // ragged, 1-D
      make(2, 9, 11, 128, 64, 8, 8, 50, TRA_FP32, TRA_DIST_2D),       // block 64, text
      make(1, 1, 1, 128, 128, 8, 16, 0, TRA_BF16, TRA_DIST_2D),       // a single token
      make(3, 7, 19, 128, 128, 5, 7, 77, TRA_FP32, TRA_DIST_1D),      // odd tiles, text, 1-D
  };
  for (size_t ci = 0; ci < good.size(); ++ci) {
    const tra_config& c = good[ci];
    const int ic = (int)ci;
    std::string why;
    expect(tra::validate_config(&c, &why) == TRA_OK, "valid config rejected", ic);
    tra::HostTables t;
    tra::build_host_tables(c, &t, true, true, true, true, c.dtype == TRA_BF16);
    const int N = c.frames * c.height * c.width, S = N + c.text_tokens;
    expect(t.N == N && t.S == S && t.NB == (S + c.block - 1) / c.block, "sizes", ic);
    // the permutation is a bijection of [0, S), text tokens last and in order
    std::vector<int> seen(S, 0);
    bool in_range = (int)t.perm.size() == S;
    for (int p = 0; in_range && p < S; ++p) {
      in_range = t.perm[p] >= 0 && t.perm[p] < S;
      if (in_range) ++seen[t.perm[p]];
    }
    expect(in_range, "perm out of range", ic);
    bool bij = in_range;
    for (int i = 0; bij && i < S; ++i) bij = seen[i] == 1;
    expect(bij, "perm not a bijection", ic);
    for (int p = N; p < S; ++p) expect(t.perm[p] == p, "text tokens reordered", ic);
    // packed coordinates agree with the permutation
    for (int p = 0; p < N; ++p) {
      const int i = t.perm[p];
      const int f = i / (c.height * c.width), x = (i / c.width) % c.height, y = i % c.width;
      if (t.coord[p] != tra::pack_coord(f, x, y)) {
        expect(false, "coord", ic);
        break;
      }
    }
    // thresholds: delta = 0 is n itself, non-increasing in delta
    const int F = c.frames;
    for (int n = 0; n <= t.n_cap; ++n) {
      expect(t.thr[(size_t)n * F] == n, "thr[n][0] != n", ic);
      for (int d = 1; d < F; ++d)
        if (t.thr[(size_t)n * F + d] > t.thr[(size_t)n * F + d - 1]) { expect(false, "thr increasing", ic); break; }
      for (int d = 1; d < F; ++d)
        if (t.thr1[(size_t)n * F + d] > t.thr1[(size_t)n * F + d - 1]) { expect(false, "thr1 increasing", ic); break; }
    }
    // block boxes hold every video token of their block; counts add up
    int video = 0, text = 0;
    for (int u = 0; u < t.NB; ++u) {
      const int32_t* bi = &t.blocks[(size_t)u * tra::kBlockInfo];
      video += bi[6];
      text += bi[9];
      for (int p = u * c.block; p < std::min(S, (u + 1) * c.block) && p < N; ++p) {
        const int i = t.perm[p];
        const int f = i / (c.height * c.width), x = (i / c.width) % c.height, y = i % c.width;
        if (f < bi[0] || f > bi[1] || x < bi[2] || x > bi[3] || y < bi[4] || y > bi[5] || i < bi[7] || i > bi[8]) {
          expect(false, "token outside its block box", ic);
          break;
        }
      }
    }
    expect(video == N && text == c.text_tokens, "block token counts", ic);
    if (c.dtype == TRA_BF16) {
      expect(t.kinfo.size() == (size_t)(t.NB + 1) * tra::kKeyInfo, "key-word table size", ic);
      for (int p = 0; p < S; ++p) {
        const uint32_t w = (uint32_t)t.kinfo[(size_t)(p / c.block) * tra::kKeyInfo + p % c.block];
        if (p >= N) {
          if (w != 1u << 31) { expect(false, "text key word", ic); break; }
          continue;
        }
        const int i = t.perm[p];
        const uint32_t base = c.distance == TRA_DIST_1D ? (uint32_t)i
                                                        : (uint32_t)((i / c.width) % c.height) | ((uint32_t)(i % c.width) << 16);
        const uint32_t flag = c.distance == TRA_DIST_1D ? 1u << 30 : 1u << 15;
        if ((w & ~flag) != base) { expect(false, "key word", ic); break; }
      }
      if (c.distance == TRA_DIST_2D) {
        // key vectors b_j: for a sample of query positions and thresholds, the
        // product with the query vector a_i (built here from its definition)
        // equals T - D for a video key of either frame, and 1 for a text key
        expect(t.kfeat.size() == (size_t)t.NB * c.block * tra::kKeyFeat, "key-feature table size", ic);
        bool bad = false;
        for (int u = 0; u < t.NB && !bad; u += 7) {
          const int i0 = t.perm[(size_t)u * c.block];
          const int f0 = i0 < N ? i0 / (c.height * c.width) : 0;
          for (int j = 0; j < c.block && !bad; ++j) {
            const int p = u * c.block + j;
            if (p >= S) break;
            double bv[tra::kKeyFeat];
            for (int k = 0; k < tra::kKeyFeat; ++k)  // stored [block][k / 4][key][k % 4]
              bv[k] = f16_value(t.kfeat[(((size_t)u * 2 + k / 4) * c.block + j) * 4 + k % 4]);
            const int i = t.perm[p];
            for (int qi = 0; qi < N && !bad; qi += 997) {
              const int qx = (qi / c.width) % c.height, qy = qi % c.width;
              for (int T : {0, 1, 37, 4096, 65535, 1 << 22}) {
                const int T2 = T / 2 + 3;  // a different threshold for the second frame
                const int a_lo = T - (qx * qx + qy * qy), a_hi = T2 - (qx * qx + qy * qy);
                const double a[tra::kKeyFeat] = {(double)(a_lo >> 11), (double)(a_lo & 2047), (double)(a_hi >> 11),
                                                 (double)(a_hi & 2047), 2048.0, 1.0, 2.0 * qx, 2.0 * qy};
                double e = 0.0;
                for (int k = 0; k < tra::kKeyFeat; ++k) e += a[k] * bv[k];
                double want;
                if (i >= N) {
                  want = 1.0;
                } else {
                  const int x = (i / c.width) % c.height, y = i % c.width;
                  const int D = (qx - x) * (qx - x) + (qy - y) * (qy - y);
                  want = (i / (c.height * c.width) != f0 ? T2 : T) - D;
                }
                if (e != want) {
                  expect(false, "key vector product", ic);
                  bad = true;
                  break;
                }
              }
            }
          }
        }
      }
    }
  }
  // tile-aligned padded blocks: NB * b positions, every token once, tokens a
  // prefix of each block, each video block inside one tile of one frame
  {
    const std::vector<tra_config> tiled = {
        make(4, 13, 37, 128, 128, 8, 16, 77, TRA_BF16, TRA_DIST_2D),
        make(7, 5, 9, 64, 128, 8, 16, 0, TRA_BF16, TRA_DIST_1D),
        make(21, 45, 80, 128, 128, 8, 16, 0, TRA_BF16, TRA_DIST_2D)};
    for (size_t ci = 0; ci < tiled.size(); ++ci) {
      tra_config c = tiled[ci];
      c.block_layout = TRA_BLOCKS_TILES;
      const int ic = 300 + (int)ci;
      std::string why;
      expect(tra::validate_config(&c, &why) == TRA_OK, "valid tiled config rejected", ic);
      tra::HostTables t;
      tra::build_host_tables(c, &t, true, true, false, true, true);
      const int N = c.frames * c.height * c.width, S = N + c.text_tokens, b = c.block;
      const int tiles = c.frames * ((c.height + c.tile_h - 1) / c.tile_h) * ((c.width + c.tile_w - 1) / c.tile_w);
      expect(t.NB == tiles + (c.text_tokens + b - 1) / b && t.P == t.NB * b && (int)t.perm.size() == t.P,
             "tiled sizes", ic);
      expect((int)t.perm_attn.size() == S, "packed order of the token calls", ic);
      std::vector<int> seen(S, 0);
      for (int u = 0; u < t.NB; ++u) {
        const int32_t* bi = &t.blocks[(size_t)u * tra::kBlockInfo];
        const int n = bi[6] + bi[9];
        for (int j = 0; j < b; ++j) {
          const int i = t.perm[(size_t)u * b + j];
          if ((j < n) != (i >= 0)) { expect(false, "tokens not a prefix of the block", ic); break; }
          if (i < 0) continue;
          if (i >= S) { expect(false, "tiled perm out of range", ic); break; }
          ++seen[i];
          if (i < N) {
            const int f = i / (c.height * c.width), x = (i / c.width) % c.height, y = i % c.width;
            if (f != bi[0] || f != bi[1] || x / c.tile_h != bi[2] / c.tile_h || y / c.tile_w != bi[4] / c.tile_w ||
                x < bi[2] || x > bi[3] || y < bi[4] || y > bi[5]) {
              expect(false, "tiled block not one tile of one frame", ic);
              break;
            }
          }
        }
      }
      for (int i = 0; i < S; ++i)
        if (seen[i] != 1) { expect(false, "tiled perm not a bijection", ic); break; }
    }
  }
  // invalid configurations are rejected before any table is built
  std::vector<tra_config> bad;
  tra_config b0 = good[1]; b0.head_dim = 96; bad.push_back(b0);
  tra_config b1 = good[1]; b1.frames = 0; bad.push_back(b1);
  tra_config b2 = good[1]; b2.frames = 65; bad.push_back(b2);
  tra_config b3 = good[1]; b3.width = 1024; bad.push_back(b3);
  tra_config b4 = good[1]; b4.block = 64; bad.push_back(b4);  // bf16 needs 128
  tra_config b5 = good[1]; b5.tau = 1.0f; bad.push_back(b5);
  tra_config b6 = good[1]; b6.text_tokens = -1; bad.push_back(b6);
  tra_config b7 = good[1]; b7.distance = 7; bad.push_back(b7);
  tra_config b8 = good[1]; b8.block_layout = TRA_BLOCKS_TILES; b8.tile_w = 8; bad.push_back(b8);
  for (size_t i = 0; i < bad.size(); ++i) {
    std::string why;
    expect(tra::validate_config(&bad[i], &why) != TRA_OK && !why.empty(), "invalid config accepted",
           100 + (int)i);
  }
  std::string why;
  expect(tra::validate_config(nullptr, &why) == TRA_ERR_INVALID_ARG, "NULL config", 200);
  std::printf(failures ? "host tables: %d failure(s)\n" : "host tables: ok\n", failures);
  return failures ? 1 : 0;
}
