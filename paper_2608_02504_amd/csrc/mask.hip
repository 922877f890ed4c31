// Token-radius block mask (App. C.1, Alg. 1) and the heaviest-first row order.
//
// One workgroup per query-block row (batch, head, u); its four waves walk the
// key blocks v.  For a key column j of block v, c_j counts the valid queries
// i of u whose radius covers j (Eq. 15):
//     (x_i - x_j)^2 + (y_i - y_j)^2 <= thr[n_i][|f_i - f_j|].
// Alg. 1 evaluates every (i, j) pair.  Here each query is first classified
// against the bounding box of v (App. C.1 uses such boxes to reject whole
// block pairs): "none" if even the nearest box point in the most favourable
// frame is outside its disk, "all" if the farthest box point in the least
// favourable frame is inside.  Only "partial" queries are tested key by key,
// so the counts -- and the mask -- are exactly Alg. 1's; the boxes only skip
// work whose outcome is already known.  Everything is integer arithmetic.
//
// Sequence-distance ablation (DIST = TRA_DIST_1D, App. C.1): a query covers
// key j iff |i - j| <= thr1[n_i][|f_i - f_j|] on raster indices; the box of a
// block is then its raster-index range, and the same none / all / partial
// argument holds because thr1 is non-increasing in delta too.
//
// Joint text-video attention (Sec. 3.2; Alg. 1's u >= B_v or v >= B_v branch):
// a block holding any text token is retained in every row, and the row of such
// a block retains every key block.
#include <climits>
#include <mutex>

#include "tra_internal.h"

namespace tra {
namespace {

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }

// Distance of a token pair from its position difference: squared Euclidean
// (x, y) for 2-D, |raster difference| (carried in the first component) for 1-D.
// (Coordinate differences are below 1024 in magnitude, so 24-bit multiplies
// are exact.)
template <int DIST>
__device__ __forceinline__ int metric(int da, int db) {
  if constexpr (DIST == TRA_DIST_1D) return abs(da);
  else return __mul24(da, da) + __mul24(db, db);
}

// Position of a packed coordinate in the metric's space.
template <int DIST>
__device__ __forceinline__ void position(int32_t c, int H, int W, int* a, int* b, int* f) {
  *f = coord_f(c);
  if constexpr (DIST == TRA_DIST_1D) {
    *a = (*f * H + coord_x(c)) * W + coord_y(c);
    *b = 0;
  } else {
    *a = coord_x(c);
    *b = coord_y(c);
  }
}

typedef short short2_t __attribute__((ext_vector_type(2)));
typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));

template <int B, int RULE, int DIST>
__global__ __launch_bounds__(256) void block_mask_kernel(
    const int32_t* __restrict__ radius_sq, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ coord, const int32_t* __restrict__ thr,
    const int32_t* __restrict__ binfo, uint8_t* __restrict__ mask, int32_t* __restrict__ cnt,
    int32_t* __restrict__ cols, int N, int S, int NB, int F, int H, int W, int n_cap) {
  constexpr int QPL = B / 64;  // queries (and keys) per lane
  extern __shared__ int32_t s_T[];         // [B * F]: s_T[q*F + delta], distance threshold of query q
  __shared__ int32_t s_c[B];               // packed coordinate of query q
  __shared__ uint8_t s_keep[kMaxBlocks];
  // per wave: the partial queries of the current key block, two per entry, as
  // 16-bit halves of four words (x, y, threshold + 1 for each of the block's two
  // frames); read back with one broadcast load per entry
  __shared__ uint32_t s_pairs[4][B / 2][4];
  // 16-bit packed distances are exact while every squared distance and
  // threshold stays below 2^15 (the plan caps H and W, not their squares)
  const bool packed16 = DIST == TRA_DIST_2D && n_cap < 32767;

  const int row = blockIdx.x;
  const int bh = row / NB, u = row - bh * NB;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int q0 = u * B;
  // a block's tokens fill its first n_video + n_text positions
  const int n_u = binfo[(size_t)u * kBlockInfo + 6];

  if (binfo[(size_t)u * kBlockInfo + 9] > 0) {
    // a text block's row keeps every key block
    for (int v = t; v < NB; v += blockDim.x) {
      if (mask) mask[(size_t)row * NB + v] = 1;
      cols[(size_t)row * NB + v] = v;
    }
    if (t == 0) cnt[row] = NB;
    return;
  }
  const int u_frames = binfo[(size_t)u * kBlockInfo + 1] - binfo[(size_t)u * kBlockInfo + 0] + 1;

  for (int qi = t; qi < B; qi += blockDim.x) {
    if (qi < n_u) {
      const int pos = q0 + qi;
      int n = radius_sq[(size_t)bh * S + perm[pos]];
      const bool full = n > n_cap;  // TRA_RADIUS_FULL and anything above the cap
      n = max(n, 0);
      s_c[qi] = coord[pos];
      for (int d = 0; d < F; ++d) s_T[qi * F + d] = full ? INT_MAX : thr[(size_t)n * F + d];
    } else {
      s_c[qi] = 0;
      for (int d = 0; d < F; ++d) s_T[qi * F + d] = -1;  // covers nothing: D >= 0 > -1
    }
  }
  __syncthreads();

  // This lane's queries, fixed for the whole row (positions in the metric's space).
  int qx[QPL], qy[QPL], qf[QPL];
  bool qvalid[QPL];
#pragma unroll
  for (int s = 0; s < QPL; ++s) {
    const int qi = lane + 64 * s;
    position<DIST>(s_c[qi], H, W, &qx[s], &qy[s], &qf[s]);
    qvalid[s] = qi < n_u;
  }

  for (int v = wave; v < NB; v += 4) {
    bool keep;
    if (v == u) {
      keep = true;  // every query keeps its own key, so the diagonal block is never empty
    } else if (binfo[(size_t)v * kBlockInfo + 9] > 0) {
      keep = true;  // text keys stay visible
    } else {
      const int32_t* bi = binfo + (size_t)v * kBlockInfo;
      const int fmin = bi[0], fmax = bi[1], n_v = bi[6];
      const int xmin = DIST == TRA_DIST_1D ? bi[7] : bi[2], xmax = DIST == TRA_DIST_1D ? bi[8] : bi[3];
      const int ymin = DIST == TRA_DIST_1D ? 0 : bi[4], ymax = DIST == TRA_DIST_1D ? 0 : bi[5];
      uint64_t all_m[QPL], part_m[QPL];
      int n_all = 0, n_reach = 0;
      bool any_part = false;
#pragma unroll
      for (int s = 0; s < QPL; ++s) {
        const int qi = lane + 64 * s;
        const int dxn = max(0, max(xmin - qx[s], qx[s] - xmax));
        const int dyn = max(0, max(ymin - qy[s], qy[s] - ymax));
        const int dxf = max(qx[s] - xmin, xmax - qx[s]);
        const int dyf = max(qy[s] - ymin, ymax - qy[s]);
        const int dmin = qf[s] < fmin ? fmin - qf[s] : (qf[s] > fmax ? qf[s] - fmax : 0);
        const int dmax = max(qf[s] - fmin, fmax - qf[s]);
        const int t_hi = s_T[qi * F + dmin];  // thresholds are non-increasing in delta
        const int t_lo = s_T[qi * F + dmax];
        const bool none = !qvalid[s] || metric<DIST>(dxn, dyn) > t_hi;
        const bool all = qvalid[s] && metric<DIST>(dxf, dyf) <= t_lo;
        all_m[s] = ballot(all);
        part_m[s] = ballot(!none && !all);
        n_all += popc(all_m[s]);
        any_part |= part_m[s] != 0;
        // partial queries whose disk over v's frames is more than a point
        n_reach += popc(ballot(!none && !all && t_hi > 0));
      }
      if (RULE == TRA_MASK_VOTE && 3 * n_all > n_u) {
        keep = true;   // every column already has c_j >= n_all > n_u / 3
      } else if (RULE == TRA_MASK_UNION && n_all > 0) {
        keep = true;
      } else if (!any_part) {
        // every column has c_j = n_all; under the vote, 3 n_all <= n_u here
        keep = false;
      } else if (RULE == TRA_MASK_VOTE && 3 * (n_all + u_frames + n_reach) <= n_u) {
        // The vote needs a column with 3 c_j > n_u.  A key j is covered by the
        // n_all queries, by partial queries with a positive threshold, and by
        // partial queries whose threshold there is 0 -- those only at their own
        // (x, y), at most one per frame of u.  So no column reaches n_u / 3 and
        // the block is dropped, exactly as Alg. 1 decides.
        keep = false;
      } else {
        int kx[QPL], ky[QPL], kf[QPL], c[QPL];
        bool kvalid[QPL];
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
          const int j = lane + 64 * s;
          kvalid[s] = j < n_v;
          const int cc = kvalid[s] ? coord[(size_t)v * B + j] : 0;
          position<DIST>(cc, H, W, &kx[s], &ky[s], &kf[s]);
          c[s] = n_all;
        }
        if (packed16 && fmax - fmin <= 1) {
          // Block v spans at most two frames, so a partial query needs two
          // thresholds (keys of frame fmin, keys of frame fmax).  The wave's
          // partial queries are listed in LDS in pairs (16-bit halves), and each
          // step tests two queries against this lane's keys with packed 16-bit
          // arithmetic: D = dx^2 + dy^2 per half, covered iff D - (T + 1) < 0,
          // the sign bits summed into a packed count per key.
          uint16_t* lst = (uint16_t*)&s_pairs[wave][0][0];
          int P = 0;
#pragma unroll
          for (int s = 0; s < QPL; ++s) {
            const uint64_t m = part_m[s];
            if ((m >> lane) & 1) {
              const int qi = lane + 64 * s;
              const int rank = P + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
              uint16_t* e = lst + (rank >> 1) * 8 + (rank & 1);
              e[0] = (uint16_t)qx[s];
              e[2] = (uint16_t)qy[s];
              e[4] = (uint16_t)(s_T[qi * F + abs(qf[s] - fmin)] + 1);
              e[6] = (uint16_t)(s_T[qi * F + abs(qf[s] - fmax)] + 1);
            }
            P += popc(m);
          }
          if ((P & 1) && lane == 0) {
            // pad the last pair with a query that covers nothing (T + 1 = 0)
            uint16_t* e = lst + (P >> 1) * 8 + 1;
            e[0] = 0;
            e[2] = 0;
            e[4] = 0;
            e[6] = 0;
          }
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          short2_t kxx[QPL], kyy[QPL];
          ushort2_t cp[QPL];
          int tf[QPL];
#pragma unroll
          for (int s = 0; s < QPL; ++s) {
            kxx[s] = (short2_t){(short)kx[s], (short)kx[s]};
            kyy[s] = (short2_t){(short)ky[s], (short)ky[s]};
            cp[s] = (ushort2_t){0, 0};
            tf[s] = kf[s] == fmin ? 2 : 3;
          }
          const int pairs = (P + 1) >> 1;
          for (int k = 0; k < pairs; ++k) {
            const uint32_t* ent = &s_pairs[wave][k][0];
            const short2_t X = __builtin_bit_cast(short2_t, ent[0]);
            const short2_t Y = __builtin_bit_cast(short2_t, ent[1]);
#pragma unroll
            for (int s = 0; s < QPL; ++s) {
              const short2_t T1 = __builtin_bit_cast(short2_t, ent[tf[s]]);
              const short2_t dx = kxx[s] - X, dy = kyy[s] - Y;
              const short2_t diff = dx * dx + dy * dy - T1;
              cp[s] += __builtin_bit_cast(ushort2_t, diff) >> (unsigned short)15;
            }
            if (RULE == TRA_MASK_UNION) {
              bool hit = false;
#pragma unroll
              for (int s = 0; s < QPL; ++s) hit |= kvalid[s] && (cp[s][0] | cp[s][1]) != 0;
              if (ballot(hit) != 0) break;  // one covered key decides the union
            }
          }
#pragma unroll
          for (int s = 0; s < QPL; ++s) c[s] += (int)cp[s][0] + (int)cp[s][1];
        } else if (fmax - fmin <= 1) {
          // Block v spans at most two frames, so a query needs two thresholds
          // here: ta for keys of frame fmin, tb for keys of frame fmax.  The
          // partial queries are then walked with their data broadcast from
          // registers (v_readlane), no LDS round trip per query.
          int ta[QPL], tb[QPL];
          bool kfirst[QPL];
#pragma unroll
          for (int s = 0; s < QPL; ++s) {
            const int qi = lane + 64 * s;
            ta[s] = s_T[qi * F + abs(qf[s] - fmin)];
            tb[s] = s_T[qi * F + abs(qf[s] - fmax)];
            kfirst[s] = kf[s] == fmin;
          }
#pragma unroll
          for (int s2 = 0; s2 < QPL; ++s2) {
            uint64_t m = part_m[s2];
            while (m) {
              const int l = __ffsll((unsigned long long)m) - 1;
              m &= m - 1;
              const int px = __builtin_amdgcn_readlane(qx[s2], l);
              const int py = __builtin_amdgcn_readlane(qy[s2], l);
              const int pa = __builtin_amdgcn_readlane(ta[s2], l);
              const int pb = __builtin_amdgcn_readlane(tb[s2], l);
#pragma unroll
              for (int s = 0; s < QPL; ++s)
                c[s] += (metric<DIST>(px - kx[s], py - ky[s]) <= (kfirst[s] ? pa : pb)) ? 1 : 0;
              if (RULE == TRA_MASK_UNION) {
                bool hit = false;
#pragma unroll
                for (int s = 0; s < QPL; ++s) hit |= kvalid[s] && c[s] > 0;
                if (ballot(hit) != 0) break;  // one covered key decides the union
              }
            }
            if (RULE == TRA_MASK_UNION && m != 0) break;
          }
        } else {
#pragma unroll
          for (int s2 = 0; s2 < QPL; ++s2) {
            uint64_t m = part_m[s2];
            while (m) {
              const int qi = __ffsll((unsigned long long)m) - 1 + 64 * s2;
              m &= m - 1;
              int px, py, pf;
              position<DIST>(s_c[qi], H, W, &px, &py, &pf);
              const int32_t* Tp = s_T + qi * F;
#pragma unroll
              for (int s = 0; s < QPL; ++s) {
                const int dx = px - kx[s], dy = py - ky[s];
                const int dl = abs(pf - kf[s]);
                c[s] += (metric<DIST>(dx, dy) <= Tp[dl]) ? 1 : 0;
              }
            }
          }
        }
        int nonempty = 0, high = 0;
#pragma unroll
        for (int s = 0; s < QPL; ++s) {
          nonempty += popc(ballot(kvalid[s] && c[s] > 0));
          high += popc(ballot(kvalid[s] && 3 * c[s] > n_u));
        }
        keep = RULE == TRA_MASK_VOTE ? (nonempty > 0 && 10 * high > 6 * nonempty) : nonempty > 0;
      }
    }
    if (lane == 0) {
      s_keep[v] = keep ? 1 : 0;
      if (mask) mask[(size_t)row * NB + v] = keep ? 1 : 0;
    }
  }
  __syncthreads();

  // Compact the retained key blocks of this row in ascending order.
  if (wave == 0) {
    int base = 0;
    for (int v0 = 0; v0 < NB; v0 += 64) {
      const int v = v0 + lane;
      const bool k = v < NB && s_keep[v];
      const uint64_t bm = ballot(k);
      const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(bm >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)bm, 0u));
      if (k) cols[(size_t)row * NB + base + rank] = v;
      base += popc(bm);
    }
    for (int i = base + lane; i < NB; i += 64) cols[(size_t)row * NB + i] = -1;
    if (lane == 0) cnt[row] = base;
  }
}

// ------------------------------------------------ heaviest-first row order
// Stable counting sort of rows by key NB - cnt (so larger cnt first, ties by
// row index): per-chunk histograms, one exclusive scan in (key, chunk) order,
// then a scatter that ranks equal keys inside a chunk by row index.

__global__ __launch_bounds__(kSortChunk) void order_hist_kernel(const int32_t* __restrict__ cnt,
                                                                int32_t* __restrict__ ws, int rows,
                                                                int NB, int chunks) {
  __shared__ int32_t h[kMaxBlocks + 1];
  for (int i = threadIdx.x; i <= NB; i += blockDim.x) h[i] = 0;
  __syncthreads();
  const int r = blockIdx.x * kSortChunk + threadIdx.x;
  if (r < rows) atomicAdd(&h[NB - min(max(cnt[r], 0), NB)], 1);
  __syncthreads();
  for (int k = threadIdx.x; k <= NB; k += blockDim.x) ws[(size_t)k * chunks + blockIdx.x] = h[k];
}

__global__ __launch_bounds__(1024) void order_scan_kernel(int32_t* __restrict__ ws, int L) {
  __shared__ int32_t part[1024];
  const int t = threadIdx.x;
  const int per = (L + 1023) / 1024;
  const int lo = min(L, t * per), hi = min(L, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += ws[i];
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int run = 0;
    for (int i = 0; i < 1024; ++i) {
      const int x = part[i];
      part[i] = run;
      run += x;
    }
  }
  __syncthreads();
  int run = part[t];
  for (int i = lo; i < hi; ++i) {
    const int x = ws[i];
    ws[i] = run;
    run += x;
  }
}

__global__ __launch_bounds__(kSortChunk) void order_scatter_kernel(const int32_t* __restrict__ cnt,
                                                                   const int32_t* __restrict__ ws,
                                                                   int32_t* __restrict__ order,
                                                                   int rows, int NB, int chunks) {
  __shared__ int32_t keys[kSortChunk];
  const int t = threadIdx.x;
  const int r = blockIdx.x * kSortChunk + t;
  const int key = r < rows ? NB - min(max(cnt[r], 0), NB) : -1;
  keys[t] = key;
  __syncthreads();
  if (r < rows) {
    int rank = 0;
    for (int s = 0; s < t; ++s) rank += keys[s] == key;
    order[ws[(size_t)key * chunks + blockIdx.x] + rank] = r;
  }
}

}  // namespace

template <int B, int RULE, int DIST>
void launch_mask_variant(const tra_plan_s& p, const int32_t* radius_sq, uint8_t* mask, int32_t* cnt,
                         int32_t* cols, hipStream_t s) {
  const int32_t* thr = DIST == TRA_DIST_1D ? p.d_thr1 : p.d_thr;
  const size_t lds = (size_t)B * p.cfg.frames * sizeof(int32_t);
  hipLaunchKernelGGL((block_mask_kernel<B, RULE, DIST>), dim3(p.rows), dim3(256), lds, s, radius_sq, p.d_perm,
                     p.d_coord, thr, p.d_blocks, mask, cnt, cols, p.N, p.S, p.NB, p.cfg.frames,
                     p.cfg.height, p.cfg.width, p.n_cap);
}

template <int B, int RULE>
void launch_mask_dist(const tra_plan_s& p, const int32_t* radius_sq, uint8_t* mask, int32_t* cnt,
                      int32_t* cols, hipStream_t s) {
  if (p.cfg.distance == TRA_DIST_1D) launch_mask_variant<B, RULE, TRA_DIST_1D>(p, radius_sq, mask, cnt, cols, s);
  else launch_mask_variant<B, RULE, TRA_DIST_2D>(p, radius_sq, mask, cnt, cols, s);
}

template <int B>
void launch_mask_rule(const tra_plan_s& p, const int32_t* radius_sq, uint8_t* mask, int32_t* cnt,
                      int32_t* cols, hipStream_t s) {
  if (p.cfg.rule == TRA_MASK_VOTE) launch_mask_dist<B, TRA_MASK_VOTE>(p, radius_sq, mask, cnt, cols, s);
  else launch_mask_dist<B, TRA_MASK_UNION>(p, radius_sq, mask, cnt, cols, s);
}

hipError_t launch_block_mask(const tra_plan_s& p, const int32_t* radius_sq, uint8_t* mask,
                             int32_t* cnt, int32_t* cols, hipStream_t s) {
  if (p.cfg.block == 128) launch_mask_rule<128>(p, radius_sq, mask, cnt, cols, s);
  else launch_mask_rule<64>(p, radius_sq, mask, cnt, cols, s);
  return hipGetLastError();
}

hipError_t launch_row_order_ws(const tra_plan_s& p, const int32_t* cnt, int32_t* order, int32_t* ws,
                               hipStream_t s) {
  const int chunks = p.sort_chunks;
  hipLaunchKernelGGL(order_hist_kernel, dim3(chunks), dim3(kSortChunk), 0, s, cnt, ws, p.rows, p.NB, chunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(order_scan_kernel, dim3(1), dim3(1024), 0, s, ws, (int)((int64_t)(p.NB + 1) * chunks));
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(order_scatter_kernel, dim3(chunks), dim3(kSortChunk), 0, s, cnt, ws, order, p.rows, p.NB,
                     chunks);
  return hipGetLastError();
}

hipError_t launch_row_order(const tra_plan_s& p, const int32_t* cnt, int32_t* order, hipStream_t s) {
  return launch_row_order_ws(p, cnt, order, p.d_sort_ws, s);
}

// ------------------------------------------------ no-allocation entry point
// The counting-sort workspace of tra_build_block_mask_noalloc: a device array
// of the library itself, one copy per GPU, held until the process ends.  In
// host code `scratch` only names the symbol; its device address on each GPU
// comes from hipGetSymbolAddress (resolve_noalloc_scratch) and only that
// address is handed to kernels.  Every order kernel writes each workspace
// entry it later reads, so no clearing is needed between calls.
static __device__ __align__(256) int32_t scratch[kNoAllocScratchInts];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t resolve_noalloc_scratch(int device, int32_t** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    int32_t* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = ptr;
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

hipError_t launch_row_order_noalloc(const tra_plan_s& p, const int32_t* cnt, int32_t* order, hipStream_t s) {
  int32_t* ws = nullptr;
  const hipError_t e = resolve_noalloc_scratch(p.device, &ws);
  if (e != hipSuccess) return e;
  return launch_row_order_ws(p, cnt, order, ws, s);
}

}  // namespace tra
