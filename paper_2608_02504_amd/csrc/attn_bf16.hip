// bf16 attention family on gfx950 matrix cores: dense attention (Eq. 1),
// block-sparse TRA attention (Eq. 16 at block granularity) and the fused
// online-softmax entropy pass (App. C.2, Alg. 2), all from one template.
//
// Work decomposition
//   One workgroup (4 waves, 256 threads) per query-block row r = (b, h, u):
//   128 queries, wave w owning queries [32w, 32w + 32).  The workgroup walks
//   the key blocks of its row (all NB for dense; cols[r][0..cnt[r]) for
//   sparse), 128 keys at a time.
//
// Per key block
//   K (128 x d) is staged row-major in LDS and V (128 x d) transposed (d x 128).
//   Each wave computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (keys are the
//   M side, its 32 queries the N side), so a lane holds 64 scores of ONE query:
//   row max and row sum are in-lane reductions plus one exchange between the two
//   lane halves.  The probabilities are converted to bf16 in registers and
//   reused directly as the B operand of O^T += V^T P^T, again 32x32x16 MFMAs
//   with fp32 accumulation.  Softmax runs in the base-2 domain with
//   alpha * log2(e) folded into one FMA per score.
//
// Entropy (Alg. 2 with the running sum kept relative to the running max)
//   x = s alpha log2(e) - m,  w = 2^x,  l = sum w,  a = sum w x.
//   On a max increase m -> m': l <- 2^{m-m'} l, a <- 2^{m-m'} (a + l (m - m')).
//   H = ln(l) - ln(2) a / l  (nats)  == log Z - sum_j p_j s_j (App. C.2).
//   Each lane keeps l and a over its own keys; the halves are added at the end.
//
// Tokens are read and written through the tile-major permutation of Sec. 3.3
// (perm[p] = raster row of tile-major position p), so the caller's tensors stay
// in raster order.
#include <cmath>

#include "tra_internal.h"

namespace tra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kBQ = 128;        // queries per workgroup (= block size)
constexpr int kBK = 128;        // keys per tile (= block size)
constexpr int kThreads = 256;
constexpr int kVtStride = kBK + 4;  // Vt row stride in bf16 (264 B: 8-byte reads spread over all banks)

struct Bf16Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  float* entropy;
  const int32_t* perm;
  const int32_t* cnt;
  const int32_t* cols;
  const int32_t* order;
  int N, NB, rows;
  float scale_log2;  // alpha * log2(e)
};

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 f = {a, b};
  bf16x2 h = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// XCD-aware row mapping: workgroups are dispatched round-robin over the 8
// XCDs, so give each XCD one contiguous range of rows.  Neighbouring query
// blocks of one head retain overlapping key blocks, which then share that
// XCD's L2.
__device__ __forceinline__ int xcd_row(int g, int R) {
  const int x = g & 7, i = g >> 3;
  const int q = R >> 3, rmd = R & 7;
  return x * q + min(x, rmd) + i;
}

template <int D, bool SPARSE, bool PV, bool ENT>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(Bf16Params P) {
  constexpr int KS = D + 8;   // K row stride in bf16 (16-byte reads spread over all banks)
  constexpr int QK_STEPS = D / 16;
  constexpr int D_TILES = D / 32;
  __shared__ __attribute__((aligned(16))) uint16_t sK[kBK * KS];
  __shared__ __attribute__((aligned(16))) uint16_t sVt[PV ? D * kVtStride : 8];

  int r;
  if (SPARSE && P.order) {
    r = P.order[blockIdx.x];
    if (r < 0 || r >= P.rows) return;  // whole workgroup leaves together
  } else {
    r = xcd_row(blockIdx.x, P.rows);
  }
  const int bh = r / P.NB, u = r - bh * P.NB;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int col = lane & 31;   // query column of this lane within the wave
  const int half = lane >> 5;  // lane half: selects k-slots / output rows
  const size_t head_off = (size_t)bh * P.N * D;

  // ---- Q fragments: B operand of S^T = K Q^T, 8 bf16 per lane per 16-deep step
  const int qpos = u * kBQ + wave * 32 + col;
  const bool qvalid = qpos < P.N;
  const int qrow = qvalid ? P.perm[qpos] : 0;
  bf16x8 qf[QK_STEPS];
  {
    const uint4* src = (const uint4*)(P.q + head_off + (size_t)qrow * D);
#pragma unroll
    for (int kk = 0; kk < QK_STEPS; ++kk) {
      uint4 x = qvalid ? src[2 * kk + half] : make_uint4(0, 0, 0, 0);
      qf[kk] = __builtin_bit_cast(bf16x8, x);
    }
  }

  f32x16 oacc[PV ? D_TILES : 1];
#pragma unroll
  for (int i = 0; i < (PV ? D_TILES : 1); ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[i][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f, a_run = 0.f;

  const int count = SPARSE ? min(max(P.cnt[r], 0), P.NB) : P.NB;
  const int32_t* colp = SPARSE ? P.cols + (size_t)r * P.NB : nullptr;

  for (int c = 0; c < count; ++c) {
    const int vb = SPARSE ? colp[c] : c;
    if (SPARSE && (vb < 0 || vb >= P.NB)) continue;  // uniform across the workgroup
    const int k0 = vb * kBK;
    const int nv = min(kBK, P.N - k0);

    __syncthreads();  // previous tile fully consumed
    // ---- K tile -> LDS, row-major.  16 threads cover one 2*D-byte row.
    {
      constexpr int CH = D / 8;              // 16-byte chunks per row
      constexpr int RPP = kThreads / CH;     // rows per pass
      const int ch = t % CH;
#pragma unroll
      for (int r0 = 0; r0 < kBK; r0 += RPP) {
        const int j = r0 + t / CH;
        uint4 x = make_uint4(0, 0, 0, 0);
        if (j < nv) x = ((const uint4*)(P.k + head_off + (size_t)P.perm[k0 + j] * D))[ch];
        *(uint4*)&sK[j * KS + ch * 8] = x;
      }
    }
    // ---- V tile -> LDS transposed: two keys per 32-bit word.
    if (PV) {
      const int pr = t & 63;   // key pair (keys 2pr, 2pr+1)
      const int g0 = t >> 6;   // first 8-wide d chunk
      const int j0 = 2 * pr, j1 = 2 * pr + 1;
      const uint4* s0 = (const uint4*)(P.v + head_off + (size_t)P.perm[k0 + min(j0, nv - 1)] * D);
      const uint4* s1 = (const uint4*)(P.v + head_off + (size_t)P.perm[k0 + min(j1, nv - 1)] * D);
#pragma unroll
      for (int g = g0; g < D / 8; g += 4) {
        uint4 a = j0 < nv ? s0[g] : make_uint4(0, 0, 0, 0);
        uint4 b = j1 < nv ? s1[g] : make_uint4(0, 0, 0, 0);
        const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
        const uint32_t bw[4] = {b.x, b.y, b.z, b.w};
        uint32_t* dst = (uint32_t*)&sVt[(g * 8) * kVtStride + j0];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // d = 8g + 2e and 8g + 2e + 1: low / high halves of the words
          dst[(2 * e) * (kVtStride / 2)] = __builtin_amdgcn_perm(bw[e], aw[e], 0x05040100u);
          dst[(2 * e + 1) * (kVtStride / 2)] = __builtin_amdgcn_perm(bw[e], aw[e], 0x07060302u);
        }
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T : 4 sub-tiles of 32 keys x 32 queries
    f32x16 s[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
      const uint16_t* kr = &sK[(kt * 32 + col) * KS + half * 8];
#pragma unroll
      for (int kk = 0; kk < QK_STEPS; ++kk) {
        const bf16x8 ka = __builtin_bit_cast(bf16x8, *(const uint4*)(kr + kk * 16));
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], s[kt], 0, 0, 0);
      }
    }
    // Output element e of sub-tile kt is key 32kt + 8(e/4) + 4*half + e%4.
    // Keys past the end of a ragged last block get a large finite negative
    // score: their weight 2^x underflows to 0 and w * x stays 0 (not 0 * inf).
    if (nv < kBK) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kt * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
          if (key >= nv) s[kt][e] = -1.0e30f;
        }
    }

    // ---- online softmax (base 2)
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * P.scale_log2);
    const float sc = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 on the first tile
    if (ENT) a_run = l_run > 0.f ? sc * (a_run + l_run * (m_run - m_new)) : 0.f;
    l_run *= sc;
    if (PV) {
#pragma unroll
      for (int i = 0; i < D_TILES; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[i][e] *= sc;
    }
    m_run = m_new;

    uint32_t pb[4][8];  // bf16 pairs of probabilities: [sub-tile][pair]
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float x0 = fmaf(s[kt][e], P.scale_log2, -m_new);
        const float x1 = fmaf(s[kt][e + 1], P.scale_log2, -m_new);
        const float w0 = __builtin_amdgcn_exp2f(x0);
        const float w1 = __builtin_amdgcn_exp2f(x1);
        l_run += w0 + w1;
        if (ENT) a_run = fmaf(w0, x0, fmaf(w1, x1, a_run));
        if (PV) pb[kt][e >> 1] = pack_bf16x2(w0, w1);
      }
    }

    // ---- O^T += V^T P^T.  k-step ks covers keys [16ks, 16ks+16); in lane half h
    // the B operand (from sub-tile ks/2, elements 8(ks%2)..+7) holds keys
    // 16ks + 4h + {0,1,2,3} and 16ks + 8 + 4h + {0,1,2,3}; the A operand (V^T
    // rows) is read with the same key order.
    if (PV) {
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const int kt = ks >> 1, eb = (ks & 1) * 4;
        const uint4 bw = make_uint4(pb[kt][eb], pb[kt][eb + 1], pb[kt][eb + 2], pb[kt][eb + 3]);
        const bf16x8 pbv = __builtin_bit_cast(bf16x8, bw);
#pragma unroll
        for (int dt = 0; dt < D_TILES; ++dt) {
          const uint16_t* vr = &sVt[(dt * 32 + col) * kVtStride + ks * 16 + 4 * half];
          const uint2 lo = *(const uint2*)vr;
          const uint2 hi = *(const uint2*)(vr + 8);
          const bf16x8 va = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pbv, oacc[dt], 0, 0, 0);
        }
      }
    }
  }

  // ---- epilogue (cross-half sums first: every lane takes part in the exchange)
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float a_tot = ENT ? a_run + __shfl_xor(a_run, 32) : 0.f;
  if (!qvalid) return;
  const size_t tok = (size_t)bh * P.N + qrow;
  if (PV) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    uint16_t* dst = P.o + tok * D;
#pragma unroll
    for (int dt = 0; dt < D_TILES; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        // elements 4g..4g+3 hold d = 32dt + 8g + 4*half + {0,1,2,3}
        const int d0 = dt * 32 + 8 * g + 4 * half;
        uint2 w;
        w.x = pack_bf16x2(oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv);
        w.y = pack_bf16x2(oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv);
        *(uint2*)(dst + d0) = w;
      }
  }
  if (half == 0) {
    if (ENT) P.entropy[tok] = 0.69314718055994531f * (__log2f(l_tot) - a_tot / l_tot);
    if (P.lse)
      P.lse[tok] = l_tot > 0.f ? 0.69314718055994531f * (m_run + __log2f(l_tot)) : -INFINITY;
  }
}

template <int D>
hipError_t launch_bf16_d(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  Bf16Params P{(const uint16_t*)a.q, (const uint16_t*)a.k, (const uint16_t*)a.v, (uint16_t*)a.o,
               a.lse, a.entropy, p.d_perm, a.cnt, a.cols, a.order, p.N, p.NB, p.rows,
               (float)(1.4426950408889634 / std::sqrt((double)D))};
  const dim3 grid(p.rows), block(kThreads);
  if (a.sparse)
    hipLaunchKernelGGL((attn_bf16_kernel<D, true, true, false>), grid, block, 0, s, P);
  else if (a.entropy && a.o)
    hipLaunchKernelGGL((attn_bf16_kernel<D, false, true, true>), grid, block, 0, s, P);
  else if (a.entropy)
    hipLaunchKernelGGL((attn_bf16_kernel<D, false, false, true>), grid, block, 0, s, P);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<D, false, true, false>), grid, block, 0, s, P);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_bf16(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  if (p.cfg.head_dim == 64) return launch_bf16_d<64>(p, a, s);
  return launch_bf16_d<128>(p, a, s);
}

}  // namespace tra
