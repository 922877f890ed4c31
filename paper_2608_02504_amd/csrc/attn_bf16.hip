// bf16 attention family on gfx950 matrix cores: dense attention (Eq. 1),
// block-sparse TRA attention (Eq. 16 at block granularity), its token-level
// form (the token mask of Eq. 15 inside the retained blocks) and the
// online-softmax entropy pass (App. C.2, Alg. 2).  Three kernels:
//   attn_k64_kernel   dense and block-sparse output, 64-key tiles, three
//                     4-wave workgroups per CU;
//   attn_bf16_kernel  token-level output (two 4-wave workgroups per CU) and the
//                     entropy pass (four), 128-key tiles;
//   attn_fused_kernel the entropy pass fused with the dense output, 8 waves
//                     splitting the keys of one query block.
//
// Layout pre-pass
//   K and V are first gathered into tile-major order (Sec. 3.3: tokens of a
//   spatial tile become contiguous) in the call's workspace, one 128-token key
//   block = one contiguous tile, padding positions zero-filled: K as 128 rows x D,
//   V transposed (D rows x 128 keys), so that both matrix operands are read
//   from LDS with plain 16-byte reads.  The attention loop then addresses
//   tiles affinely.  Q is gathered and O scattered through the same
//   permutation inside the kernel, so callers keep raster order.
//
// Work decomposition
//   The unit of work is a query-block row r = (b, h, u): 128 queries, wave w of
//   a 4-wave workgroup owning queries [32w, 32w + 32), walking the key blocks
//   of the row (all NB for dense; cols[r][0..cnt[r]) for sparse).  Every kernel
//   is persistent: as many workgroups as can be resident, each taking rows
//   from a row queue (per-XCD contiguous ranges with stealing, see next_row)
//   until it is drained.  Several workgroups share a CU, so a SIMD can run one
//   workgroup's matrix phase while another is in its softmax.  Block-sparse
//   calls take work units instead of rows: long rows are cut into pieces whose
//   partial results a merge kernel combines, and each XCD's segment of the
//   unit table lists its split pieces first, piece-major, so that the
//   workgroups of one XCD walk the same key range (see plan_units_kernel).
//
// Per tile (split barriers)
//   K and V^T go from HBM straight into LDS (global_load_lds_dwordx4 from a
//   scalar tile base, no register staging), 16-byte chunks XOR-swizzled per
//   row so that operand reads hit every bank once.  The next K tile streams in
//   during softmax + PV, the next V^T tile during QK^T + softmax.  Scheduling
//   hints keep four LDS operand reads in flight ahead of the MFMAs.
//
// Matrix work (v_mfma_f32_32x32x16_bf16, fp32 accumulation)
//   S^T = K Q^T: keys are the M side and the wave's 32 queries the N side, so a
//   lane holds the scores of ONE query (row max / row sum are in-lane plus one
//   cross-half lane swap).  The bf16 probabilities stay in registers as the B
//   operand of O^T += V^T P^T; K rows are loaded in an order that leaves every
//   lane half holding 8 consecutive keys, the k-slice a V^T row chunk covers.
//
// Softmax and entropy (Alg. 2 with the running sum kept relative to the max)
//   x = s alpha log2(e) - m,  w = 2^x,  l = sum w,  a = sum w x.
//   On a max increase m -> m': l <- 2^{m-m'} l, a <- 2^{m-m'} (a + l (m - m')).
//   H = ln(l) - ln(2) a / l  (nats)  == log Z - sum_j p_j s_j (App. C.2).
//   Each lane keeps l and a over its own keys; the halves are added at the end.
#include <algorithm>
#include <climits>
#include <cmath>

#include "tra_internal.h"

namespace tra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kBQ = 128;       // queries per workgroup (= block size)
constexpr int kBK = 128;       // keys per tile (= block size)
constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 f = {a, b};
  bf16x2 h = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// XOR swizzle of the 16-byte chunks of LDS row `row` (one K row of D*2 bytes =
// CH chunks, or one V^T row of 128 keys = 16 chunks): 16 consecutive rows read
// at one logical chunk, which is what the 16 lanes of one LDS cycle of an
// operand read ask for, land in 16 distinct bank groups.
template <int CH>
__device__ __forceinline__ int swz(int row) {
  if constexpr (CH == 16) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);  // CH == 8: two rows per 256 B
}

// vmcnt-only wait (expcnt and lgkmcnt left unconstrained), gfx9 encoding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations,
// then s_barrier.  __syncthreads() would also drain every outstanding global
// load (its release fence), which would stall on the tile loads that are
// meant to stay in flight across the barrier; tile readiness is instead
// established with explicit vmcnt waits before the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ------------------------------------------------------------ layout pre-pass
// Both gathers take (batch, head) pairs bh = blockIdx.y, blockIdx.y + gridDim.y, ...
// (the grid's y extent is capped at kGatherMaxY).
constexpr int kGatherMaxY = 65535;

// kt[bh][p][:] = k[bh][perm[p]][:], 0 where perm[p] < 0 (a padding position).
// Grid: (16-byte chunks of one head / 256, pairs); thread = one chunk.
template <int D>
__global__ __launch_bounds__(256) void gather_k_kernel(const uint4* __restrict__ k, uint4* __restrict__ kt,
                                                       const int32_t* __restrict__ perm, int N, int n_pad,
                                                       int bhs) {
  constexpr int CH = D / 8;
  const int idx = blockIdx.x * 256 + threadIdx.x;  // < n_pad * CH < 2^24
  if (idx >= n_pad * CH) return;
  const int p = idx / CH, c = idx % CH;
  const int tok = perm[p];
  for (size_t bh = blockIdx.y; bh < (size_t)bhs; bh += gridDim.y)
    kt[bh * n_pad * CH + idx] = tok >= 0 ? k[(bh * N + tok) * CH + c] : make_uint4(0, 0, 0, 0);
}

// V transposed per key block, tile-major: for tile-major position p = 128 b + j,
// vt[bh][b][d][j] = v[bh][perm[p]][d] (0 at a padding position), so key block b of a
// head is one contiguous D x 128 tile with the key index fastest.  One
// workgroup per 64 positions (of one pair at a time), through LDS.
template <int D>
__global__ __launch_bounds__(256) void gather_vt_kernel(const uint16_t* __restrict__ v,
                                                        uint16_t* __restrict__ vt,
                                                        const int32_t* __restrict__ perm, int N,
                                                        int n_pad, int bhs) {
  constexpr int TOK = 64, CH = D / 8, LS = D + 2;
  __shared__ uint16_t tile[TOK * LS];
  const int p0 = blockIdx.x * TOK, t = threadIdx.x;
  for (int bh = blockIdx.y; bh < bhs; bh += gridDim.y) {
    __syncthreads();  // the previous pair's reads of the tile are done
    for (int i = t; i < TOK * CH; i += 256) {
      const int j = i / CH, c = i - j * CH;
      uint4 x = make_uint4(0, 0, 0, 0);
      const int tok = perm[p0 + j];
      if (tok >= 0) x = *(const uint4*)(v + ((size_t)bh * N + tok) * D + c * 8);
      const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        tile[j * LS + c * 8 + 2 * e] = (uint16_t)(w[e] & 0xFFFFu);
        tile[j * LS + c * 8 + 2 * e + 1] = (uint16_t)(w[e] >> 16);
      }
    }
    __syncthreads();
    for (int i = t; i < D * (TOK / 8); i += 256) {
      const int d = i / (TOK / 8), tc = i - d * (TOK / 8);
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)tile[(tc * 8 + 2 * e) * LS + d] | ((uint32_t)tile[(tc * 8 + 2 * e + 1) * LS + d] << 16);
      const int p = p0 + tc * 8;
      *(uint4*)(vt + (size_t)bh * n_pad * D + ((size_t)(p / kBK) * D + d) * kBK + p % kBK) =
          make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// ------------------------------------------------------------ attention
template <int D>
struct Geo {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int QK_STEPS = D / 16;
  static constexpr int D_TILES = D / 32;
};

// One 16-byte HBM -> LDS copy per lane (global_load_lds_dwordx4 with a scalar
// base): lane i reads sbase + voff_i and its 16 bytes land at LDS address
// lds_base + 16 i.  Issued as inline assembly so the compiler does not track
// it: its conservative tracking of LDS-writing loads would wait for every tile
// in flight before any LDS read.  Completion is established by the explicit
// vmcnt waits before the barriers that publish a tile, so the loads stay in
// flight across unrelated LDS work.  Nothing else in these kernels uses m0.
// The LDS address is lds_base + LDS_STEP, formed in m0 by the same statement
// so that no per-step copy of it is kept live.
template <int LDS_STEP>
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_add_u32 m0, %2, %3\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_base), "i"(LDS_STEP)
               : "memory", "m0", "scc");
}

// A tile (K: 128 rows x D; V^T: D rows x 128 keys; 32 KB or 16 KB, contiguous
// in HBM) is copied by the 4 waves in 4 KB steps: step n of wave w fills LDS
// bytes [4096 n + 1024 w, +1024) from HBM bytes 4096 n + tile_lane_off.  A
// 4 KB step spans 16 K rows (D = 128) or 32 (D = 64), or 16 V^T rows, so row
// mod 16 and with it the swizzle is the same in every step: the per-lane
// offset is fixed and only the scalar base moves.
template <int D>
struct TileCopy {
  static constexpr int STEPS = kBK * D * 2 / 4096;
};

// Lane offset within a 4 KB step of a K tile: row wave * RPI + lane / CH,
// physical chunk lane % CH, which holds logical chunk (lane % CH) ^ swz(row).
template <int D>
__device__ __forceinline__ uint32_t k_lane_off(int wave, int lane) {
  constexpr int CH = D / 8, RPI = 64 / CH;
  const int row = wave * RPI + lane / CH;
  return row * D * 2 + (((lane % CH) ^ swz<CH>(row)) << 4);
}

// Lane offset within a 4 KB step of a V^T tile (rows of 128 keys = 16 chunks):
// row wave * 4 + lane / 16, physical chunk lane % 16.
__device__ __forceinline__ uint32_t vt_lane_off(int wave, int lane) {
  const int row = wave * 4 + lane / 16;
  return row * kBK * 2 + (((lane % 16) ^ swz<16>(row)) << 4);
}

template <int N>
__device__ __forceinline__ void issue_steps(uint32_t lds_wave, const uint8_t* tile, uint32_t lane_off) {
  if constexpr (N > 0) {
    issue_steps<N - 1>(lds_wave, tile, lane_off);
    dma16<(N - 1) * 4096>(tile + (N - 1) * 4096, lane_off, lds_wave);
  }
}

template <int D>
__device__ __forceinline__ void issue_tile(uint32_t lds_wave, const uint8_t* tile, uint32_t lane_off) {
  issue_steps<TileCopy<D>::STEPS>(lds_wave, tile, lane_off);
}

// max / sum of a value over the two lane halves (lanes l and l ^ 32), with
// one cross-half swap instead of an LDS round trip
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ bf16x8 lds_read16(const lds_u8* base, uint32_t off) {
  return __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) uint4*)(base + off));
}

// Hides a value from the optimiser, so that offsets derived from it are
// recomputed next to their use instead of being hoisted out of the tile loop
// and kept live in registers.
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

// LDS byte offset of logical 16-byte chunk 2k + h of a row whose chunks are
// XOR-swizzled by sw: (2k + h) ^ sw == 2k ^ (h ^ sw), so with
// base = row_bytes + ((h ^ sw) << 4) the offset is base ^ (k << 5): one XOR per
// read (the row bytes are a multiple of 128, above the chunk bits).
__device__ __forceinline__ uint32_t chunk_off(uint32_t base, int k) { return base ^ (uint32_t)(k << 5); }

// One MFMA step of S^T = K Q^T for sub-tile kt and k-step kk.
template <int D>
__device__ __forceinline__ void qk_step(f32x16& s, const lds_u8* __restrict__ kbuf, uint32_t koff_kk,
                                        const bf16x8 (&qf)[Geo<D>::QK_STEPS], int kt, int kk) {
  const bf16x8 ka = lds_read16(kbuf, koff_kk + kt * 32 * D * 2);
  s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], s, 0, 0, 0);
}

// Scheduling pattern for a run of n MFMAs each fed by `reads` LDS reads: the
// first `ahead` MFMAs' operands are requested up front, then every MFMA is
// followed by the reads of the MFMA `ahead` places later, so LDS latency hides
// behind matrix work.
template <int n, int reads, int ahead>
__device__ __forceinline__ void sched_reads_ahead() {
#pragma unroll
  for (int i = 0; i < ahead; ++i) __builtin_amdgcn_sched_group_barrier(0x100, reads, 0);
#pragma unroll
  for (int i = 0; i < n - ahead; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, reads, 0);
  }
#pragma unroll
  for (int i = 0; i < ahead; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
}

template <int D>
__device__ __forceinline__ void qk_tile(f32x16 (&s)[4], const lds_u8* __restrict__ kbuf, uint32_t kbase,
                                        const bf16x8 (&qf)[Geo<D>::QK_STEPS]) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
  kbase = opaque(kbase);
  // k-step outer, sub-tile inner: four independent accumulation chains
#pragma unroll
  for (int kk = 0; kk < Geo<D>::QK_STEPS; ++kk) {
    const uint32_t off = chunk_off(kbase, kk);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) qk_step<D>(s[kt], kbuf, off, qf, kt, kk);
  }
  sched_reads_ahead<4 * Geo<D>::QK_STEPS, 1, 4>();
}

// Keys past the end of a ragged last block get a large finite negative score:
// their weight 2^x underflows to 0 and w * x stays 0 (not 0 * inf).
// Output element e of sub-tile kt is key 32kt + 16(e/8) + 8*half + e%8 (the
// K rows are loaded in that order: krow in the kernel).  The select is done with
// integer arithmetic (sign of key - nv as a bit mask) so that no per-element
// lane mask is materialised in scalar registers.
__device__ __forceinline__ void mask_tail(f32x16 (&s)[4], int nv, int half) {
  const int base = 8 * half - nv;
  const uint32_t neg = __float_as_uint(-1.0e30f);
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint32_t keep = (uint32_t)((kt * 32 + 16 * (e >> 3) + (e & 7) + base) >> 31);
      s[kt][e] = __uint_as_float(((__float_as_uint(s[kt][e]) & keep) | (neg & ~keep)));
    }
}

// lr is the sum of the weights as rounded to the bf16 probabilities that PV
// multiplies (the output is normalised by it, so that the bf16 weights form an
// exact convex combination: a query dominated by one key gets that key's value
// to fp32 rounding); l is the fp32 sum (log-sum-exp, entropy).
struct RowState {
  float m, l, a, lr;  // running max (log2 units), sum of weights, entropy sum, rounded sum
};

// acc + the two bf16 probabilities packed in p, in fp32 (one v_dot2 with 1.0).
__device__ __forceinline__ float add_bf16_pair(uint32_t p, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p), __builtin_bit_cast(bf16x2, 0x3F803F80u),
                                         acc, false);
}

// Floor of the running max (log2 units), far below any real score and far
// above the masked ones (-1e30 times the scale): a tile whose keys are all
// masked for a query then leaves m at the floor and gives its masked keys
// weight 2^(-1e29) = 0.  Without it m would be the masked value itself, and
// s * scale - m, formed by one fma from the exact product, would leave the
// product's rounding error (~1e22) instead of 0 -- an infinite weight.
constexpr float kMaxFloor = -1.0e20f;

// Lazy rescaling: the exponent reference m of a query moves only when a tile's
// max exceeds it by more than kMaxSlack (log2 units).  Weights then stay below
// 2^kMaxSlack = 256 (fine for the fp32 sums and the bf16 probabilities), the
// normalisation by l at the end is unchanged, and the O rescale -- and with it
// most of the max bookkeeping -- runs on the first tiles of a row only.
constexpr float kMaxSlack = 8.0f;

// In the 128-key kernel (entropy pass, token-level attention), tiles after a
// wave's first take their weights against the current reference
// without forming the tile max: a lane's sum of weights at most kFastSum bounds
// every weight by it (they are positive), so nothing can overflow -- weights up
// to 2^20 keep O, l and the bf16 probabilities far inside the fp32 / bf16
// range for any |v| below 2^80.  Only when some lane's sum exceeds it (or is
// not finite) is the tile redone from its max, which moves the reference; on
// the method's inputs that is a fraction of a percent of the tiles.  The
// reference is always some earlier tile's max, so the largest weight of a row
// is at least 1 and nothing that matters underflows.
constexpr float kFastSum = 1048576.0f;  // 2^20

// New exponent reference of one query from its tile max (log2 units).
__device__ __forceinline__ float next_reference(float m, float tile_max_scaled) {
  const float m_new = tile_max_scaled > m + kMaxSlack ? tile_max_scaled : m;
  return fmaxf(m_new, kMaxFloor);
}

// Max of a score tile folded into the running state; returns the factor that
// rescales everything accumulated so far (0 on the first tile).
template <bool ENT>
__device__ __forceinline__ float tile_max(const f32x16 (&s)[4], float scale_log2, RowState& st) {
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
  mx = max_halves(mx);
  const float m_new = next_reference(st.m, mx * scale_log2);
  const float sc = __builtin_amdgcn_exp2f(st.m - m_new);
  if (ENT) st.a = st.l > 0.f ? sc * (st.a + st.l * (st.m - m_new)) : 0.f;
  st.l *= sc;
  st.lr *= sc;
  st.m = m_new;
  return sc;
}

// Weights of sub-tile kt: w = 2^(s alpha log2e - m), summed into l (and w x into
// a); bf16 pairs into pb[8kt .. 8kt+7].
// With PV the rounded pairs are also added to the four accumulation chains
// lr4, which a caller carries over all sub-tiles of a tile (one long chain of
// dot products would stall the wave on their latency); with LF the fp32
// weights into lsum.  tile_exp: the same for one sub-tile, with its own
// chains, their total added to lrsum.
template <bool PV, bool ENT, bool LF = true>
__device__ __forceinline__ void tile_exp_acc(const f32x16& s, float scale_log2, float m, float& lsum,
                                             float& asum, float (&lr4)[4], uint32_t* pb) {
#pragma unroll
  for (int e = 0; e < 16; e += 2) {
    const float x0 = fmaf(s[e], scale_log2, -m);
    const float x1 = fmaf(s[e + 1], scale_log2, -m);
    const float w0 = __builtin_amdgcn_exp2f(x0);
    const float w1 = __builtin_amdgcn_exp2f(x1);
    if (LF) lsum += w0 + w1;
    if (ENT) asum = fmaf(w0, x0, fmaf(w1, x1, asum));
    if (PV) {
      pb[e >> 1] = pack_bf16x2(w0, w1);
      lr4[(e >> 1) & 3] = add_bf16_pair(pb[e >> 1], lr4[(e >> 1) & 3]);
    }
  }
}

template <bool PV, bool ENT, bool LF = true>
__device__ __forceinline__ void tile_exp(const f32x16& s, float scale_log2, float m, float& lsum,
                                         float& asum, float& lrsum, uint32_t* pb) {
  float lr4[4] = {0.f, 0.f, 0.f, 0.f};
  tile_exp_acc<PV, ENT, LF>(s, scale_log2, m, lsum, asum, lr4, pb);
  if (PV) lrsum += (lr4[0] + lr4[1]) + (lr4[2] + lr4[3]);
}

// O^T += V^T P^T.  k-step ks covers keys [16ks, 16ks+16); in lane half h the
// B operand (sub-tile ks/2, elements 8(ks%2)..+7) holds the 8 consecutive keys
// 16ks + 8h + {0..7}, and the A operand row d = 32dt + (lane % 32) of V^T is the
// 16-byte chunk (2ks + h) of that row in LDS.
template <int D>
__device__ __forceinline__ void pv_step(f32x16& oacc, const lds_u8* __restrict__ vbuf, uint32_t voff_ks,
                                        const uint32_t (&pb)[32], int ks, int dt) {
  const int kt = ks >> 1, eb = (ks & 1) * 4;
  const uint4 bw = make_uint4(pb[kt * 8 + eb], pb[kt * 8 + eb + 1], pb[kt * 8 + eb + 2], pb[kt * 8 + eb + 3]);
  const bf16x8 va = lds_read16(vbuf, voff_ks + dt * 32 * kBK * 2);
  oacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, __builtin_bit_cast(bf16x8, bw), oacc, 0, 0, 0);
}

// ------------------------------------------------------------ token mask inside a tile
// Inputs of the token-level variant (Eq. 15 inside the listed blocks).
struct TokArgs {
  const int32_t* radius_sq;  // [B*Ha][S] per-token squared radii, raster order
  const int32_t* thr;        // [(n_cap + 1) * F] thresholds (2-D or 1-D per the plan)
  const int32_t* kinfo;      // [NB][kKeyInfo] key distance words, then frames
  const int32_t* binfo;      // [NB][kBlockInfo] block boxes
  const int32_t* coord;      // [S] packed (f, x, y) per tile-major position
  const uint16_t* kfeat;     // 2-D: [NB][128][kKeyFeat] f16 key vectors of the token mask
  int Nv, F, n_cap;
};

typedef short short2_t __attribute__((ext_vector_type(2)));
typedef int int4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int4v lds_read_i4(const lds_u8* base, uint32_t off) {
  return *(const __attribute__((address_space(3))) int4v*)(base + off);
}

// Distance between a query and a key from their distance words: 2-D squared
// Euclidean distance of the packed (x, y) (packed 16-bit subtract, then a
// 16-bit dot product), or |i - j| of raster indices for the 1-D ablation.
template <int TOK>
__device__ __forceinline__ int token_metric(int qw, int kw) {
  if constexpr ((TOK & 3) == 2) {
    return abs(qw - kw);
  } else {
    const short2_t d = __builtin_bit_cast(short2_t, qw) - __builtin_bit_cast(short2_t, kw);
    return __builtin_amdgcn_sdot2(d, d, 0, false);
  }
}

// Token mask of one score tile for this lane's query: element e of sub-tile
// kt is key 32 kt + 16 (e / 8) + 8 half + e % 8 of the block; it keeps its
// score iff the query covers the key (distance <= the query's threshold for
// the key's frame: t_lo for the block's first frame, t_hi for its second) or
// the key is a text token, else gets the same large negative score as the
// ragged tail.  kinfo: the block's 128 key words (distance word, second-frame
// flag at bit 15 for 2-D / 30 for 1-D, text flag at bit 31; the text test is
// compiled in only for plans with text tokens, TOK & 4).  One code path for
// every block: a second, single-frame specialisation would not fit the
// kernel's registers alongside it.
template <int TOK>
__device__ __forceinline__ void token_mask(f32x16 (&s)[4], const lds_u8* __restrict__ kinfo, int half,
                                           int qw, int t_lo, int t_hi) {
  const uint32_t neg = __float_as_uint(-1.0e30f);
  constexpr int kFrameBit = (TOK & 3) == 2 ? 30 : 15;
  constexpr uint32_t kWordMask = (TOK & 3) == 2 ? 0x3FFFFFFFu : 0x7FFF7FFFu;
  constexpr bool kText = (TOK & 4) != 0;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int g = 0; g < 2; ++g) {
#pragma unroll
      for (int h4 = 0; h4 < 2; ++h4) {
        const int k0 = kt * 32 + 16 * g + 8 * half + 4 * h4;  // 4 consecutive keys
        const int4v w = lds_read_i4(kinfo, 4 * k0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int dist = token_metric<TOK>(qw, (int)((uint32_t)w[j] & kWordMask));
          const bool keep = (kText && w[j] < 0) || dist <= (((w[j] >> kFrameBit) & 1) ? t_hi : t_lo);
          const int e = 8 * g + 4 * h4 + j;
          s[kt][e] = keep ? s[kt][e] : __uint_as_float(neg);
        }
      }
    }
}

// 2-D token mask of one score tile as a matrix product: E^T = B_K A_Q^T on a
// 32x32x8 f16 MFMA per 32-key sub-tile, with the keys' vectors b_j (8 f16
// integers each, from the plan's key-feature table, stored half-major so that
// a lane half's reads are consecutive; rows in the same krow order as the K
// operand so that E lines up with S element by element) and
// this lane's query vector a_i, so that E_ij = T_i(frame of j) - D_ij (1 for a
// text key).  The key is covered iff E_ij >= 0; every term is an integer and
// every partial sum stays below 2^24, so the test is exact.  Lane half h holds
// components 4h..4h+3 of both vectors: a_i = (h_lo, l_lo, h_hi, l_hi | 2048, 1,
// 2x_i, 2y_i) with T - x_i^2 - y_i^2 = 2048 h + l for the thresholds of the
// block's first and second frame (a query covering every key gets T = 2^22,
// beyond any squared distance on a 1023 x 1023 frame).
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void token_mask_mfma(f32x16 (&s)[4], const lds_u8* __restrict__ kfeat, int krow,
                                                int half, int qw, int t_lo, int t_hi) {
  const int qx = qw & 0xFFFF, qy = qw >> 16;
  const int sq = qx * qx + qy * qy;
  const int a_lo = min(t_lo, 1 << 22) - sq, a_hi = min(t_hi, 1 << 22) - sq;
  const f16x4 qa = {(_Float16)(half ? 2048 : a_lo >> 11), (_Float16)(half ? 1 : a_lo & 2047),
                    (_Float16)(half ? 2 * qx : a_hi >> 11), (_Float16)(half ? 2 * qy : a_hi & 2047)};
  const uint32_t neg = __float_as_uint(-1.0e30f);
  f32x16 zero;
#pragma unroll
  for (int e = 0; e < 16; ++e) zero[e] = 0.f;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const uint32_t off = half * (kBK * 8) + (32 * kt + krow) * 8;  // [half][key][4] f16
    const f16x4 ka = __builtin_bit_cast(f16x4, *(const __attribute__((address_space(3))) uint2*)(kfeat + off));
    const f32x16 e = __builtin_amdgcn_mfma_f32_32x32x8f16(ka, qa, zero, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 16; ++i) s[kt][i] = e[i] >= 0.f ? s[kt][i] : __uint_as_float(neg);
  }
}

// Row queue of the persistent attention kernels (thread 0 of a workgroup only).  Without a
// caller order the rows are split into 8 contiguous ranges, one per XCD (the
// workgroup with index b runs on XCD b mod 8), each drained through its own
// counter: the rows an XCD has in flight are neighbouring query blocks of one
// head, which share most key tiles in its L2.  A workgroup whose range is
// drained takes rows from the next ranges in turn, so an XCD that runs at a
// higher clock ends up doing more rows.  With a caller order, one counter walks
// it (entries outside [0, rows) are skipped).  Returns -1 once all is drained.
// ctr: kRowCounters ints, zero before the launch; counter x at ctr[16 x].
__device__ __forceinline__ int next_row(int32_t* ctr, const int32_t* __restrict__ order, int rows, int xcd,
                                            int& steal) {
  if (order) {
    for (;;) {
      const int k = atomicAdd(&ctr[0], 1);
      if (k >= rows) return -1;
      const int r = order[k];
      if (r >= 0 && r < rows) return r;
    }
  }
  const int per = rows / 8, rem = rows % 8;
  while (steal < 8) {
    const int qd = (xcd + steal) & 7;
    const int beg = qd * per + min(qd, rem), n = per + (qd < rem ? 1 : 0);
    const int k = atomicAdd(&ctr[qd * 16], 1);
    if (k < n) return beg + k;
    ++steal;
  }
  return -1;
}

// Zeroes the row-queue counters (a kernel rather than a memset, so that the
// launch sequence also replays correctly inside a captured graph).
__global__ void reset_row_counters(int32_t* ctr) {
  if (threadIdx.x < kRowCounters) ctr[threadIdx.x] = 0;
}


// ------------------------------------------------------------ softmax and copy helpers
// Row max of a score tile as a max3 tree (short dependency chains), folded into
// the running state like tile_max.
template <bool ENT>
__device__ __forceinline__ float tile_max_tree(const f32x16 (&s)[4], float scale_log2, RowState& st) {
  float m4[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const float a = fmaxf(fmaxf(s[kt][0], s[kt][1]), s[kt][2]);
    const float b = fmaxf(fmaxf(s[kt][3], s[kt][4]), s[kt][5]);
    const float c = fmaxf(fmaxf(s[kt][6], s[kt][7]), s[kt][8]);
    const float d = fmaxf(fmaxf(s[kt][9], s[kt][10]), s[kt][11]);
    const float e = fmaxf(fmaxf(s[kt][12], s[kt][13]), s[kt][14]);
    m4[kt] = fmaxf(fmaxf(fmaxf(a, b), fmaxf(c, d)), fmaxf(e, s[kt][15]));
  }
  float mx = fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]));
  mx = max_halves(mx);
  const float m_new = next_reference(st.m, mx * scale_log2);
  const float sc = __builtin_amdgcn_exp2f(st.m - m_new);
  if (ENT) st.a = st.l > 0.f ? sc * (st.a + st.l * (st.m - m_new)) : 0.f;
  st.l *= sc;
  st.lr *= sc;
  st.m = m_new;
  return sc;
}

// dma16 pinned between two steps of a computation: it is issued after `after`
// has been computed and before `before` is next used (both pass through the
// statement untouched), so the compiler keeps it at that point of the
// instruction stream instead of hoisting it next to the other copies.
template <int LDS_STEP>
__device__ __forceinline__ void dma16_between(const void* sbase, uint32_t voff, uint32_t lds_base, float after,
                                              float& before) {
  asm volatile("s_add_u32 m0, %3, %4\n\tglobal_load_lds_dwordx4 %1, %2"
               : "+v"(before)
               : "v"(voff), "s"(sbase), "s"(lds_base), "i"(LDS_STEP), "v"(after)
               : "memory", "m0", "scc");
}

// Copy steps [J, JEND) of a tile (4 KB each), pinned after `after` and before
// `before` is next used.
template <int J, int JEND>
__device__ __forceinline__ void copies_after(float after, float& before, uint32_t lds, const uint8_t* src,
                                             uint32_t off) {
  if constexpr (J < JEND) {
    dma16_between<J * 4096>(src + J * 4096, off, lds, after, before);
    copies_after<J + 1, JEND>(after, before, lds, src, off);
  }
}

// S^T = K Q^T for one tile with NC copy steps of `src` issued in between, one
// after every (QK_STEPS / NC)-th k-step, pinned by the LDS-read order.
template <int D, int NC>
__device__ __forceinline__ void qk_tile_copies(f32x16 (&s)[4], const lds_u8* __restrict__ kbuf, uint32_t kbase,
                                               const bf16x8 (&qf)[Geo<D>::QK_STEPS], uint32_t lds,
                                               const uint8_t* src, uint32_t off) {
  constexpr int KK = Geo<D>::QK_STEPS;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
  kbase = opaque(kbase);
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const uint32_t o = chunk_off(kbase, kk);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) qk_step<D>(s[kt], kbuf, o, qf, kt, kk);
    if constexpr (NC > 0) {
      if (kk % (KK / NC) == KK / NC - 1) {
        switch (kk / (KK / NC)) {
          case 0: dma16<0 * 4096>(src + 0 * 4096, off, lds); break;
          case 1: dma16<1 * 4096>(src + 1 * 4096, off, lds); break;
          case 2: dma16<2 * 4096>(src + 2 * 4096, off, lds); break;
          case 3: dma16<3 * 4096>(src + 3 * 4096, off, lds); break;
          case 4: dma16<4 * 4096>(src + 4 * 4096, off, lds); break;
          case 5: dma16<5 * 4096>(src + 5 * 4096, off, lds); break;
          case 6: dma16<6 * 4096>(src + 6 * 4096, off, lds); break;
          default: dma16<7 * 4096>(src + 7 * 4096, off, lds); break;
        }
      }
    }
  }
  sched_reads_ahead<4 * KK, 1, 4>();
}

// O^T += V^T P^T for one tile with NC copy steps of `src` issued in between,
// one after every (8 / NC)-th k-step, pinned by the LDS-read order (a copy
// statement is a memory barrier for the compiler).
template <int D, int NC>
__device__ __forceinline__ void pv_tile_copies(f32x16 (&oacc)[Geo<D>::D_TILES], const lds_u8* __restrict__ vbuf,
                                               uint32_t vbase, const uint32_t (&pb)[32], uint32_t lds,
                                               const uint8_t* src, uint32_t off) {
  const uint32_t vb0 = opaque(vbase);
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    const uint32_t o = chunk_off(vb0, ks);
#pragma unroll
    for (int dt = 0; dt < Geo<D>::D_TILES; ++dt) pv_step<D>(oacc[dt], vbuf, o, pb, ks, dt);
    if constexpr (NC > 0) {
      if (ks % (8 / NC) == 8 / NC - 1) {
        switch (ks / (8 / NC)) {
          case 0: dma16<0 * 4096>(src + 0 * 4096, off, lds); break;
          case 1: dma16<1 * 4096>(src + 1 * 4096, off, lds); break;
          case 2: dma16<2 * 4096>(src + 2 * 4096, off, lds); break;
          case 3: dma16<3 * 4096>(src + 3 * 4096, off, lds); break;
          case 4: dma16<4 * 4096>(src + 4 * 4096, off, lds); break;
          case 5: dma16<5 * 4096>(src + 5 * 4096, off, lds); break;
          case 6: dma16<6 * 4096>(src + 6 * 4096, off, lds); break;
          default: dma16<7 * 4096>(src + 7 * 4096, off, lds); break;
        }
      }
    }
  }
  sched_reads_ahead<8 * Geo<D>::D_TILES, 1, 4>();
}

// Weights of score pairs [P, PEND) of a tile (pair P = 8 kt + e / 2):
// w = 2^(s alpha log2e - m) into the bf16 pairs pb[P], w summed into lp[kt]
// (and w x into ap[kt]), four independent chains.  NC tile-copy steps of
// `src` (4 KB each) are issued in between, spread evenly over the pairs and
// pinned there by data dependences: a burst of the four waves' copies would
// stall each wave on the memory queue, spread out they drain while the
// exponentials run.  C counts the copy steps issued so far.
template <int D, bool PV, bool ENT, int P0, int PEND, int NC, int P = P0>
__device__ __forceinline__ void exp_pairs(f32x16 (&s)[4], float c, float m, float (&lp)[4], float (&ap)[4],
                                          float (&lr)[4], uint32_t* pb, uint32_t lds, const uint8_t* src,
                                          uint32_t off) {
  if constexpr (P < PEND) {
    constexpr int kt = P / 8, e = (P % 8) * 2;
    const float x0 = fmaf(s[kt][e], c, -m);
    const float x1 = fmaf(s[kt][e + 1], c, -m);
    const float w0 = __builtin_amdgcn_exp2f(x0);
    const float w1 = __builtin_amdgcn_exp2f(x1);
    lp[kt] += w0 + w1;
    if (ENT) ap[kt] = fmaf(w0, x0, fmaf(w1, x1, ap[kt]));
    if (PV) {
      pb[P] = pack_bf16x2(w0, w1);
      lr[kt] = add_bf16_pair(pb[P], lr[kt]);
    }
    // copies [C, C_NEXT) follow this pair: ceil(NC (pairs done) / pairs in range)
    constexpr int C = ((P - P0) * NC + (PEND - P0) - 1) / (PEND - P0);
    constexpr int C_NEXT = ((P + 1 - P0) * NC + (PEND - P0) - 1) / (PEND - P0);
    if constexpr (C_NEXT > C) {
      if constexpr (P + 1 < 32) {
        constexpr int kt2 = (P + 1) / 8, e2 = ((P + 1) % 8) * 2;
        float nxt = s[kt2][e2];
        copies_after<C, C_NEXT>(w0, nxt, lds, src, off);
        s[kt2][e2] = nxt;
      } else {
        float nxt = lp[kt];
        copies_after<C, C_NEXT>(w0, nxt, lds, src, off);
        lp[kt] = nxt;
      }
    }
    exp_pairs<D, PV, ENT, P0, PEND, NC, P + 1>(s, c, m, lp, ap, lr, pb, lds, src, off);
  }
}

// One query-block row r of the 128-key-tile kernel.  LDS: smemK / smemV the K
// and V^T tiles, smemKinfo (token variant) the key words of the current and
// the next tile (a 1 KB copy each, of which the first 512 B are the tile's),
// smemCols the row's key-block list (NB entries for the sparse variant), read
// once so that the tile loop issues no global loads of its own (a wait for one
// would also drain the tiles in flight); the token variant then keeps each
// query's thresholds by frame distance after it, [128][F] uint16.
template <int D, bool SPARSE, bool PV, bool ENT, int TOK>
__device__ __forceinline__ void bf16_row(
    int r, uint8_t* smemK, uint8_t* smemV, uint8_t* smemKinfo, int32_t* smemCols,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile,
    const uint16_t* __restrict__ vtile, uint16_t* __restrict__ o, float* __restrict__ lse,
    float* __restrict__ entropy, const int32_t* __restrict__ perm, const int32_t* __restrict__ cnt,
    const int32_t* __restrict__ cols, int N, int n_pad, int NB, float scale_log2, const TokArgs& tk) {
  using G = Geo<D>;
  uint16_t* thrq = (uint16_t*)(smemCols + ((NB + 3) & ~3));
  const int bh = r / NB, u = r - bh * NB;
  // (opaque: the lane arithmetic below is redone per row instead of being
  // hoisted out of the persistent row loop, where it would stay live and spill)
  const int t = (int)opaque(threadIdx.x), lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int col = lane & 31, half = lane >> 5;
  const size_t head_off = (size_t)bh * N * D;
  constexpr size_t kTileBytes = (size_t)kBK * D * 2;
  const uint8_t* Kb = (const uint8_t*)(ktile + (size_t)bh * n_pad * D);
  const uint8_t* Vb = (const uint8_t*)(vtile + (size_t)bh * n_pad * D);  // V^T tiles of this head
  const uint32_t k_lds = (uint32_t)(uintptr_t)smemK + wave * 1024;
  const uint32_t v_lds = (uint32_t)(uintptr_t)smemV + wave * 1024;
  const uint32_t k_off = k_lane_off<D>(wave, lane);
  const uint32_t v_off = vt_lane_off(wave, lane);

  const int qpos = u * kBQ + wave * 32 + col;
  const int qtok = perm[qpos];  // -1 at a padding position
  const bool qvalid = qtok >= 0;
  const int qrow = qvalid ? qtok : 0;
  bf16x8 qf[G::QK_STEPS];
  {
    const uint4* src = (const uint4*)(q + head_off + (size_t)qrow * D);
#pragma unroll
    for (int kk = 0; kk < G::QK_STEPS; ++kk) {
      uint4 x = qvalid ? src[2 * kk + half] : make_uint4(0, 0, 0, 0);
      qf[kk] = __builtin_bit_cast(bf16x8, x);
    }
  }
  const int count = SPARSE ? min(max(cnt[r], 0), NB) : NB;
  if constexpr (SPARSE) {
    const int32_t* colp = cols + (size_t)r * NB;
    for (int j = t; j < count; j += kThreads) smemCols[j] = colp[j];
  }
  // token variant: this lane's query as a distance word and frame; a text
  // query or a full radius covers every key (thresholds then INT_MAX)
  [[maybe_unused]] int tq_word = 0, tq_f = 0;
  [[maybe_unused]] bool tq_all = true;
  const int qi = wave * 32 + col;
  if constexpr (TOK != 0) {
    if (qvalid && qrow < tk.Nv) {
      int n = tk.radius_sq[(size_t)bh * N + qrow];
      tq_all = n > tk.n_cap;
      n = max(n, 0);
      const int32_t c = tk.coord[qpos];
      tq_f = coord_f(c);
      tq_word = (TOK & 3) == 2 ? qrow : (coord_x(c) | (coord_y(c) << 16));
      if (!tq_all)
        for (int d = half; d < tk.F; d += 2) thrq[qi * tk.F + d] = (uint16_t)tk.thr[(size_t)n * tk.F + d];
    }
  }
  // retire the Q and list loads before any tile load is in flight, so that no
  // compiler wait for them lands inside the tile loop (it would also drain the
  // tiles), and publish the list
  wait_vm<0>();
  lds_barrier();
  // QK^T operand rows: lane (row m = lane % 32) loads key row krow(m)
  // of each 32-key sub-tile, chosen so that lane half h ends up holding the 8
  // consecutive keys 8h..8h+7 (and 16+8h..) of the sub-tile: output row
  // R = 8(e/4) + 4h + e%4 must be key 16(e/8) + 8h + e%8, i.e. rows 4..7 and
  // 8..11 of every 16 swap places.
  const int krow = (col & ~15) | ((col & 15) ^ (((col >> 2) & 3) == 1 || ((col >> 2) & 3) == 2 ? 12 : 0));
  const uint32_t kbase = krow * D * 2 + ((half ^ swz<G::CH>(krow)) << 4);
  // V^T operand: row d = 32dt + (lane % 32) (dt as an immediate), chunk 2ks + h
  const uint32_t vbase = col * kBK * 2 + ((half ^ swz<16>(col)) << 4);

  // Next list position at or after i holding a valid key block, or count;
  // entries outside [0, NB) are skipped.  *b receives the block id.
  auto next_valid = [&](int i, int* b) -> int {
    if (!SPARSE) {
      *b = i;
      return i;
    }
    for (; i < count; ++i) {
      const int c = smemCols[i];
      if (c >= 0 && c < NB) {
        *b = c;
        return i;
      }
    }
    *b = 0;
    return count;
  };

  f32x16 oacc[PV ? G::D_TILES : 1];
#pragma unroll
  for (int i = 0; i < (PV ? G::D_TILES : 1); ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[i][e] = 0.f;
  RowState st{-INFINITY, 0.f, 0.f, 0.f};

  // token variant: wave 0 copies each tile's key info (1 KB) right after its
  // K steps, into the buffer of the tile's parity, so "K landed" covers it
  [[maybe_unused]] const uint32_t kinfo_lds = (uint32_t)(uintptr_t)smemKinfo;
  // per tile: 2-D the key vectors (2 KB, two copies), 1-D the key words (one 1 KB copy)
  constexpr int kKeyBufBytes = (TOK & 3) == 1 ? kBK * kKeyFeat * 2 : 1024;
  constexpr int kKeyCopies = (TOK & 3) == 1 ? 2 : 1;
  auto issue_kinfo = [&](int b, int parity) {
    if constexpr ((TOK & 3) == 1) {  // 2-D: the block's 128 key vectors, 2 KB
      if (wave == 0) {
        const uint8_t* src = (const uint8_t*)(tk.kfeat + (size_t)b * kBK * kKeyFeat);
        dma16<0>(src, lane * 16, kinfo_lds + parity * kKeyBufBytes);
        dma16<1024>(src + 1024, lane * 16, kinfo_lds + parity * kKeyBufBytes);
      }
    } else if constexpr (TOK != 0) {
      if (wave == 0) dma16<0>((const uint8_t*)(tk.kinfo + (size_t)b * kKeyInfo), lane * 16, kinfo_lds + parity * kKeyBufBytes);
    }
  };
  int b_cur;
  int i = next_valid(0, &b_cur);
  int parity = 0;
  bool fresh = true;  // no tile of the row done by this wave yet
  if (i < count) {
    b_cur = __builtin_amdgcn_readfirstlane(b_cur);
    issue_tile<D>(k_lds, Kb + b_cur * kTileBytes, k_off);
    issue_kinfo(b_cur, 0);
    if (PV) issue_tile<D>(v_lds, Vb + b_cur * kTileBytes, v_off);
    for (;;) {
      int b_nxt;
      const int i_nxt = next_valid(i + 1, &b_nxt);
      const bool has_next = i_nxt < count;
      b_nxt = __builtin_amdgcn_readfirstlane(b_nxt);
      wait_vm<PV ? TileCopy<D>::STEPS : 0>();  // K_i landed (V_i may still be in flight)
      lds_barrier();
      // token variant: classify this lane's query against the block's box
      // ("none": no key of the block covered; "all": every video key covered)
      // with its thresholds for the block's nearest and farthest frames; a
      // wave none of whose queries covers a key skips the tile's matrix work,
      // a wave all of whose queries cover every key skips the key test
      bool wave_skip = false, wave_test = false;
      int t_lo = INT_MAX, t_hi = INT_MAX;
      int n_keys = N - b_cur * kBK;  // keys of the block holding a token (its first n_keys)
      if constexpr (TOK != 0) {
        const int32_t* bi = tk.binfo + (size_t)b_cur * kBlockInfo;
        const int fmin = bi[0], fmax = bi[1], n_video = bi[6], n_text = bi[9];
        n_keys = n_video + n_text;
        bool none = !qvalid, all = true;
        if (qvalid && n_video > 0 && !tq_all) {
          t_lo = thrq[qi * tk.F + abs(tq_f - fmin)];
          t_hi = thrq[qi * tk.F + abs(tq_f - fmax)];
          int dmin, dmax;
          if constexpr ((TOK & 3) == 2) {
            const int rmin = bi[7], rmax = bi[8];
            dmin = max(0, max(rmin - tq_word, tq_word - rmax));
            dmax = max(tq_word - rmin, rmax - tq_word);
          } else {
            const int qx = tq_word & 0xFFFF, qy = tq_word >> 16;
            const int dxn = max(0, max(bi[2] - qx, qx - bi[3])), dyn = max(0, max(bi[4] - qy, qy - bi[5]));
            const int dxf = max(qx - bi[2], bi[3] - qx), dyf = max(qy - bi[4], bi[5] - qy);
            dmin = dxn * dxn + dyn * dyn;
            dmax = dxf * dxf + dyf * dyf;
          }
          none = n_text == 0 && dmin > max(t_lo, t_hi);
          all = dmax <= min(t_lo, t_hi);
        }
        wave_skip = __ballot(!none) == 0;
        wave_test = __ballot(!all) != 0;
      }
      f32x16 s[4];
      if (!wave_skip) qk_tile<D>(s, (const lds_u8*)smemK, kbase, qf);
      lds_barrier();  // every wave is done with K_i
      if (has_next) {
        issue_tile<D>(k_lds, Kb + b_nxt * kTileBytes, k_off);
        issue_kinfo(b_nxt, parity ^ 1);
      }
      float sc = 1.f;
      uint32_t pb[32];
      if (!wave_skip) {
        if constexpr (TOK != 0) {
          if (wave_test) {
            const lds_u8* ki = (const lds_u8*)smemKinfo + parity * kKeyBufBytes;
            if constexpr ((TOK & 3) == 1) token_mask_mfma(s, ki, krow, half, tq_word, t_lo, t_hi);
            else token_mask<TOK>(s, ki, half, tq_word, t_lo, t_hi);
          }
        }
        if (n_keys < kBK) mask_tail(s, n_keys, half);
        float lsum = 0.f, asum = 0.f, lrsum = 0.f;
        bool exact = fresh;
        // (the rounded weights' four sum chains run over all four sub-tiles)
        if (!exact) {  // weights against the current reference (kFastSum)
          float lr4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) tile_exp_acc<PV, ENT>(s[kt], scale_log2, st.m, lsum, asum, lr4, pb + 8 * kt);
          if (PV) lrsum = (lr4[0] + lr4[1]) + (lr4[2] + lr4[3]);
          exact = __ballot(!((PV ? lrsum : lsum) <= kFastSum)) != 0;
        }
        if (exact) {  // the wave's first tile, or a weight past 2^20: from the tile max
          sc = tile_max<ENT>(s, scale_log2, st);
          lsum = asum = 0.f;
          float lr4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) tile_exp_acc<PV, ENT>(s[kt], scale_log2, st.m, lsum, asum, lr4, pb + 8 * kt);
          if (PV) lrsum = (lr4[0] + lr4[1]) + (lr4[2] + lr4[3]);
        }
        fresh = false;
        st.l += lsum;
        if (PV) st.lr += lrsum;
        if (ENT) st.a += asum;
      }
      if constexpr (PV) {
        // V_i landed (K_{i+1} -- and for wave 0 of the token variant its key
        // info -- may still be in flight)
        if (has_next && TOK != 0 && wave == 0) wait_vm<TileCopy<D>::STEPS + kKeyCopies>();
        else if (has_next) wait_vm<TileCopy<D>::STEPS>();
        else wait_vm<0>();
        lds_barrier();
        if (!wave_skip) {
          if (__ballot(sc != 1.0f) != 0) {
#pragma unroll
            for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
              for (int e = 0; e < 16; ++e) oacc[dt][e] *= sc;
          }
          const uint32_t vb0 = opaque(vbase);
#pragma unroll
          for (int ks = 0; ks < 8; ++ks) {
            const uint32_t off = chunk_off(vb0, ks);
#pragma unroll
            for (int dt = 0; dt < G::D_TILES; ++dt) pv_step<D>(oacc[dt], (const lds_u8*)smemV, off, pb, ks, dt);
          }
          sched_reads_ahead<8 * G::D_TILES, 1, 4>();
        }
        lds_barrier();  // every wave is done with V_i
        if (has_next) issue_tile<D>(v_lds, Vb + b_nxt * kTileBytes, v_off);
      }
      if (!has_next) break;
      i = i_nxt;
      b_cur = b_nxt;
      parity ^= 1;
    }
  }

  const float l_tot = sum_halves(st.l);
  const float a_tot = ENT ? sum_halves(st.a) : 0.f;
  const float lr_tot = PV ? sum_halves(st.lr) : 0.f;
  if (!qvalid) return;
  const size_t tok = (size_t)bh * N + qrow;
  if (PV) {
    const float inv = lr_tot > 0.f ? 1.f / lr_tot : 0.f;
    uint16_t* dst = o + tok * D;
#pragma unroll
    for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = dt * 32 + 8 * g + 4 * half;
        uint2 w;
        w.x = pack_bf16x2(oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv);
        w.y = pack_bf16x2(oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv);
        *(uint2*)(dst + d0) = w;
      }
  }
  if (half == 0) {
    if (ENT) entropy[tok] = 0.69314718055994531f * (__log2f(l_tot) - a_tot / l_tot);
    if (lse) lse[tok] = l_tot > 0.f ? 0.69314718055994531f * (st.m + __log2f(l_tot)) : -INFINITY;
  }
}

// TOK (sparse only): 0 block granular; 1 token mask with the 2-D distance,
// 2 with the 1-D sequence distance (Eq. 15 inside the listed blocks); + 4 when
// the plan has text tokens (text keys stay visible).
// Persistent: as many workgroups as can be resident, each taking rows from the
// row queue until it is drained (the first barrier of every row, after its list
// is staged, orders the next s_row write after every wave's read).
template <int D, bool SPARSE, bool PV, bool ENT, int OCC, int TOK = 0>
__global__ __launch_bounds__(kThreads, OCC) void attn_bf16_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile,
    const uint16_t* __restrict__ vtile, uint16_t* __restrict__ o, float* __restrict__ lse,
    float* __restrict__ entropy, const int32_t* __restrict__ perm, const int32_t* __restrict__ cnt,
    const int32_t* __restrict__ cols, const int32_t* __restrict__ order, int N, int n_pad, int NB,
    int rows, float scale_log2, TokArgs tk, int32_t* __restrict__ ctr) {
  constexpr int TILE = kBK * D * 2;
  __shared__ __attribute__((aligned(1024))) uint8_t smemK[TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t smemV[PV ? TILE : 16];
  __shared__ __attribute__((aligned(16))) uint8_t smemKinfo[(TOK & 3) == 1 ? 2 * kBK * kKeyFeat * 2 : TOK ? 2 * 1024 : 16];
  extern __shared__ int32_t smemCols[];
  __shared__ int s_row, s_steal;  // thread 0's queue state lives in LDS, not in a register
  if (threadIdx.x == 0) s_steal = 0;
  for (;;) {
    if (threadIdx.x == 0) {
      int steal = s_steal;
      s_row = next_row(ctr, SPARSE ? order : nullptr, rows, blockIdx.x & 7, steal);
      s_steal = steal;
    }
    __syncthreads();
    const int r = s_row;
    if (r < 0) break;
    bf16_row<D, SPARSE, PV, ENT, TOK>(r, smemK, smemV, smemKinfo, smemCols, q, ktile, vtile, o, lse, entropy,
                                      perm, cnt, cols, N, n_pad, NB, scale_log2, tk);
  }
}

// ------------------------------------------------------------ 64-key tiles
// Dense / block-sparse attention with each 128-key block taken as two 64-key
// tiles: per wave 32 scores and 16 probability pairs in flight instead of 64
// and 32, and 32 KB of LDS per workgroup, so three workgroups (three waves per
// SIMD) share a CU.  The V^T half-tile rows are 128 bytes, strided by the
// block's 256-byte rows in HBM; their 16-byte chunks are XOR-swizzled so that
// the PV operand reads hit every bank once.
constexpr int kKT = 64;  // keys per tile

// Lane offset within a 4 KB step of a V^T half-tile: row wave * 8 + lane / 8
// of the step (32 rows of 64 keys), physical chunk lane % 8, which holds logical
// chunk (lane % 8) ^ swz<8>(row); rows are 256 bytes apart in HBM.
__device__ __forceinline__ uint32_t vt64_lane_off(int wave, int lane) {
  const int row = wave * 8 + lane / 8;
  return row * 256 + (((lane % 8) ^ swz<8>(row)) << 4);
}

template <int N, int SRC_STEP>
__device__ __forceinline__ void issue_steps_strided(uint32_t lds_wave, const uint8_t* tile, uint32_t lane_off) {
  if constexpr (N > 0) {
    issue_steps_strided<N - 1, SRC_STEP>(lds_wave, tile, lane_off);
    dma16<(N - 1) * 4096>(tile + (N - 1) * SRC_STEP, lane_off, lds_wave);
  }
}

// One work unit of a row: list positions [beg, end) of row r (the whole row
// for dense).  slot < 0: the unit is the whole row and writes the normalised
// output (and lse).  slot >= 0: one piece of a split row; it writes its
// unnormalised output, running max and sums to partial slot `slot` for the
// merge kernel.  LSE: also keep the fp32 sum of the weights for the
// log-sum-exp output.
template <int D, bool SPARSE, bool LSE>
__device__ __forceinline__ void k64_row(
    int r, int beg, int end, int slot, uint8_t* smemK, uint8_t* smemV, int32_t* smemCols,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile, const uint16_t* __restrict__ vtile,
    uint16_t* __restrict__ o, float* __restrict__ lse, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ cols, const int32_t* __restrict__ bcount, int N, int n_pad, int NB,
    float scale_log2, float* __restrict__ part, float* __restrict__ pstats) {
  using G = Geo<D>;
  constexpr int KT_BYTES = kKT * D * 2;            // one 64-key tile of K or V^T
  constexpr int STEPS = KT_BYTES / 4096;           // 4 KB copy steps per tile
  const int bh = r / NB, u = r - bh * NB;
  // (opaque: the lane arithmetic below is redone per row instead of being
  // hoisted out of the persistent row loop, where it would stay live and spill)
  const int t = (int)opaque(threadIdx.x), lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int col = lane & 31, half = lane >> 5;
  const size_t head_off = (size_t)bh * N * D;
  constexpr size_t kBlockBytes = (size_t)kBK * D * 2;
  const uint8_t* Kb = (const uint8_t*)(ktile + (size_t)bh * n_pad * D);
  const uint8_t* Vb = (const uint8_t*)(vtile + (size_t)bh * n_pad * D);
  const uint32_t k_lds = (uint32_t)(uintptr_t)smemK + wave * 1024;
  const uint32_t v_lds = (uint32_t)(uintptr_t)smemV + wave * 1024;
  const uint32_t k_off = k_lane_off<D>(wave, lane);
  const uint32_t v_off = vt64_lane_off(wave, lane);

  const int qpos = u * kBQ + wave * 32 + col;
  const int qtok = perm[qpos];  // -1 at a padding position
  const bool qvalid = qtok >= 0;
  const int qrow = qvalid ? qtok : 0;
  bf16x8 qf[G::QK_STEPS];
  {
    const uint4* src = (const uint4*)(q + head_off + (size_t)qrow * D);
#pragma unroll
    for (int kk = 0; kk < G::QK_STEPS; ++kk) {
      uint4 x = qvalid ? src[2 * kk + half] : make_uint4(0, 0, 0, 0);
      qf[kk] = __builtin_bit_cast(bf16x8, x);
    }
  }
  const int count = SPARSE ? end - beg : NB;
  if constexpr (SPARSE) {
    // a valid entry is staged with its block's token count in the high half
    // (the tokens fill the block's first positions), an invalid one as -1
    const int32_t* colp = cols + (size_t)r * NB + beg;
    for (int j = t; j < count; j += kThreads) {
      const int c = colp[j];
      int e = -1;
      if (c >= 0 && c < NB) e = c | ((bcount ? bcount[c] : min(kBK, N - c * kBK)) << 16);
      smemCols[j] = e;
    }
  }
  wait_vm<0>();
  lds_barrier();
  const int krow = (col & ~15) | ((col & 15) ^ (((col >> 2) & 3) == 1 || ((col >> 2) & 3) == 2 ? 12 : 0));
  const uint32_t kbase = krow * D * 2 + ((half ^ swz<G::CH>(krow)) << 4);
  // V^T operand: row d = 32 dt + (lane % 32) of the half-tile (128-byte rows), chunk 2 ks + h
  const uint32_t vbase = col * kKT * 2 + ((half ^ swz<8>(col)) << 4);

  // Tile i of the row: block list[i / 2], keys [64 (i % 2), +64) of it; a
  // list entry outside [0, NB) and a half holding no token are skipped.
  // Returns the tile as (2 block + half) | (its keys holding a token) << 16,
  // or -1 past the end.
  auto next_valid = [&](int i, int* pos) -> int {
    for (; i < 2 * count; ++i) {
      int c, n;
      if constexpr (SPARSE) {
        const int e = smemCols[i >> 1];
        c = e & 0xFFFF;
        n = e >> 16;  // -1 for an invalid entry
      } else {
        c = i >> 1;
        n = min(kBK, N - c * kBK);
      }
      const int nv = n - (i & 1) * kKT;
      if (nv > 0) {
        *pos = i;
        return __builtin_amdgcn_readfirstlane((2 * c + (i & 1)) | (min(nv, kKT) << 16));
      }
    }
    *pos = 2 * count;
    return -1;
  };
  auto k_src = [&](int bt) {
    bt &= 0xFFFF;
    return Kb + (bt >> 1) * kBlockBytes + (bt & 1) * KT_BYTES;
  };
  auto v_src = [&](int bt) {
    bt &= 0xFFFF;
    return Vb + (bt >> 1) * kBlockBytes + (bt & 1) * (kKT * 2);
  };
  auto issue_k = [&](int bt) { issue_steps<STEPS>(k_lds, k_src(bt), k_off); };
  auto issue_v = [&](int bt) { issue_steps_strided<STEPS, 32 * 256>(v_lds, v_src(bt), v_off); };

  f32x16 oacc[G::D_TILES];
#pragma unroll
  for (int i = 0; i < G::D_TILES; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[i][e] = 0.f;
  RowState st{-INFINITY, 0.f, 0.f, 0.f};

  int pos;
  int bt_cur = next_valid(0, &pos);
  int bt_nxt = bt_cur >= 0 ? next_valid(pos + 1, &pos) : -1;
  if (bt_cur >= 0) {
    issue_k(bt_cur);
    issue_v(bt_cur);
    for (;;) {
      const bool has_next = bt_nxt >= 0;
      wait_vm<STEPS>();  // K tile landed (V^T may still be in flight)
      lds_barrier();
      f32x16 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
      {
        const uint32_t kb = opaque(kbase);
        const lds_u8* kbuf = (const lds_u8*)smemK;
#pragma unroll
        for (int kk = 0; kk < G::QK_STEPS; ++kk) {
          const uint32_t off = chunk_off(kb, kk);
#pragma unroll
          for (int kt = 0; kt < 2; ++kt) qk_step<D>(s[kt], kbuf, off, qf, kt, kk);
        }
        sched_reads_ahead<2 * G::QK_STEPS, 1, 4>();
      }
      lds_barrier();  // every wave is done with the K tile
      if (has_next) issue_k(bt_nxt);
      const int nv = bt_cur >> 16;  // keys of this tile holding a token (the first nv, > 0)
      if (nv < kKT) {
        const int base = 8 * half - nv;
        const uint32_t neg = __float_as_uint(-1.0e30f);
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const uint32_t keep = (uint32_t)((kt * 32 + 16 * (e >> 3) + (e & 7) + base) >> 31);
            s[kt][e] = __uint_as_float(((__float_as_uint(s[kt][e]) & keep) | (neg & ~keep)));
          }
      }
      // (the tile max is always formed here: skipping it as the 128-key
      // kernel does keeps the score tile live through the exponentials, and at
      // this kernel's 168 registers the compiler then keeps one LDS read in
      // flight instead of four -- 2-8 % slower)
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
      mx = max_halves(mx);
      const float m_new = next_reference(st.m, mx * scale_log2);
      const float sc = __builtin_amdgcn_exp2f(st.m - m_new);
      if (LSE) st.l *= sc;
      st.lr *= sc;
      st.m = m_new;
      uint32_t pb[16];
      float lsum = 0.f, asum = 0.f;
      // the rounded weights' four sum chains run over both sub-tiles, the
      // first one seeded with the running sum
      float lr4[4] = {st.lr, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
        tile_exp_acc<true, false, LSE>(s[kt], scale_log2, st.m, lsum, asum, lr4, pb + 8 * kt);
      if (LSE) st.l += lsum;
      st.lr = (lr4[0] + lr4[1]) + (lr4[2] + lr4[3]);
      if (has_next) wait_vm<STEPS>();  // V^T landed (the next K tile may still be in flight)
      else wait_vm<0>();
      lds_barrier();
      if (__ballot(sc != 1.0f) != 0) {
#pragma unroll
        for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[dt][e] *= sc;
      }
      {
        const uint32_t vb0 = opaque(vbase);
        const lds_u8* vbuf = (const lds_u8*)smemV;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const uint32_t off = chunk_off(vb0, ks);
          const int kt = ks >> 1, eb = (ks & 1) * 4;
          const uint4 bw = make_uint4(pb[kt * 8 + eb], pb[kt * 8 + eb + 1], pb[kt * 8 + eb + 2], pb[kt * 8 + eb + 3]);
#pragma unroll
          for (int dt = 0; dt < G::D_TILES; ++dt) {
            const bf16x8 va = lds_read16(vbuf, off + dt * 32 * kKT * 2);
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, __builtin_bit_cast(bf16x8, bw), oacc[dt], 0, 0, 0);
          }
        }
        sched_reads_ahead<4 * G::D_TILES, 1, 4>();
      }
      lds_barrier();  // every wave is done with the V^T tile
      if (has_next) issue_v(bt_nxt);
      if (!has_next) break;
      bt_cur = bt_nxt;
      bt_nxt = next_valid(pos + 1, &pos);
    }
  }

  const float lr_tot = sum_halves(st.lr);
  const float l_tot = LSE ? sum_halves(st.l) : 0.f;
  if (SPARSE && slot >= 0) {
    // a piece of a split row: O relative to 2^m, unnormalised, [slot][query][D]
    const int qi = wave * 32 + col;
    float* po = part + ((size_t)slot * kBQ + qi) * D;
#pragma unroll
    for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *(float4*)(po + dt * 32 + 8 * g + 4 * half) =
            make_float4(oacc[dt][4 * g], oacc[dt][4 * g + 1], oacc[dt][4 * g + 2], oacc[dt][4 * g + 3]);
    if (half == 0) {
      float* ps = pstats + (size_t)slot * 3 * kBQ;
      ps[qi] = st.m;
      ps[kBQ + qi] = lr_tot;
      ps[2 * kBQ + qi] = l_tot;
    }
    return;
  }
  if (!qvalid) return;
  const size_t tok = (size_t)bh * N + qrow;
  const float inv = lr_tot > 0.f ? 1.f / lr_tot : 0.f;
  uint16_t* dst = o + tok * D;
#pragma unroll
  for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d0 = dt * 32 + 8 * g + 4 * half;
      uint2 w;
      w.x = pack_bf16x2(oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv);
      w.y = pack_bf16x2(oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv);
      *(uint2*)(dst + d0) = w;
    }
  if (LSE && half == 0) lse[tok] = l_tot > 0.f ? 0.69314718055994531f * (st.m + __log2f(l_tot)) : -INFINITY;
}

// Queue of work units (thread 0 of a workgroup only): with `single`, one
// counter walks the units in table order (the caller's row order); otherwise
// XCD x drains its segment [seg[x], seg[x + 1]) of the table, then takes units
// from the other segments in turn, as next_row.  Returns -1 once all is
// drained.
__device__ __forceinline__ int next_unit(int32_t* ctr, bool single, int n, const int32_t* __restrict__ seg, int xcd,
                                         int& steal) {
  if (single) {
    const int k = atomicAdd(&ctr[0], 1);
    return k < n ? k : -1;
  }
  while (steal < 8) {
    const int qd = (xcd + steal) & 7;
    const int beg = seg[qd], cnt = seg[qd + 1] - beg;
    const int k = atomicAdd(&ctr[qd * 16], 1);
    if (k < cnt) return beg + k;
    ++steal;
  }
  return -1;
}

// Persistent kernel: as many workgroups as fit on the GPU (three per CU), each
// taking work from a queue until it is drained: rows (dense), or the units of
// the work-unit table (block-sparse; see plan_units_kernel).  Every unit starts
// with a workgroup barrier (after its block list is staged), which also orders
// the next s_row write after every wave's read of the current one.
template <int D, bool SPARSE, bool LSE>
__global__ __launch_bounds__(kThreads, 3) void attn_k64_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile, const uint16_t* __restrict__ vtile,
    uint16_t* __restrict__ o, float* __restrict__ lse, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ cols, const int32_t* __restrict__ bcount, const int4* __restrict__ units,
    const int32_t* __restrict__ unit_hdr, bool ordered, int N, int n_pad, int NB, int rows, float scale_log2,
    int32_t* __restrict__ ctr, float* __restrict__ part, float* __restrict__ pstats) {
  constexpr int KT_BYTES = kKT * D * 2;
  __shared__ __attribute__((aligned(1024))) uint8_t smemK[KT_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t smemV[KT_BYTES];
  extern __shared__ int32_t smemCols[];
  __shared__ int s_row, s_steal;  // thread 0's queue state lives in LDS, not in a register
  const int n_work = SPARSE ? unit_hdr[0] : rows;
  if (threadIdx.x == 0) s_steal = 0;
  for (;;) {
    if (threadIdx.x == 0) {
      int steal = s_steal;
      s_row = SPARSE ? next_unit(ctr, ordered, n_work, unit_hdr + 4, blockIdx.x & 7, steal)
                     : next_row(ctr, nullptr, rows, blockIdx.x & 7, steal);
      s_steal = steal;
    }
    __syncthreads();
    const int w = s_row;
    if (w < 0) break;
    if constexpr (SPARSE) {
      const int4 un = units[w];
      if (un.x < 0) {  // a placeholder unit (never written by a consistent plan): nothing to do
        __syncthreads();
        continue;
      }
      k64_row<D, true, LSE>(un.x, un.y, un.z, un.w, smemK, smemV, smemCols, q, ktile, vtile, o, lse, perm, cols,
                            bcount, N, n_pad, NB, scale_log2, part, pstats);
    } else {
      k64_row<D, false, LSE>(w, 0, NB, -1, smemK, smemV, smemCols, q, ktile, vtile, o, lse, perm, cols, bcount,
                             N, n_pad, NB, scale_log2, part, pstats);
    }
  }
}

// Work units of a block-sparse call (one workgroup of 1024 threads).  With T
// the total list length and G the attention grid, L = max(kSplitMin, ceil(T /
// (G kSplitPerWG))) (doubled while the pieces would exceed the workspace's
// partial slots, which its capacity, 2 G kSplitPerWG + 1 slots, rules out),
// and a row of c > L entries becomes ceil(c / L) units of near-equal
// length, each writing a partial slot, so that no unit holds more than about
// 1 / kSplitPerWG of a workgroup's share of the work and the rows the call
// waits on at its end are short, while short rows are never cut into pieces
// whose fixed costs (query load, partial write, merge) would dominate.  Rows of
// at most L entries are one unit each (and give the same result as an unsplit
// call).
//
// Unit order.  With the caller's row order, units follow it (a row's pieces
// consecutive) and one counter walks them.  Otherwise the rows are cut into
// eight contiguous segments, one per XCD queue (hdr[4 + x] .. hdr[5 + x]), and
// inside a segment the pieces of its split rows come first, piece-major (piece
// 0 of every split row, then piece 1, ...; a row with fewer pieces than the
// segment's most leaves placeholder units), then its other rows in row order.
// Long rows keep most of their lists alike (rows whose queries mostly have
// the full radius keep every block), so the split pieces a queue's workgroups
// run side by side walk the same key blocks, and the L2 serves them to all.
// The last 1 / kTailDiv of a segment's whole rows run longest first (bucketed
// by length, in no fixed order inside a bucket), so that the units its
// workgroups finish on are the short ones and few of them wait idle at the end
// of the call; the rows before them keep row order, whose neighbouring rows
// share key blocks.  A whole row's result does not depend on where it runs.
//
// Writes units[U] = {row, list begin, list end, slot or -1} (row -1: a
// placeholder), splits[P] = {row, first slot, pieces, 0} and hdr = {U, P, L,
// 0, segment starts x 9}, and zeroes the attention kernel's queue counters.  A split row has c / L < pieces < 2 c / L, so P <= T
// / L <= G kSplitPerWG; with the placeholders U <= rows + max(G kSplitPerWG,
// ceil(NB / kSplitMin) slots / 2): the call's workspace holds tables of these
// bounds (entries past a capacity are never written).
constexpr int kSplitPerWG = 16;
constexpr int kSplitMin = 48;
constexpr int kPlanStagedRows = 32768;  // rows whose lengths plan_units_kernel keeps in LDS (64 KB)
constexpr int kTailDiv = 8;              // the tail: the last eighth of a segment's whole rows
constexpr int kTailBins = 256;           // length buckets of the tail's order

// Length bucket of a whole row (0 <= c <= L) in the tail's order.
__device__ __forceinline__ int tail_bin(int c, int L) { return min(kTailBins - 1, c * kTailBins / (L + 1)); }

__global__ __launch_bounds__(1024) void plan_units_kernel(const int32_t* __restrict__ cnt,
                                                          const int32_t* __restrict__ order, int rows, int NB,
                                                          int n_wg, int4* __restrict__ units, int units_cap,
                                                          int4* __restrict__ splits, int splits_cap,
                                                          int slots_cap, int32_t* __restrict__ hdr,
                                                          int32_t* __restrict__ ctr) {
  __shared__ long long s_red[1024];
  __shared__ int s_scan[3][1024];
  __shared__ int s_seg[4][1024];  // per thread, segmented: split rows, other rows, max pieces
  __shared__ int s_base[9];
  __shared__ int s_tail[8][kTailBins];  // per segment: tail rows per length bucket, then their slots
  __shared__ uint16_t s_len[kPlanStagedRows];  // the row lengths, read once with coalesced loads
  const int t = threadIdx.x;
  if (t < kRowCounters) ctr[t] = 0;  // the attention kernel's queue counters, zeroed here for it
  const bool segmented = order == nullptr;
  // (each thread's walk below is a contiguous range of rows, which would read
  // the counts with one dependent-latency load per row in every pass)
  const bool staged = rows <= kPlanStagedRows;
  if (staged) {
#pragma unroll 8
    for (int r = t; r < rows; r += 1024) s_len[r] = (uint16_t)min(max(cnt[r], 0), NB);
    __syncthreads();
  }
  // this thread's positions [k0, k1) of the walk: in segment t / 128 for the
  // per-XCD queues, else 1/1024 of the caller's order
  int k0, k1;
  if (segmented) {
    const int x = t >> 7, ls = t & 127;
    const int r0 = (int)((long long)rows * x / 8), r1 = (int)((long long)rows * (x + 1) / 8);
    const int per = (r1 - r0 + 127) / 128;
    k0 = min(r1, r0 + ls * per);
    k1 = min(r1, k0 + per);
  } else {
    const int per = (rows + 1023) / 1024;
    k0 = min(rows, t * per);
    k1 = min(rows, k0 + per);
  }
  auto row_at = [&](int k) { return order ? order[k] : k; };
  auto len_of = [&](int r) {
    return (r >= 0 && r < rows) ? (staged ? (int)s_len[r] : min(max(cnt[r], 0), NB)) : -1;
  };
  long long tot = 0;
  for (int k = k0; k < k1; ++k) tot += max(len_of(row_at(k)), 0);
  s_red[t] = tot;
  __syncthreads();
  for (int st = 512; st > 0; st >>= 1) {
    if (t < st) s_red[t] += s_red[t + st];
    __syncthreads();
  }
  const long long total = s_red[0];
  const long long share = (long long)max(n_wg, 1) * kSplitPerWG;
  int L = (int)max((long long)kSplitMin, (total + share - 1) / share);
  // per thread: units, slots and split rows of its positions; L doubles until
  // the pieces of the split rows fit the partial slots
  int nu, ns, np, nw, pmx;
  for (;;) {
    nu = ns = np = nw = pmx = 0;
    for (int k = k0; k < k1; ++k) {
      const int c = len_of(row_at(k));
      if (c < 0) continue;
      const int pieces = c > L ? (c + L - 1) / L : 1;
      nu += pieces;
      if (pieces > 1) {
        ns += pieces;
        ++np;
        pmx = max(pmx, pieces);
      } else {
        ++nw;
      }
    }
    __syncthreads();
    s_red[t] = ns;
    __syncthreads();
    for (int st = 512; st > 0; st >>= 1) {
      if (t < st) s_red[t] += s_red[t + st];
      __syncthreads();
    }
    if (s_red[0] <= slots_cap || L >= NB) break;
    L = min(2 * L, NB);
  }
  s_scan[0][t] = nu;
  s_scan[1][t] = ns;
  s_scan[2][t] = np;
  s_seg[0][t] = np;
  s_seg[1][t] = nw;
  s_seg[2][t] = pmx;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {  // inclusive scans; s_seg within 128-thread segments
    int a0 = 0, a1 = 0, a2 = 0, g0 = 0, g1 = 0, g2 = 0;
    if (t >= off) {
      a0 = s_scan[0][t - off];
      a1 = s_scan[1][t - off];
      a2 = s_scan[2][t - off];
    }
    if ((t & 127) >= off) {
      g0 = s_seg[0][t - off];
      g1 = s_seg[1][t - off];
      g2 = s_seg[2][t - off];
    }
    __syncthreads();
    s_scan[0][t] += a0;
    s_scan[1][t] += a1;
    s_scan[2][t] += a2;
    s_seg[0][t] += g0;
    s_seg[1][t] += g1;
    s_seg[2][t] = max(s_seg[2][t], g2);
    __syncthreads();
  }
  // segment starts: segment x holds (its most pieces) x (its split rows)
  // piece-major units, then its other rows
  if (t == 0) {
    int b = 0;
    for (int x = 0; x < 8; ++x) {
      s_base[x] = b;
      const int last = x * 128 + 127;
      b += segmented ? s_seg[2][last] * s_seg[0][last] + s_seg[1][last] : 0;
    }
    s_base[8] = b;
  }
  __syncthreads();
  int sb = s_scan[1][t] - ns, pb = s_scan[2][t] - np;
  if (segmented) {
    const int x = t >> 7, last = x * 128 + 127;
    const int n_split = s_seg[0][last], p_most = s_seg[2][last];
    const int base = s_base[x];
    const int n_whole = s_seg[1][last];
    const int keep = n_whole - n_whole / kTailDiv;  // whole rows of rank >= keep form the tail
    // the tail's order: rows per length bucket, then each bucket's first slot
    // counted from the longest bucket down
    for (int i = t; i < 8 * kTailBins; i += 1024) s_tail[i / kTailBins][i % kTailBins] = 0;
    __syncthreads();
    {
      int kw = s_seg[1][t] - nw;
      for (int k = k0; k < k1; ++k) {
        const int c = len_of(row_at(k));
        if (c < 0 || c > L) continue;
        if (kw >= keep) atomicAdd(&s_tail[x][tail_bin(c, L)], 1);
        ++kw;
      }
    }
    __syncthreads();
    if (t < 8) {
      int run = 0;
      for (int b = kTailBins - 1; b >= 0; --b) {
        const int n = s_tail[t][b];
        s_tail[t][b] = run;
        run += n;
      }
    }
    __syncthreads();
    int ks = s_seg[0][t] - np, kw = s_seg[1][t] - nw;  // ranks of this thread's first rows
    for (int k = k0; k < k1; ++k) {
      const int r = row_at(k);
      const int c = len_of(r);
      if (c < 0) continue;
      const int pieces = c > L ? (c + L - 1) / L : 1;
      if (pieces == 1) {
        const int rank = kw < keep ? kw : keep + atomicAdd(&s_tail[x][tail_bin(c, L)], 1);
        const int pos = base + p_most * n_split + rank;
        if (pos < units_cap) units[pos] = make_int4(r, 0, c, -1);
        ++kw;
        continue;
      }
      const bool fits = sb + pieces <= slots_cap && pb < splits_cap;  // always, by the bounds above
      for (int s = 0; s < p_most; ++s) {
        int4 un = make_int4(-1, 0, 0, -1);
        if (s < pieces && fits)
          un = make_int4(r, c * s / pieces, c * (s + 1) / pieces, sb + s);  // c s < 2^24: 32-bit
        const int pos = base + s * n_split + ks;
        if (pos < units_cap) units[pos] = un;
      }
      if (fits) splits[pb] = make_int4(r, sb, pieces, 0);
      ++ks;
      sb += pieces;
      ++pb;
    }
    if (t == 1023) {
      hdr[0] = min(s_base[8], units_cap);
      hdr[1] = min(s_scan[2][1023], splits_cap);
      hdr[2] = L;
      hdr[3] = 0;
      for (int i = 0; i < 9; ++i) hdr[4 + i] = min(s_base[i], units_cap);
    }
    return;
  }
  int ub = s_scan[0][t] - nu;
  for (int k = k0; k < k1; ++k) {
    const int r = row_at(k);
    const int c = len_of(r);
    if (c < 0) continue;
    const int pieces = c > L ? (c + L - 1) / L : 1;
    // (past a capacity -- impossible by the bounds above -- the row stays one
    // unit and its other entries become placeholders the kernel skips)
    const bool split = pieces > 1 && sb + pieces <= slots_cap && pb < splits_cap;
    for (int s = 0; s < pieces; ++s) {
      const int b0 = c * s / pieces, b1 = c * (s + 1) / pieces;  // c s < 2^24: 32-bit
      int4 un = make_int4(r, b0, b1, split ? sb + s : -1);
      if (!split && pieces > 1) un = s == 0 ? make_int4(r, 0, c, -1) : make_int4(-1, 0, 0, -1);
      if (ub + s < units_cap) units[ub + s] = un;
    }
    if (split) splits[pb] = make_int4(r, sb, pieces, 0);
    ub += pieces;
    if (pieces > 1) {
      sb += pieces;
      ++pb;
    }
  }
  if (t == 1023) {
    hdr[0] = min(s_scan[0][1023], units_cap);
    hdr[1] = min(s_scan[2][1023], splits_cap);
    hdr[2] = L;
    hdr[3] = 0;
  }
}

// Merges the pieces of the split rows: m = max over pieces of m_p (pieces
// with no weight skipped), w_p = 2^(m_p - m), o = sum_p w_p O_p / sum_p w_p lr_p
// (the rounded sums the pieces' bf16 weights add up to), lse = ln 2 (m +
// log2 sum_p w_p l_p).  One workgroup per split row at a time; thread t takes
// query t / 2 and half t % 2 of its D outputs.
template <int D, bool LSE>
__global__ __launch_bounds__(256) void merge_split_rows_kernel(const int4* __restrict__ splits,
                                                               const int32_t* __restrict__ hdr,
                                                               const float* __restrict__ part,
                                                               const float* __restrict__ pstats,
                                                               uint16_t* __restrict__ o, float* __restrict__ lse,
                                                               const int32_t* __restrict__ perm, int N, int NB) {
  constexpr int HD = D / 2;
  const int n_split = hdr[1];
  const int t = threadIdx.x, qi = t >> 1, hd = t & 1;
  for (int sp = blockIdx.x; sp < n_split; sp += gridDim.x) {
    const int4 e = splits[sp];
    const int r = e.x, slot0 = e.y, pieces = e.z;
    const int bh = r / NB, u = r - bh * NB;
    const int qtok = perm[u * kBQ + qi];  // -1 at a padding position
    if (qtok < 0) continue;
    float m = -INFINITY;
#pragma unroll 4
    for (int p = 0; p < pieces; ++p) {
      const float* ps = pstats + (size_t)(slot0 + p) * 3 * kBQ;
      if (ps[kBQ + qi] > 0.f) m = fmaxf(m, ps[qi]);
    }
    float acc[HD];
#pragma unroll
    for (int j = 0; j < HD; ++j) acc[j] = 0.f;
    float lr = 0.f, lf = 0.f;
#pragma unroll 2  // two pieces' loads in flight
    for (int p = 0; p < pieces; ++p) {
      const float* ps = pstats + (size_t)(slot0 + p) * 3 * kBQ;
      const float lrp = ps[kBQ + qi];
      if (!(lrp > 0.f)) continue;
      const float w = __builtin_amdgcn_exp2f(ps[qi] - m);
      lr += w * lrp;
      if (LSE) lf += w * ps[2 * kBQ + qi];
      const float4* src = (const float4*)(part + ((size_t)(slot0 + p) * kBQ + qi) * D + hd * HD);
#pragma unroll
      for (int j = 0; j < HD / 4; ++j) {
        const float4 x = src[j];
        acc[4 * j] += w * x.x;
        acc[4 * j + 1] += w * x.y;
        acc[4 * j + 2] += w * x.z;
        acc[4 * j + 3] += w * x.w;
      }
    }
    const size_t tok = (size_t)bh * N + qtok;
    const float inv = lr > 0.f ? 1.f / lr : 0.f;
    uint2* dst = (uint2*)(o + tok * D + hd * HD);
#pragma unroll
    for (int j = 0; j < HD / 4; ++j) {
      uint2 w2;
      w2.x = pack_bf16x2(acc[4 * j] * inv, acc[4 * j + 1] * inv);
      w2.y = pack_bf16x2(acc[4 * j + 2] * inv, acc[4 * j + 3] * inv);
      dst[j] = w2;
    }
    if (LSE && hd == 0) lse[tok] = lf > 0.f ? 0.69314718055994531f * (m + __log2f(lf)) : -INFINITY;
  }
}

// Grid of a persistent attention kernel: as many workgroups as can be resident
// at once (the occupancy its registers and LDS allow), capped by the row count.
template <typename K>
int resident_grid(K kernel, size_t lds_bytes, const tra_plan_s& p, int threads = kThreads) {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, lds_bytes) != hipSuccess || per_cu < 1)
    per_cu = 1;
  return std::min(p.rows, per_cu * std::max(p.n_cu, 1));
}

template <int D>
int k64_sparse_grid_cap_d(const tra_plan_s& p) {
  const size_t lds_bytes = (size_t)p.NB * sizeof(int32_t);
  int a = 0, b = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, attn_k64_kernel<D, true, true>, kThreads, lds_bytes) !=
      hipSuccess)
    a = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, attn_k64_kernel<D, true, false>, kThreads, lds_bytes) !=
      hipSuccess)
    b = 1;
  return std::max(1, std::max(a, b)) * std::max(p.n_cu, 1);
}

template <int D, bool SPARSE, bool LSE>
void launch_k64_lse(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  const size_t lds_bytes = SPARSE ? (size_t)p.NB * sizeof(int32_t) : 0;
  int grid = resident_grid(attn_k64_kernel<D, SPARSE, LSE>, lds_bytes, p);
  if (SPARSE) {
    grid = std::min(grid, p.split_wg_cap);
    hipLaunchKernelGGL(plan_units_kernel, dim3(1), dim3(1024), 0, s, a.cnt, a.order, p.rows, p.NB, grid,
                       (int4*)p.d_units, p.units_cap, (int4*)p.d_splits, p.splits_cap, p.slots_cap, p.d_unit_hdr,
                       p.d_row_ctr);
  } else {
    hipLaunchKernelGGL(reset_row_counters, dim3(1), dim3(kRowCounters), 0, s, p.d_row_ctr);
  }
  if (a.ev_start) (void)hipEventRecord(a.ev_start, s);
  hipLaunchKernelGGL((attn_k64_kernel<D, SPARSE, LSE>), dim3(grid), dim3(kThreads), lds_bytes, s,
                     (const uint16_t*)a.q, p.d_kt, p.d_vt, (uint16_t*)a.o, a.lse, p.d_perm, a.cols,
                     p.cfg.block_layout == TRA_BLOCKS_TILES ? p.d_bcount : nullptr, (const int4*)p.d_units,
                     p.d_unit_hdr, a.order != nullptr, p.S, p.n_pad, p.NB, p.rows, scale_log2, p.d_row_ctr,
                     p.d_part, p.d_pstats);
  if (a.ev_stop) (void)hipEventRecord(a.ev_stop, s);
  if (SPARSE)
    hipLaunchKernelGGL((merge_split_rows_kernel<D, LSE>), dim3(std::max(1, std::min(p.splits_cap, 1024))),
                       dim3(256), 0, s, (const int4*)p.d_splits, p.d_unit_hdr, p.d_part, p.d_pstats,
                       (uint16_t*)a.o, a.lse, p.d_perm, p.S, p.NB);
}

template <int D, bool SPARSE>
void launch_k64(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  if (a.lse) launch_k64_lse<D, SPARSE, true>(p, a, s);
  else launch_k64_lse<D, SPARSE, false>(p, a, s);
}

// ------------------------------------------------------------ fused entropy + dense output
// The warm-up step's call (App. C.2, Alg. 2 with O): entropy and the dense
// output in one pass.  Its per-wave state (scores, P, O, Q and the entropy
// sum) does not fit the 128 registers a wave has when two of the 4-wave
// workgroups above share a CU, so this kernel keeps two waves per SIMD a
// different way, with matrix and vector work overlapped on purpose:
//
// One workgroup of 8 waves per query-block row, in two groups of 4 waves that
// share the row's 128 queries and split its key tiles (group g takes key
// blocks g, g + 2, ...); wave w4 of either group owns queries
// [32 w4, 32 w4 + 32) with its own running state, and the two groups' states
// (m, l, a, O) are merged at the end with the online-softmax rescaling.  Each
// group alternates a matrix phase (PV of its previous tile, QK^T of the
// current one) and a vector phase (softmax and entropy of the current tile,
// O rescale), group 1 one phase behind group 0, every phase split by a mid
// and a closing workgroup barrier.  So on every SIMD one wave keeps the matrix
// core busy while the other runs its softmax.
//
//   matrix phase i:  PV(i-1) | mid | QK^T(i), copies of V^T(i) in between
//   vector phase i:  copies of K(i+1) in between the row max and the first
//                    half of the exponentials | mid | second half, O rescale
// V^T(i) goes into the group's V buffer once PV(i-1) is done (mid barrier of
// matrix phase i) and is waited for at the end of vector phase i; K(i+1)
// goes into its K buffer once QK^T(i) is done (end of matrix phase i) and is
// waited for before the mid barrier of matrix phase i+1, so each copy has
// about one and a half phases to land.
constexpr int kFusedThreads = 512;

// One query-block row r of the fused kernel.  smem: per group a K tile, then a
// V^T tile; smemState: group 1's (m, l, a, lr) per query, for the merge.
template <int D>
__device__ __forceinline__ void fused_row(int r, uint8_t* smem, float* smemState,
                                          const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile,
                                          const uint16_t* __restrict__ vtile, uint16_t* __restrict__ o,
                                          float* __restrict__ entropy, const int32_t* __restrict__ perm, int N,
                                          int n_pad, int NB, float scale_log2) {
  using G = Geo<D>;
  constexpr int TILE = kBK * D * 2;
  constexpr int GROUP_BYTES = 2 * TILE;  // K tile, then V^T tile
  constexpr int KS = TileCopy<D>::STEPS;
  const int bh = r / NB, u = r - bh * NB;
  // (opaque: the lane arithmetic below is redone per row instead of being
  // hoisted out of the persistent row loop, where it would stay live and spill)
  const int t = (int)opaque(threadIdx.x), lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int g = wave >> 2, w4 = wave & 3;
  const int col = lane & 31, half = lane >> 5;
  const size_t head_off = (size_t)bh * N * D;
  constexpr size_t kTileBytes = (size_t)kBK * D * 2;
  const uint8_t* Kb = (const uint8_t*)(ktile + (size_t)bh * n_pad * D);
  const uint8_t* Vb = (const uint8_t*)(vtile + (size_t)bh * n_pad * D);
  uint8_t* gbuf = smem + g * GROUP_BYTES;
  const uint32_t k_lds = (uint32_t)(uintptr_t)gbuf + w4 * 1024;
  const uint32_t v_lds = k_lds + TILE;
  const uint32_t k_off = k_lane_off<D>(w4, lane);
  const uint32_t v_off = vt_lane_off(w4, lane);
  const lds_u8* kbuf = (const lds_u8*)gbuf;
  const lds_u8* vbuf = (const lds_u8*)(gbuf + TILE);

  const int qpos = u * kBQ + w4 * 32 + col;
  const bool qvalid = qpos < N;
  const int qrow = qvalid ? perm[qpos] : 0;
  bf16x8 qf[G::QK_STEPS];
  {
    const uint4* src = (const uint4*)(q + head_off + (size_t)qrow * D);
#pragma unroll
    for (int kk = 0; kk < G::QK_STEPS; ++kk) {
      uint4 x = qvalid ? src[2 * kk + half] : make_uint4(0, 0, 0, 0);
      qf[kk] = __builtin_bit_cast(bf16x8, x);
    }
  }
  const int krow = (col & ~15) | ((col & 15) ^ (((col >> 2) & 3) == 1 || ((col >> 2) & 3) == 2 ? 12 : 0));
  const uint32_t kbase = krow * D * 2 + ((half ^ swz<G::CH>(krow)) << 4);
  const uint32_t vbase = col * kBK * 2 + ((half ^ swz<16>(col)) << 4);

  f32x16 oacc[G::D_TILES];
#pragma unroll
  for (int i = 0; i < G::D_TILES; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[i][e] = 0.f;
  RowState st{-INFINITY, 0.f, 0.f, 0.f};
  uint32_t pb[32];
  f32x16 s[4];

  // Group g's phases matrix 0, vector 0, ..., vector n-1, matrix n run in
  // slots g, g + 1, ...; both groups count n_slots slots of two barriers each.
  const int n_g = (NB - g + 1) >> 1;
  const int n_half = (NB + 1) >> 1;
  const int n_slots = (NB & 1) ? 2 * n_half + 1 : 2 * n_half + 2;

  int b_cur = g;  // key block of this group's tile i: 2 i + g
  if (n_g > 0) issue_tile<D>(k_lds, Kb + b_cur * kTileBytes, k_off);
  wait_vm<0>();
  lds_barrier();
  if (g == 1) {  // group 1 idles in slot 0
    lds_barrier();
    lds_barrier();
  }

  for (int i = 0; i < n_g; ++i) {
    const bool has_next = i + 1 < n_g;
    const int b_nxt = b_cur + 2;
    // ---- matrix phase i
    if (i > 0) pv_tile_copies<D, 0>(oacc, vbuf, vbase, pb, v_lds, Vb, v_off);
    wait_vm<0>();  // this wave's part of K(i) has landed
    lds_barrier();
    qk_tile_copies<D, KS>(s, kbuf, kbase, qf, v_lds, Vb + b_cur * kTileBytes, v_off);
    lds_barrier();
    // ---- vector phase i
    if (N - b_cur * kBK < kBK) mask_tail(s, N - b_cur * kBK, half);
    const float sc = tile_max_tree<true>(s, scale_log2, st);
    float lp[4] = {0.f, 0.f, 0.f, 0.f}, ap[4] = {0.f, 0.f, 0.f, 0.f}, lr[4] = {0.f, 0.f, 0.f, 0.f};
    if (has_next)
      exp_pairs<D, true, true, 0, 16, KS>(s, scale_log2, st.m, lp, ap, lr, pb, k_lds, Kb + b_nxt * kTileBytes,
                                          k_off);
    else
      exp_pairs<D, true, true, 0, 16, 0>(s, scale_log2, st.m, lp, ap, lr, pb, k_lds, Kb, k_off);
    lds_barrier();
    exp_pairs<D, true, true, 16, 32, 0>(s, scale_log2, st.m, lp, ap, lr, pb, k_lds, Kb, k_off);
    st.l += (lp[0] + lp[1]) + (lp[2] + lp[3]);
    st.a += (ap[0] + ap[1]) + (ap[2] + ap[3]);
    st.lr += (lr[0] + lr[1]) + (lr[2] + lr[3]);
    if (__ballot(sc != 1.0f) != 0) {
#pragma unroll
      for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[dt][e] *= sc;
    }
    if (has_next) wait_vm<KS>();  // V^T(i) has landed; K(i+1) may still be in flight
    else wait_vm<0>();
    lds_barrier();
    b_cur = b_nxt;
  }
  // ---- matrix phase n: PV of the last tile
  if (n_g > 0) pv_tile_copies<D, 0>(oacc, vbuf, vbase, pb, v_lds, Vb, v_off);
  lds_barrier();
  lds_barrier();
  for (int k = g + 2 * n_g + 1; k < n_slots; ++k) {
    lds_barrier();
    lds_barrier();
  }

  // ---- merge group 1 into group 0.  Every tile copy has completed (the last
  // vector phase waits for all of them), so group 1's buffers take its O.
  float l_tot = sum_halves(st.l);
  float a_tot = sum_halves(st.a);
  float lr_tot = sum_halves(st.lr);
  const int qi = w4 * 32 + col;
  if (g == 1) {
    float4* dst = (float4*)(smem + GROUP_BYTES);
#pragma unroll
    for (int j = 0; j < 4 * G::D_TILES; ++j)
      dst[j * 256 + w4 * 64 + lane] = make_float4(oacc[j >> 2][4 * (j & 3)], oacc[j >> 2][4 * (j & 3) + 1],
                                                  oacc[j >> 2][4 * (j & 3) + 2], oacc[j >> 2][4 * (j & 3) + 3]);
    if (half == 0) {
      smemState[qi] = st.m;
      smemState[kBQ + qi] = l_tot;
      smemState[2 * kBQ + qi] = a_tot;
      smemState[3 * kBQ + qi] = lr_tot;
    }
  }
  lds_barrier();
  if (g == 1) return;
  {
    const float m1 = smemState[qi], l1 = smemState[kBQ + qi], a1 = smemState[2 * kBQ + qi];
    const float lr1 = smemState[3 * kBQ + qi];
    // a group state with l = 0 saw no key (m = -inf) and contributes nothing
    const float m = l1 > 0.f ? (l_tot > 0.f ? fmaxf(st.m, m1) : m1) : st.m;
    const float s0 = l_tot > 0.f ? __builtin_amdgcn_exp2f(st.m - m) : 0.f;
    const float s1 = l1 > 0.f ? __builtin_amdgcn_exp2f(m1 - m) : 0.f;
    const float e0 = l_tot > 0.f ? s0 * (a_tot + l_tot * (st.m - m)) : 0.f;
    const float e1 = l1 > 0.f ? s1 * (a1 + l1 * (m1 - m)) : 0.f;
    a_tot = e0 + e1;
    l_tot = s0 * l_tot + s1 * l1;
    lr_tot = s0 * lr_tot + s1 * lr1;
    const float4* src = (const float4*)(smem + GROUP_BYTES);
#pragma unroll
    for (int j = 0; j < 4 * G::D_TILES; ++j) {
      const float4 x = src[j * 256 + w4 * 64 + lane];
      f32x16& acc = oacc[j >> 2];
      const int e = 4 * (j & 3);
      acc[e] = s0 * acc[e] + s1 * x.x;
      acc[e + 1] = s0 * acc[e + 1] + s1 * x.y;
      acc[e + 2] = s0 * acc[e + 2] + s1 * x.z;
      acc[e + 3] = s0 * acc[e + 3] + s1 * x.w;
    }
  }

  if (!qvalid) return;
  const size_t tok = (size_t)bh * N + qrow;
  const float inv = lr_tot > 0.f ? 1.f / lr_tot : 0.f;
  uint16_t* dst = o + tok * D;
#pragma unroll
  for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int d0 = dt * 32 + 8 * gq + 4 * half;
      uint2 w;
      w.x = pack_bf16x2(oacc[dt][4 * gq] * inv, oacc[dt][4 * gq + 1] * inv);
      w.y = pack_bf16x2(oacc[dt][4 * gq + 2] * inv, oacc[dt][4 * gq + 3] * inv);
      *(uint2*)(dst + d0) = w;
    }
  if (half == 0) entropy[tok] = 0.69314718055994531f * (__log2f(l_tot) - a_tot / l_tot);
}

// Persistent: one workgroup per CU, taking rows from the per-XCD row queues
// until they are drained (the first barrier of every row orders the next
// s_row write after every wave's read of the current one).
template <int D>
__global__ __launch_bounds__(kFusedThreads, 1) void attn_fused_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile,
    const uint16_t* __restrict__ vtile, uint16_t* __restrict__ o, float* __restrict__ entropy,
    const int32_t* __restrict__ perm, int N, int n_pad, int NB, int rows, float scale_log2,
    int32_t* __restrict__ ctr) {
  constexpr int TILE = kBK * D * 2;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[4 * TILE];
  __shared__ float smemState[4 * kBQ];
  __shared__ int s_row, s_steal;
  if (threadIdx.x == 0) s_steal = 0;
  for (;;) {
    if (threadIdx.x == 0) {
      int steal = s_steal;
      s_row = next_row(ctr, nullptr, rows, blockIdx.x & 7, steal);
      s_steal = steal;
    }
    __syncthreads();
    const int r = s_row;
    if (r < 0) break;
    fused_row<D>(r, smem, smemState, q, ktile, vtile, o, entropy, perm, N, n_pad, NB, scale_log2);
  }
}

template <int D>
void launch_fused_entropy_output(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  const int grid = resident_grid(attn_fused_kernel<D>, 0, p, kFusedThreads);
  hipLaunchKernelGGL(reset_row_counters, dim3(1), dim3(kRowCounters), 0, s, p.d_row_ctr);
  if (a.ev_start) (void)hipEventRecord(a.ev_start, s);
  hipLaunchKernelGGL((attn_fused_kernel<D>), dim3(grid), dim3(kFusedThreads), 0, s, (const uint16_t*)a.q,
                     p.d_kt, p.d_vt, (uint16_t*)a.o, a.entropy, p.d_perm, p.S, p.n_pad, p.NB, p.rows,
                     scale_log2, p.d_row_ctr);
  if (a.ev_stop) (void)hipEventRecord(a.ev_stop, s);
}

template <int D, bool SPARSE, bool PV, bool ENT, int TOK = 0>
void launch_variant(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  size_t lds_bytes = SPARSE ? (size_t)((p.NB + 3) & ~3) * sizeof(int32_t) : 0;
  if (TOK != 0) lds_bytes += (size_t)kBQ * p.cfg.frames * sizeof(uint16_t);
  const TokArgs tk{a.radius_sq, p.cfg.distance == TRA_DIST_1D ? p.d_thr1 : p.d_thr, p.d_kinfo, p.d_blocks,
                   p.d_coord, p.d_kfeat, p.N, p.cfg.frames, p.n_cap};
  const int grid = resident_grid(attn_bf16_kernel<D, SPARSE, PV, ENT, 2, TOK>, lds_bytes, p);
  hipLaunchKernelGGL(reset_row_counters, dim3(1), dim3(kRowCounters), 0, s, p.d_row_ctr);
  if (a.ev_start) (void)hipEventRecord(a.ev_start, s);
  hipLaunchKernelGGL((attn_bf16_kernel<D, SPARSE, PV, ENT, 2, TOK>), dim3(grid), dim3(kThreads), lds_bytes, s,
                     (const uint16_t*)a.q, p.d_kt, p.d_vt, (uint16_t*)a.o, a.lse, a.entropy, p.d_perm,
                     a.cnt, a.cols, a.order, p.S, p.n_pad, p.NB, p.rows, scale_log2, tk, p.d_row_ctr);
  if (a.ev_stop) (void)hipEventRecord(a.ev_stop, s);
}

template <int D>
hipError_t launch_bf16_d(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const int bhs = p.cfg.batch * p.cfg.heads;
  const unsigned gy = (unsigned)std::min(bhs, kGatherMaxY);
  hipLaunchKernelGGL((gather_k_kernel<D>), dim3((unsigned)((p.n_pad * (D / 8) + 255) / 256), gy), dim3(256), 0, s,
                     (const uint4*)a.k, (uint4*)p.d_kt, p.d_perm, p.S, p.n_pad, bhs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.v) {
    hipLaunchKernelGGL((gather_vt_kernel<D>), dim3(p.n_pad / 64, gy), dim3(256), 0, s,
                       (const uint16_t*)a.v, p.d_vt, p.d_perm, p.S, p.n_pad, bhs);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const bool text = p.S > p.N;
  if (a.sparse && a.radius_sq && p.cfg.distance == TRA_DIST_1D && text) launch_variant<D, true, true, false, 6>(p, a, s);
  else if (a.sparse && a.radius_sq && p.cfg.distance == TRA_DIST_1D) launch_variant<D, true, true, false, 2>(p, a, s);
  else if (a.sparse && a.radius_sq && text) launch_variant<D, true, true, false, 5>(p, a, s);
  else if (a.sparse && a.radius_sq) launch_variant<D, true, true, false, 1>(p, a, s);
  else if (a.sparse) launch_k64<D, true>(p, a, s);
  else if (a.entropy && a.o) launch_fused_entropy_output<D>(p, a, s);
  else if (a.entropy) launch_variant<D, false, false, true>(p, a, s);
  else launch_k64<D, false>(p, a, s);
  return hipGetLastError();
}

}  // namespace

int k64_sparse_grid_cap(const tra_plan_s& p) {
  return p.cfg.head_dim == 64 ? k64_sparse_grid_cap_d<64>(p) : k64_sparse_grid_cap_d<128>(p);
}

void split_capacities(int grid_cap, int rows, int NB, int head_dim, int* units_cap, int* splits_cap,
                      int* slots_cap) {
  (void)head_dim;
  const long long share = (long long)grid_cap * kSplitPerWG;
  // a split row of c entries has fewer than 2 c / L pieces, and L >= T / share,
  // L >= kSplitMin: at most 2 share pieces, and at most 2 rows ceil(NB / kSplitMin)
  *slots_cap = (int)std::min<long long>(2 * share + 1, 2LL * rows * ((NB + kSplitMin - 1) / kSplitMin) + 1);
  *splits_cap = (int)std::min<long long>(INT_MAX, share + 1);
  // piece-major segments: at most ceil(NB / kSplitMin) units per split row,
  // and at most slots / 2 split rows
  const long long seg = (long long)((NB + kSplitMin - 1) / kSplitMin) * (*slots_cap / 2 + 1);
  *units_cap = (int)std::min<long long>(INT_MAX, rows + std::max(share, seg) + 1);
}

hipError_t launch_attention_bf16(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  if (p.cfg.head_dim == 64) return launch_bf16_d<64>(p, a, s);
  return launch_bf16_d<128>(p, a, s);
}

}  // namespace tra
