// bf16 attention family on gfx950 matrix cores: dense attention (Eq. 1),
// block-sparse TRA attention (Eq. 16 at block granularity) and the fused
// online-softmax entropy pass (App. C.2, Alg. 2), all from one template.
//
// Layout pre-pass
//   K and V are first gathered into tile-major order (Sec. 3.3: tokens of a
//   spatial tile become contiguous) in the plan's workspace, one 128-token key
//   block = one contiguous 32 KB tile, rows past N zero-filled.  The attention
//   loop then addresses tiles affinely.  Q is gathered and O scattered through
//   the same permutation inside the kernel, so callers keep raster order.
//
// Work decomposition
//   One workgroup (4 waves, 256 threads) per query-block row r = (b, h, u):
//   128 queries, wave w owning queries [32w, 32w + 32).  It walks the key
//   blocks of its row (all NB for dense; cols[r][0..cnt[r]) for sparse), 128
//   keys per tile.  Two workgroups share a CU (64 KB of LDS each), so every
//   SIMD runs one workgroup's matrix phase while the other is in its softmax.
//
// Per tile (split barriers)
//   K and V go from HBM straight into LDS (global_load_lds_dwordx4, no register
//   staging), 16-byte chunks XOR-swizzled per row so K reads and transposed V
//   reads hit every bank once.  The next K tile streams in during softmax + PV,
//   the next V tile during QK^T + softmax.  Scheduling hints keep several LDS
//   operand reads in flight ahead of the MFMAs.
//
// Matrix work (v_mfma_f32_32x32x16_bf16, fp32 accumulation)
//   S^T = K Q^T: keys are the M side and the wave's 32 queries the N side, so a
//   lane holds 64 scores of ONE query (row max / row sum are in-lane plus one
//   exchange between lane halves).  The bf16 probabilities stay in registers
//   as the B operand of O^T += V^T P^T; the V^T operand comes from LDS through
//   ds_read_b64_tr_b16, which transposes 16-bit elements across lanes.
//
// Softmax and entropy (Alg. 2 with the running sum kept relative to the max)
//   x = s alpha log2(e) - m,  w = 2^x,  l = sum w,  a = sum w x.
//   On a max increase m -> m': l <- 2^{m-m'} l, a <- 2^{m-m'} (a + l (m - m')).
//   H = ln(l) - ln(2) a / l  (nats)  == log Z - sum_j p_j s_j (App. C.2).
//   Each lane keeps l and a over its own keys; the halves are added at the end.
#include <cmath>
#include <type_traits>

#include "tra_internal.h"

namespace tra {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kBQ = 128;       // queries per workgroup (= block size)
constexpr int kBK = 128;       // keys per tile (= block size)
constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 f = {a, b};
  bf16x2 h = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// XOR swizzle of the 16-byte chunks of LDS row `row` (one key).  Row length is
// D*2 bytes = CH chunks.  Requirements: (a) 16 consecutive rows read at one
// logical chunk land in distinct banks (QK^T operand reads); (b) 4 aligned
// consecutive rows read at 4 aligned consecutive chunks land in distinct
// banks (transposed V reads).
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

// ------------------------------------------------------------ layout pre-pass
// dst[bh][p][:] = src[bh][perm[p]][:] for p < N, 0 for N <= p < n_pad.
__global__ __launch_bounds__(256) void gather_kv_kernel(const uint4* __restrict__ k,
                                                        const uint4* __restrict__ v,
                                                        uint4* __restrict__ kt, uint4* __restrict__ vt,
                                                        const int32_t* __restrict__ perm, int N,
                                                        int n_pad, int ch, long long total) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const long long per_head = (long long)n_pad * ch;
  const long long bh = idx / per_head;
  const long long rem = idx - bh * per_head;
  const int p = (int)(rem / ch), c = (int)(rem - (long long)p * ch);
  uint4 zk = make_uint4(0, 0, 0, 0), zv = zk;
  if (p < N) {
    const long long s = (bh * N + perm[p]) * ch + c;
    zk = k[s];
    if (v) zv = v[s];
  }
  kt[idx] = zk;
  if (v) vt[idx] = zv;
}

// ------------------------------------------------------------ attention
template <int D>
struct Geo {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int LPT = kBK * CH / kThreads;  // direct loads per thread per tile
  static constexpr int RPI = 64 / CH;              // rows covered by one wave-wide load
  static constexpr int QK_STEPS = D / 16;
  static constexpr int D_TILES = D / 32;
};

// Direct HBM -> LDS copy of one contiguous tile (kBK rows x D): load n of this
// thread fills LDS slots [(4n + wave) * 64, +64), i.e. row (4n + wave) * RPI +
// lane / CH, physical chunk lane % CH, which holds logical chunk
// (lane % CH) ^ swz(row).
template <int D>
__device__ __forceinline__ void issue_tile(uint16_t* lds, const uint16_t* tile, int wave, int lane) {
  using G = Geo<D>;
  const int lrow0 = wave * G::RPI + lane / G::CH;
  const int lphys = lane % G::CH;
#pragma unroll
  for (int n = 0; n < G::LPT; ++n) {
    const int row = n * 4 * G::RPI + lrow0;
    const int c = lphys ^ swz<G::CH>(row);
    __builtin_amdgcn_global_load_lds((const void*)(tile + row * D + c * 8),
                                     (lds_void*)(lds + (n * 4 + wave) * 64 * 8), 16, 0, 0);
  }
}

typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ bf16x8 lds_read16(const lds_u8* base, uint32_t off) {
  return __builtin_bit_cast(bf16x8, *(const __attribute__((address_space(3))) uint4*)(base + off));
}

// One MFMA step of S^T = K Q^T for sub-tile kt: keys 32kt + (lane % 32).
template <int D>
__device__ __forceinline__ void qk_step(f32x16& s, const lds_u8* kbuf, const uint32_t (&koff)[Geo<D>::QK_STEPS],
                                        const bf16x8 (&qf)[Geo<D>::QK_STEPS], int kt, int kk) {
  const bf16x8 ka = lds_read16(kbuf, koff[kk] + kt * 32 * D * 2);
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
__device__ __forceinline__ void qk_tile(f32x16 (&s)[4], const lds_u8* kbuf,
                                        const uint32_t (&koff)[Geo<D>::QK_STEPS],
                                        const bf16x8 (&qf)[Geo<D>::QK_STEPS]) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
  // k-step outer, sub-tile inner: four independent accumulation chains
#pragma unroll
  for (int kk = 0; kk < Geo<D>::QK_STEPS; ++kk)
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) qk_step<D>(s[kt], kbuf, koff, qf, kt, kk);
  sched_reads_ahead<4 * Geo<D>::QK_STEPS, 1, 4>();
}

// Keys past the end of a ragged last block get a large finite negative score:
// their weight 2^x underflows to 0 and w * x stays 0 (not 0 * inf).
// Output element e of sub-tile kt is key 32kt + 8(e/4) + 4*half + e%4.
__device__ __forceinline__ void mask_tail(f32x16 (&s)[4], int nv, int half) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = kt * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
      if (key >= nv) s[kt][e] = -1.0e30f;
    }
}

struct RowState {
  float m, l, a;  // running max (log2 units), sum of weights, entropy sum
};

// Max of a score tile folded into the running state; returns the factor that
// rescales everything accumulated so far (0 on the first tile).
template <bool ENT>
__device__ __forceinline__ float tile_max(const f32x16 (&s)[4], float scale_log2, RowState& st) {
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(st.m, mx * scale_log2);
  const float sc = __builtin_amdgcn_exp2f(st.m - m_new);
  if (ENT) st.a = st.l > 0.f ? sc * (st.a + st.l * (st.m - m_new)) : 0.f;
  st.l *= sc;
  st.m = m_new;
  return sc;
}

// Weights of sub-tile kt: w = 2^(s alpha log2e - m), summed into l (and w x into
// a); bf16 pairs into pb[8kt .. 8kt+7].
template <bool PV, bool ENT>
__device__ __forceinline__ void tile_exp(const f32x16& s, float scale_log2, float m, float& lsum,
                                         float& asum, uint32_t* pb) {
#pragma unroll
  for (int e = 0; e < 16; e += 2) {
    const float x0 = fmaf(s[e], scale_log2, -m);
    const float x1 = fmaf(s[e + 1], scale_log2, -m);
    const float w0 = __builtin_amdgcn_exp2f(x0);
    const float w1 = __builtin_amdgcn_exp2f(x1);
    lsum += w0 + w1;
    if (ENT) asum = fmaf(w0, x0, fmaf(w1, x1, asum));
    if (PV) pb[e >> 1] = pack_bf16x2(w0, w1);
  }
}

// O^T += V^T P^T.  k-step ks covers keys [16ks, 16ks+16); in lane half h the B
// operand (sub-tile ks/2, elements 8(ks%2)..+7) holds keys 16ks + 4h + {0..3}
// and 16ks + 8 + 4h + {0..3}.  ds_read_b64_tr_b16 gives output lane i (of a
// 16-lane group) element (i%4) of the 8-byte rows addressed by lanes i/4 + 4k,
// k = 0..3: so lane j of group g addresses key 16ks + 4h + j/4 (+8 for the
// second read) at d = 32dt + 16(g%2) + 4(j%4), and lane i receives
// d = 32dt + (lane % 32) with keys 16ks + 4h + {0..3} (+8).
template <int D>
__device__ __forceinline__ void pv_step(f32x16& oacc, const lds_u8* vbuf, const uint32_t (&voff)[2][Geo<D>::D_TILES],
                                        const uint32_t (&pb)[32], int ks, int dt) {
  const int kt = ks >> 1, eb = (ks & 1) * 4;
  const uint4 bw = make_uint4(pb[kt * 8 + eb], pb[kt * 8 + eb + 1], pb[kt * 8 + eb + 2], pb[kt * 8 + eb + 3]);
  const uint32_t o0 = voff[0][dt] + ks * 16 * D * 2, o1 = voff[1][dt] + ks * 16 * D * 2;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vbuf + o0));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vbuf + o1));
  const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
  const uint4 va4 = make_uint4(l2.x, l2.y, h2.x, h2.y);
  oacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, va4),
                                                 __builtin_bit_cast(bf16x8, bw), oacc, 0, 0, 0);
}

// Main attention kernel.  One workgroup per query-block row, two workgroups per
// CU (64 KB of LDS each: one K and one V tile).  Split barriers let the next
// K tile stream in during softmax + PV and the next V tile during QK^T +
// softmax; each SIMD interleaves one workgroup's matrix phase with the other's
// vector phase.  OCC is the workgroups-per-CU bound the registers are sized
// for (the fused entropy + output variant needs one per CU to avoid spills).
template <int D, bool SPARSE, bool PV, bool ENT, int OCC>
__global__ __launch_bounds__(kThreads, OCC) void attn_bf16_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ ktile,
    const uint16_t* __restrict__ vtile, uint16_t* __restrict__ o, float* __restrict__ lse,
    float* __restrict__ entropy, const int32_t* __restrict__ perm, const int32_t* __restrict__ cnt,
    const int32_t* __restrict__ cols, const int32_t* __restrict__ order, int N, int n_pad, int NB,
    int rows, float scale_log2) {
  using G = Geo<D>;
  constexpr int TILE = kBK * D * 2;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[(PV ? 2 : 1) * TILE];  // [K][V]
  lds_u8* lds = (lds_u8*)smem;

  int r = blockIdx.x;
  if (SPARSE && order) {
    r = order[blockIdx.x];
    if (r < 0 || r >= rows) return;
  }
  const int bh = r / NB, u = r - bh * NB;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int col = lane & 31, half = lane >> 5;
  const size_t head_off = (size_t)bh * N * D;
  const uint16_t* Kb = ktile + (size_t)bh * n_pad * D;
  const uint16_t* Vb = vtile + (size_t)bh * n_pad * D;

  const int qpos = u * kBQ + wave * 32 + col;
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
  uint32_t koff[G::QK_STEPS];
  {
    const int sw = swz<G::CH>(col);
#pragma unroll
    for (int kk = 0; kk < G::QK_STEPS; ++kk) koff[kk] = col * D * 2 + (((2 * kk + half) ^ sw) << 4);
  }
  uint32_t voff[2][G::D_TILES];
  {
    const int grp = lane >> 4, j = lane & 15;
    const int kj = 4 * half + (j >> 2);
    const int dq = 16 * (grp & 1) + 4 * (j & 3);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int key = kj + 8 * h;
      const int sw = swz<G::CH>(key);
#pragma unroll
      for (int dt = 0; dt < G::D_TILES; ++dt) {
        const int d = 32 * dt + dq;
        voff[h][dt] = key * D * 2 + ((((d >> 3) ^ sw) << 3) + (d & 7)) * 2;
      }
    }
  }

  const int count = SPARSE ? min(max(cnt[r], 0), NB) : NB;
  const int32_t* colp = SPARSE ? cols + (size_t)r * NB : nullptr;
  auto blk = [&](int i) -> int { return SPARSE ? min(max(colp[i], 0), NB - 1) : i; };

  f32x16 oacc[PV ? G::D_TILES : 1];
#pragma unroll
  for (int i = 0; i < (PV ? G::D_TILES : 1); ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[i][e] = 0.f;
  RowState st{-INFINITY, 0.f, 0.f};

  if (count > 0) {
    int b_cur = blk(0);
    issue_tile<D>((uint16_t*)smem, Kb + (size_t)b_cur * kBK * D, wave, lane);
    if (PV) issue_tile<D>((uint16_t*)(smem + TILE), Vb + (size_t)b_cur * kBK * D, wave, lane);
    for (int i = 0; i < count; ++i) {
      const bool has_next = i + 1 < count;
      const int b_nxt = has_next ? blk(i + 1) : 0;
      wait_vm<PV ? G::LPT : 0>();  // K_i landed (V_i may still be in flight)
      __syncthreads();
      f32x16 s[4];
      qk_tile<D>(s, lds, koff, qf);
      __syncthreads();  // every wave is done with K_i
      if (has_next) issue_tile<D>((uint16_t*)smem, Kb + (size_t)b_nxt * kBK * D, wave, lane);
      if (N - b_cur * kBK < kBK) mask_tail(s, N - b_cur * kBK, half);
      const float sc = tile_max<ENT>(s, scale_log2, st);
      uint32_t pb[32];
      float lsum = 0.f, asum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        tile_exp<PV, ENT>(s[kt], scale_log2, st.m, lsum, asum, pb + 8 * kt);
      }
      st.l += lsum;
      if (ENT) st.a += asum;
      if constexpr (PV) {
        if (has_next) wait_vm<G::LPT>();  // V_i landed (K_{i+1} may still be in flight)
        else wait_vm<0>();
        __syncthreads();
        if (__ballot(sc != 1.0f) != 0) {
#pragma unroll
          for (int dt = 0; dt < G::D_TILES; ++dt)
#pragma unroll
            for (int e = 0; e < 16; ++e) oacc[dt][e] *= sc;
        }
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
#pragma unroll
          for (int dt = 0; dt < G::D_TILES; ++dt) pv_step<D>(oacc[dt], lds + TILE, voff, pb, ks, dt);
        sched_reads_ahead<8 * G::D_TILES, 2, 4>();
        __syncthreads();  // every wave is done with V_i
        if (has_next) issue_tile<D>((uint16_t*)(smem + TILE), Vb + (size_t)b_nxt * kBK * D, wave, lane);
      }
      b_cur = b_nxt;
    }
  }

  const float l_tot = st.l + __shfl_xor(st.l, 32);
  const float a_tot = ENT ? st.a + __shfl_xor(st.a, 32) : 0.f;
  if (!qvalid) return;
  const size_t tok = (size_t)bh * N + qrow;
  if (PV) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
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

template <int D, bool SPARSE, bool PV, bool ENT>
void launch_variant(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  // the fused entropy + output variant needs more than the 256 VGPRs a wave
  // gets at two workgroups per CU
  constexpr int kOcc = (PV && ENT) ? 1 : 2;
  hipLaunchKernelGGL((attn_bf16_kernel<D, SPARSE, PV, ENT, kOcc>), dim3(p.rows), dim3(kThreads), 0, s,
                     (const uint16_t*)a.q, p.d_kt, p.d_vt, (uint16_t*)a.o, a.lse, a.entropy, p.d_perm,
                     a.cnt, a.cols, a.order, p.N, p.n_pad, p.NB, p.rows,
                     (float)(1.4426950408889634 / std::sqrt((double)D)));
}

template <int D>
hipError_t launch_bf16_d(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const int ch = D / 8;
  const long long total = (long long)p.cfg.batch * p.cfg.heads * p.n_pad * ch;
  hipLaunchKernelGGL(gather_kv_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     (const uint4*)a.k, (const uint4*)a.v, (uint4*)p.d_kt, (uint4*)p.d_vt, p.d_perm,
                     p.N, p.n_pad, ch, total);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.sparse) launch_variant<D, true, true, false>(p, a, s);
  else if (a.entropy && a.o) launch_variant<D, false, true, true>(p, a, s);
  else if (a.entropy) launch_variant<D, false, false, true>(p, a, s);
  else launch_variant<D, false, true, false>(p, a, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_bf16(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  if (p.cfg.head_dim == 64) return launch_bf16_d<64>(p, a, s);
  return launch_bf16_d<128>(p, a, s);
}

}  // namespace tra
