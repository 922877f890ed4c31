// fp32 attention family (dense, block-sparse, token-level sparse, fused
// entropy) for fp32 workloads.  Scalar fp32 arithmetic with one thread per
// query row; the bf16 path is the MFMA kernel.  One workgroup per query-block
// row.  The token-level variant (Eq. 16 with the token mask of Eq. 15 inside
// the listed blocks) tests every (query, key) pair with the plan's integer
// thresholds, as the block-mask kernel does.
//
// Online softmax with the entropy accumulator of Alg. 2 (App. C.2), kept
// relative to the running maximum m: per row l = sum_j e^{s_j - m} and
// a = sum_j e^{s_j - m} (s_j - m); when m grows to m', l <- e^{m-m'} l and
// a <- e^{m-m'} (a + l (m - m')).  At the end H = log l - a / l, which equals
// log Z - sum_j p_j s_j (the fused-entropy identity of App. C.2), and
// lse = m + log l.
#include <cmath>

#include "tra_internal.h"

namespace tra {
namespace {

struct F32Params {
  const float* q;
  const float* k;
  const float* v;
  float* o;
  float* lse;
  float* entropy;
  const int32_t* perm;
  const int32_t* cnt;
  const int32_t* cols;
  const int32_t* order;
  const int32_t* bcount;  // tokens of each block (tile-aligned layout), NULL: packed
  int N, NB, rows;
  float alpha;
  // token-level attention only
  const int32_t* radius_sq;
  const int32_t* thr;  // [(n_cap + 1) * F], 2-D or 1-D thresholds per the plan
  int Nv, F, H, W, n_cap;
};

// Does video query i (radius n, raster index) cover video key j (raster
// index)?  DIST as in the block mask: 2-D squared distance or 1-D |i - j|.
template <int DIST>
__device__ __forceinline__ bool covers(const F32Params& P, int i, int n, int j) {
  const int HW = P.H * P.W;
  const int fi = i / HW, fj = j / HW;
  int dist;
  if (DIST == TRA_DIST_1D) {
    dist = abs(i - j);
  } else {
    const int dx = (i / P.W) % P.H - (j / P.W) % P.H, dy = i % P.W - j % P.W;
    dist = dx * dx + dy * dy;
  }
  return dist <= P.thr[(size_t)n * P.F + abs(fi - fj)];
}

constexpr int kSub = 32;  // keys staged in LDS at a time

// TOK: 0 block-granular, 1 token mask with 2-D distance, 2 with 1-D distance.
template <int D, int B, bool SPARSE, bool PV, bool ENT, int TOK = 0>
__global__ __launch_bounds__(B) void attn_f32_kernel(F32Params P) {
  __shared__ float sK[kSub][D + 1];
  __shared__ float sV[PV ? kSub : 1][PV ? D + 1 : 1];
  __shared__ int sPos[kSub];  // raster index of each staged key

  int r = blockIdx.x;
  if (SPARSE && P.order) {
    r = P.order[blockIdx.x];
    if (r < 0 || r >= P.rows) return;  // whole workgroup leaves together
  }
  const int bh = r / P.NB, u = r - bh * P.NB;
  const int t = threadIdx.x;
  const int qpos = u * B + t;
  const int qtok = P.perm[qpos];  // -1 at a padding position
  const bool qvalid = qtok >= 0;
  const int qrow = qvalid ? qtok : 0;
  const size_t head_off = (size_t)bh * P.N * D;

  float qr[D];
#pragma unroll
  for (int d = 0; d < D; ++d) qr[d] = qvalid ? P.q[head_off + (size_t)qrow * D + d] : 0.f;
  float acc[PV ? D : 1];
#pragma unroll
  for (int d = 0; d < (PV ? D : 1); ++d) acc[d] = 0.f;
  float m = -INFINITY, l = 0.f, a = 0.f;
  // token mask: a text query (or a FULL radius) covers every key
  int n_i = 0;
  bool all_keys = true;
  if (TOK && qvalid && qrow < P.Nv) {
    n_i = P.radius_sq[(size_t)bh * P.N + qrow];
    all_keys = n_i > P.n_cap;
    n_i = max(n_i, 0);
  }

  const int count = SPARSE ? min(max(P.cnt[r], 0), P.NB) : P.NB;
  for (int c = 0; c < count; ++c) {
    const int vb = SPARSE ? P.cols[(size_t)r * P.NB + c] : c;
    if (vb < 0 || vb >= P.NB) continue;  // uniform across the workgroup
    const int nv = P.bcount ? P.bcount[vb] : min(B, P.N - vb * B);  // a block's tokens fill its first positions
    for (int j0 = 0; j0 < nv; j0 += kSub) {
      const int ns = min(kSub, nv - j0);
      __syncthreads();
      for (int e = t; e < kSub * D; e += B) {
        const int j = e / D, d = e - j * D;
        float kv = 0.f, vv = 0.f;
        if (j < ns) {
          const size_t off = head_off + (size_t)P.perm[vb * B + j0 + j] * D + d;
          kv = P.k[off];
          if (PV) vv = P.v[off];
        }
        sK[j][d] = kv;
        if (PV) sV[j][d] = vv;
      }
      if (TOK && t < kSub) sPos[t] = t < ns ? P.perm[vb * B + j0 + t] : 0;
      __syncthreads();
      float s[kSub];
      float mc = -INFINITY;
#pragma unroll
      for (int j = 0; j < kSub; ++j) {
        float dot = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) dot = fmaf(qr[d], sK[j][d], dot);
        bool keep = j < ns;
        if (TOK && keep && !all_keys && sPos[j] < P.Nv)
          keep = covers<TOK == 2 ? TRA_DIST_1D : TRA_DIST_2D>(P, qrow, n_i, sPos[j]);
        s[j] = keep ? dot * P.alpha : -INFINITY;
        mc = fmaxf(mc, s[j]);
      }
      if (TOK && mc == -INFINITY) continue;  // no covered key here: nothing to add
      const float mn = fmaxf(m, mc);
      const float sc = expf(m - mn);  // 0 on the first sub-tile (m = -inf)
      if (ENT) a = l > 0.f ? sc * (a + l * (m - mn)) : 0.f;
      l *= sc;
      if (PV) {
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] *= sc;
      }
      for (int j = 0; j < ns; ++j) {
        const float x = s[j] - mn;
        const float p = expf(x);
        l += p;
        if (ENT) a = fmaf(p, x, a);
        if (PV) {
#pragma unroll
          for (int d = 0; d < D; ++d) acc[d] = fmaf(p, sV[j][d], acc[d]);
        }
      }
      m = mn;
    }
  }
  if (!qvalid) return;
  const size_t tok = (size_t)bh * P.N + qrow;
  if (PV) {
    const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) P.o[tok * D + d] = acc[d] * inv;
  }
  if (ENT) P.entropy[tok] = logf(l) - a / l;
  if (P.lse) P.lse[tok] = l > 0.f ? m + logf(l) : -INFINITY;
}

template <int D, int B>
hipError_t launch_f32_db(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const bool one_d = p.cfg.distance == TRA_DIST_1D;
  F32Params P{(const float*)a.q, (const float*)a.k, (const float*)a.v, (float*)a.o, a.lse,
              a.entropy, p.d_perm, a.cnt, a.cols, a.order,
              a.sparse && p.cfg.block_layout == TRA_BLOCKS_TILES ? p.d_bcount : nullptr, p.S, p.NB, p.rows,
              1.0f / sqrtf((float)D), a.radius_sq, one_d ? p.d_thr1 : p.d_thr, p.N,
              p.cfg.frames, p.cfg.height, p.cfg.width, p.n_cap};
  const dim3 grid(p.rows), block(B);
  if (a.ev_start) (void)hipEventRecord(a.ev_start, s);
  if (a.sparse && a.radius_sq && one_d)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, true, true, false, 2>), grid, block, 0, s, P);
  else if (a.sparse && a.radius_sq)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, true, true, false, 1>), grid, block, 0, s, P);
  else if (a.sparse)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, true, true, false>), grid, block, 0, s, P);
  else if (a.entropy && a.o)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, false, true, true>), grid, block, 0, s, P);
  else if (a.entropy)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, false, false, true>), grid, block, 0, s, P);
  else
    hipLaunchKernelGGL((attn_f32_kernel<D, B, false, true, false>), grid, block, 0, s, P);
  if (a.ev_stop) (void)hipEventRecord(a.ev_stop, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_f32(const tra_plan_s& p, const AttnArgs& a, hipStream_t s) {
  const int D = p.cfg.head_dim, B = p.cfg.block;
  if (D == 64 && B == 64) return launch_f32_db<64, 64>(p, a, s);
  if (D == 64 && B == 128) return launch_f32_db<64, 128>(p, a, s);
  if (D == 128 && B == 64) return launch_f32_db<128, 64>(p, a, s);
  return launch_f32_db<128, 128>(p, a, s);
}

}  // namespace tra
