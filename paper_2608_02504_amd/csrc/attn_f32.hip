// fp32 attention family (dense, block-sparse, fused entropy) for fp32
// workloads.  Scalar fp32 arithmetic with one thread per query row; the bf16
// path is the MFMA kernel.  One workgroup per query-block row.
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
  int N, NB, rows;
  float alpha;
};

constexpr int kSub = 32;  // keys staged in LDS at a time

template <int D, int B, bool SPARSE, bool PV, bool ENT>
__global__ __launch_bounds__(B) void attn_f32_kernel(F32Params P) {
  __shared__ float sK[kSub][D + 1];
  __shared__ float sV[PV ? kSub : 1][PV ? D + 1 : 1];

  int r = blockIdx.x;
  if (SPARSE && P.order) {
    r = P.order[blockIdx.x];
    if (r < 0 || r >= P.rows) return;  // whole workgroup leaves together
  }
  const int bh = r / P.NB, u = r - bh * P.NB;
  const int t = threadIdx.x;
  const int qpos = u * B + t;
  const bool qvalid = qpos < P.N;
  const int qrow = qvalid ? P.perm[qpos] : 0;
  const size_t head_off = (size_t)bh * P.N * D;

  float qr[D];
#pragma unroll
  for (int d = 0; d < D; ++d) qr[d] = qvalid ? P.q[head_off + (size_t)qrow * D + d] : 0.f;
  float acc[PV ? D : 1];
#pragma unroll
  for (int d = 0; d < (PV ? D : 1); ++d) acc[d] = 0.f;
  float m = -INFINITY, l = 0.f, a = 0.f;

  const int count = SPARSE ? min(max(P.cnt[r], 0), P.NB) : P.NB;
  for (int c = 0; c < count; ++c) {
    const int vb = SPARSE ? P.cols[(size_t)r * P.NB + c] : c;
    if (vb < 0 || vb >= P.NB) continue;  // uniform across the workgroup
    const int nv = min(B, P.N - vb * B);
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
      __syncthreads();
      float s[kSub];
      float mc = -INFINITY;
#pragma unroll
      for (int j = 0; j < kSub; ++j) {
        float dot = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) dot = fmaf(qr[d], sK[j][d], dot);
        s[j] = j < ns ? dot * P.alpha : -INFINITY;
        mc = fmaxf(mc, s[j]);
      }
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
  F32Params P{(const float*)a.q, (const float*)a.k, (const float*)a.v, (float*)a.o, a.lse,
              a.entropy, p.d_perm, a.cnt, a.cols, a.order, p.S, p.NB, p.rows,
              1.0f / sqrtf((float)D)};
  const dim3 grid(p.rows), block(B);
  if (a.sparse)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, true, true, false>), grid, block, 0, s, P);
  else if (a.entropy && a.o)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, false, true, true>), grid, block, 0, s, P);
  else if (a.entropy)
    hipLaunchKernelGGL((attn_f32_kernel<D, B, false, false, true>), grid, block, 0, s, P);
  else
    hipLaunchKernelGGL((attn_f32_kernel<D, B, false, true, false>), grid, block, 0, s, P);
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
