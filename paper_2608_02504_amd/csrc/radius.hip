// Entropy -> budget -> squared radius, one thread per (batch, head, token).
//
//  K_hat = ceil(tau * exp(H))                       Sec. 3.1, Eq. 8 (fp64)
//    or, lognormal mapping (App. A.2, Eq. lognormal_budget_appendix), with S keys
//    per row: K_hat = ceil(S * Phibar(sqrt(2 (log S - H)) - Phi^{-1}(tau)))
//  C(n)  = sum_t #{(x', y') in frame : (x-x')^2 + (y-y')^2 <= thr[n][|t-f|]}
//                                                   Sec. 3.2, Eq. 13
//  n     = min{n in [0, n_cap] : C(n) >= K_hat}, else FULL        Eq. 14
//
// The counts come from the lookup table of App. C.1 over query coordinate and
// radius: table[(f', x', y')][n] = C(n) for n in [0, n_cap], built once per
// plan.  C is symmetric under f -> F-1-f, x -> H-1-x and y -> W-1-y (the
// frame and the clip are), so the table covers one octant of the grid,
// ceil(F/2) x ceil(H/2) x ceil(W/2) positions (331 MB at 21 x 45 x 80).  It
// is filled from a per-frame disk-count table of one quadrant of the frame,
// and the search is a bisection on a monotone row of the table: 13 loads per
// query at n_cap = 8,177.  Plans whose table would exceed a size limit keep
// only C(n_cap) per position and count the other radii on the fly (exact
// lattice counts, row by row).  Counts are exact integers either way.
#include "tra_internal.h"

namespace tra {
namespace {

// floor(sqrt(v)) for 0 <= v < 2^24, exact.
__device__ __forceinline__ int isqrt_floor(int v) {
  int r = (int)sqrtf((float)v);
  while (r * r > v) --r;
  while ((r + 1) * (r + 1) <= v) ++r;
  return r;
}

// Lattice points (x', y') of an H x W frame with (x-x')^2 + (y-y')^2 <= T.
__device__ int disk_count(int x, int y, int T, int H, int W) {
  int w = isqrt_floor(T);                        // half-width of the row dx = 0
  const int dx_end = min(w, max(x, H - 1 - x));  // rows beyond |dx| > sqrt(T) are empty
  int total = 0;
  for (int dx = 0; dx <= dx_end; ++dx) {
    const int rem = T - dx * dx;
    while (w * w > rem) --w;                     // half-width shrinks as |dx| grows
    const int row = min(W - 1, y + w) - max(0, y - w) + 1;
    if (x + dx <= H - 1) total += row;
    if (dx > 0 && x - dx >= 0) total += row;
  }
  return total;
}

// C(n) of Eq. 13 for the query in frame f, with frame_disk(T) the lattice
// points of one frame within squared distance T of the query's (x, y).
template <typename DiskFn>
__device__ int grid_count_with(int f, int n, const int32_t* __restrict__ thr, int F, DiskFn frame_disk) {
  const int32_t* t = thr + (size_t)n * F;
  int total = 0;
  for (int d = 0; d < F; ++d) {
    const int mult = (f - d >= 0) + (d > 0 && f + d <= F - 1);  // frames at distance d
    if (mult == 0) break;                                       // no frame this far
    const int T = t[d];
    if (T == 0) {
      // thr is non-increasing in d: every frame at distance >= d keeps only the
      // query's own pixel position.
      const int closer = min(f, d - 1) + min(F - 1 - f, d - 1) + 1;  // frames at distance < d (d >= 1 here)
      total += F - (d == 0 ? 0 : closer);
      break;
    }
    total += mult * frame_disk(T);
  }
  return total;
}

__device__ int grid_count(int f, int x, int y, int n, const int32_t* __restrict__ thr, int F,
                          int H, int W) {
  return grid_count_with(f, n, thr, F, [&](int T) { return disk_count(x, y, T, H, W); });
}

// Disk counts of the positions of one quadrant of the frame, every squared
// radius: disk[((x * wh) + y) * (n_cap + 1) + T] for x < hh, y < wh.
__global__ __launch_bounds__(256) void disk_table_kernel(int32_t* __restrict__ disk, int H, int W, int hh, int wh,
                                                         int n_cap) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)hh * wh * (n_cap + 1)) return;
  const int T = (int)(i % (n_cap + 1));
  const int p = (int)(i / (n_cap + 1));
  disk[i] = disk_count(p / wh, p % wh, T, H, W);
}

// The count table over one octant of the grid: ctab[((f * hh + x) * wh + y) *
// (n_cap + 1) + n] = C(n) at (f, x, y), f < fh, x < hh, y < wh.
__global__ __launch_bounds__(256) void count_table_kernel(int32_t* __restrict__ ctab, const int32_t* __restrict__ disk,
                                                          const int32_t* __restrict__ thr, int F, int fh, int hh,
                                                          int wh, int n_cap) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)fh * hh * wh * (n_cap + 1)) return;
  const int n = (int)(i % (n_cap + 1));
  const long long p = i / (n_cap + 1);
  const int y = (int)(p % wh), x = (int)((p / wh) % hh), f = (int)(p / ((long long)wh * hh));
  const int32_t* drow = disk + (size_t)(x * wh + y) * (n_cap + 1);
  ctab[i] = grid_count_with(f, n, thr, F, [&](int T) { return drow[T]; });
}

// C(n_cap) of every video position (raster order), the count at the largest
// candidate radius: a query whose budget exceeds it gets the full radius.  A
// per-plan lookup table, filled once when the plan is created.
__global__ __launch_bounds__(256) void cap_count_kernel(const int32_t* __restrict__ thr, int32_t* __restrict__ out,
                                                        int N, int F, int H, int W, int n_cap) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  const int f = i / (H * W), x = (i / W) % H, y = i % W;
  out[i] = grid_count(f, x, y, n_cap, thr, F, H, W);
}

template <int MAP>
__global__ __launch_bounds__(256) void budget_radius_kernel(
    const float* __restrict__ entropy, int32_t* __restrict__ budget, int32_t* __restrict__ radius_sq,
    const int32_t* __restrict__ thr, const int32_t* __restrict__ cap_count, const int32_t* __restrict__ ctab,
    int total, int S, int N, int F, int H, int W, int n_cap, double tau, double z_tau) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int i = idx % S;  // token: raster index for video, >= N for text
  if (i >= N) {
    // text token: no radius (joint attention keeps its rows dense)
    if (budget) budget[idx] = S;
    radius_sq[idx] = TRA_RADIUS_FULL;
    return;
  }
  const double h = (double)entropy[idx];
  double kd;
  if (h != h) {
    kd = h;  // NaN entropy: keep everything (below)
  } else if (MAP == TRA_BUDGET_LOGNORMAL) {
    const double sigma = sqrt(2.0 * fmax(0.0, log((double)S) - h));
    kd = ceil((double)S * (0.5 * erfc((sigma - z_tau) * 0.70710678118654752)));
  } else {
    kd = ceil(tau * exp(h));
  }
  int khat;
  if (kd != kd || kd >= (double)S) khat = S;  // NaN entropy: keep everything
  else if (kd < 1.0) khat = 1;
  else khat = (int)kd;
  if (budget) budget[idx] = khat;

  const int f = i / (H * W), x = (i / W) % H, y = i % W;
  // this position's row of the count table (its octant image), if the plan has one
  const int32_t* crow = nullptr;
  if (ctab) {
    const int hh = (H + 1) >> 1, wh = (W + 1) >> 1;
    const int fq = min(f, F - 1 - f), xq = min(x, H - 1 - x), yq = min(y, W - 1 - y);
    crow = ctab + ((size_t)(fq * hh + xq) * wh + yq) * (n_cap + 1);
  }
  int n;
  const int c_cap = crow ? crow[n_cap] : cap_count[i];
  if (khat <= F) {
    n = 0;  // C(0) = F: the query's own position in every frame
  } else if (c_cap < khat) {
    n = TRA_RADIUS_FULL;
  } else {
    // Smallest n with C(n) >= khat by bisection: C(0) = F < khat, and
    // C(n_cap) >= khat.
    int lo = 0, hi = n_cap;
    while (hi - lo > 1) {
      const int mid = lo + ((hi - lo) >> 1);
      const int c = crow ? crow[mid] : grid_count(f, x, y, mid, thr, F, H, W);
      if (c >= khat) hi = mid;
      else lo = mid;
    }
    n = hi;
  }
  radius_sq[idx] = n;
}

}  // namespace

size_t count_table_bytes(const tra_plan_s& p) {
  const size_t fh = (p.cfg.frames + 1) / 2, hh = (p.cfg.height + 1) / 2, wh = (p.cfg.width + 1) / 2;
  return fh * hh * wh * ((size_t)p.n_cap + 1) * sizeof(int32_t);
}

hipError_t fill_count_table(const tra_plan_s& p, int32_t* ctab, int32_t* disk_tmp, hipStream_t s) {
  const int F = p.cfg.frames, H = p.cfg.height, W = p.cfg.width;
  const int fh = (F + 1) / 2, hh = (H + 1) / 2, wh = (W + 1) / 2;
  const long long nd = (long long)hh * wh * (p.n_cap + 1);
  const long long nc = (long long)fh * nd;
  hipLaunchKernelGGL(disk_table_kernel, dim3((unsigned)((nd + 255) / 256)), dim3(256), 0, s, disk_tmp, H, W, hh, wh,
                     p.n_cap);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(count_table_kernel, dim3((unsigned)((nc + 255) / 256)), dim3(256), 0, s, ctab, disk_tmp,
                     p.d_thr, F, fh, hh, wh, p.n_cap);
  return hipGetLastError();
}

hipError_t fill_cap_counts(const tra_plan_s& p, int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(cap_count_kernel, dim3((p.N + 255) / 256), dim3(256), 0, s, p.d_thr, out, p.N,
                     p.cfg.frames, p.cfg.height, p.cfg.width, p.n_cap);
  return hipGetLastError();
}

hipError_t launch_budget_radius(const tra_plan_s& p, const float* entropy, int32_t* budget,
                                int32_t* radius_sq, hipStream_t s) {
  const int total = p.cfg.batch * p.cfg.heads * p.S;
  const int threads = 256;
  const dim3 grid((total + threads - 1) / threads);
  if (p.cfg.budget_map == TRA_BUDGET_LOGNORMAL)
    hipLaunchKernelGGL(budget_radius_kernel<TRA_BUDGET_LOGNORMAL>, grid, dim3(threads), 0, s, entropy,
                       budget, radius_sq, p.d_thr, p.d_cap_count, p.d_ctab, total, p.S, p.N, p.cfg.frames,
                       p.cfg.height, p.cfg.width, p.n_cap, p.cfg.tau, p.z_tau);
  else
    hipLaunchKernelGGL(budget_radius_kernel<TRA_BUDGET_UNIFORM>, grid, dim3(threads), 0, s, entropy,
                       budget, radius_sq, p.d_thr, p.d_cap_count, p.d_ctab, total, p.S, p.N, p.cfg.frames,
                       p.cfg.height, p.cfg.width, p.n_cap, p.cfg.tau, p.z_tau);
  return hipGetLastError();
}

}  // namespace tra
