// Ratio scan of the mirror family G(r) = {-1, -r, +r, +1} (Sec. 3.4 Eq. (18); the sensitivity study of
// Sec. 4.5.3): for samples x[0..n) (pooled rotated weights), every ratio r_i and every clip candidate
// c_j,
//   s       = c_j * max|x|,
//   level   = sign(x) * (1 if |x / s| > (1 + r_i) / 2 else r_i)   (zero positive),
//   sse[i][j] = sum (x - s * level)^2,
// then per ratio the first minimiser best[i] over j and nmse[i] = sse[i][best[i]] / sum x^2.
//
// Every term is formed with the same rounded fp64 operations in the same order as the definition
// (quotient, threshold compare, product, difference, square; no fused multiply-add), so each term is
// the same number on any IEEE fp64 machine; only the order of the n-term sums is this kernel's
// (a fixed tree, the same on every run).
//
// Three launches: the statistics (max|x|, sum x^2) by one workgroup, the squared errors by one
// workgroup per (ratio, candidate) reading x from the L2 (a diagnostic over ~10^5 samples: the
// quotient, not the bandwidth, bounds it), the per-ratio minimum by one thread per ratio.  The
// ratios and candidates travel as kernel arguments (a chunk of kScanRatiosPerLaunch ratios per
// launch), so the call needs no device copies and no scratch.
#include <hip/hip_runtime.h>

#include "qift_internal.h"

namespace qift {
namespace {

constexpr int kStatThreads = 1024, kSseThreads = 256;

struct ScanTable {
  double r[kScanRatiosPerLaunch];
  double c[kScanMaxCands];
};

template <int NT>
__device__ __forceinline__ double block_reduce(double v, double* red, bool is_max) {
  const int t = threadIdx.x;
  red[t] = v;
  __syncthreads();
#pragma unroll
  for (int h = NT / 2; h > 0; h >>= 1) {
    if (t < h) red[t] = is_max ? fmax(red[t], red[t + h]) : red[t] + red[t + h];
    __syncthreads();
  }
  const double out = red[0];
  __syncthreads();
  return out;
}

__global__ __launch_bounds__(kStatThreads) void k_scan_stats(const double* __restrict__ x, int64_t n,
                                                            double* __restrict__ stats) {
#pragma clang fp contract(off)
  __shared__ double red[kStatThreads];
  double a = 0.0, ss = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += kStatThreads) {
    const double v = x[i];
    a = fmax(a, fabs(v));
    ss += v * v;
  }
  a = block_reduce<kStatThreads>(a, red, true);
  ss = block_reduce<kStatThreads>(ss, red, false);
  if (threadIdx.x == 0) {
    stats[0] = a;
    stats[1] = ss;
  }
}

// workgroup (candidate j, ratio i0 + blockIdx.y)
__global__ __launch_bounds__(kSseThreads) void k_scan_sse(const double* __restrict__ x, int64_t n,
                                                         const double* __restrict__ stats, ScanTable tab, int i0,
                                                         int n_cands, double* __restrict__ sse) {
#pragma clang fp contract(off)
  __shared__ double red[kSseThreads];
  const int j = blockIdx.x, ii = blockIdx.y;
  const double r = tab.r[ii];
  const double a = stats[0];
  const double s = tab.c[j] * a;
  const double thr = 0.5 * (r + 1.0);
  double acc = 0.0;
  if (a > 0.0) {
    for (int64_t k = threadIdx.x; k < n; k += kSseThreads) {
      const double v = x[k];
      const double u = v / s;
      const double mag = fabs(u) > thr ? 1.0 : r;
      const double lev = u >= 0.0 ? mag : -mag;
      const double p = s * lev;
      const double d = v - p;
      acc += d * d;
    }
  }
  acc = block_reduce<kSseThreads>(acc, red, false);
  if (threadIdx.x == 0) sse[(int64_t)(i0 + ii) * n_cands + j] = acc;
}

__global__ void k_scan_best(const double* __restrict__ sse, const double* __restrict__ stats, int n_ratios,
                            int n_cands, double* __restrict__ nmse, int32_t* __restrict__ best) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_ratios) return;
  const double* row = sse + (int64_t)i * n_cands;
  int bj = 0;
  double be = row[0];
  for (int j = 1; j < n_cands; ++j)
    if (row[j] < be) {
      be = row[j];
      bj = j;
    }
  best[i] = bj;
  const double ss = stats[1];
  nmse[i] = ss > 0.0 ? be / ss : 0.0;
}

}  // namespace

hipError_t launch_ratio_scan(const double* x, int64_t n, const double* ratios, int n_ratios, const double* cands,
                             int n_cands, double* sse, double* nmse, int32_t* best, double* stats, hipStream_t s) {
  hipLaunchKernelGGL(k_scan_stats, dim3(1), dim3(kStatThreads), 0, s, x, n, stats);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  ScanTable tab;
  for (int j = 0; j < kScanMaxCands; ++j) tab.c[j] = j < n_cands ? cands[j] : 0.0;
  for (int i0 = 0; i0 < n_ratios; i0 += kScanRatiosPerLaunch) {
    const int cnt = n_ratios - i0 < kScanRatiosPerLaunch ? n_ratios - i0 : kScanRatiosPerLaunch;
    for (int i = 0; i < kScanRatiosPerLaunch; ++i) tab.r[i] = i < cnt ? ratios[i0 + i] : 0.0;
    hipLaunchKernelGGL(k_scan_sse, dim3((unsigned)n_cands, (unsigned)cnt), dim3(kSseThreads), 0, s, x, n, stats,
                       tab, i0, n_cands, sse);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_scan_best, dim3((unsigned)((n_ratios + 63) / 64)), dim3(64), 0, s, sse, stats, n_ratios,
                     n_cands, nmse, best);
  return hipGetLastError();
}

}  // namespace qift
