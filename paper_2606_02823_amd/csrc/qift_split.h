// The second pass of a linear split over K: the int32 partial sums of S K-ranges, written by the
// first pass to a caller workspace as [S][M][np] (np = N rounded up to 4), are added and the epilogue
// of Sec. 1 applied.  The sums are integers, so the order of the additions changes nothing.
#pragma once

#include "qift_mma.h"

namespace qift {
namespace split {

inline int64_t round4(int64_t n) { return (n + 3) / 4 * 4; }

// Bytes of the partial sums, 256-byte aligned so that what follows them in a workspace is too.
inline size_t part_bytes(int S, int64_t M, int64_t N) {
  return ((size_t)S * (size_t)M * (size_t)round4(N) * 4 + 255) / 256 * 256;
}

// One thread per 4 outputs of a token.  The partial sums were written by workgroups on every XCD and
// come from past the L2, so a thread issues its loads (scales, code sums, four ranges at a time)
// before it uses any of them.  The per-token code sums are asum[m] when given, else the ps_n values
// psum[m * ps_m + p * ps_p], p < ps_n.
template <int FMT>
__global__ __launch_bounds__(64) void k_split_sum(const int32_t* __restrict__ part, int S, int M, int N,
                                                  const float* __restrict__ sx, const int32_t* __restrict__ asum,
                                                  const int32_t* __restrict__ psum, int ps_n, int ps_m, int ps_p,
                                                  const uint16_t* __restrict__ sw, uint16_t* __restrict__ y,
                                                  int32_t* __restrict__ acc_out) {
  const int np = (N + 3) & ~3, nq = np / 4;
  const int q = blockIdx.x * 64 + threadIdx.x;
  if (q >= M * nq) return;
  const int m = q / nq, n0 = (q - m * nq) * 4;
  const float s_x = sx[m];
  uint2 swq;
  if (n0 + 3 < N) {
    swq = *reinterpret_cast<const uint2*>(sw + n0);   // s_w is 16-byte aligned, n0 a multiple of 4
  } else {
    uint32_t h[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) h[r] = n0 + r < N ? sw[n0 + r] : 0u;
    swq = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
  }
  int sq = 0;
  if (asum) {
    sq = asum[m];
  } else {
    const int32_t* __restrict__ pm = psum + (size_t)m * ps_m;
    int p = 0;
    for (; p + 4 <= ps_n; p += 4) {
      int c[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) c[i] = pm[(p + i) * ps_p];
      sq += (c[0] + c[1]) + (c[2] + c[3]);
    }
    for (; p < ps_n; ++p) sq += pm[p * ps_p];
  }
  const int32_t* __restrict__ pz = part + (size_t)m * np + n0;
  const size_t zs = (size_t)M * np;
  mma::v4i D = mma::v4i{0, 0, 0, 0};
  int z = 0;
  for (; z + 4 <= S; z += 4) {
    int4 v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = *reinterpret_cast<const int4*>(pz + (size_t)(z + i) * zs);
#pragma unroll
    for (int i = 0; i < 4; ++i) D += mma::v4i{v[i].x, v[i].y, v[i].z, v[i].w};
  }
  for (; z < S; ++z) {
    const int4 v = *reinterpret_cast<const int4*>(pz + (size_t)z * zs);
    D += mma::v4i{v.x, v.y, v.z, v.w};
  }
  mma::store4_sw<FMT>(D, m, n0, N, s_x, sq, swq, y, acc_out);
}

template <int FMT>
hipError_t launch_sum(const int32_t* part, int S, int64_t M, int64_t N, const float* sx, const int32_t* asum,
                      const int32_t* psum, int ps_n, int ps_m, int ps_p, const uint16_t* sw, uint16_t* y,
                      int32_t* acc_out, hipStream_t s) {
  const int64_t quads = M * (round4(N) / 4);
  hipLaunchKernelGGL((k_split_sum<FMT>), dim3((unsigned)((quads + 63) / 64)), dim3(64), 0, s, part, S, (int)M,
                     (int)N, sx, asum, psum, ps_n, ps_m, ps_p, sw, y, acc_out);
  return hipGetLastError();
}

}  // namespace split
}  // namespace qift
