// Skinny decode linear: y = s_w[n] s_x[m] sum_k level[n,k] q[m,k] for a few dozen tokens (Sec. 1: the
// decode regime streams the packed weights; Sec. 3.6: small signed integer levels, exact int32
// accumulation on the int8 MFMA), in one pass over the weights.
//
// The 16-token decode kernel stages every token's codes in LDS, which holds at most 16 tokens of
// K = 4096 (fewer for longer K); beyond that the weights would have to stream once per block of
// tokens.  Here every weight byte is read once: a workgroup owns T 16-row tiles, its 8 waves cut K
// into 8 slices, and each wave issues all of its slice's weight loads at once, then walks its 256-k
// units.  Per unit a lane reads the 64 codes of its k-group for each of its TT token tiles (token
// 16 tt + lane mod 16) straight from memory (they stay in the L2: every workgroup reads the same
// M x K codes), decodes each weight operand once and applies it to the TT token tiles.  The next
// unit's codes are loaded during this unit's MFMAs.  MNZ is decoded by bit plane into two
// accumulators (planes 0 and 3 at factor 1, planes 1 and 2 at factor 4); plane t's code operand is
// dword t of each of the four 16-byte code groups, a register selection.  The K-slices meet in LDS;
// the code sums (when not given) come from the same code loads.
#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"

namespace qift {
namespace {

using namespace mma;

constexpr int kSkSlices = 8;

// VGPRs of a lane's accumulators, weight groups (U units of T tiles) and one unit's codes
template <int FMT, int T, int TT, int U>
constexpr int sk_regs() { return T * TT * (FMT == FMT_MNZ ? 2 : 1) * 4 + U * T * (FMT == FMT_W4 ? 2 : 1) * 4 + TT * 16; }
// a second code buffer (the next unit's loads in flight during this unit's MFMAs) where it fits
template <int FMT, int T, int TT, int U>
constexpr bool sk_double() { return sk_regs<FMT, T, TT, U>() + TT * 16 <= 224; }

template <int T, int TT>
constexpr size_t sk_shmem() { return (size_t)T * TT * kSkSlices * 64 * 16 + kSkSlices * 64 * 4; }

__device__ __forceinline__ uint32_t dw(const uint4& v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

template <int FMT, int T, int TT, int U>
__global__ __launch_bounds__(64 * kSkSlices) void k_skinny(const uint32_t* __restrict__ P,
                                                           const uint16_t* __restrict__ sw, int N, int K,
                                                           const int8_t* __restrict__ act,
                                                           const float* __restrict__ sx,
                                                           const int32_t* __restrict__ asum, int M,
                                                           uint16_t* __restrict__ y, int32_t* __restrict__ acc_out) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr bool PLANAR = FMT == FMT_MNZ;
  constexpr int NA = PLANAR ? 2 : 1;
  constexpr int UM = U;   // units per slice (the host picks U >= NC)
  constexpr bool DB = sk_double<FMT, T, TT, U>();
  extern __shared__ __align__(16) unsigned char smem[];
  v4i* red = reinterpret_cast<v4i*>(smem);                                        // [T][TT][slices][64]
  int* s_sum = reinterpret_cast<int*>(smem + (size_t)T * TT * kSkSlices * 64 * 16);   // [slices][64]

  const int tid = threadIdx.x, lane = tid & 63;
  const int slice = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int tile0 = blockIdx.x * T;
  const int rowbytes = FMT == FMT_W4 ? K / 2 : K / 4;
  const int NC = (K + kSkSlices * 256 - 1) / (kSkSlices * 256);   // units per slice (host: NC <= UM)
  const int kq0 = slice * NC * 256;

  // every weight group of the slice, up front (zeros for rows past N and k past K)
  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(P, (uint32_t)N * (uint32_t)rowbytes);
  uint4 w[UM][T][NH];
#pragma unroll
  for (int u = 0; u < UM; ++u)
#pragma unroll
    for (int j = 0; j < T; ++j) {
      const int n = (tile0 + j) * 16 + r16;
      const int k0 = kq0 + (u << 8) + (g << 6);
      const bool ok = u < NC && k0 < K && n < N;
      const uint32_t off = ok ? (uint32_t)n * (uint32_t)rowbytes + (uint32_t)(FMT == FMT_W4 ? k0 / 2 : k0 / 4)
                              : dev::kOutOfRange;
#pragma unroll
      for (int h = 0; h < NH; ++h) w[u][j][h] = dev::bload16(wrs, off + 16 * h);
    }

  // the lane's 64 codes of unit u for each token tile (zeros for tokens past M and k past K)
  const __amdgpu_buffer_rsrc_t ars = dev::make_rsrc(act, (uint32_t)M * (uint32_t)K);
  auto load_b = [&](int u, uint4 (&b)[TT][4]) {
    const int k0 = kq0 + (u << 8) + (g << 6);
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int m = 16 * tt + r16;
      const uint32_t base = u < NC && k0 < K && m < M ? (uint32_t)m * (uint32_t)K + (uint32_t)k0 : dev::kOutOfRange;
#pragma unroll
      for (int i = 0; i < 4; ++i) b[tt][i] = dev::bload16(ars, base + 16 * i);
    }
  };

  v4i acc[T][TT][NA];
#pragma unroll
  for (int j = 0; j < T; ++j)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
      for (int a = 0; a < NA; ++a) acc[j][tt][a] = v4i{0, 0, 0, 0};
  int qs[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) qs[tt] = 0;

  uint4 bq[DB ? 2 : 1][TT][4];
  load_b(0, bq[0]);
#pragma unroll
  for (int u = 0; u < UM; ++u) {
    if (u < NC) {   // wave-uniform
      if (DB && u + 1 < UM && u + 1 < NC) load_b(u + 1, bq[(u + 1) & 1]);   // in flight during this unit
      const uint4(&b)[TT][4] = bq[DB ? (u & 1) : 0];
      if (!asum) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
          for (int i = 0; i < 4; ++i) qs[tt] = sum16_i8(b[tt][i], qs[tt]);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        v4i bop[TT];
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) {
          if constexpr (PLANAR)   // plane s: codes of k = 16 i + 4 s + (0..3) of group i
            bop[tt] = v4i{(int)dw(b[tt][0], s), (int)dw(b[tt][1], s), (int)dw(b[tt][2], s), (int)dw(b[tt][3], s)};
          else
            bop[tt] = v4i{(int)b[tt][s].x, (int)b[tt][s].y, (int)b[tt][s].z, (int)b[tt][s].w};
        }
#pragma unroll
        for (int j = 0; j < T; ++j) {
          const v4i a = PLANAR ? decode_plane2(w[u][j][0], s) : decode_unit<FMT>(w[u][j], s);
#pragma unroll
          for (int tt = 0; tt < TT; ++tt) {
            const int ai = PLANAR && (s == 1 || s == 2) ? 1 : 0;
            acc[j][tt][ai] = mfma_i8(a, bop[tt], acc[j][tt][ai]);
          }
        }
      }
      // one buffer: the next unit's codes are requested once this unit's MFMAs have their operands
      if (!DB && u + 1 < UM && u + 1 < NC) load_b(u + 1, bq[0]);
    }
  }

  // the K-slices meet in LDS; per token, the code sums of the slice (the four k-groups added)
#pragma unroll
  for (int j = 0; j < T; ++j)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      v4i sacc = acc[j][tt][0];
      if constexpr (PLANAR) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sacc[r] += acc[j][tt][1][r] >> 2;   // exact: 4 times an integer sum
      }
      red[((j * TT + tt) * kSkSlices + slice) * 64 + lane] = sacc;
    }
  if (!asum) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      int v = qs[tt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) s_sum[slice * 64 + 16 * tt + lane] = v;
    }
  }
  __syncthreads();
  for (int p = slice; p < T * TT; p += kSkSlices) {   // wave-uniform
    const int j = p / TT, tt = p - j * TT;
    v4i D = red[(p * kSkSlices) * 64 + lane];
#pragma unroll
    for (int q = 1; q < kSkSlices; ++q) D += red[(p * kSkSlices + q) * 64 + lane];
    const int m = 16 * tt + r16, n0 = (tile0 + j) * 16 + 4 * g;
    if (m < M && n0 < N) {
      int sq;
      if (asum) {
        sq = asum[m];
      } else {
        sq = 0;
#pragma unroll
        for (int q = 0; q < kSkSlices; ++q) sq += s_sum[q * 64 + m];
      }
      store4<FMT>(D, m, n0, N, sx[m], sq, sw, y, acc_out);
    }
  }
}

template <int FMT, int T, int TT, int U>
hipError_t launch_sk(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act, const float* sx,
                     const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out, hipStream_t s) {
  constexpr size_t shmem = sk_shmem<T, TT>();
  static_assert(shmem <= 160 * 1024, "LDS");
  if constexpr (shmem > 65536) {
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_skinny<FMT, T, TT, U>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
  }
  const int64_t tiles = (N + 15) / 16;
  hipLaunchKernelGGL((k_skinny<FMT, T, TT, U>), dim3((unsigned)((tiles + T - 1) / T)), dim3(64 * kSkSlices), shmem, s,
                     P, sw, (int)N, (int)K, act, sx, asum, (int)M, y, acc_out);
  return hipGetLastError();
}

// (T, U): T tiles per workgroup, enough to keep the grid near one workgroup per CU (every workgroup
// reads all M x K codes), and U >= NC units, as far as the registers allow: at most 16 16-byte weight
// groups (U T, twice that for W4), and for MNZ at four token tiles (two accumulators each) neither
// (4, 2) nor (2, 4) (measured to spill).
template <int FMT, int TT>
hipError_t launch_sk_tu(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                        const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                        hipStream_t s) {
  constexpr bool W4 = FMT == FMT_W4;
  constexpr bool wide = FMT == FMT_MNZ && TT == 4;
  const int64_t nc = (K + kSkSlices * 256 - 1) / (kSkSlices * 256);   // units per slice
  const int64_t want = ((N + 15) / 16 + 255) / 256;
#define QIFT_SK(T_, U_) launch_sk<FMT, T_, TT, U_>(P, sw, N, K, act, sx, asum, M, y, acc_out, s)
  if (nc <= 1 && want >= 3) return QIFT_SK(4, 1);
  if constexpr (!W4 && !wide) {
    if (nc <= 2 && want >= 3) return QIFT_SK(4, 2);
  }
  if (nc <= 2 && want >= 2) return QIFT_SK(2, 2);
  if constexpr (!W4 && !wide) {
    if (nc <= 4 && want >= 2) return QIFT_SK(2, 4);
  }
  if (nc <= 2) return QIFT_SK(1, 2);
  if (nc <= 4) return QIFT_SK(1, 4);
  return QIFT_SK(1, 8);
#undef QIFT_SK
}

template <int FMT>
hipError_t launch_skinny_fmt(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                             const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                             hipStream_t s) {
  if (M < 1 || M > kSkinnyMaxM || K > kSkinnyMaxK) return hipErrorInvalidValue;
  if (M <= 16) return launch_sk_tu<FMT, 1>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
  if (M <= 32) return launch_sk_tu<FMT, 2>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
  return launch_sk_tu<FMT, 4>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
}

}  // namespace

hipError_t launch_skinny(int fmt, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                         const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                         hipStream_t s) {
  switch (fmt) {
    case mma::FMT_MNZ: return launch_skinny_fmt<mma::FMT_MNZ>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
    case mma::FMT_POT: return launch_skinny_fmt<mma::FMT_POT>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
    case mma::FMT_W4: return launch_skinny_fmt<mma::FMT_W4>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qift
