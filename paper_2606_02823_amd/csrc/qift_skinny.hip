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
// unit's codes are loaded during this unit's MFMAs.  MNZ up to 32 tokens is decoded by bit plane into
// two accumulators (planes 0 and 3 at factor 1, planes 1 and 2 at factor 4); plane t's code operand
// is dword t of each of the four 16-byte code groups, a register selection.  From 33 tokens on every
// weight operand serves four token tiles and MNZ takes the plain decode (one accumulator, so that a
// workgroup holds four tiles: gate|up at 64 tokens 42.9 -> 25.0 us).  The K-slices meet in LDS; the
// code sums (when not given) come from the same code loads.
//
// Split over K (SPLIT, with a workspace): every workgroup reads all M x K codes, and the address unit
// that turns those loads into requests bounds this kernel (busy 81 % of the time for down at 64
// tokens), so a linear with K > 4096 and few 16-row tiles (down) takes four tiles per workgroup and
// gives each workgroup a range of K instead: workgroup (x, z) writes its int32 partial sums of tile
// group x over unit range z to the workspace, and the second pass (qift_split.h) adds the ranges (integers: exact in any
// order) and applies the epilogue (down at 64 tokens: 28.9 -> 16.4 us).
#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"
#include "qift_split.h"

namespace qift {
namespace {

using namespace mma;

constexpr int kSkSlices = 8;

// VGPRs of a lane's accumulators (MNZ by bit plane below four token tiles: two per tile pair), weight
// groups (U units of T tiles) and one unit's codes
template <int FMT, int T, int TT, int U>
constexpr int sk_regs() {
  return T * TT * (FMT == FMT_MNZ && TT < 4 ? 2 : 1) * 4 + U * T * (FMT == FMT_W4 ? 2 : 1) * 4 + TT * 16;
}
// a second code buffer (the next unit's loads in flight during this unit's MFMAs) where it fits
template <int FMT, int T, int TT, int U>
constexpr bool sk_double() { return sk_regs<FMT, T, TT, U>() + TT * 16 <= 224; }

template <int T, int TT>
constexpr size_t sk_shmem() { return (size_t)T * TT * kSkSlices * 64 * 16 + kSkSlices * 64 * 4; }

__device__ __forceinline__ uint32_t dw(const uint4& v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

// us: units (256 k) per K-range (all of K's units without SPLIT); with SPLIT, part receives the partial
// sums [ranges][M][np] and psum the code sums of each range [ranges][M] (when asum is null).
template <int FMT, int T, int TT, int U, bool SPLIT>
__global__ __launch_bounds__(64 * kSkSlices) void k_skinny(const uint32_t* __restrict__ P,
                                                           const uint16_t* __restrict__ sw, int N, int K,
                                                           const int8_t* __restrict__ act,
                                                           const float* __restrict__ sx,
                                                           const int32_t* __restrict__ asum, int M,
                                                           uint16_t* __restrict__ y, int32_t* __restrict__ acc_out,
                                                           int us, int np, int32_t* __restrict__ part,
                                                           int32_t* __restrict__ psum) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  // MNZ by bit plane (two accumulators) up to two token tiles; at four the plain decode (one
  // accumulator, the operand decoded once for four token tiles) lets a workgroup take four tiles
  constexpr bool PLANAR = FMT == FMT_MNZ && TT < 4;
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
  // this workgroup's units [ub, ue) of the row's UT, cut into 8 slices of NC (host: NC <= UM)
  const int zs = SPLIT ? (int)blockIdx.y : 0;
  const int UT = (K + 255) / 256;
  const int ub = zs * us, ue = ub + us < UT ? ub + us : UT;
  const int kend = ue * 256 < K ? ue * 256 : K;   // k past the range
  const int NC = (ue - ub + kSkSlices - 1) / kSkSlices;
  const int kq0 = (ub + slice * NC) * 256;

  // every weight group of the slice, up front (zeros for rows past N and k past K)
  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(P, (uint32_t)N * (uint32_t)rowbytes);
  uint4 w[UM][T][NH];
#pragma unroll
  for (int u = 0; u < UM; ++u)
#pragma unroll
    for (int j = 0; j < T; ++j) {
      const int n = (tile0 + j) * 16 + r16;
      const int k0 = kq0 + (u << 8) + (g << 6);
      const bool ok = u < NC && k0 < kend && n < N;
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
      const uint32_t base = u < NC && k0 < kend && m < M ? (uint32_t)m * (uint32_t)K + (uint32_t)k0 : dev::kOutOfRange;
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
    if constexpr (SPLIT) {
      if (m < M && n0 < np)
        *reinterpret_cast<int4*>(part + ((size_t)zs * M + m) * np + n0) = make_int4(D[0], D[1], D[2], D[3]);
      if (!asum && blockIdx.x == 0 && j == 0 && g == 0 && m < M) {   // the range's code sums, once
        int sq = 0;
#pragma unroll
        for (int q = 0; q < kSkSlices; ++q) sq += s_sum[q * 64 + m];
        psum[zs * M + m] = sq;
      }
    } else if (m < M && n0 < N) {
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
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_skinny<FMT, T, TT, U, false>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
  }
  const int64_t tiles = (N + 15) / 16;
  const int ut = (int)((K + 255) / 256);
  hipLaunchKernelGGL((k_skinny<FMT, T, TT, U, false>), dim3((unsigned)((tiles + T - 1) / T)), dim3(64 * kSkSlices),
                     shmem, s, P, sw, (int)N, (int)K, act, sx, asum, (int)M, y, acc_out, ut, 0, nullptr, nullptr);
  return hipGetLastError();
}

// (T, U): T tiles per workgroup, enough to keep the grid near one workgroup per CU (every workgroup
// reads all M x K codes), and U >= NC units, as far as the registers allow: at most 16 16-byte weight
// groups (U T, twice that for W4).
template <int FMT, int TT>
hipError_t launch_sk_tu(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                        const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                        hipStream_t s) {
  constexpr bool W4 = FMT == FMT_W4;
  const int64_t nc = (K + kSkSlices * 256 - 1) / (kSkSlices * 256);   // units per slice
  const int64_t want = ((N + 15) / 16 + 255) / 256;
#define QIFT_SK(T_, U_) launch_sk<FMT, T_, TT, U_>(P, sw, N, K, act, sx, asum, M, y, acc_out, s)
  if (nc <= 1 && want >= 3) return QIFT_SK(4, 1);
  if constexpr (!W4) {
    if (nc <= 2 && want >= 3) return QIFT_SK(4, 2);
  }
  if (nc <= 2 && want >= 2) return QIFT_SK(2, 2);
  if constexpr (!W4) {
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

// ---- split over K (W2 formats, with a workspace)

// The split of a linear: T = 4 tiles per workgroup, S ranges of us units each, chosen for about one
// workgroup per CU with at most two units per slice; S = 0 for K <= 4096 (the codes per workgroup are
// few enough: measured faster unsplit) and when a linear has tiles enough without a split (gate|up).
// Also for up to 16 tokens whose codes the decode kernel cannot stage in LDS (it would read them from
// memory per 16-row tile instead).
struct SkSplit {
  int T = 0, S = 0, us = 0, np = 0;
};

inline SkSplit split_plan(int fmt, int64_t N, int64_t K, int64_t M) {
  SkSplit p;
  if (fmt == FMT_W4 || M < 1 || M > kSkinnyMaxM || K > kSkinnyMaxK || N < 1 || K < 1) return p;
  const int T = 4;
  const int64_t tiles = (N + 15) / 16, gx = (tiles + T - 1) / T;
  const int ut = (int)((K + 255) / 256);
  if (ut <= 16) return p;
  int S = (int)((256 + gx / 2) / gx);
  if (S < 2) return p;
  const int min_s = (ut + kSkSlices * 2 - 1) / (kSkSlices * 2);   // at most two units per slice
  if (S < min_s) S = min_s;
  if (S > ut) S = ut;
  const int us = (ut + S - 1) / S;
  p.T = T;
  p.us = us;
  p.S = (ut + us - 1) / us;   // every range holds at least one unit
  p.np = (int)((N + 3) / 4 * 4);
  if (p.S < 2) p.S = 0;
  return p;
}

inline size_t split_part_bytes(const SkSplit& p, int64_t M, int64_t N) { return split::part_bytes(p.S, M, N); }

template <int FMT, int T, int TT>
hipError_t launch_split_t(const SkSplit& p, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K,
                          const int8_t* act, const float* sx, const int32_t* asum, int64_t M, uint16_t* y,
                          int32_t* acc_out, void* ws, hipStream_t s) {
  constexpr size_t shmem = sk_shmem<T, TT>();
  static_assert(shmem <= 160 * 1024, "LDS");
  if constexpr (shmem > 65536) {
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_skinny<FMT, T, TT, 2, true>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
  }
  int32_t* part = static_cast<int32_t*>(ws);
  int32_t* psum = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(ws) + split_part_bytes(p, M, N));
  const int64_t tiles = (N + 15) / 16;
  hipLaunchKernelGGL((k_skinny<FMT, T, TT, 2, true>), dim3((unsigned)((tiles + T - 1) / T), (unsigned)p.S),
                     dim3(64 * kSkSlices), shmem, s, P, sw, (int)N, (int)K, act, sx, asum, (int)M, y, acc_out, p.us,
                     p.np, part, psum);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // code sums of range z at psum[z M + m]
  return split::launch_sum<FMT>(part, p.S, M, N, sx, asum, psum, p.S, 1, (int)M, sw, y, acc_out, s);
}

template <int FMT>
hipError_t launch_split_fmt(const SkSplit& p, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K,
                            const int8_t* act, const float* sx, const int32_t* asum, int64_t M, uint16_t* y,
                            int32_t* acc_out, void* ws, hipStream_t s) {
#define QIFT_SPLIT(T_, TT_) launch_split_t<FMT, T_, TT_>(p, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s)
  if (M <= 32) return M <= 16 ? QIFT_SPLIT(4, 1) : QIFT_SPLIT(4, 2);
  return QIFT_SPLIT(4, 4);
#undef QIFT_SPLIT
}

}  // namespace

size_t skinny_workspace(int fmt, int64_t N, int64_t K, int64_t M) {
  if (M <= kCodesMaxM) {   // up to 16 tokens only where the decode kernel's LDS does not hold the codes
    const size_t cs = fmt == FMT_MNZ ? codes_shmem_mnz(M, N, K) : fmt == FMT_POT ? codes_shmem_pot(M, N, K) : 0;
    if (cs != 0 && cs <= 160 * 1024) return 0;
  }
  const SkSplit p = split_plan(fmt, N, K, M);
  if (p.S == 0) return 0;
  return split_part_bytes(p, M, N) + (size_t)p.S * (size_t)M * 4;
}

hipError_t launch_skinny_ws(int fmt, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                            const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out, void* ws,
                            hipStream_t s) {
  const SkSplit p = split_plan(fmt, N, K, M);
  if (ws == nullptr || p.S == 0) return launch_skinny(fmt, P, sw, N, K, act, sx, asum, M, y, acc_out, s);
  switch (fmt) {
    case FMT_MNZ: return launch_split_fmt<FMT_MNZ>(p, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s);
    case FMT_POT: return launch_split_fmt<FMT_POT>(p, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s);
    default: return launch_skinny(fmt, P, sw, N, K, act, sx, asum, M, y, acc_out, s);
  }
}

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
