// Offline weight quantizer: the step before packing.
//
// Per output row n of W [N][K] (fp32):
//   W_rot[n, :] = (I_{K/b} (x) H_b) W[n, :] / sqrt(b)      (Sec. 3.1, fp64)
// then one scale per row and the nearest level of the format's set against the
// stored fp16 scale (Sec. 3.3, Sec. 3.5, Sec. 4.5.1):
//   MNZ  s = RMS(W_rot[n, :]), s_w = fp16(s / 2), level in {-3,-1,+1,+3} by
//        the midpoints 0 and +-2 of u = w / s_w (Eqs. (13)-(14));
//   PoT  s_w = fp16 of the first minimiser, over the 64 candidates
//        linspace(0.2, 1, 64) * max|row| / 4, of sum (w - s * level(w, s))^2,
//        level in {-4,-1,+1,+4} by |u| > 5/2 (Eq. (17));
//   W4   s_w = fp16(max|row| / 7), q = clip(rne(w / s_w), -7, 7) (Eq. (1));
//   G(r) the mirror family {-1, -r, +r, +1} (Sec. 3.4 Eq. (18)) with the PoT scale search (outer
//        level 1: candidates linspace(0.2, 1, 64) * max|row|), the outer level where |u| > (1 + r) / 2;
//        written as codes 0..3 of the ascending levels (the level-table linear's input).
// Readings: a value on a midpoint takes the inner level, zero the positive one;
// a row whose stored scale is 0 gets level +1 (W2) or 0 (W4).
//
// One 256-thread workgroup per row; thread t holds elements 16 t .. 16 t + 15
// of every 4096-element tile in fp64 registers, rotated with the butterfly
// kernels of the activation quantizer (natural layout in and out).  The
// rotation is not exact for arbitrary fp32 rows, so its last bits depend on
// the summation order; the level and scale decisions are the paper's, taken
// in fp64 on these values.
#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"

namespace qift {
using mma::FMT_MNZ;
using mma::FMT_POT;
using mma::FMT_W4;
namespace {

constexpr int FMT_MIRROR = 3;   // G(r): a run-time inner level r, codes out

// fp64 -> IEEE binary16 bits, round to nearest, ties to even, overflow to infinity (from the bit
// fields: 10 fraction bits kept, the rest rounded; below 2^-14 in units of 2^-24).
__device__ __forceinline__ uint16_t half_bits_rne(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  const uint64_t a = b & 0x7FFFFFFFFFFFFFFFull;
  if (a >= 0x7FF0000000000000ull) return sign | (a > 0x7FF0000000000000ull ? 0x7E00u : 0x7C00u);
  const int E = (int)(a >> 52) - 1023;
  if (E < -26) return sign;   // below 2^-26: under half of the smallest subnormal
  const uint64_t m = (a & 0xFFFFFFFFFFFFFull) | 0x10000000000000ull;   // value = m * 2^(E - 52)
  if (E > 15) return sign | 0x7C00u;
  uint64_t r, rem, half;
  if (E < -14) {
    const int sh = 28 - E;   // value / 2^-24 = m >> sh
    r = m >> sh;
    rem = m & ((1ull << sh) - 1);
    half = 1ull << (sh - 1);
  } else {
    r = ((uint64_t)(E + 15) << 10) | ((m >> 42) & 0x3FFu);
    rem = m & ((1ull << 42) - 1);
    half = 1ull << 41;
  }
  if (rem > half || (rem == half && (r & 1))) ++r;   // a carry runs into the exponent; 0x7C00 is infinity
  return sign | (uint16_t)r;
}

__device__ __forceinline__ double half_value(uint16_t h) { return (double)__half2float(__ushort_as_half(h)); }

// Candidate c_j of the PoT scale search: j * (0.8 / 63) + 0.2, the last one exactly 1
__device__ __forceinline__ double pot_candidate(int j) {
  const double step = (1.0 - 0.2) / 63.0;
  return j == 63 ? 1.0 : (double)j * step + 0.2;
}

// sum over a wave in a fixed order (quads, half rows, rows, then the four rows); every lane gets it
__device__ __forceinline__ double wave_sum_f64(double x) {
  x += QIFT_DPP_F64(x, 0xb1);    // quad_perm [1,0,3,2]
  x += QIFT_DPP_F64(x, 0x4e);    // quad_perm [2,3,0,1]
  x += QIFT_DPP_F64(x, 0x141);   // row_half_mirror
  x += QIFT_DPP_F64(x, 0x140);   // row_mirror: every lane of a row holds the row's sum
  auto row = [&](int l) {
    return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(x), l),
                            __builtin_amdgcn_readlane(__double2loint(x), l));
  };
  return (row(0) + row(16)) + (row(32) + row(48));
}

// sum of a per-thread fp64 value over the workgroup; red holds 4 doubles; all threads get the sum
__device__ __forceinline__ double group_sum(double v, double* red) {
  v = wave_sum_f64(v);
  __syncthreads();   // red is free
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// The stored value of a two-magnitude set: MNZ levels +-1 / +-3, PoT +-1 / +-4, G(r) the codes
// 1 / 0 (negative) and 2 / 3 (positive) of the ascending levels -1, -r, +r, +1.
template <int FMT>
__device__ __forceinline__ int level_of(bool nonneg, bool outer) {
  if constexpr (FMT == FMT_MIRROR) return nonneg ? (outer ? 3 : 2) : (outer ? 0 : 1);
  const int mag = outer ? (FMT == FMT_MNZ ? 3 : 4) : 1;
  return nonneg ? mag : -mag;
}

template <int FMT, int NTILES, int LC>
__global__ __launch_bounds__(256) void k_quant_weights(const float* __restrict__ W, int K, int L_rt, double sqrtb,
                                                       double rin, int8_t* __restrict__ levels,
                                                       uint16_t* __restrict__ scales) {
  using S = dev::Tile<256, 16>;
  __shared__ double xch[S::LDS_DOUBLES];
  __shared__ double red[4];
  __shared__ double red64[4][64];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int L = LC > 0 ? LC : L_rt;
  const int64_t n = blockIdx.x;

  // ---- load (a thread's 16 elements of a tile are all below K or all past it: K % 64 == 0)
  double v[NTILES][16];
  bool valid[NTILES];
  {
    const __amdgpu_buffer_rsrc_t r = dev::make_rsrc(W + n * K, (uint32_t)K * 4u);
#pragma unroll
    for (int tau = 0; tau < NTILES; ++tau) {
      const int base = tau * S::T + 16 * t;
      valid[tau] = base < K;
      const uint32_t off = valid[tau] ? (uint32_t)base * 4u : dev::kOutOfRange;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint4 d = dev::bload16(r, off + 16u * c);
        v[tau][4 * c + 0] = (double)__uint_as_float(d.x);
        v[tau][4 * c + 1] = (double)__uint_as_float(d.y);
        v[tau][4 * c + 2] = (double)__uint_as_float(d.z);
        v[tau][4 * c + 3] = (double)__uint_as_float(d.w);
      }
    }
  }
  // ---- rotate every block of b (blocks past K are zeros and stay zeros), then / sqrt(b)
  dev::BlockSync sync;
  // sqrt(b) a power of two (b = 4^k): dividing by it is the exact product with its reciprocal
  int sqe;
  const bool sq_pow2 = frexp(sqrtb, &sqe) == 0.5;
  const double inv_sqrtb = 1.0 / sqrtb;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    if (tau > 0) __syncthreads();   // the previous tile's last exchange reads are done
    dev::fwht_tile_s<256, 16, true>(v[tau], xch, t, L, sync);
    if (sq_pow2) {
#pragma unroll
      for (int e = 0; e < 16; ++e) v[tau][e] = v[tau][e] * inv_sqrtb;
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) v[tau][e] = v[tau][e] / sqrtb;
    }
  }

  // ---- scale
  double amax = 0.0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau)
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[tau][e]));   // zeros past K change nothing
  uint16_t sw = 0;
  if constexpr (FMT == FMT_MNZ) {
    double ss = 0.0;
#pragma unroll
    for (int tau = 0; tau < NTILES; ++tau)
#pragma unroll
      for (int e = 0; e < 16; ++e) ss += v[tau][e] * v[tau][e];
    const double s = sqrt(group_sum(ss, red) / (double)K);
    sw = half_bits_rne(s / 2.0);
  } else if constexpr (FMT == FMT_W4) {
    amax = dev::wave_max(amax);
    __syncthreads();
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    const double a = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
    sw = half_bits_rne(a / 7.0);
  } else {
    amax = dev::wave_max(amax);
    __syncthreads();
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    const double a = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
    // PoT: levels 1, 4 at s = c max / 4, midpoint 5/2; G(r): levels r, 1 at s = c max, midpoint (1 + r) / 2
    const double thr = FMT == FMT_MIRROR ? 0.5 * (rin + 1.0) : 2.5;
    const double m_in = FMT == FMT_MIRROR ? rin : 1.0, m_out = FMT == FMT_MIRROR ? 1.0 : 4.0;
    if (a > 0.0) {
      // squared error of each candidate (one candidate per iteration, the waves' partial sums into
      // LDS), then the first minimum
#pragma unroll 1
      for (int j = 0; j < 64; ++j) {
        const double s = FMT == FMT_MIRROR ? pot_candidate(j) * a : pot_candidate(j) * a / 4.0;
        // The outer level is taken where the rounded quotient |w| / s exceeds thr.  The sign of
        // fma(-thr, s, |w|) is the exact sign of |w| - thr s, which decides the same way except for
        // |w| / s within half an ulp of thr above it (the quotient rounds down to thr there; an ulp of
        // thr <= 5/2 is at most 2^-51): those few values, and only those, within 2^-51 s above the
        // threshold, are decided by the division itself (a wave-uniform branch, rarely taken).
        uint32_t outer[NTILES], near_any = 0;
#pragma unroll
        for (int tau = 0; tau < NTILES; ++tau) {
          outer[tau] = 0;
          uint32_t nr = 0;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const double r = fma(-thr, s, fabs(v[tau][e]));
            outer[tau] |= (uint32_t)(r > 0.0) << e;
            nr |= (uint32_t)(r > 0.0 && r <= 0x1p-51 * s) << e;
          }
          near_any |= valid[tau] ? nr : 0u;
        }
        if (__any(near_any != 0)) {
#pragma unroll
          for (int tau = 0; tau < NTILES; ++tau)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const double r = fma(-thr, s, fabs(v[tau][e]));
              if (valid[tau] && r > 0.0 && r <= 0x1p-51 * s) {
                const bool o = fabs(v[tau][e] / s) > thr;
                outer[tau] = (outer[tau] & ~(1u << e)) | ((uint32_t)o << e);
              }
            }
        }
        double acc = 0.0;
#pragma unroll
        for (int tau = 0; tau < NTILES; ++tau) {
          if (!valid[tau]) continue;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const double w = v[tau][e];
            const double mag = (outer[tau] >> e) & 1u ? m_out : m_in;
            const double d = w - s * (w >= 0.0 ? mag : -mag);
            acc += d * d;
          }
        }
        acc = wave_sum_f64(acc);
        if (lane == 0) red64[wave][j] = acc;
      }
      __syncthreads();
      double best_err = 0.0;
      int best_j = 0;
      for (int j = 0; j < 64; ++j) {
        const double e = (red64[0][j] + red64[1][j]) + (red64[2][j] + red64[3][j]);
        if (j == 0 || e < best_err) {
          best_err = e;
          best_j = j;
        }
      }
      sw = half_bits_rne(FMT == FMT_MIRROR ? pot_candidate(best_j) * a : pot_candidate(best_j) * a / 4.0);
    }
  }
  if (t == 0) scales[n] = sw;

  // ---- levels against the stored scale, decided as by the rounded quotient u = w / s_w:
  //   MNZ |u| > 2 -> 3, PoT |u| > 2.5 -> 4 (else 1, sign of w), W4 q = clamp(rint(u), -7, 7).
  // Without the division where the decision is clear: for the two-level sets the exact sign of
  // fma(-thr, s_w, |w|) (the quotient and the real ratio can disagree only within 2^-51 s_w above
  // the threshold); for W4 the product with 1/s_w rounded to q0, kept when the residual w - q0 s_w
  // lies clearly inside half a step.  The rest (a wave-uniform branch, rarely taken) divide.
  const double s_w = half_value(sw);
  const double inv_sw = s_w > 0.0 ? 1.0 / s_w : 0.0;
  const double thr = FMT == FMT_MNZ ? 2.0 : FMT == FMT_POT ? 2.5 : 0.5 * (rin + 1.0);
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    if (!valid[tau]) continue;
    int q[16];
    uint32_t nr = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const double w = v[tau][e];
      if constexpr (FMT == FMT_W4) {
        const double q0 = rint(w * inv_sw);
        const double res = fma(-q0, s_w, w);
        q[e] = (int)fmin(fmax(q0, -7.0), 7.0);
        nr |= (uint32_t)(fabs(res) >= (0.5 - 0x1p-45) * s_w) << e;
      } else {
        const double r = fma(-thr, s_w, fabs(w));
        q[e] = level_of<FMT>(w >= 0.0, r > 0.0);
        nr |= (uint32_t)(r > 0.0 && r <= 0x1p-51 * s_w) << e;
      }
    }
    if (s_w > 0.0) {
      if (__any(nr != 0)) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          if ((nr >> e) & 1u) {
            const double u = v[tau][e] / s_w;
            if constexpr (FMT == FMT_W4) {
              q[e] = (int)fmin(fmax(rint(u), -7.0), 7.0);
            } else {
              q[e] = level_of<FMT>(u >= 0.0, fabs(u) > thr);
            }
          }
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) q[e] = FMT == FMT_W4 ? 0 : FMT == FMT_MIRROR ? 2 : 1;
    }
    uint32_t wd[4] = {0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 16; ++e) wd[e >> 2] |= ((uint32_t)q[e] & 0xFFu) << (8 * (e & 3));
    *reinterpret_cast<uint4*>(levels + n * K + tau * S::T + 16 * t) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
  }
}

template <int FMT, int NTILES, int LC>
hipError_t launch_l(const float* W, int64_t N, int64_t K, int L, double sqrtb, double r, int8_t* levels,
                    uint16_t* scales, hipStream_t s) {
  hipLaunchKernelGGL((k_quant_weights<FMT, NTILES, LC>), dim3((unsigned)N), dim3(256), 0, s, W, (int)K, L, sqrtb,
                     r, levels, scales);
  return hipGetLastError();
}

// block exponents compiled as constants: 12, 11, 8 and 6; anything else at run time
template <int FMT, int NTILES>
hipError_t launch_nt(const float* W, int64_t N, int64_t K, int L, double sqrtb, double r, int8_t* levels,
                     uint16_t* scales, hipStream_t s) {
  switch (L) {
    case 12: return launch_l<FMT, NTILES, 12>(W, N, K, L, sqrtb, r, levels, scales, s);
    case 11: return launch_l<FMT, NTILES, 11>(W, N, K, L, sqrtb, r, levels, scales, s);
    case 8: return launch_l<FMT, NTILES, 8>(W, N, K, L, sqrtb, r, levels, scales, s);
    case 6: return launch_l<FMT, NTILES, 6>(W, N, K, L, sqrtb, r, levels, scales, s);
    default: return launch_l<FMT, NTILES, 0>(W, N, K, L, sqrtb, r, levels, scales, s);
  }
}

template <int FMT>
hipError_t launch_fmt(const float* W, int64_t N, int64_t K, int L, double sqrtb, double r, int8_t* levels,
                      uint16_t* scales, hipStream_t s) {
  switch ((K + 4095) / 4096) {
    case 1: return launch_nt<FMT, 1>(W, N, K, L, sqrtb, r, levels, scales, s);
    case 2: return launch_nt<FMT, 2>(W, N, K, L, sqrtb, r, levels, scales, s);
    case 3: return launch_nt<FMT, 3>(W, N, K, L, sqrtb, r, levels, scales, s);
    case 4: return launch_nt<FMT, 4>(W, N, K, L, sqrtb, r, levels, scales, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_quantize_weights(const float* W, int64_t N, int64_t K, int block, int fmt, int8_t* levels,
                                   uint16_t* scales, hipStream_t s) {
  const int L = dev::ilog2c(block);
  const double sqrtb = sqrt((double)block);
  switch (fmt) {
    case FMT_MNZ: return launch_fmt<FMT_MNZ>(W, N, K, L, sqrtb, 0.0, levels, scales, s);
    case FMT_POT: return launch_fmt<FMT_POT>(W, N, K, L, sqrtb, 0.0, levels, scales, s);
    case FMT_W4: return launch_fmt<FMT_W4>(W, N, K, L, sqrtb, 0.0, levels, scales, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_quantize_weights_mirror(const float* W, int64_t N, int64_t K, int block, double r, int8_t* codes,
                                          uint16_t* scales, hipStream_t s) {
  return launch_fmt<FMT_MIRROR>(W, N, K, dev::ilog2c(block), sqrt((double)block), r, codes, scales, s);
}

}  // namespace qift
