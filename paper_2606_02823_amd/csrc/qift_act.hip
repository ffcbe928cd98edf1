// Online Hadamard rotation + per-token symmetric INT4 quantization.
//
// Per token (Sec. 3.1; Sec. 4.1 "Quantization configuration"):
//   X = (I_{K/b} (x) H_b) x          exact: fp16 inputs are integer multiples
//                                     of 2^-24 below 2^40 units, so every fp64
//                                     butterfly sum (at most 2^13 terms) is an
//                                     integer below 2^53 units;
//   A = max|X|,  q = sign(X) min(7, rne(7|X| / (cA))),  s_x = cA / (7 sqrt(b)).
//
// Design for gfx950: one workgroup per token.  Each thread keeps 16
// consecutive elements of every 16*NT-element tile of the token in registers
// (fp64), does the four butterfly stages on bits 0-3 in registers, and moves
// to the next group of four index bits with an LDS exchange (padded against
// bank conflicts).  The whole token stays in registers until the absmax is
// known, so x is read from HBM once and act_q written once (16 B per thread).
// Rounding is decided exactly: an fp64 estimate of the quotient is corrected
// with int64 remainders, and exact halves go to even.
#include <hip/hip_fp16.h>

#include "qift_internal.h"

namespace qift {
namespace {

template <int NT>
struct TileShape {
  static constexpr int T = 16 * NT;                  // elements per tile
  static constexpr int TB = (NT == 256) ? 12 : 13;   // log2(T)
  static constexpr int LDS = T + T / 8;              // padded length in doubles
};

// padded LDS slot of tile element i: two spare doubles after every 16
__device__ __forceinline__ int pad_idx(int i) { return i + 2 * (i >> 4); }

// Tile element held in register e by thread t when index bits [w, w+4) are in registers.
__device__ __forceinline__ int win_idx(int t, int e, int w) {
  return (t & ((1 << w) - 1)) | (e << w) | ((t >> w) << (w + 4));
}

// Butterflies on the register bits r in [r_lo, r_hi) (register bit r <-> index bit w + r).
__device__ __forceinline__ void stages(double (&v)[16], int r_lo, int r_hi) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (r >= r_lo && r < r_hi) {
      const int h = 1 << r;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        if (!(e & h)) {
          const double a = v[e], b = v[e + h];
          v[e] = a + b;
          v[e + h] = a - b;
        }
      }
    }
  }
}

template <int NT>
__device__ __forceinline__ void store_win(double* lds, const double (&v)[16], int t, int w) {
#pragma unroll
  for (int e = 0; e < 16; ++e) lds[pad_idx(win_idx(t, e, w))] = v[e];
}

template <int NT>
__device__ __forceinline__ void load_win(const double* lds, double (&v)[16], int t, int w) {
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = lds[pad_idx(win_idx(t, e, w))];
}

template <int NT, int NTILES>
__global__ __launch_bounds__(NT) void k_rotate_quant_act(const uint16_t* __restrict__ x, int64_t K,
                                                         int L, int num, int den, double denom,
                                                         int8_t* __restrict__ act_q,
                                                         float* __restrict__ act_scale,
                                                         int32_t* __restrict__ act_sum) {
  using S = TileShape<NT>;
  __shared__ double lds[S::LDS];
  __shared__ double red_d[NT / 64];
  __shared__ int red_i[NT / 64];

  const int t = threadIdx.x;
  const int64_t m = blockIdx.x;
  const uint16_t* xr = x + m * K;

  double v[NTILES][16];
  double amax = 0.0;

#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    const int64_t base = (int64_t)tau * S::T + 16 * t;
    if (base < K) {
      const uint4* src = reinterpret_cast<const uint4*>(xr + base);
      const uint4 a = src[0], b = src[1];
      const uint32_t d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const uint16_t h = (uint16_t)(d[e >> 1] >> (16 * (e & 1)));
        v[tau][e] = (double)__half2float(__ushort_as_half(h));
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) v[tau][e] = 0.0;
    }

    // index bits 0..3 are register bits in the natural layout
    stages(v[tau], 0, L < 4 ? L : 4);
    if (L > 4) {
      int cur = 0;
#pragma unroll
      for (int wb = 4; wb <= 12; wb += 4) {
        if (wb < L) {
          const int wr = wb < S::TB - 4 ? wb : S::TB - 4;   // register window start
          store_win<NT>(lds, v[tau], t, cur);
          __syncthreads();
          load_win<NT>(lds, v[tau], t, wr);
          const int hi = (wb + 4 < L ? wb + 4 : L);
          stages(v[tau], wb - wr, hi - wr);
          cur = wr;
        }
      }
      store_win<NT>(lds, v[tau], t, cur);
      __syncthreads();
      load_win<NT>(lds, v[tau], t, 0);
      __syncthreads();   // the next tile reuses the buffer
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[tau][e]));
  }

  // absmax of the token: wave butterfly, then across waves
  const int lane = t & 63, wave = t >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) amax = fmax(amax, __shfl_xor(amax, off, 64));
  if (lane == 0) red_d[wave] = amax;
  __syncthreads();
  double A = red_d[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) A = fmax(A, red_d[w]);

  // exact integer rounding: q0 = floor((t + num A) / d) with t = 14 den |X|, d = 2 num A,
  // in units of 2^-24; an exact half (zero remainder) with odd q0 goes down to even.
  const int64_t Ai = (int64_t)(A * 0x1p24);
  const int64_t dd = 2 * (int64_t)num * Ai;
  const int64_t off = (int64_t)num * Ai;
  const double est_mul = Ai > 0 ? (14.0 * den) / (2.0 * num * A) : 0.0;
  int qsum = 0;

#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    const int64_t base = (int64_t)tau * S::T + 16 * t;
    uint32_t packed[4] = {0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const double val = v[tau][e];
      const double ax = fabs(val);
      int q0 = 0;
      if (Ai > 0) {
        const int64_t xi = (int64_t)(ax * 0x1p24);
        const int64_t tt = 14 * (int64_t)den * xi + off;
        int64_t qh = (int64_t)(ax * est_mul + 0.5);
        int64_t r = tt - qh * dd;
        if (r < 0) { --qh; r += dd; }
        else if (r >= dd) { ++qh; r -= dd; }
        if (r == 0 && (qh & 1)) --qh;
        q0 = (int)(qh < 7 ? qh : 7);
      }
      const int q = val < 0.0 ? -q0 : q0;
      qsum += q;
      packed[e >> 2] |= ((uint32_t)q & 0xFFu) << (8 * (e & 3));
    }
    if (base < K) {
      *reinterpret_cast<uint4*>(act_q + m * K + base) =
          make_uint4(packed[0], packed[1], packed[2], packed[3]);
    }
  }

#pragma unroll
  for (int o = 32; o > 0; o >>= 1) qsum += __shfl_xor(qsum, o, 64);
  if (lane == 0) red_i[wave] = qsum;
  __syncthreads();
  if (t == 0) {
    int s = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) s += red_i[w];
    act_sum[m] = s;
    act_scale[m] = (float)((A * (double)num) / denom);
  }
}

template <int NT>
hipError_t launch_nt(const uint16_t* x, int64_t M, int64_t K, int L, int num, int den, double denom,
                     int8_t* q, float* sc, int32_t* sum, hipStream_t s) {
  const int64_t T = 16 * NT;
  const int nt = (int)((K + T - 1) / T);
  const dim3 grid((unsigned)M), block(NT);
  switch (nt) {
    case 1: hipLaunchKernelGGL((k_rotate_quant_act<NT, 1>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    case 2: hipLaunchKernelGGL((k_rotate_quant_act<NT, 2>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    case 3: hipLaunchKernelGGL((k_rotate_quant_act<NT, 3>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    case 4: hipLaunchKernelGGL((k_rotate_quant_act<NT, 4>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rotate_quant_act(const uint16_t* x, int64_t M, int64_t K, int block, int clip_num,
                                   int clip_den, int8_t* act_q, float* act_scale, int32_t* act_sum,
                                   hipStream_t s) {
  int L = 0;
  while ((1 << L) < block) ++L;
  // the fixed divisor of the per-token scale, (den * 7) * sqrt(b), rounded in that order
  const double denom = ((double)clip_den * 7.0) * sqrt((double)block);
  if (block <= 4096 && K <= 4 * 4096)
    return launch_nt<256>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
  return launch_nt<512>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
}

}  // namespace qift
