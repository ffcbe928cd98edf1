// Device-side exact block Walsh-Hadamard transform and INT4 rounding of one
// token, shared by the stand-alone activation quantizer and the fused decode
// linear.
//
// Exactness: every finite fp16 value is an integer multiple of 2^-24 with
// magnitude below 2^40 units; a +-1 combination of at most 2^13 of them stays
// below 2^53 units, so every fp64 butterfly sum is exact whatever the order.
//
// Layout: a tile of T = NT * E elements; thread t holds E consecutive elements
// (natural layout, element 16t+e for E = 16).  The butterflies on the EB index
// bits held in registers run in registers; the next EB index bits are brought
// into registers by an exchange through LDS (two spare doubles after every 16
// to spread the banks).
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qift {
namespace dev {

constexpr int ilog2c(int v) { return v <= 1 ? 0 : 1 + ilog2c(v >> 1); }

// Raw buffer loads.  A buffer resource (base, size in bytes; wave-uniform)
// makes the hardware return zero for any offset at or past the end, so masked
// lanes get zeros from an out-of-range offset instead of an exec-masked
// branch: every load then issues unconditionally and the in-order
// vector-memory counter waits for exactly the loads a value depends on.
constexpr uint32_t kOutOfRange = 0x80000000u;   // past every buffer (sizes stay below 2^31)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // raw (stride 0) buffer, 32-bit data format word as used for gfx9 untyped loads
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

template <int NT, int E>
struct Tile {
  static constexpr int EB = ilog2c(E);
  static constexpr int T = NT * E;
  static constexpr int TB = ilog2c(T);
  static constexpr int LDS_DOUBLES = T + T / 8;
};

__device__ __forceinline__ int pad_idx(int i) { return i + 2 * (i >> 4); }

// butterflies on register bits r in [r_lo, r_hi)
template <int E>
__device__ __forceinline__ void reg_stages(double (&v)[E], int r_lo, int r_hi) {
#pragma unroll
  for (int r = 0; r < ilog2c(E); ++r) {
    if (r >= r_lo && r < r_hi) {
      const int h = 1 << r;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (!(e & h)) {
          const double a = v[e], b = v[e + h];
          v[e] = a + b;
          v[e + h] = a - b;
        }
      }
    }
  }
}

// Window W: register e of thread t holds tile element
//   i = (t & (2^W - 1)) | (e << W) | ((t >> W) << (W + 4)),
// i.e. index bits [W, W + 4) are in registers (W = 0 is the natural layout,
// element 16t + e).  With W a compile-time constant and W = 0 or W >= 4, the
// padded LDS slot is a per-thread base plus a compile-time offset per e.
template <int W>
__device__ __forceinline__ int win_pbase(int t) {
  if constexpr (W == 0) {
    return 18 * t;
  } else {
    static_assert(W >= 4, "window");
    const int base = (t & ((1 << W) - 1)) | ((t >> W) << (W + 4));
    return base + 2 * (base >> 4);
  }
}
template <int W>
constexpr int win_step() { return W == 0 ? 1 : (1 << W) + (1 << (W - 3)); }

template <int W>
__device__ __forceinline__ void lds_store_w(double* lds, const double (&v)[16], int t) {
  double* p = lds + win_pbase<W>(t);
#pragma unroll
  for (int e = 0; e < 16; ++e) p[e * win_step<W>()] = v[e];
}

template <int W>
__device__ __forceinline__ void lds_load_w(const double* lds, double (&v)[16], int t) {
  const double* p = lds + win_pbase<W>(t);
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = p[e * win_step<W>()];
}

// In-place transform of one tile over index bits [0, L) (block 2^L, L <= TB).
// Natural layout on entry and on exit.  All NT threads must call it.
// Index bits are brought into registers four at a time: windows 0, 4, 8 and,
// for 8192-element tiles, 9 (its only new bit is 12).
template <int NT, int E>
__device__ __forceinline__ void fwht_tile(double (&v)[E], double* lds, int t, int L) {
  static_assert(E == 16, "16 elements per thread");
  using S = Tile<NT, E>;
  static_assert(S::TB == 12 || S::TB == 13, "tile of 4096 or 8192");
  reg_stages<E>(v, 0, L < 4 ? L : 4);
  if (L <= 4) return;
  lds_store_w<0>(lds, v, t);
  __syncthreads();
  lds_load_w<4>(lds, v, t);
  reg_stages<E>(v, 0, (L < 8 ? L : 8) - 4);
  if (L > 8) {
    lds_store_w<4>(lds, v, t);
    __syncthreads();
    lds_load_w<8>(lds, v, t);
    reg_stages<E>(v, 0, (L < 12 ? L : 12) - 8);
    if constexpr (S::TB == 13) {
      if (L > 12) {
        lds_store_w<8>(lds, v, t);
        __syncthreads();
        lds_load_w<9>(lds, v, t);
        reg_stages<E>(v, 3, 4);   // register bit 3 of window 9 is index bit 12
        lds_store_w<9>(lds, v, t);
      } else {
        lds_store_w<8>(lds, v, t);
      }
    } else {
      lds_store_w<8>(lds, v, t);
    }
  } else {
    lds_store_w<4>(lds, v, t);
  }
  __syncthreads();
  lds_load_w<0>(lds, v, t);
  __syncthreads();
}

// Per-token rounding constants: q = sign(X) min(7, rne(7 den |X| / (num A))).
struct QuantParams {
  double A;        // max |X| (natural units)
  double c1;       // 7 den / (num A), fp64 (estimate only)
  int64_t Ai;      // A in units of 2^-24
  int num, den;
};

__device__ __forceinline__ QuantParams make_qparams(double A, int num, int den) {
  QuantParams p;
  p.A = A;
  p.Ai = (int64_t)(A * 0x1p24);
  p.c1 = p.Ai > 0 ? (7.0 * den) / ((double)num * A) : 0.0;
  p.num = num;
  p.den = den;
  return p;
}

// Exact rounding near a half-integer: t = 14 den |X| + num A and d = 2 num A
// in units of 2^-24; q = floor(t / d), lowered to even on an exact half.
// Rarely executed, so it is kept out of line (the inlined copies per element
// made the kernels larger than the instruction cache).
__device__ __attribute__((noinline)) int quant_exact(double ax, double f, int64_t Ai, int num, int den) {
  const int64_t xi = (int64_t)(ax * 0x1p24);
  const int64_t t = 14 * (int64_t)den * xi + (int64_t)num * Ai;
  const int64_t d = 2 * (int64_t)num * Ai;
  int64_t q = (int64_t)f;
  int64_t r = t - q * d;
  while (r < 0) { --q; r += d; }
  while (r >= d) { ++q; r -= d; }
  if (r == 0 && (q & 1)) --q;
  return (int)(q < 7 ? q : 7);
}

// Exact rounding of one magnitude.  The fp64 quotient v = |X| c1 is within
// 1e-13 of the exact 7 den |X| / (num A) (v <= 112), so when its fractional
// part is farther than 1e-9 from 1/2 the nearest integer is decided;
// otherwise the exact int64 remainder decides.
__device__ __forceinline__ int quant_mag(double ax, const QuantParams& p) {
  const double v = ax * p.c1;       // c1 = 0 when A = 0, giving q = 0
  const double f = floor(v);
  const double fr = v - f;
  if (fabs(fr - 0.5) <= 1e-9 && p.Ai > 0) return quant_exact(ax, f, p.Ai, p.num, p.den);
  const double r = fr > 0.5 ? f + 1.0 : f;
  return (int)fmin(r, 7.0);
}

__device__ __forceinline__ int quant_one(double val, const QuantParams& p) {
  const int q0 = quant_mag(fabs(val), p);
  return val < 0.0 ? -q0 : q0;
}

// Block-wide max of a non-negative double; red must hold NT/64 doubles.
template <int NT>
__device__ __forceinline__ double block_max(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double r = red[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) r = fmax(r, red[w]);
  return r;
}

template <int NT>
__device__ __forceinline__ int block_sum(int v, int* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int r = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) r += red[w];
  return r;
}

// Raw fp16 bits of one token as held by thread t: 16 consecutive elements of
// each tile (two 16-byte loads per tile).  Issuing these loads before other
// long-latency loads lets the rotation start as soon as x arrives: the
// vector-memory counter retires loads in order.
template <int NTILES>
struct TokenRaw {
  uint4 d[NTILES][2];
};

template <int NT, int NTILES>
__device__ __forceinline__ void load_token_raw(TokenRaw<NTILES>& raw, const uint16_t* xr, int64_t K) {
  using S = Tile<NT, 16>;
  const int t = threadIdx.x;
  const __amdgpu_buffer_rsrc_t r = make_rsrc(xr, (uint32_t)(K * 2));
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    const int64_t base = (int64_t)tau * S::T + 16 * t;   // elements past K read as zeros
    const uint32_t off = base < K ? (uint32_t)(base * 2) : kOutOfRange;
    raw.d[tau][0] = bload16(r, off);
    raw.d[tau][1] = bload16(r, off + 16);
  }
}

__device__ __forceinline__ void unpack_fp16(double (&v)[16], const uint4 (&d)[2]) {
  const uint32_t w[8] = {d[0].x, d[0].y, d[0].z, d[0].w, d[1].x, d[1].y, d[1].z, d[1].w};
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const uint16_t h = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
    v[e] = (double)__half2float(__ushort_as_half(h));
  }
}

// Rotate + quantize one token of K <= NTILES * T elements from its raw bits.
// Writes the int8 codes (16 per thread per tile, natural order, one 16-byte
// store) to dst (global or LDS, 16-byte aligned rows) and returns sum_q and
// the scale.  All NT threads must call it.
template <int NT, int NTILES>
__device__ __forceinline__ void quant_token_raw(const TokenRaw<NTILES>& raw, int64_t K, int L, int num, int den,
                                                double denom, double* lds, double* red_d, int* red_i,
                                                int8_t* dst, int& sum_q, float& scale) {
  using S = Tile<NT, 16>;
  const int t = threadIdx.x;
  double v[NTILES][16];
  double amax = 0.0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    unpack_fp16(v[tau], raw.d[tau]);
    fwht_tile<NT, 16>(v[tau], lds, t, L);
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[tau][e]));
  }
  const double A = block_max<NT>(amax, red_d);
  const QuantParams p = make_qparams(A, num, den);
  int qs = 0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    const int64_t base = (int64_t)tau * S::T + 16 * t;
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int q = quant_one(v[tau][e], p);
      qs += q;
      w[e >> 2] |= ((uint32_t)q & 0xFFu) << (8 * (e & 3));
    }
    if (base < K) *reinterpret_cast<uint4*>(dst + base) = make_uint4(w[0], w[1], w[2], w[3]);
  }
  sum_q = block_sum<NT>(qs, red_i);
  scale = (float)((A * (double)num) / denom);
}

template <int NT, int NTILES>
__device__ __forceinline__ void quant_token(const uint16_t* xr, int64_t K, int L, int num, int den,
                                            double denom, double* lds, double* red_d, int* red_i,
                                            int8_t* dst, int& sum_q, float& scale) {
  TokenRaw<NTILES> raw;
  load_token_raw<NT, NTILES>(raw, xr, K);
  quant_token_raw<NT, NTILES>(raw, K, L, num, den, denom, lds, red_d, red_i, dst, sum_q, scale);
}

}  // namespace dev
}  // namespace qift
