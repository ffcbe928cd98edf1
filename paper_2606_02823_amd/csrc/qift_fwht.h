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
// bits held in registers run in registers; blocks of up to 64 finish with two
// quad-DPP stages on lane bits 0 and 1; larger blocks bring the next EB index
// bits into registers by an exchange through LDS (two spare doubles after
// every 16 to spread the banks).
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

__device__ __forceinline__ uint2 bload8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return make_uint2(v[0], v[1]);
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

// Butterflies on lane bit B (B = 0, 1) of the natural layout, i.e. on index
// bit 4 + B: the partner value comes from lane ^ (1 << B) of the same quad by
// a DPP move, and sum / difference become one exact fma with a sign that
// depends on the lane: self + partner, or partner - self for the upper lane.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  return __hiloint2double(__builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, 0xf, 0xf, false),
                          __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, 0xf, 0xf, false));
}

// Lane index within the wave, from the count of mask bits below the lane, made afresh at each use: it
// reads no work-item id register and no earlier value, so nothing derived from it is kept live (or
// spilled) across a caller's loops.
__device__ __forceinline__ int lane_id() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

template <int B, int E>
__device__ __forceinline__ void lane_stage(double (&v)[E]) {
  constexpr int CTRL = B == 0 ? 0xB1 : 0x4E;   // quad_perm [1,0,3,2] / [2,3,0,1]
  // the lane index as an opaque value: the sign is made here, not hoisted out of a caller's loop
  // (where it would stay live, or spill, across everything else the loop does)
  int ln = threadIdx.x;
  asm volatile("" : "+v"(ln));
  const double sgn = ((ln >> B) & 1) ? -1.0 : 1.0;
#pragma unroll
  for (int e = 0; e < E; ++e) v[e] = fma(v[e], sgn, dpp_f64<CTRL>(v[e]));
}

// Window W: register e of thread t holds tile element
//   i = (t & (2^W - 1)) | (e << W) | ((t >> W) << (W + 4)),
// i.e. index bits [W, W + 4) are in registers (W = 0 is the natural layout,
// element 16t + e).  LDS slot of element i: i + 2 (i/16) (two spare doubles
// per 16, the fastest of the paddings measured for these exchanges).  With W
// a compile-time constant and W = 0 or W >= 4 the slot is a per-thread base
// plus a compile-time offset per e.
template <int W>
__device__ __forceinline__ int win_elem(int t) {
  return W == 0 ? 16 * t : ((t & ((1 << W) - 1)) | ((t >> W) << (W + 4)));
}
template <int W>
__device__ __forceinline__ int win_pbase(int t) {
  static_assert(W == 0 || W >= 4, "window");
  const int base = win_elem<W>(t);
  return base + 2 * (base >> 4);
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
// Natural layout on entry.  With NATURAL the values are back in the natural
// layout on exit; otherwise they stay in the last window used, which is
// returned (0, 4, 8 or 9) so the caller can address elements with
// win_elem/win_step.  All NT threads must call it.
struct BlockSync {
  __device__ void operator()() const { __syncthreads(); }
};

// Bits of the per-device error word that bounded waits set when they give up
// (read back by the host through qift_device_error).
constexpr uint32_t kErrGroupWait = 1u;   // a wave barrier inside a workgroup (GroupSync)
constexpr uint32_t kErrChainWait = 2u;   // a wait for another workgroup's result (decode chain)

__device__ __forceinline__ void flag_error(uint32_t* err, uint32_t bit) {
  if (err) __hip_atomic_fetch_or(err, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Barrier among the first NW waves of a workgroup that leaves its other waves
// running: lane 0 of each wave bumps a counter in LDS once the wave's LDS
// accesses have completed, and the wave spins until the counter reaches the
// next multiple of NW.  The counter is zeroed once before first use (under a
// full workgroup barrier) and never reset.  All NW waves make the same
// sequence of calls, so every wait ends; the spin is bounded all the same
// (limit iterations): a wave that gives up sets kErrGroupWait in *err and
// carries on, so the kernel still exits and the host learns that its
// results are not to be trusted.
template <int NW>
struct GroupSync {
  unsigned* ctr;
  unsigned target;
  int limit;
  uint32_t* err;
  __device__ void operator()() {
    target += NW;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    for (int spin = 0;; ++spin) {
      const unsigned c = __builtin_amdgcn_readfirstlane(
          __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
      if (c >= target) break;
      if (spin >= limit) {
        if ((threadIdx.x & 63) == 0) flag_error(err, kErrGroupWait);
        break;
      }
    }
    asm volatile("" ::: "memory");
  }
};

// Workgroup barrier that waits only for this wave's LDS accesses (not for its
// outstanding global loads, which a plain __syncthreads would also drain).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int NT, int E, bool NATURAL, typename Sync>
__device__ __forceinline__ int fwht_tile_s(double (&v)[E], double* lds, int t, int L, Sync& sync) {
  static_assert(E == 16, "16 elements per thread");
  using S = Tile<NT, E>;
  static_assert(S::TB == 12 || S::TB == 13, "tile of 4096 or 8192");
  reg_stages<E>(v, 0, L < 4 ? L : 4);
  if (L <= 4) return 0;
  if (L <= 6) {
    // index bits 4 and 5 are lane bits 0 and 1: quad DPP, no exchange, natural layout throughout
    lane_stage<0>(v);
    if (L == 6) lane_stage<1>(v);
    return 0;
  }
  int w = 4;
  lds_store_w<0>(lds, v, t);
  sync();
  lds_load_w<4>(lds, v, t);
  reg_stages<E>(v, 0, (L < 8 ? L : 8) - 4);
  if (L > 8) {
    // a thread's window-4 slots were read only by itself, so it may overwrite them at once
    lds_store_w<4>(lds, v, t);
    sync();
    lds_load_w<8>(lds, v, t);
    reg_stages<E>(v, 0, (L < 12 ? L : 12) - 8);
    w = 8;
    if constexpr (S::TB == 13) {
      if (L > 12) {
        lds_store_w<8>(lds, v, t);
        sync();
        lds_load_w<9>(lds, v, t);
        reg_stages<E>(v, 3, 4);   // register bit 3 of window 9 is index bit 12
        w = 9;
      }
    }
  }
  if constexpr (NATURAL) {
    if (w == 4) lds_store_w<4>(lds, v, t);
    else if (w == 8) lds_store_w<8>(lds, v, t);
    else lds_store_w<9>(lds, v, t);
    sync();
    lds_load_w<0>(lds, v, t);
    return 0;
  }
  return w;
}

template <int NT, int E, bool NATURAL>
__device__ __forceinline__ int fwht_tile(double (&v)[E], double* lds, int t, int L) {
  BlockSync sync;
  return fwht_tile_s<NT, E, NATURAL>(v, lds, t, L, sync);
}

// Per-token rounding constants: q = sign(X) min(7, rne(7 den |X| / (num A))).
struct QuantParams {
  double A;        // max |X| (natural units)
  double c1;       // 7 den / (num A), fp64 (estimate only)
  int num, den;
};

__device__ __forceinline__ QuantParams make_qparams(double A, int num, int den) {
  QuantParams p;
  p.A = A;
  p.c1 = A > 0.0 ? (7.0 * den) / ((double)num * A) : 0.0;
  p.num = num;
  p.den = den;
  return p;
}

// Exact rounding near a half-integer, on the fp64 values |X| <= A taken as rationals:
// t = 14 den |X| + num A and d = 2 num A, q = floor(t / d), lowered to even on an exact half.
// Both are normal doubles (every nonzero rotated value is a sum of fp16 or bf16 values, at
// least 2^-133): |X| = mx 2^ex, A = ma 2^ea with 53-bit integer mantissas and ea >= ex, so in
// units of 2^ex, t and d are integers below 2^70 when ea - ex <= 12 (beyond that, 7 den |X| /
// (num A) < 112 2^-11 and q = 0).  Rarely executed, so it is kept out of line (the inlined
// copies per element made the kernels larger than the instruction cache).
__device__ __attribute__((noinline)) int quant_exact(double ax, double A, int num, int den, double f) {
  if (!(f < 8.0)) return 7;   // clamps anyway (and keeps q and t below in range)
  if (!(ax > 0.0)) return 0;
  typedef unsigned __int128 u128;
  const uint64_t bx = (uint64_t)__double_as_longlong(ax), ba = (uint64_t)__double_as_longlong(A);
  const uint64_t mx = (bx & 0xFFFFFFFFFFFFFull) | (1ull << 52), ma = (ba & 0xFFFFFFFFFFFFFull) | (1ull << 52);
  const int s = (int)((ba >> 52) & 0x7FF) - (int)((bx >> 52) & 0x7FF);
  if (s > 12) return 0;
  const u128 t = (u128)(14u * (unsigned)den) * mx + (((u128)(unsigned)num * ma) << s);
  const u128 d = ((u128)(2u * (unsigned)num) * ma) << s;
  int q = (int)f;             // within one of the exact quotient: each loop runs at most twice
  for (int it = 0; it < 4 && q > 0 && (u128)q * d > t; ++it) --q;
  for (int it = 0; it < 4 && (u128)(q + 1) * d <= t; ++it) ++q;
  if ((u128)q * d == t && (q & 1)) --q;
  return q < 7 ? q : 7;
}

// Rounding of 16 values.  The fp64 quotient v = X c1 is within 1e-13 of the
// exact 7 den X / (num A) (|v| <= 112), so unless v lies within 1e-9 of a
// half-integer its nearest integer is rint(v); round-half-even is odd-symmetric,
// so rounding the signed quotient gives sign(X) times the rounded magnitude.
// That branch-free fast path covers all 16 values; only when some lane of the
// wave has a value that close to a half (a wave-uniform, rare branch) are those
// values redone with the exact integer test.
__device__ __forceinline__ void quant16(const double (&v)[16], const QuantParams& p, int (&q)[16]) {
  int near = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const double vv = v[e] * p.c1;   // c1 = 0 when A = 0, giving q = 0
    // vv + 1.5 * 2^52 rounds vv to the nearest integer (ties to even) into the low word as a
    // two's-complement int32, since |vv| < 2^31; subtracting the constant again gives that
    // integer as a double, exactly
    const double tt = vv + 0x1.8p52;
    const double r = tt - 0x1.8p52;
    near |= fabs(vv - r) > 0.5 - 1e-9;
    q[e] = min(max(__double2loint(tt), -7), 7);   // one v_med3_i32
  }
  if (__any(near)) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const double ax = fabs(v[e]);
      const double vv = ax * p.c1;
      if (p.A > 0.0 && fabs(vv - rint(vv)) > 0.5 - 1e-9) {
        const int qq = quant_exact(ax, p.A, p.num, p.den, floor(vv));
        q[e] = v[e] < 0.0 ? -qq : qq;
      }
    }
  }
}

// Wave-wide max / sum with DPP moves inside rows of 16 lanes and lane reads
// across the four rows (no LDS traffic).
#define QIFT_DPP_F64(x, CTRL)                                                                  \
  __hiloint2double(__builtin_amdgcn_update_dpp(__double2hiint(x), __double2hiint(x), CTRL, 0xf, 0xf, false), \
                   __builtin_amdgcn_update_dpp(__double2loint(x), __double2loint(x), CTRL, 0xf, 0xf, false))

__device__ __forceinline__ double wave_max(double x) {
  x = fmax(x, QIFT_DPP_F64(x, 0xb1));    // quad_perm [1,0,3,2]
  x = fmax(x, QIFT_DPP_F64(x, 0x4e));    // quad_perm [2,3,0,1]
  x = fmax(x, QIFT_DPP_F64(x, 0x141));   // row_half_mirror
  x = fmax(x, QIFT_DPP_F64(x, 0x140));   // row_mirror
  double r = x;
#pragma unroll
  for (int row = 1; row < 4; ++row)
    r = fmax(r, __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(x), row * 16),
                                 __builtin_amdgcn_readlane(__double2loint(x), row * 16)));
  return r;   // lane 0 holds the wave maximum (the others hold partial results)
}

__device__ __forceinline__ int wave_sum(int x) {
  x += __builtin_amdgcn_update_dpp(x, x, 0xb1, 0xf, 0xf, false);
  x += __builtin_amdgcn_update_dpp(x, x, 0x4e, 0xf, 0xf, false);
  x += __builtin_amdgcn_update_dpp(x, x, 0x141, 0xf, 0xf, false);
  x += __builtin_amdgcn_update_dpp(x, x, 0x140, 0xf, 0xf, false);
  return __builtin_amdgcn_readlane(x, 0) + __builtin_amdgcn_readlane(x, 16) + __builtin_amdgcn_readlane(x, 32) +
         __builtin_amdgcn_readlane(x, 48);
}

// Block-wide max of a non-negative double; red must hold NT/64 doubles.
template <int NT>
__device__ __forceinline__ double block_max(double v, double* red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();   // red may still be read from a previous call
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double r = red[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) r = fmax(r, red[w]);
  return r;
}

template <int NT>
__device__ __forceinline__ int block_sum(int v, int* red) {
  v = wave_sum(v);
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

// bf16 bits are the upper half of the fp32 value: exact in fp32, then in fp64
__device__ __forceinline__ void unpack_bf16(double (&v)[16], const uint4 (&d)[2]) {
  const uint32_t w[8] = {d[0].x, d[0].y, d[0].z, d[0].w, d[1].x, d[1].y, d[1].z, d[1].w};
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const uint32_t bits = (e & 1) ? (w[e >> 1] & 0xFFFF0000u) : (w[e >> 1] << 16);
    v[e] = (double)__uint_as_float(bits);
  }
}

template <bool BF16>
__device__ __forceinline__ void unpack16(double (&v)[16], const uint4 (&d)[2]) {
  if constexpr (BF16) unpack_bf16(v, d);
  else unpack_fp16(v, d);
}

// Rotate + quantize one token of K <= NTILES * T elements from its raw bits.
// Writes the int8 codes (16 per thread per tile, natural order, one 16-byte
// store) to dst (global or LDS, 16-byte aligned rows) and returns sum_q and
// the scale.  All NT threads must call it.
template <int NT, int NTILES, bool BF16 = false>
__device__ __forceinline__ void quant_token_raw(const TokenRaw<NTILES>& raw, int64_t K, int L, int num, int den,
                                                double denom, double* lds, double* red_d, int* red_i,
                                                int8_t* dst, int& sum_q, float& scale) {
  using S = Tile<NT, 16>;
  const int t = threadIdx.x;
  double v[NTILES][16];
  double amax = 0.0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    unpack16<BF16>(v[tau], raw.d[tau]);
    fwht_tile<NT, 16, true>(v[tau], lds, t, L);
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[tau][e]));
  }
  const double A = block_max<NT>(amax, red_d);
  const QuantParams p = make_qparams(A, num, den);
  int qs = 0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    const int64_t base = (int64_t)tau * S::T + 16 * t;
    int q[16];
    quant16(v[tau], p, q);
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      qs += q[e];
      w[e >> 2] |= ((uint32_t)q[e] & 0xFFu) << (8 * (e & 3));
    }
    if (base < K) *reinterpret_cast<uint4*>(dst + base) = make_uint4(w[0], w[1], w[2], w[3]);
  }
  sum_q = block_sum<NT>(qs, red_i);
  scale = (float)((A * (double)num) / denom);
}

// Byte position of code k in LDS.  Natural: k.  Planar (PLANAR = true): inside
// each 64-k chunk, k = 16i + 4t + b goes to 16t + 4i + b, so that the 16 codes
// {16i + 4t + b : i, b} that meet bit-plane t of four consecutive packed W2
// words in one MFMA are 16 contiguous bytes (qift_mma.h).
template <bool PLANAR>
__device__ __forceinline__ int code_pos(int k) {
  if constexpr (PLANAR) return (k & ~63) | ((k & 0x0C) << 2) | ((k & 0x30) >> 2) | (k & 3);
  else return k;
}

template <int W, bool PLANAR = false>
__device__ __forceinline__ void store_codes(int8_t* dst, const int (&q)[16], int t) {
  if constexpr (W == 0) {
    // natural layout: the thread's 16 codes are k = 16t .. 16t + 15, i.e. four packed words
    uint32_t wd[4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
      wd[a] = ((uint32_t)q[4 * a] & 0xFFu) | (((uint32_t)q[4 * a + 1] & 0xFFu) << 8) |
              (((uint32_t)q[4 * a + 2] & 0xFFu) << 16) | ((uint32_t)q[4 * a + 3] << 24);
    if constexpr (PLANAR) {
      // word a (k = 16t + 4a + b) goes to 16a + 4 (t mod 4) + b of the 64-k chunk t / 4
      int8_t* d = dst + 64 * (t >> 2) + 4 * (t & 3);
#pragma unroll
      for (int a = 0; a < 4; ++a) *reinterpret_cast<uint32_t*>(d + 16 * a) = wd[a];
    } else {
      *reinterpret_cast<uint4*>(dst + 16 * t) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
    }
  } else {
    const int base = win_elem<W>(t);
#pragma unroll
    for (int e = 0; e < 16; ++e) dst[code_pos<PLANAR>(base + e * (1 << W))] = (int8_t)q[e];
  }
}

// Rotate + quantize one token held in registers by the 256 threads of the
// first four waves of a workgroup, synchronizing only those waves (sync), so
// that other waves of the workgroup keep running.  Every tile is transformed
// once and stays in registers until the absmax is known; tiles alternate
// between two exchange buffers (xch0, xch1), so a tile's first exchange never
// overwrites slots a slower wave still reads from the tile before (the
// exchange of the tile in between orders them).  Codes go to dst (16-byte
// aligned) bytewise from the layout the transform ends in, at code_pos<PLANAR>;
// elements past K are skipped.  Returns A = max |X|; each wave's sum of codes
// lands in red_i[wave] (red_d holds 4 doubles).  LC > 0 fixes the block
// exponent L = LC at compile time (every butterfly stage and exchange is then
// straight-line code); LC = 0 takes L at run time.  With xch0 == xch1 (one
// exchange buffer) every tile after the first starts with a sync instead.
template <int NTILES, int LC, bool PLANAR, typename Sync, bool BF16 = false>
__device__ __forceinline__ double quant_token_group(const TokenRaw<NTILES>& raw, int64_t K, int L_rt, int num,
                                                    int den, double* xch0, double* xch1, double* red_d,
                                                    int* red_i, Sync& sync, int8_t* dst, bool xbf16 = false) {
  using S = Tile<256, 16>;
  const int L = LC > 0 ? LC : L_rt;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  double v[NTILES][16];
  double amax = 0.0;
  int wend = 0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    if (BF16 || xbf16) unpack_bf16(v[tau], raw.d[tau]);   // x bf16: a wave-uniform run-time choice
    else unpack_fp16(v[tau], raw.d[tau]);
    if (tau > 0 && xch0 == xch1 && L > 6) sync();   // the previous tile's exchange reads are done
    wend = fwht_tile_s<256, 16, false>(v[tau], (tau & 1) ? xch1 : xch0, t, L, sync);
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[tau][e]));
  }
  amax = wave_max(amax);
  if (lane == 0) red_d[wave] = amax;
  sync();
  const double A = fmax(fmax(red_d[0], red_d[1]), fmax(red_d[2], red_d[3]));
  const QuantParams p = make_qparams(A, num, den);
  int qs = 0;
#pragma unroll
  for (int tau = 0; tau < NTILES; ++tau) {
    int q[16];
    quant16(v[tau], p, q);
#pragma unroll
    for (int e = 0; e < 16; ++e) qs += q[e];
    int8_t* tile_dst = dst + tau * S::T;
    if ((int64_t)(tau + 1) * S::T <= K) {
      if (wend == 0) store_codes<0, PLANAR>(tile_dst, q, t);
      else if (wend == 4) store_codes<4, PLANAR>(tile_dst, q, t);
      else store_codes<8, PLANAR>(tile_dst, q, t);
    } else if (wend == 0) {
      // K is a multiple of 64: a thread's 16 consecutive elements are all in or all past K
      if ((int64_t)tau * S::T + 16 * t < K) store_codes<0, PLANAR>(tile_dst, q, t);
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = wend == 4 ? win_elem<4>(t) + (e << 4) : win_elem<8>(t) + (e << 8);
        if ((int64_t)tau * S::T + i < K) tile_dst[code_pos<PLANAR>(i)] = (int8_t)q[e];
      }
    }
  }
  qs = wave_sum(qs);
  if (lane == 0) red_i[wave] = qs;
  return A;
}

template <int NT, int NTILES, bool BF16 = false>
__device__ __forceinline__ void quant_token(const uint16_t* xr, int64_t K, int L, int num, int den,
                                            double denom, double* lds, double* red_d, int* red_i,
                                            int8_t* dst, int& sum_q, float& scale) {
  TokenRaw<NTILES> raw;
  load_token_raw<NT, NTILES>(raw, xr, K);
  quant_token_raw<NT, NTILES, BF16>(raw, K, L, num, den, denom, lds, red_d, red_i, dst, sum_q, scale);
}

}  // namespace dev
}  // namespace qift
