// Online Hadamard rotation + per-token symmetric INT4 quantization.
//
// Per token (Sec. 3.1; Sec. 4.1 "Quantization configuration"):
//   X = (I_{K/b} (x) H_b) x  exactly,  A = max|X|,
//   q = sign(X) min(7, rne(7|X| / (cA))),  s_x = cA / (7 sqrt(b)),  sum = sum q.
//
// Tokens of K <= 16384 with blocks b <= 4096 (k_act_tokens): a persistent
// grid of 256-thread workgroups, each walking tokens blockIdx.x, + gridDim.x,
// ... (for tokens of up to two 4096-element tiles with the next token's fp16
// loads in flight while the current one is rotated).  Each thread keeps 16 consecutive elements of every 4096-element
// tile of the token in fp64 registers (the whole token stays on chip until
// its absmax is known); the butterflies run in registers (quad DPP for index
// bits 4-5 of blocks up to 64) with LDS exchanges between groups of four
// index bits; values are quantized in the layout the transform ends in,
// their codes scattered into the exchange buffer in natural order and copied
// out with 16-byte stores.  The block exponent is a template constant for
// common block sizes.
//
// Larger tokens (k_rotate_quant_act): one 512-thread workgroup per token,
// returning to the natural layout before quantizing.  See qift_fwht.h for
// the exactness argument and the rounding decision.
//
// A few tokens of several tiles (k_act_wide, M <= kActWideMaxM): one workgroup of four waves per
// tile and token, the tiles rotated at once (each group of four waves with its own exchange buffer
// and wave barrier), one workgroup barrier for the token's max, each group quantizing its own tile:
// a token's latency is that of one tile instead of NTILES (down's 14336-wide input at 16 tokens:
// the tiles one after another took about 10 us).  The same transform and rounding as above, so the
// codes, scales and sums are the same.
#include "qift_fwht.h"
#include "qift_internal.h"

namespace qift {
namespace {

// tokens up to which a tokens' tiles are rotated at once (k_act_wide); beyond, one tile after another
// by the persistent k_act_tokens, whose grid keeps more tokens in flight
constexpr int64_t kActWideMaxM = 256;

template <int NT, int NTILES, bool BF16>
__global__ __launch_bounds__(NT) void k_rotate_quant_act(const uint16_t* __restrict__ x, int64_t K, int L,
                                                         int num, int den, double denom,
                                                         int8_t* __restrict__ act_q,
                                                         float* __restrict__ act_scale,
                                                         int32_t* __restrict__ act_sum) {
  using S = dev::Tile<NT, 16>;
  __shared__ double lds[S::LDS_DOUBLES];
  __shared__ double red_d[NT / 64];
  __shared__ int red_i[NT / 64];
  const int64_t m = blockIdx.x;
  int sum_q;
  float scale;
  dev::quant_token<NT, NTILES, BF16>(x + m * K, K, L, num, den, denom, lds, red_d, red_i, act_q + m * K,
                                   sum_q, scale);
  if (threadIdx.x == 0) {
    if (act_sum) act_sum[m] = sum_q;
    act_scale[m] = scale;
  }
}

template <int NTILES, int LC, bool BF16>
__global__ __launch_bounds__(256) void k_act_tokens(const uint16_t* __restrict__ x, int M, int64_t K, int L,
                                                    int num, int den, double denom, int8_t* __restrict__ act_q,
                                                    float* __restrict__ act_scale, int32_t* __restrict__ act_sum) {
  using S = dev::Tile<256, 16>;
  static_assert(NTILES * S::T <= S::LDS_DOUBLES * 8, "the codes of a token fit in the exchange buffer");
  __shared__ double xch[S::LDS_DOUBLES];
  __shared__ double red_d[4];
  __shared__ int red_i[4];
  const int t = threadIdx.x;
  dev::BlockSync sync;
  int8_t* codes = reinterpret_cast<int8_t*>(xch);   // natural-order codes, once the transform is done
  int m = blockIdx.x;                               // gridDim.x <= M
  // tokens of up to two tiles keep the next token's loads in flight; longer ones need those registers
  constexpr bool kPrefetch = NTILES <= 2;
  dev::TokenRaw<NTILES> raw;
  dev::load_token_raw<256, NTILES>(raw, x + (int64_t)m * K, K);
  for (; m < M; m += gridDim.x) {
    dev::TokenRaw<NTILES> cur = raw;
    if (kPrefetch && m + (int)gridDim.x < M)
      dev::load_token_raw<256, NTILES>(raw, x + (int64_t)(m + gridDim.x) * K, K);
    __syncthreads();   // the previous token's codes have been copied out and its partial sums read
    const double A = dev::quant_token_group<NTILES, LC, false, dev::BlockSync, BF16>(cur, K, L, num, den, xch, xch,
                                                                                   red_d, red_i, sync, codes);
    __syncthreads();   // codes and partial sums are in LDS
#pragma unroll
    for (int tau = 0; tau < NTILES; ++tau) {
      const int64_t base = (int64_t)tau * S::T + 16 * t;
      if (base < K) *reinterpret_cast<uint4*>(act_q + (int64_t)m * K + base) = *reinterpret_cast<const uint4*>(codes + base);
    }
    if (t == 0) {
      act_scale[m] = (float)((A * (double)num) / denom);
      if (act_sum) act_sum[m] = red_i[0] + red_i[1] + red_i[2] + red_i[3];
    }
    if (!kPrefetch && m + (int)gridDim.x < M)
      dev::load_token_raw<256, NTILES>(raw, x + (int64_t)(m + gridDim.x) * K, K);
  }
}

template <int NTILES, int LC, bool BF16>
__global__ __launch_bounds__(256 * NTILES) void k_act_wide(const uint16_t* __restrict__ x, int64_t K, int L, int num,
                                                           int den, double denom, int8_t* __restrict__ act_q,
                                                           float* __restrict__ act_scale,
                                                           int32_t* __restrict__ act_sum, int wait_limit,
                                                           uint32_t* __restrict__ err) {
  using S = dev::Tile<256, 16>;
  extern __shared__ __align__(16) double xch_all[];   // NTILES exchange buffers of S::LDS_DOUBLES
  __shared__ double red_d[4 * NTILES];
  __shared__ int red_i[4 * NTILES];
  __shared__ unsigned ctr[NTILES];
  const int gi = threadIdx.x >> 8, t = threadIdx.x & 255, lane = t & 63, w = t >> 6;
  if (threadIdx.x < NTILES) ctr[threadIdx.x] = 0u;
  __syncthreads();
  dev::GroupSync<4> gs{ctr + gi, 0u, wait_limit, err};
  const int m = blockIdx.x;
  const int Lc = LC > 0 ? LC : L;
  double* xch = xch_all + gi * S::LDS_DOUBLES;
  // tile gi of token m: 16 consecutive elements per thread (zeros past K)
  const __amdgpu_buffer_rsrc_t r = dev::make_rsrc(x + (int64_t)m * K, (uint32_t)(K * 2));
  const int64_t base = (int64_t)gi * S::T + 16 * t;
  const uint32_t off = base < K ? (uint32_t)(base * 2) : dev::kOutOfRange;
  const uint4 raw[2] = {dev::bload16(r, off), dev::bload16(r, off + 16)};
  double v[16];
  dev::unpack16<BF16>(v, raw);
  const int wend = dev::fwht_tile_s<256, 16, false>(v, xch, t, Lc, gs);
  double amax = 0.0;
#pragma unroll
  for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[e]));
  amax = dev::wave_max(amax);
  if (lane == 0) red_d[4 * gi + w] = amax;
  __syncthreads();   // every group's maxima are in
  double A = red_d[0];
#pragma unroll
  for (int k = 1; k < 4 * NTILES; ++k) A = fmax(A, red_d[k]);
  const dev::QuantParams p = dev::make_qparams(A, num, den);
  int q[16];
  dev::quant16(v, p, q);
  int qs = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) qs += q[e];
  // the codes in natural order through the group's exchange buffer (its exchange reads are done
  // once every wave of the group has passed the wave barrier), then 16 bytes per thread
  gs();
  int8_t* codes = reinterpret_cast<int8_t*>(xch);
  if (wend == 0) dev::store_codes<0>(codes, q, t);
  else if (wend == 4) dev::store_codes<4>(codes, q, t);
  else dev::store_codes<8>(codes, q, t);
  gs();
  if (base < K) *reinterpret_cast<uint4*>(act_q + (int64_t)m * K + base) = *reinterpret_cast<const uint4*>(codes + 16 * t);
  qs = dev::wave_sum(qs);
  if (lane == 0) red_i[4 * gi + w] = qs;
  __syncthreads();
  if (threadIdx.x == 0) {
    act_scale[m] = (float)((A * (double)num) / denom);
    if (act_sum) {
      int sum = 0;
#pragma unroll
      for (int k = 0; k < 4 * NTILES; ++k) sum += red_i[k];
      act_sum[m] = sum;
    }
  }
}

template <int NTILES, int LC, bool BF16>
hipError_t launch_wide_l(const uint16_t* x, int64_t M, int64_t K, int L, int num, int den, double denom, int8_t* q,
                         float* sc, int32_t* sum, hipStream_t s) {
  constexpr size_t shmem = (size_t)NTILES * dev::Tile<256, 16>::LDS_DOUBLES * 8;
  // the dynamic LDS this instance takes (the kernel's static LDS comes on top of it)
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_act_wide<NTILES, LC, BF16>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((k_act_wide<NTILES, LC, BF16>), dim3((unsigned)M), dim3(256 * NTILES), shmem, s, x, K, L, num,
                     den, denom, q, sc, sum, wait_limit(), device_error_word());
  return hipGetLastError();
}

template <int NTILES, int LC, bool BF16>
hipError_t launch_tokens_l(const uint16_t* x, int64_t M, int64_t K, int L, int num, int den, double denom,
                           int8_t* q, float* sc, int32_t* sum, hipStream_t s) {
  // persistent grid: every workgroup that fits on the chip at once (queried once per instance)
  static const int resident = [] {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(&k_act_tokens<NTILES, LC, BF16>),
                                                     256, 0) != hipSuccess || per_cu < 1)
      per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
      cus = 256;
    return per_cu * cus;
  }();
  const unsigned grid = (unsigned)(M < resident ? M : resident);
  hipLaunchKernelGGL((k_act_tokens<NTILES, LC, BF16>), dim3(grid), dim3(256), 0, s, x, (int)M, K, L, num, den, denom, q,
                     sc, sum);
  return hipGetLastError();
}

// block exponents compiled as constants: 12, 11, 8 and 6; anything else at run time
template <int NTILES, bool BF16>
hipError_t launch_tokens(const uint16_t* x, int64_t M, int64_t K, int L, int num, int den, double denom,
                         int8_t* q, float* sc, int32_t* sum, hipStream_t s) {
  if constexpr (NTILES > 1) {
    if (M <= kActWideMaxM) {
      switch (L) {
        case 12: return launch_wide_l<NTILES, 12, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
        case 11: return launch_wide_l<NTILES, 11, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
        case 8: return launch_wide_l<NTILES, 8, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
        case 6: return launch_wide_l<NTILES, 6, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
        default: return launch_wide_l<NTILES, 0, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
      }
    }
  }
  switch (L) {
    case 12: return launch_tokens_l<NTILES, 12, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
    case 11: return launch_tokens_l<NTILES, 11, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
    case 8: return launch_tokens_l<NTILES, 8, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
    case 6: return launch_tokens_l<NTILES, 6, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
    default: return launch_tokens_l<NTILES, 0, BF16>(x, M, K, L, num, den, denom, q, sc, sum, s);
  }
}

template <int NT, bool BF16>
hipError_t launch_nt(const uint16_t* x, int64_t M, int64_t K, int L, int num, int den, double denom,
                     int8_t* q, float* sc, int32_t* sum, hipStream_t s) {
  const int64_t T = 16 * NT;
  const int nt = (int)((K + T - 1) / T);
  const dim3 grid((unsigned)M), block(NT);
  switch (nt) {
    case 1: hipLaunchKernelGGL((k_rotate_quant_act<NT, 1, BF16>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    case 2: hipLaunchKernelGGL((k_rotate_quant_act<NT, 2, BF16>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    case 3: hipLaunchKernelGGL((k_rotate_quant_act<NT, 3, BF16>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    case 4: hipLaunchKernelGGL((k_rotate_quant_act<NT, 4, BF16>), grid, block, 0, s, x, K, L, num, den, denom, q, sc, sum); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

double act_denominator(int block, int clip_den) {
  // the fixed divisor of the per-token scale, (den * 7) * sqrt(b), rounded in that order
  return ((double)clip_den * 7.0) * sqrt((double)block);
}

template <bool BF16>
hipError_t launch_rqa(const uint16_t* x, int64_t M, int64_t K, int block, int clip_num, int clip_den, int8_t* act_q,
                      float* act_scale, int32_t* act_sum, hipStream_t s) {
  const int L = dev::ilog2c(block);
  const double denom = act_denominator(block, clip_den);
  if (block <= 4096 && K <= 4 * 4096) {
    switch ((K + 4095) / 4096) {
      case 1: return launch_tokens<1, BF16>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
      case 2: return launch_tokens<2, BF16>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
      case 3: return launch_tokens<3, BF16>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
      default: return launch_tokens<4, BF16>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
    }
  }
  return launch_nt<512, BF16>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
}

hipError_t launch_rotate_quant_act(const uint16_t* x, int64_t M, int64_t K, int block, int clip_num,
                                   int clip_den, int8_t* act_q, float* act_scale, int32_t* act_sum,
                                   hipStream_t s, bool bf16) {
  return bf16 ? launch_rqa<true>(x, M, K, block, clip_num, clip_den, act_q, act_scale, act_sum, s)
              : launch_rqa<false>(x, M, K, block, clip_num, clip_den, act_q, act_scale, act_sum, s);
}

}  // namespace qift
