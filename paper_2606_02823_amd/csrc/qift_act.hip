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
#include "qift_fwht.h"
#include "qift_internal.h"

namespace qift {
namespace {

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
