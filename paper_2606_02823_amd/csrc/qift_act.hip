// Online Hadamard rotation + per-token symmetric INT4 quantization.
//
// Per token (Sec. 3.1; Sec. 4.1 "Quantization configuration"):
//   X = (I_{K/b} (x) H_b) x  exactly,  A = max|X|,
//   q = sign(X) min(7, rne(7|X| / (cA))),  s_x = cA / (7 sqrt(b)),  sum = sum q.
//
// One workgroup per token: each thread keeps 16 consecutive elements of every
// 16*NT-element tile of the token in fp64 registers (the whole token stays
// on chip until its absmax is known), the butterflies run in registers with
// LDS exchanges between groups of four index bits, and each thread writes its
// 16 codes with one 16-byte store.  See qift_fwht.h for the exactness
// argument and the rounding decision.
#include "qift_fwht.h"
#include "qift_internal.h"

namespace qift {
namespace {

template <int NT, int NTILES>
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
  dev::quant_token<NT, NTILES>(x + m * K, K, L, num, den, denom, lds, red_d, red_i, act_q + m * K,
                                   sum_q, scale);
  if (threadIdx.x == 0) {
    act_sum[m] = sum_q;
    act_scale[m] = scale;
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

double act_denominator(int block, int clip_den) {
  // the fixed divisor of the per-token scale, (den * 7) * sqrt(b), rounded in that order
  return ((double)clip_den * 7.0) * sqrt((double)block);
}

hipError_t launch_rotate_quant_act(const uint16_t* x, int64_t M, int64_t K, int block, int clip_num,
                                   int clip_den, int8_t* act_q, float* act_scale, int32_t* act_sum,
                                   hipStream_t s) {
  const int L = dev::ilog2c(block);
  const double denom = act_denominator(block, clip_den);
  if (block <= 4096 && K <= 4 * 4096)
    return launch_nt<256>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
  return launch_nt<512>(x, M, K, L, clip_num, clip_den, denom, act_q, act_scale, act_sum, s);
}

}  // namespace qift
