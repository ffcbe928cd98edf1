// Fused decode linear instances for the PoT-MNZ (W2, levels {-4,-1,1,4} x s) weight format.
#include "qift_fused.h"

namespace qift {

hipError_t launch_fused_pot(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const uint16_t* x,
                          int block, int clip_num, int clip_den, int64_t M, uint16_t* y, int32_t* acc_out,
                          int8_t* act_q, float* act_scale, int32_t* act_sum, hipStream_t s) {
  return launch_fused_fmt<mma::FMT_POT>(P, sw, N, K, x, block, clip_num, clip_den, M, y, acc_out, act_q, act_scale,
                                   act_sum, s);
}

}  // namespace qift
