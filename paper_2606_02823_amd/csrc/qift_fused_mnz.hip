// Fused decode linear and decode-on-codes instances for the MNZ (W2, levels {-3,-1,1,3} x s/2) weight format.
#include "qift_fused.h"

namespace qift {

hipError_t launch_fused_mnz(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const uint16_t* x,
                          int block, int clip_num, int clip_den, int64_t M, uint16_t* y, int32_t* acc_out,
                          int8_t* act_q, float* act_scale, int32_t* act_sum, bool bf16, hipStream_t s) {
  return launch_fused_fmt<mma::FMT_MNZ>(P, sw, N, K, x, block, clip_num, clip_den, M, y, acc_out, act_q, act_scale,
                                   act_sum, bf16, s);
}

hipError_t launch_codes_mnz(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act_q,
                          const float* act_scale, const int32_t* act_sum, int64_t M, uint16_t* y, int32_t* acc_out,
                          hipStream_t s) {
  return launch_codes_fmt<mma::FMT_MNZ>(P, sw, N, K, act_q, act_scale, act_sum, M, y, acc_out, s);
}

size_t codes_shmem_mnz(int64_t M, int64_t N, int64_t K) { return codes_shmem_fmt<mma::FMT_MNZ>(M, N, K); }

}  // namespace qift
