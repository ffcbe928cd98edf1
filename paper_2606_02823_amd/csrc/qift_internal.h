// Internal declarations shared by the C-ABI layer and the kernel launchers.
// Launchers enqueue work only; all argument checks happen in qift_api.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qift {

// Packing (qift_pack.hip)
hipError_t launch_pack_w2(const int8_t* levels, int64_t N, int64_t K, int fmt, uint32_t* packed,
                          int32_t* invalid_count, hipStream_t s);
hipError_t launch_pack_w4(const int8_t* levels, int64_t N, int64_t K, uint32_t* packed,
                          int32_t* invalid_count, hipStream_t s);

// Rotation + INT4 quantization (qift_act.hip)
hipError_t launch_rotate_quant_act(const uint16_t* x, int64_t M, int64_t K, int block, int clip_num,
                                   int clip_den, int8_t* act_q, float* act_scale, int32_t* act_sum,
                                   hipStream_t s);

// Quantized linear (qift_linear.hip).  fmt selects the decode.
hipError_t launch_linear(int fmt, const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K,
                         const int8_t* act_q, const float* act_scale, const int32_t* act_sum, int64_t M,
                         uint16_t* out, int32_t* acc_out, hipStream_t s);

// Largest M served by the skinny decode kernel.
constexpr int64_t kDecodeMaxM = 64;
// Largest K accepted by the activation quantizer.
constexpr int64_t kActMaxK = 32768;

}  // namespace qift
