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

// Offline weight rotation + per-row scale + nearest level (qift_wquant.hip); fmt is a format constant
// of qift_mma.h, block a power of two up to 4096 dividing K <= kWquantMaxK.
constexpr int64_t kWquantMaxK = 16384;
hipError_t launch_quantize_weights(const float* W, int64_t N, int64_t K, int block, int fmt, int8_t* levels,
                                   uint16_t* scales, hipStream_t s);
// The same for the mirror family {-1, -r, +r, +1}, 0 < r < 1: codes 0..3 of the ascending levels.
hipError_t launch_quantize_weights_mirror(const float* W, int64_t N, int64_t K, int block, double r, int8_t* codes,
                                          uint16_t* scales, hipStream_t s);

// Ratio scan of the mirror family over fp64 samples (qift_scan.hip); ratios and cands are host arrays
// of at most kScanMaxRatios / kScanMaxCands values.
constexpr int kScanRatiosPerLaunch = 32, kScanMaxCands = 256, kScanMaxRatios = 1024;
hipError_t launch_ratio_scan(const double* x, int64_t n, const double* ratios, int n_ratios, const double* cands,
                             int n_cands, double* sse, double* nmse, int32_t* best, double* stats, hipStream_t s);

// KV4 cache quantizer and decode attention over it (qift_kv4.hip); head dimension 128, Hq / Hkv in
// {1, 2, 4, 8}; cache rows [B][T][Hkv] or, head_major, [B][Hkv][T]; ws holds
// kv4_attention_workspace(B, Hq, T) bytes.
size_t kv4_attention_workspace(int64_t B, int64_t Hq, int64_t T);
hipError_t launch_kv4_quant(const uint16_t* x, int64_t groups, uint8_t* codes, float* scales, uint8_t* zeros,
                            hipStream_t s);
hipError_t launch_kv4_attention(const uint16_t* q, int64_t B, int Hq, int Hkv, int64_t T, int head_major,
                                const uint8_t* kc, const float* ks, const uint8_t* kz, const uint8_t* vc,
                                const float* vs, const uint8_t* vz, uint16_t* y, void* ws, hipStream_t s);

// Linear over a four-level fp16 table (qift_lut.hip): lut holds the table entries exactly
hipError_t launch_lut_linear(const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K, const double lut[4],
                             const int8_t* act_q, const float* act_scale, int64_t M, uint16_t* out, hipStream_t s);

// Rotation + INT4 quantization (qift_act.hip)
hipError_t launch_rotate_quant_act(const uint16_t* x, int64_t M, int64_t K, int block, int clip_num,
                                   int clip_den, int8_t* act_q, float* act_scale, int32_t* act_sum,
                                   hipStream_t s, bool bf16 = false);   // x fp16, or bf16 bits

// Quantized linear (qift_linear.hip).  fmt selects the decode.  ws (nullable): at M > 64 the GEMM split
// over K where gemm_split_workspace(fmt, N, M, K) (its bytes) is not 0, else for MNZ and PoT weights the
// FP4 x FP6 MFMA kernel with gemm_f4_workspace(N, M, K) bytes.
size_t gemm_split_workspace(int fmt, int64_t N, int64_t M, int64_t K);
hipError_t launch_linear(int fmt, const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K,
                         const int8_t* act_q, const float* act_scale, const int32_t* act_sum, int64_t M,
                         uint16_t* out, int32_t* acc_out, void* ws, hipStream_t s);

// MNZ and PoT prefill on the FP4 x FP6 scaled MFMA (qift_prefill_f4.hip): act_q re-coded to FP6
// into ws (gemm_f4_workspace(N, M, K) bytes), then the GEMM, split over K into int32 partial sums in
// ws where its tiles are few; results identical to the int8 kernel.
constexpr int64_t kGemmF4MinM = 65;
size_t gemm_f4_workspace(int64_t N, int64_t M, int64_t K);
hipError_t launch_gemm_f4(int fmt, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K,
                          const int8_t* act_q, const float* sx, const int32_t* asum, int64_t M, uint16_t* y,
                          int32_t* acc_out, void* ws, hipStream_t s);

// Fused rotation + quantization + linear for a few decode tokens, one launcher
// per weight format (qift_fused_<fmt>.hip).
#define QIFT_FUSED_LAUNCHER(NAME)                                                                          \
  hipError_t NAME(const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K, const uint16_t* x, \
                  int block, int clip_num, int clip_den, int64_t M, uint16_t* out, int32_t* acc_out,       \
                  int8_t* act_q, float* act_scale, int32_t* act_sum, bool bf16, hipStream_t s)
QIFT_FUSED_LAUNCHER(launch_fused_mnz);
QIFT_FUSED_LAUNCHER(launch_fused_pot);
QIFT_FUSED_LAUNCHER(launch_fused_w4);
#undef QIFT_FUSED_LAUNCHER

// The same decode kernel as the linear on precomputed codes (M <= kCodesMaxM), one launcher per
// weight format; codes_shmem_<fmt> gives its LDS bytes (0 outside its limits), and the launcher
// returns hipErrorInvalidValue when they exceed 160 KiB.
#define QIFT_CODES_LAUNCHER(NAME)                                                                            \
  hipError_t NAME(const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K, const int8_t* act_q, \
                  const float* act_scale, const int32_t* act_sum, int64_t M, uint16_t* out, int32_t* acc_out, \
                  hipStream_t s)
QIFT_CODES_LAUNCHER(launch_codes_mnz);
QIFT_CODES_LAUNCHER(launch_codes_pot);
QIFT_CODES_LAUNCHER(launch_codes_w4);
#undef QIFT_CODES_LAUNCHER
size_t codes_shmem_mnz(int64_t M, int64_t N, int64_t K);
size_t codes_shmem_pot(int64_t M, int64_t N, int64_t K);
size_t codes_shmem_w4(int64_t M, int64_t N, int64_t K);

// Streaming-read probe (qift_probe.hip): reads bytes (a multiple of 16) once; workgroup b XORs the
// words of the 64 KiB segment b into partials[b].
constexpr size_t kReadProbeSegment = 65536;
size_t read_probe_slots(size_t bytes);
hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* partials, hipStream_t s);

// (den * 7) * sqrt(b): the fixed divisor of the per-token activation scale.
double act_denominator(int block, int clip_den);

// The per-device error word of the bounded device waits (qift_api.hip): its device address on the
// current device (nullptr if it cannot be resolved; the kernels then skip the report), and the spin
// limit of the waves' in-workgroup barriers (a test hook lowers it so that the waits give up).
uint32_t* device_error_word();
int wait_limit();
constexpr int kDefaultWaitLimit = 1 << 22;

// Persistent decode chain (qift_chain.h, qift_chain_<fmt>.hip): one link of a prepared chain as the
// kernel reads it (written to device memory by the prepare call).  A link whose output another link
// reads also writes it into the exchange copy ty[r mod 2] [M][ystride] of call r (and kUnwritten into
// the other copy); its consumers read element k of token m from tx[r mod 2][m][xoff + k].
struct ChainDesc {
  const uint32_t* P;     // packed words [N][K/16] (W2) or [N][K/8] (W4)
  const uint16_t* sw;    // fp16 s_w [N]
  const uint16_t* tx;    // the producer's exchange copies (nullptr: the chain input)
  uint16_t* ty;          // this link's exchange copies [2][M][ystride] (nullptr: no link reads this output)
  uint16_t* y;           // fp16 output [M][N]
  int32_t* acc;          // nullable int32 [M][N]
  double denom;          // (den * 7) * sqrt(block)
  int32_t N, K, L, num, den, in_link, xoff, xstride, ystride, tiles;
};
constexpr int kChainMaxM = 4;
// The fp16 pattern that marks an exchange value not yet written (a NaN no output carries there).
constexpr unsigned kUnwritten = 0xFFFFu;
// Hadamard blocks of the chain's links: 64, 256, 2048 and 4096 (the block exponent is compiled in)
inline bool chain_block_ok(int block) { return block == 64 || block == 256 || block == 2048 || block == 4096; }
constexpr int kChainMaxK = 16384;
constexpr int kChainMaxLinks = 4096;
constexpr int kChainSlots = 16;                    // per-token reduction slots (12 waves rotate long links)
constexpr int kChainTailBytes = 32 + 96 * kChainSlots + 32 + 64 + 8 * 256;
constexpr int kChainXchBytes = (4096 + 512) * 8;   // one rotation exchange buffer (a 4096-tile, padded)
// LDS rotation region: the activation group's exchange buffer, and for a chain with a link of more
// than one rotation tile (K > 4096) the two weight-wave groups' as well; aliased by the K-slice
// partial sums (8 slices x 7, W4 3, tiles).
inline int chain_region0(int max_tiles, bool w4) {
  const int own = (max_tiles > 1 ? 3 : 1) * kChainXchBytes, part = 8 * (w4 ? 3 : 7) * 1024;
  return own > part ? own : part;
}
inline size_t chain_lds_bytes(int64_t M, int64_t Kmax, int region0) {
  return (size_t)((M * (Kmax + 16) + 15) & ~int64_t(15)) + (size_t)region0 + kChainTailBytes;
}
#define QIFT_CHAIN_LAUNCHER(NAME)                                                                                \
  hipError_t NAME(const ChainDesc* links, int n_links, const uint16_t* x0, int M, int Kmax, int region0, int grid, \
                  unsigned* counters, hipStream_t s)
QIFT_CHAIN_LAUNCHER(launch_chain_mnz);
QIFT_CHAIN_LAUNCHER(launch_chain_pot);
QIFT_CHAIN_LAUNCHER(launch_chain_w4);
#undef QIFT_CHAIN_LAUNCHER

// Limits of the fused entry point.
constexpr int64_t kFusedMaxM = 4;
constexpr int64_t kCodesMaxM = 16;   // one MFMA column block of tokens
// Skinny decode linear (qift_skinny.hip): up to 64 tokens in one pass over the weights, codes read
// from memory by the K-slice waves.
constexpr int64_t kSkinnyMaxM = 64;
constexpr int64_t kSkinnyMaxK = 16384;
hipError_t launch_skinny(int fmt, const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K,
                         const int8_t* act_q, const float* act_scale, const int32_t* act_sum, int64_t M,
                         uint16_t* out, int32_t* acc_out, hipStream_t s);
// The same split over K for W2 weights (MNZ, PoT) whose few 16-row tiles would leave every workgroup
// reading all M x K codes for 16 or 32 rows (M <= 64; up to 16 tokens only where the decode kernel on
// codes does not fit): ws holds skinny_workspace(fmt, N, K, M) bytes (0: no split for this linear;
// then, or with ws null, the call above).
size_t skinny_workspace(int fmt, int64_t N, int64_t K, int64_t M);
hipError_t launch_skinny_ws(int fmt, const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K,
                            const int8_t* act_q, const float* act_scale, const int32_t* act_sum, int64_t M,
                            uint16_t* out, int32_t* acc_out, void* ws, hipStream_t s);
constexpr int64_t kFusedMaxK = 16384;
constexpr int kFusedMaxBlock = 4096;
// Largest K accepted by the activation quantizer.
constexpr int64_t kActMaxK = 32768;

}  // namespace qift
