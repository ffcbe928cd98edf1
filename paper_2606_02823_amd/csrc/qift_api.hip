// C ABI of libqift: host-side validation, then dispatch to the launchers.
// Every check runs before the first HIP call, so an error return means
// nothing was enqueued (and these paths run on machines without a GPU).
#include <math.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "../../include/qift.h"
#include "qift_fwht.h"   // ilog2c
#include "qift_internal.h"

// The error word of the bounded device waits: one per device (each device holds its own copy of
// this variable), set by kernels whose waits give up, read and cleared by qift_device_error.
__device__ uint32_t qift_device_error_bits;

namespace {

thread_local int g_last_hip = 0;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int hip_status(hipError_t e) {
  if (e == hipSuccess) return QIFT_OK;
  g_last_hip = (int)e;
  return QIFT_ERR_HIP;
}

inline bool is_w2(int32_t fmt) { return fmt == QIFT_W2_MNZ || fmt == QIFT_W2_POT; }
// 2-bit formats that pack into QW2v1 words (the integer sets and the level-table codes)
inline bool is_qw2(int32_t fmt) { return is_w2(fmt) || fmt == QIFT_W2_LUT; }

// IEEE binary16 bits -> double, exactly (non-finite values come back as inf / nan)
double half_bits_to_double(uint16_t h) {
  const int sign = h >> 15, e = (h >> 10) & 31, f = h & 1023;
  double v;
  if (e == 31) v = f ? NAN : INFINITY;
  else if (e == 0) v = ldexp((double)f, -24);
  else v = ldexp((double)(1024 + f), e - 25);
  return sign ? -v : v;
}

inline bool shape_ok(int64_t N, int64_t K) {
  // K: multiple of 64; sizes kept below 2^31 per dimension (int indexing inside tiles)
  return N >= 1 && K >= 64 && K % 64 == 0 && N < (int64_t(1) << 31) && K < (int64_t(1) << 31);
}

// Clip ratio num/den of a Hadamard spec: flags 0 is 1/1, else QIFT_CLIP(num, den) with
// 1 <= num <= den <= 16 and no other bits set.
bool parse_clip(int32_t flags, int* num, int* den) {
  if (flags == 0) {
    *num = *den = 1;
    return true;
  }
  if (flags & ~0xFFFF) return false;
  *num = (flags >> 8) & 0xFF;
  *den = flags & 0xFF;
  return *num >= 1 && *num <= *den && *den <= 16;
}

// Flags of an activation spec: the clip ratio, and QIFT_SPEC_BF16 (the tokens are bf16 values).
bool parse_act_flags(int32_t flags, int* num, int* den, bool* bf16) {
  *bf16 = (flags & QIFT_SPEC_BF16) != 0;
  return parse_clip(flags & ~QIFT_SPEC_BF16, num, den);
}

int check_linear(const qift_packed_w* w, bool want_w4, const int8_t* act_q, const float* act_scale,
                 const int32_t* act_sum, int64_t M, const uint16_t* out, const int32_t* acc_out) {
  if (!w || !act_q || !act_scale || !out || !w->packed || !w->scales) return QIFT_ERR_NULL;
  if (w->layout != QIFT_LAYOUT_V1) return QIFT_ERR_FORMAT;
  if (want_w4 ? w->fmt != QIFT_W4_SYM : !is_w2(w->fmt)) return QIFT_ERR_FORMAT;
  if (!shape_ok(w->N, w->K) || M < 1 || M >= (int64_t(1) << 31)) return QIFT_ERR_SHAPE;
  // exact int32 accumulation: |acc| <= 7 * 7 * K stays far below 2^31 for K < 2^24
  if (w->K >= (int64_t(1) << 24)) return QIFT_ERR_SHAPE;
  // buffer-resource loads address each operand with 32-bit offsets below 2^31
  if (qift_packed_bytes(w->fmt, w->N, w->K) >= (size_t(1) << 31)) return QIFT_ERR_SHAPE;
  if (!aligned16(w->packed) || !aligned16(act_q) || !aligned16(w->scales) || !aligned16(act_scale) ||
      (act_sum && !aligned16(act_sum)) || !aligned16(out) || (acc_out && !aligned16(acc_out)))
    return QIFT_ERR_ALIGN;
  return QIFT_OK;
}

// The out-of-set level counter of the packers: one int32 per device in device memory, allocated by
// the first pack call on that device (an offline call) and kept until the process ends.  The mutex
// is held from the launch until the count has been read back, so concurrent pack calls never share
// a count.
std::mutex g_pack_mu;
constexpr int kMaxDevices = 64;
int32_t* g_pack_ctr[kMaxDevices] = {};

template <typename Launch>
int pack_checked(Launch launch, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_pack_mu);
  int dev = 0;
  int st = hip_status(hipGetDevice(&dev));
  if (st != QIFT_OK) return st;
  if (dev < 0 || dev >= kMaxDevices) return hip_status(hipErrorInvalidDevice);
  if (!g_pack_ctr[dev]) {
    st = hip_status(hipMalloc(reinterpret_cast<void**>(&g_pack_ctr[dev]), sizeof(int32_t)));
    if (st != QIFT_OK) return st;
  }
  st = hip_status(launch(g_pack_ctr[dev]));
  if (st != QIFT_OK) return st;
  int32_t bad = 0;
  st = hip_status(hipMemcpyAsync(&bad, g_pack_ctr[dev], sizeof(bad), hipMemcpyDeviceToHost, stream));
  if (st == QIFT_OK) st = hip_status(hipStreamSynchronize(stream));
  if (st != QIFT_OK) return st;
  return bad ? QIFT_ERR_CODE : QIFT_OK;
}

int linear_common(const qift_packed_w* w, bool w4, const int8_t* act_q, const float* act_scale,
                  const int32_t* act_sum, int64_t M, uint16_t* out, int32_t* acc_out, void* ws,
                  size_t ws_bytes, qift_stream_t stream) {
  int st = check_linear(w, w4, act_q, act_scale, act_sum, M, out, acc_out);
  if (st != QIFT_OK) return st;
  // the workspace is optional: none selects the int8 kernels, one of at least qift_workspace_bytes
  // the FP4 x FP6 prefill kernel where that query is not 0
  const size_t need = qift_workspace_bytes(w, M);
  if (ws_bytes > 0 && (!ws || ws_bytes < need)) return QIFT_ERR_WORKSPACE;
  if (ws && !aligned16(ws)) return QIFT_ERR_ALIGN;
  void* use = ws_bytes > 0 && need > 0 ? ws : nullptr;
  return hip_status(qift::launch_linear(w->fmt, w->packed, w->scales, w->N, w->K, act_q, act_scale,
                                        act_sum, M, out, acc_out, use, (hipStream_t)stream));
}

std::mutex g_err_mu;
uint32_t* g_err_word[kMaxDevices] = {};
bool g_err_tried[kMaxDevices] = {};
std::atomic<int> g_wait_limit{qift::kDefaultWaitLimit};

}  // namespace

namespace qift {

uint32_t* device_error_word() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_err_mu);
  if (!g_err_tried[dev]) {
    // the device address of this device's copy of the symbol (resolved once per device)
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(qift_device_error_bits)) == hipSuccess) g_err_word[dev] = (uint32_t*)p;
    g_err_tried[dev] = true;
  }
  return g_err_word[dev];
}

int wait_limit() { return g_wait_limit.load(std::memory_order_relaxed); }

}  // namespace qift

extern "C" {

size_t qift_packed_bytes(int32_t fmt, int64_t N, int64_t K) {
  if (!shape_ok(N, K)) return 0;
  if (is_qw2(fmt)) return (size_t)(N * (K / 4));
  if (fmt == QIFT_W4_SYM) return (size_t)(N * (K / 2));
  return 0;
}

int qift_pack_w2(const int8_t* levels, const uint16_t* scales, int64_t N, int64_t K, int32_t fmt,
                 uint32_t* packed, qift_packed_w* out, qift_stream_t stream) {
  if (!levels || !packed) return QIFT_ERR_NULL;
  if (!is_qw2(fmt)) return QIFT_ERR_FORMAT;
  if (!shape_ok(N, K)) return QIFT_ERR_SHAPE;
  if (!aligned16(levels) || !aligned16(packed) || (scales && !aligned16(scales))) return QIFT_ERR_ALIGN;
  const hipStream_t s = (hipStream_t)stream;
  const int st = pack_checked([&](int32_t* ctr) { return qift::launch_pack_w2(levels, N, K, fmt, packed, ctr, s); }, s);
  if (st == QIFT_OK && out) *out = qift_packed_w{fmt, QIFT_LAYOUT_V1, N, K, packed, scales};
  return st;
}

int qift_pack_w4(const int8_t* levels, const uint16_t* scales, int64_t N, int64_t K, uint32_t* packed,
                 qift_packed_w* out, qift_stream_t stream) {
  if (!levels || !packed) return QIFT_ERR_NULL;
  if (!shape_ok(N, K)) return QIFT_ERR_SHAPE;
  if (!aligned16(levels) || !aligned16(packed) || (scales && !aligned16(scales))) return QIFT_ERR_ALIGN;
  const hipStream_t s = (hipStream_t)stream;
  const int st = pack_checked([&](int32_t* ctr) { return qift::launch_pack_w4(levels, N, K, packed, ctr, s); }, s);
  if (st == QIFT_OK && out) *out = qift_packed_w{QIFT_W4_SYM, QIFT_LAYOUT_V1, N, K, packed, scales};
  return st;
}

int qift_quantize_weights(const float* W, int64_t N, qift_hadamard_spec spec, int32_t fmt, int8_t* levels,
                          uint16_t* scales, qift_stream_t stream) {
  if (!W || !levels || !scales) return QIFT_ERR_NULL;
  if (fmt != QIFT_W2_MNZ && fmt != QIFT_W2_POT && fmt != QIFT_W4_SYM) return QIFT_ERR_FORMAT;
  if (!shape_ok(N, spec.K) || spec.K > qift::kWquantMaxK) return QIFT_ERR_SHAPE;
  // 32-bit offsets of the level stores and row loads
  if (N * spec.K >= (int64_t(1) << 31)) return QIFT_ERR_SHAPE;
  const int32_t b = spec.block;
  if (b < 2 || b > 4096 || (b & (b - 1)) || spec.K % b) return QIFT_ERR_SPEC;
  if (spec.flags != 0) return QIFT_ERR_SPEC;
  if (!aligned16(W) || !aligned16(levels) || !aligned16(scales)) return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_quantize_weights(W, N, spec.K, b, fmt, levels, scales, (hipStream_t)stream));
}

int qift_quantize_weights_mirror(const float* W, int64_t N, qift_hadamard_spec spec, double r, int8_t* codes,
                                 uint16_t* scales, qift_stream_t stream) {
  if (!W || !codes || !scales) return QIFT_ERR_NULL;
  if (!shape_ok(N, spec.K) || spec.K > qift::kWquantMaxK) return QIFT_ERR_SHAPE;
  if (N * spec.K >= (int64_t(1) << 31)) return QIFT_ERR_SHAPE;
  const int32_t b = spec.block;
  if (b < 2 || b > 4096 || (b & (b - 1)) || spec.K % b) return QIFT_ERR_SPEC;
  if (spec.flags != 0) return QIFT_ERR_SPEC;
  if (!(r > 0.0 && r < 1.0)) return QIFT_ERR_SPEC;   // also rejects NaN
  if (!aligned16(W) || !aligned16(codes) || !aligned16(scales)) return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_quantize_weights_mirror(W, N, spec.K, b, r, codes, scales, (hipStream_t)stream));
}

int qift_ratio_scan(const double* x, int64_t n, const double* ratios, int32_t n_ratios, const double* cands,
                    int32_t n_cands, double* sse, double* nmse, int32_t* best, double* stats,
                    qift_stream_t stream) {
  if (!x || !ratios || !cands || !sse || !nmse || !best || !stats) return QIFT_ERR_NULL;
  if (n < 1 || n >= (int64_t(1) << 40)) return QIFT_ERR_SHAPE;
  if (n_ratios < 1 || n_ratios > qift::kScanMaxRatios || n_cands < 1 || n_cands > qift::kScanMaxCands)
    return QIFT_ERR_SHAPE;
  for (int32_t i = 0; i < n_ratios; ++i)
    if (!(ratios[i] > 0.0 && ratios[i] < 1.0)) return QIFT_ERR_SPEC;
  for (int32_t j = 0; j < n_cands; ++j)
    if (!(cands[j] > 0.0 && cands[j] <= 1e300)) return QIFT_ERR_SPEC;   // positive and finite
  if (!aligned16(x) || !aligned16(sse) || !aligned16(nmse) || !aligned16(best) || !aligned16(stats))
    return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_ratio_scan(x, n, ratios, n_ratios, cands, n_cands, sse, nmse, best, stats,
                                            (hipStream_t)stream));
}

int qift_kv4_quant(const uint16_t* x, int64_t groups, int32_t head_dim, uint8_t* codes, float* scales,
                   uint8_t* zeros, qift_stream_t stream) {
  if (!x || !codes || !scales || !zeros) return QIFT_ERR_NULL;
  if (head_dim != 128 || groups < 1 || groups >= (int64_t(1) << 40)) return QIFT_ERR_SHAPE;
  // x is read with 16-byte loads; codes (4-byte words) and scales (fp32) need 4 bytes; zero-points are
  // single bytes, so a cache view at any token position (e.g. one appended decode token) is accepted
  auto aligned4 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; };
  if (!aligned16(x) || !aligned4(codes) || !aligned4(scales)) return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_kv4_quant(x, groups, codes, scales, zeros, (hipStream_t)stream));
}

namespace {
bool kv4_attn_shape_ok(int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim, int64_t T) {
  if (head_dim != 128 || B < 1 || B > 65535 || Hkv < 1 || Hkv > 65535 || Hq < Hkv || Hq % Hkv) return false;
  const int32_t G = Hq / Hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8) return false;
  // 32-bit offsets into one sequence's cache: T Hkv 64 bytes of codes below 2^31
  return T >= 1 && T * Hkv * 64 < (int64_t(1) << 31);
}
}  // namespace

size_t qift_kv4_attention_workspace_bytes(int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim, int64_t T) {
  if (!kv4_attn_shape_ok(B, Hq, Hkv, head_dim, T)) return 0;
  return qift::kv4_attention_workspace(B, Hq, T);
}

int qift_kv4_attention_decode(const uint16_t* q, int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim, int64_t T,
                              int32_t layout, const uint8_t* k_codes, const float* k_scales, const uint8_t* k_zeros,
                              const uint8_t* v_codes, const float* v_scales, const uint8_t* v_zeros, uint16_t* out,
                              void* workspace, size_t workspace_bytes, qift_stream_t stream) {
  if (!q || !k_codes || !k_scales || !k_zeros || !v_codes || !v_scales || !v_zeros || !out) return QIFT_ERR_NULL;
  if (!kv4_attn_shape_ok(B, Hq, Hkv, head_dim, T)) return QIFT_ERR_SHAPE;
  if (layout != QIFT_KV4_TOKEN_MAJOR && layout != QIFT_KV4_HEAD_MAJOR) return QIFT_ERR_SPEC;
  if (!workspace || workspace_bytes < qift::kv4_attention_workspace(B, Hq, T)) return QIFT_ERR_WORKSPACE;
  if (!aligned16(q) || !aligned16(k_codes) || !aligned16(k_scales) || !aligned16(k_zeros) || !aligned16(v_codes) ||
      !aligned16(v_scales) || !aligned16(v_zeros) || !aligned16(out) || !aligned16(workspace))
    return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_kv4_attention(q, B, Hq, Hkv, T, layout == QIFT_KV4_HEAD_MAJOR, k_codes, k_scales, k_zeros, v_codes, v_scales,
                                               v_zeros, out, workspace, (hipStream_t)stream));
}

}  // extern "C"

// The device scratch of qift_kv4_attention_decode_noalloc: the split-T partial records.  Each GPU
// holds its own copy for the life of the process; host code reaches it only through the device
// address resolved below (the symbol's name is a host-side stand-in).
static __device__ __align__(256) unsigned char scratch[QIFT_KV4_SCRATCH_BYTES];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kScratchDevices] = {};

// The current device's address of scratch, resolved once per device with that device current.
int scratch_address(void** out) {
  int dev = 0;
  int st = hip_status(hipGetDevice(&dev));
  if (st != QIFT_OK) return st;
  if (dev < 0 || dev >= kScratchDevices) return hip_status(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    st = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (st != QIFT_OK) return st;
    if (!p) return hip_status(hipErrorInvalidSymbol);
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return QIFT_OK;
}
}  // namespace

extern "C" {

int qift_kv4_attention_decode_noalloc(const uint16_t* q, int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim,
                                      int64_t T, int32_t layout, const uint8_t* k_codes, const float* k_scales,
                                      const uint8_t* k_zeros, const uint8_t* v_codes, const float* v_scales,
                                      const uint8_t* v_zeros, uint16_t* out, qift_stream_t stream) {
  if (!q || !k_codes || !k_scales || !k_zeros || !v_codes || !v_scales || !v_zeros || !out) return QIFT_ERR_NULL;
  if (!kv4_attn_shape_ok(B, Hq, Hkv, head_dim, T)) return QIFT_ERR_SHAPE;
  if (layout != QIFT_KV4_TOKEN_MAJOR && layout != QIFT_KV4_HEAD_MAJOR) return QIFT_ERR_SPEC;
  // every record the call writes fits in the array (no record has to start at zero: each call
  // writes all of the records its merge reads)
  if (qift::kv4_attention_workspace(B, Hq, T) > (size_t)QIFT_KV4_SCRATCH_BYTES) return QIFT_ERR_WORKSPACE;
  if (!aligned16(q) || !aligned16(k_codes) || !aligned16(k_scales) || !aligned16(k_zeros) || !aligned16(v_codes) ||
      !aligned16(v_scales) || !aligned16(v_zeros) || !aligned16(out))
    return QIFT_ERR_ALIGN;
  void* ws = nullptr;
  const int st = scratch_address(&ws);
  if (st != QIFT_OK) return st;
  return hip_status(qift::launch_kv4_attention(q, B, Hq, Hkv, T, layout == QIFT_KV4_HEAD_MAJOR, k_codes, k_scales,
                                               k_zeros, v_codes, v_scales, v_zeros, out, ws, (hipStream_t)stream));
}


namespace {
int rotate_quant_act(const uint16_t* x, int64_t M, qift_hadamard_spec spec, int8_t* act_q, float* act_scale,
                     int32_t* act_sum, qift_stream_t stream, bool bf16) {
  if (!x || !act_q || !act_scale) return QIFT_ERR_NULL;
  if (M < 1 || M >= (int64_t(1) << 31) || spec.K < 64 || spec.K % 64 || spec.K > qift::kActMaxK)
    return QIFT_ERR_SHAPE;
  const int32_t b = spec.block;
  if (b < 2 || b > 8192 || (b & (b - 1)) || spec.K % b) return QIFT_ERR_SPEC;
  int num, den;
  bool flag_bf16 = false;
  if (!parse_act_flags(spec.flags, &num, &den, &flag_bf16)) return QIFT_ERR_SPEC;
  if (!aligned16(x) || !aligned16(act_q) || !aligned16(act_scale) || (act_sum && !aligned16(act_sum)))
    return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_rotate_quant_act(x, M, spec.K, b, num, den, act_q, act_scale, act_sum,
                                                  (hipStream_t)stream, bf16 || flag_bf16));
}
}  // namespace

int qift_rotate_quant_act(const uint16_t* x, int64_t M, qift_hadamard_spec spec, int8_t* act_q,
                          float* act_scale, int32_t* act_sum, qift_stream_t stream) {
  return rotate_quant_act(x, M, spec, act_q, act_scale, act_sum, stream, false);
}

int qift_w2a4_lut_linear(const qift_packed_w* w, const uint16_t* lut, const int8_t* act_q, const float* act_scale,
                         int64_t M, uint16_t* out, qift_stream_t stream) {
  if (!w || !lut || !act_q || !act_scale || !out || !w->packed || !w->scales) return QIFT_ERR_NULL;
  if (w->layout != QIFT_LAYOUT_V1 || w->fmt != QIFT_W2_LUT) return QIFT_ERR_FORMAT;
  // K: whole 256-k blocks, and at most 2^14 for the exact fp64 combination; token blocks of 16 in grid.y
  if (!shape_ok(w->N, w->K) || w->K % 256 || w->K > 16384 || M < 1 || M > 16 * 65535) return QIFT_ERR_SHAPE;
  if (qift_packed_bytes(w->fmt, w->N, w->K) >= (size_t(1) << 31)) return QIFT_ERR_SHAPE;
  double L[4];
  for (int i = 0; i < 4; ++i) {
    L[i] = half_bits_to_double(lut[i]);
    if (!(fabs(L[i]) <= 256.0)) return QIFT_ERR_SPEC;   // also rejects inf and nan
  }
  if (!aligned16(w->packed) || !aligned16(w->scales) || !aligned16(act_q) || !aligned16(act_scale) ||
      !aligned16(out))
    return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_lut_linear(w->packed, w->scales, w->N, w->K, L, act_q, act_scale, M, out,
                                            (hipStream_t)stream));
}

int qift_rotate_quant_act_bf16(const uint16_t* x, int64_t M, qift_hadamard_spec spec, int8_t* act_q,
                               float* act_scale, int32_t* act_sum, qift_stream_t stream) {
  return rotate_quant_act(x, M, spec, act_q, act_scale, act_sum, stream, true);
}

int qift_w2a4_linear(const qift_packed_w* w, const int8_t* act_q, const float* act_scale, int64_t M, uint16_t* out,
                     qift_stream_t stream) {
  return linear_common(w, false, act_q, act_scale, nullptr, M, out, nullptr, nullptr, 0, stream);
}

int qift_w2a4_linear_ex(const qift_packed_w* w, const int8_t* act_q, const float* act_scale,
                        const int32_t* act_sum, int64_t M, uint16_t* out, int32_t* acc_out,
                        void* workspace, size_t workspace_bytes, qift_stream_t stream) {
  return linear_common(w, false, act_q, act_scale, act_sum, M, out, acc_out, workspace, workspace_bytes,
                       stream);
}

int qift_w4a4_linear(const qift_packed_w* w, const int8_t* act_q, const float* act_scale, int64_t M, uint16_t* out,
                     qift_stream_t stream) {
  return linear_common(w, true, act_q, act_scale, nullptr, M, out, nullptr, nullptr, 0, stream);
}

int qift_w4a4_linear_ex(const qift_packed_w* w, const int8_t* act_q, const float* act_scale,
                        const int32_t* act_sum, int64_t M, uint16_t* out, int32_t* acc_out,
                        void* workspace, size_t workspace_bytes, qift_stream_t stream) {
  return linear_common(w, true, act_q, act_scale, act_sum, M, out, acc_out, workspace, workspace_bytes,
                       stream);
}

int qift_rotate_quant_linear(const qift_packed_w* w, const uint16_t* x, int64_t M, qift_hadamard_spec spec,
                             uint16_t* out, int32_t* acc_out, int8_t* act_q, float* act_scale,
                             int32_t* act_sum, qift_stream_t stream) {
  if (!w || !x || !out || !w->packed || !w->scales) return QIFT_ERR_NULL;
  const int given = (act_q != nullptr) + (act_scale != nullptr) + (act_sum != nullptr);
  if (given != 0 && given != 3) return QIFT_ERR_NULL;
  if (w->layout != QIFT_LAYOUT_V1 || !(is_w2(w->fmt) || w->fmt == QIFT_W4_SYM)) return QIFT_ERR_FORMAT;
  if (!shape_ok(w->N, w->K) || M < 1 || M > qift::kFusedMaxM || w->K > qift::kFusedMaxK) return QIFT_ERR_SHAPE;
  if (qift_packed_bytes(w->fmt, w->N, w->K) >= (size_t(1) << 31)) return QIFT_ERR_SHAPE;
  const int32_t b = spec.block;
  if (spec.K != w->K || b < 2 || b > qift::kFusedMaxBlock || (b & (b - 1)) || spec.K % b) return QIFT_ERR_SPEC;
  int num, den;
  bool bf16 = false;
  if (!parse_act_flags(spec.flags, &num, &den, &bf16)) return QIFT_ERR_SPEC;
  if (!aligned16(w->packed) || !aligned16(w->scales) || !aligned16(x) || !aligned16(out) ||
      (acc_out && !aligned16(acc_out)) || (act_q && !aligned16(act_q)) ||
      (act_scale && !aligned16(act_scale)) || (act_sum && !aligned16(act_sum)))
    return QIFT_ERR_ALIGN;
  auto launch = w->fmt == QIFT_W2_MNZ ? qift::launch_fused_mnz
               : w->fmt == QIFT_W2_POT ? qift::launch_fused_pot
                                       : qift::launch_fused_w4;
  return hip_status(launch(w->packed, w->scales, w->N, w->K, x, b, num, den, M, out, acc_out, act_q, act_scale,
                           act_sum, bf16, (hipStream_t)stream));
}

// ---- decode chain -------------------------------------------------------------------------------

namespace {
size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
constexpr size_t kChainCounterBytes = 256;   // the arrival count and the run number, padded

// Host-side checks of a chain and the device link table (every check before any HIP call).  With a
// workspace base, the exchange buffers of the links whose output another link reads (two copies of
// the fp16 output, rows padded to 8 values) are laid out after the table and the counters;
// *ws_bytes receives the workspace size either way.
int chain_build(const qift_chain_link* links, int32_t n, int64_t M, int64_t K0, unsigned char* ws,
                std::vector<qift::ChainDesc>& d, size_t* ws_bytes, int64_t* kmax_out, int* region0) {
  if (!links) return QIFT_ERR_NULL;
  if (n < 1 || n > qift::kChainMaxLinks) return QIFT_ERR_SHAPE;
  if (M < 1 || M > qift::kChainMaxM || K0 < 64 || K0 % 64 || K0 > qift::kChainMaxK) return QIFT_ERR_SHAPE;
  const int32_t fmt = links[0].w.fmt;
  if (!(is_w2(fmt) || fmt == QIFT_W4_SYM)) return QIFT_ERR_FORMAT;
  d.assign((size_t)n, qift::ChainDesc{});
  std::vector<char> consumed((size_t)n, 0);
  int64_t kmax = 0;
  for (int32_t i = 0; i < n; ++i) {
    const qift_chain_link& l = links[i];
    const qift_packed_w& w = l.w;
    if (!w.packed || !w.scales || !l.out) return QIFT_ERR_NULL;
    if (w.layout != QIFT_LAYOUT_V1 || w.fmt != fmt) return QIFT_ERR_FORMAT;
    // N below 2^26 keeps the kernel's tile split (tiles x (CUs + 1)) in 32 bits
    if (!shape_ok(w.N, w.K) || w.K > qift::kChainMaxK || w.N >= (int64_t(1) << 26)) return QIFT_ERR_SHAPE;
    if (qift_packed_bytes(fmt, w.N, w.K) >= (size_t(1) << 31) || M * w.N * 8 >= (int64_t(1) << 31))
      return QIFT_ERR_SHAPE;
    const int32_t b = l.block;
    int num, den;
    if (!qift::chain_block_ok(b) || w.K % b || l.reserved != 0 || !parse_clip(l.flags, &num, &den))
      return QIFT_ERR_SPEC;
    if (l.in_link < -1 || l.in_link >= i) return QIFT_ERR_SHAPE;
    if (l.in_link < 0) {
      if (w.K != K0 || l.in_offset != 0) return QIFT_ERR_SHAPE;
    } else {
      const int64_t Nin = links[l.in_link].w.N;
      if (l.in_offset < 0 || l.in_offset % 8 || l.in_offset + w.K > Nin) return QIFT_ERR_SHAPE;
      consumed[(size_t)l.in_link] = 1;
    }
    if (!aligned16(w.packed) || !aligned16(w.scales) || !aligned16(l.out) || (l.acc_out && !aligned16(l.acc_out)))
      return QIFT_ERR_ALIGN;
    // the outputs of different links are disjoint
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(l.out), a1 = a0 + (uintptr_t)(M * w.N * 2);
    for (int32_t j = 0; j < i; ++j) {
      const uintptr_t b0 = reinterpret_cast<uintptr_t>(links[j].out), b1 = b0 + (uintptr_t)(M * links[j].w.N * 2);
      if (a0 < b1 && b0 < a1) return QIFT_ERR_SHAPE;
    }
    qift::ChainDesc& e = d[(size_t)i];
    e.P = w.packed;
    e.sw = w.scales;
    e.y = l.out;
    e.acc = l.acc_out;
    e.denom = qift::act_denominator(b, den);
    e.N = (int32_t)w.N;
    e.K = (int32_t)w.K;
    e.L = qift::dev::ilog2c(b);
    e.num = num;
    e.den = den;
    e.in_link = l.in_link;
    e.xoff = (int32_t)l.in_offset;
    e.ystride = (int32_t)((w.N + 7) & ~int64_t(7));
    e.tiles = (int32_t)((w.N + 15) / 16);
    kmax = w.K > kmax ? w.K : kmax;
  }
  // workspace: link table, counters, then the exchange buffers of the links that are read
  size_t off = align256((size_t)n * sizeof(qift::ChainDesc)) + kChainCounterBytes;
  for (int32_t i = 0; i < n; ++i) {
    if (!consumed[(size_t)i]) continue;
    d[(size_t)i].ty = ws ? reinterpret_cast<uint16_t*>(ws + off) : nullptr;
    off += align256(2 * (size_t)M * (size_t)d[(size_t)i].ystride * 2);
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t in = d[(size_t)i].in_link;
    if (in >= 0) {
      d[(size_t)i].tx = d[(size_t)in].ty;
      d[(size_t)i].xstride = d[(size_t)in].ystride;
    }
  }
  *ws_bytes = off;
  *region0 = qift::chain_region0((int)((kmax + 4095) / 4096), fmt == QIFT_W4_SYM);
  if (qift::chain_lds_bytes(M, kmax, *region0) > 160 * 1024) return QIFT_ERR_SHAPE;
  *kmax_out = kmax;
  return QIFT_OK;
}
}  // namespace

size_t qift_chain_workspace_bytes(const qift_chain_link* links, int32_t n_links, int64_t M) {
  std::vector<qift::ChainDesc> d;
  size_t bytes = 0;
  int64_t kmax = 0;
  int r0 = 0;
  if (!links || n_links < 1 || n_links > qift::kChainMaxLinks) return 0;
  if (chain_build(links, n_links, M, links[0].w.K, nullptr, d, &bytes, &kmax, &r0) != QIFT_OK) return 0;
  return bytes;
}

int qift_chain_prepare(const qift_chain_link* links, int32_t n_links, int64_t M, int64_t K0, void* workspace,
                       size_t workspace_bytes, qift_chain* chain, qift_stream_t stream) {
  if (!links || !workspace || !chain) return QIFT_ERR_NULL;
  if (!aligned16(workspace)) return QIFT_ERR_ALIGN;
  std::vector<qift::ChainDesc> d;
  size_t need = 0;
  int64_t kmax = 0;
  int r0 = 0;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  int st = chain_build(links, n_links, M, K0, ws, d, &need, &kmax, &r0);
  if (st != QIFT_OK) return st;
  if (workspace_bytes < need) return QIFT_ERR_WORKSPACE;
  int dev = 0, cus = 0;
  st = hip_status(hipGetDevice(&dev));
  if (st == QIFT_OK) st = hip_status(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  if (st != QIFT_OK) return st;
  if (cus < 1) return hip_status(hipErrorInvalidDevice);
  const hipStream_t s = (hipStream_t)stream;
  const size_t table = align256((size_t)n_links * sizeof(qift::ChainDesc));
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws + table);
  static const uint32_t start[2] = {0u, 1u};   // arrival count 0, run number 1
  st = hip_status(hipMemcpyAsync(ws, d.data(), (size_t)n_links * sizeof(qift::ChainDesc), hipMemcpyHostToDevice, s));
  // every exchange value starts as not written (0xFFFF)
  if (st == QIFT_OK) st = hip_status(hipMemsetAsync(ws + table, 0xFF, need - table, s));
  if (st == QIFT_OK) st = hip_status(hipMemcpyAsync(counters, start, sizeof(start), hipMemcpyHostToDevice, s));
  if (st == QIFT_OK) st = hip_status(hipStreamSynchronize(s));
  if (st != QIFT_OK) return st;
  *chain = qift_chain{links[0].w.fmt, n_links, (int32_t)M, (int32_t)K0, cus, (int32_t)kmax, r0, 0, ws, counters};
  return QIFT_OK;
}

int qift_decode_chain(const qift_chain* c, const uint16_t* x, qift_stream_t stream) {
  if (!c || !x || !c->table || !c->counters) return QIFT_ERR_NULL;
  if (c->n_links < 1 || c->n_links > qift::kChainMaxLinks || c->M < 1 || c->M > qift::kChainMaxM || c->grid < 1 ||
      c->kmax < 64 || c->kmax > qift::kChainMaxK || c->K0 < 64 || c->K0 > c->kmax || c->region0 < 0 ||
      qift::chain_lds_bytes(c->M, c->kmax, c->region0) > 160 * 1024)
    return QIFT_ERR_SHAPE;
  if (!(is_w2(c->fmt) || c->fmt == QIFT_W4_SYM)) return QIFT_ERR_FORMAT;
  if (!aligned16(x) || !aligned16(c->table) || !aligned16(c->counters)) return QIFT_ERR_ALIGN;
  auto launch = c->fmt == QIFT_W2_MNZ ? qift::launch_chain_mnz : c->fmt == QIFT_W2_POT ? qift::launch_chain_pot
                                                                                       : qift::launch_chain_w4;
  return hip_status(launch(static_cast<const qift::ChainDesc*>(c->table), c->n_links, x, c->M, c->kmax, c->region0,
                           c->grid, reinterpret_cast<unsigned*>(c->counters), (hipStream_t)stream));
}

int qift_hbm_read_probe(const void* buf, size_t bytes, uint32_t* partials, qift_stream_t stream) {
  if (!buf || !partials) return QIFT_ERR_NULL;
  if (bytes == 0 || bytes % 16 || qift::read_probe_slots(bytes) > 0x7fffffffu) return QIFT_ERR_SHAPE;
  if (!aligned16(buf) || (reinterpret_cast<uintptr_t>(partials) & 3u)) return QIFT_ERR_ALIGN;
  return hip_status(qift::launch_read_probe(buf, bytes, partials, (hipStream_t)stream));
}

size_t qift_workspace_bytes(const qift_packed_w* w, int64_t M) {
  if (!w || !shape_ok(w->N, w->K) || M < 1 || M >= (int64_t(1) << 31)) return 0;
  if (w->fmt != QIFT_W2_MNZ && w->fmt != QIFT_W2_POT && w->fmt != QIFT_W4_SYM) return 0;
  // the GEMM split over K where its tiles are few (and a wide linear from 33 tokens on)
  const size_t split = qift::gemm_split_workspace(w->fmt, w->N, M, w->K);
  if (split != 0 || w->fmt == QIFT_W4_SYM) return split;
  if (M <= qift::kSkinnyMaxM)   // the skinny linear split over K
    return qift::skinny_workspace(w->fmt, w->N, w->K, M);
  // the FP4 x FP6 kernel
  return qift::gemm_f4_workspace(w->N, M, w->K);
}

const char* qift_status_string(int status) {
  switch (status) {
    case QIFT_OK: return "ok";
    case QIFT_ERR_NULL: return "null pointer argument";
    case QIFT_ERR_SHAPE: return "invalid shape (M, N >= 1; K a positive multiple of 64; limits)";
    case QIFT_ERR_SPEC: return "invalid Hadamard block or clip ratio";
    case QIFT_ERR_FORMAT: return "wrong level-set format or layout for this call";
    case QIFT_ERR_CODE: return "level outside the format's level set (nothing usable was packed)";
    case QIFT_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case QIFT_ERR_HIP: return "HIP launch failed";
    case QIFT_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

int qift_last_hip_error(void) { return g_last_hip; }

int qift_device_error(uint32_t* bits, int32_t clear, qift_stream_t stream) {
  if (!bits) return QIFT_ERR_NULL;
  *bits = 0;
  uint32_t* word = qift::device_error_word();
  if (!word) return hip_status(hipErrorInvalidSymbol);
  const hipStream_t s = (hipStream_t)stream;
  int st = hip_status(hipMemcpyAsync(bits, word, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
  if (st == QIFT_OK && clear) st = hip_status(hipMemsetAsync(word, 0, sizeof(uint32_t), s));
  if (st == QIFT_OK) st = hip_status(hipStreamSynchronize(s));
  return st;
}

int qift_set_wait_limit(int32_t spins) {
  if (spins < 0) return QIFT_ERR_SHAPE;
  g_wait_limit.store(spins == 0 ? qift::kDefaultWaitLimit : spins, std::memory_order_relaxed);
  return QIFT_OK;
}

const char* qift_version(void) { return "qift 0.1 gfx950"; }

}  // extern "C"
