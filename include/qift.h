/*
 * qift.h - C ABI of the MI355X (gfx950) rotated W2A4 quantized linear.
 *
 * The operation (Qift, arXiv 2606.02823):
 *
 *   y[m, n] = s_w[n] * s_x[m] * sum_k level[n, k] * q[m, k]
 *
 * where level[n, :] is a row of a weight matrix quantized to a fixed
 * four-level set with one scale per output channel and no zero-point
 * (Sec. 3.3, Sec. 3.5), q[m, :] is the per-token INT4 quantization of the
 * Hadamard-rotated activation (Sec. 3.1; Sec. 4.1 "Quantization
 * configuration"), and both scales are applied after the exact integer
 * accumulation (Sec. 1; Sec. 3.6).
 *
 * Level sets ("formats"):
 *   QIFT_W2_MNZ  mirror no-zero {-1.5,-0.5,+0.5,+1.5}*s, stored as the odd
 *                integers {-3,-1,+1,+3} with the half scale s_w = s/2
 *                (Sec. 3.3 Eqs. (13)-(14)).
 *   QIFT_W2_POT  power-of-two no-zero {-4,-1,+1,+4}*s_w (Sec. 3.3 Eq. (17)).
 *   QIFT_W4_SYM  symmetric 4-bit integers -7..7 (Eq. (1) with b = 4, used on
 *                the symmetric range); the sibling format of the L-layer
 *                W2/W4 schedule (Sec. 4.4).
 *   QIFT_W2_LUT  any four levels given as an fp16 table indexed by the 2-bit
 *                code, for the non-integer reference grids of Sec. 3.3
 *                (Lloyd-Max Eq. (9), NF2 Eq. (10)); only qift_pack_w2 (with
 *                the codes 0..3 as "levels") and qift_w2a4_lut_linear take it.
 *
 * Conventions shared by every call:
 *   - fp16 values travel as uint16_t bit patterns (IEEE binary16).
 *   - Matrices are row-major and dense: x, act_q and y are [M][K] or [M][N];
 *     weights are [N][K] (output x input).
 *   - Every pointer argument is DEVICE memory owned by the caller unless the
 *     comment says "host".  The library keeps no pointer after a call
 *     returns and never frees caller memory; the only memory it allocates
 *     itself is one 4-byte counter per device for the offline pack calls.
 *     Buffers must stay alive until the work enqueued on the stream has
 *     completed.
 *   - Device pointers must be 16-byte aligned (QIFT_ERR_ALIGN otherwise).
 *   - K must be a positive multiple of 64; M >= 1; N >= 1 (no alignment).
 *   - Every call enqueues asynchronously on the caller's stream and returns
 *     a status; only the offline pack calls synchronize (to report
 *     QIFT_ERR_CODE).  Argument validation happens on the host before any
 *     HIP call, so an error return means nothing was enqueued.  Faults inside
 *     kernels surface at the caller's next synchronization.  No C++ exception
 *     crosses this interface.
 *   - Apart from that counter, a thread-local copy of the last HIP error and
 *     the per-device error word of the bounded device waits
 *     (qift_device_error), the library is stateless; calls are thread-safe.
 */
#ifndef QIFT_H
#define QIFT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t (a pointer to the runtime's opaque stream). */
typedef struct ihipStream_t *qift_stream_t;

/* ---- status codes ----------------------------------------------------- */
enum {
  QIFT_OK = 0,
  QIFT_ERR_NULL = -1,      /* a required pointer is NULL                    */
  QIFT_ERR_SHAPE = -2,     /* M < 1, N < 1, K % 64 != 0, or beyond a limit  */
  QIFT_ERR_SPEC = -3,      /* bad Hadamard block or clip ratio              */
  QIFT_ERR_FORMAT = -4,    /* wrong level-set format or layout for the call */
  QIFT_ERR_CODE = -5,      /* a level outside the format's set (pack calls)  */
  QIFT_ERR_ALIGN = -6,     /* a device pointer is not 16-byte aligned       */
  QIFT_ERR_HIP = -7,       /* a HIP launch failed: see qift_last_hip_error  */
  QIFT_ERR_WORKSPACE = -8  /* workspace smaller than qift_workspace_bytes   */
};

/* ---- level-set formats and packed layouts ----------------------------- */
enum { QIFT_W2_MNZ = 0, QIFT_W2_POT = 1, QIFT_W4_SYM = 2, QIFT_W2_LUT = 3 };

/*
 * QIFT_LAYOUT_V1 word layouts (uint32 words, little-endian, row-major):
 *
 *   W2 ("QW2v1"), words [N][K/16]: 2-bit code c = index of the level in the
 *     ascending list of its set (MNZ: level = 2c - 3, the unsigned code of
 *     the fractional-midpoint quantizer of Sec. 3.3 Eqs. (15)-(16); PoT:
 *     {-4,-1,+1,+4} -> 0..3, so bit 1 is the sign and the magnitude is 4
 *     exactly when both bits agree).  Weight k = 16j + 4t + b (t, b in 0..3)
 *     occupies bits [8b + 2t, 8b + 2t + 1] of word j; hence
 *     (word >> 2t) & 0x03030303 holds the codes of k = 16j+4t .. 16j+4t+3 in
 *     its four byte lanes.
 *
 *   W4 ("QW4v1"), words [N][K/8]: nibble u = q + 8 (1..15).  Weight
 *     k = 8j + 4t + b (t in 0..1, b in 0..3) occupies bits
 *     [8b + 4t, 8b + 4t + 3] of word j.
 */
enum { QIFT_LAYOUT_V1 = 1 };

/* Packed weight matrix: a non-owning view (all pointers device). */
typedef struct {
  int32_t fmt;             /* QIFT_W2_MNZ, QIFT_W2_POT or QIFT_W4_SYM         */
  int32_t layout;          /* QIFT_LAYOUT_V1                                  */
  int64_t N, K;            /* output and input features                       */
  const uint32_t *packed;  /* words, qift_packed_bytes(fmt, N, K) bytes       */
  const uint16_t *scales;  /* fp16 s_w[N]; for MNZ this is the half scale s/2 */
} qift_packed_w;

/*
 * Online rotation + activation quantizer settings.
 *   K        input features of the token (K % block == 0).
 *   block    Hadamard block b: a power of two in [2, 8192].  The rotation is
 *            block-diagonal, I_{K/b} (x) H_b, with the Sylvester matrix
 *            H_b[i][j] = (-1)^popcount(i & j) (deterministic, no random signs;
 *            Sec. 4.1 "Quantization configuration").
 *   flags    0: the normalized rotation H_b / sqrt(b) with clip ratio 1 (the
 *            plain absmax/7 scale).  QIFT_CLIP(num, den): clip ratio
 *            c = num / den of the symmetric INT4 quantizer, 1 <= num <= den
 *            <= 16, decided exactly (QIFT_CLIP(9, 10) is the paper's 0.9
 *            setting, Sec. 4.1).  QIFT_SPEC_BF16 may be or-ed in by the calls
 *            that rotate activations (qift_rotate_quant_act,
 *            qift_rotate_quant_linear): x then holds bf16 values.  Any other
 *            value is QIFT_ERR_SPEC.
 */
typedef struct {
  int64_t K;
  int32_t block;
  int32_t flags;
} qift_hadamard_spec;

#define QIFT_CLIP(num, den) ((int32_t)((((num) & 0xFF) << 8) | ((den) & 0xFF)))
#define QIFT_SPEC_BF16 ((int32_t)(1 << 16))

/* Bytes of packed words: N*K/4 (W2) or N*K/2 (W4); 0 for an invalid query. */
size_t qift_packed_bytes(int32_t fmt, int64_t N, int64_t K);

/*
 * Pack decoded W2 levels into QW2v1 words (Sec. 3.3: a fixed four-level set
 * with a per-output-channel scale, no zero-point).
 *   levels   int8 [N][K], each in {-3,-1,+1,+3} (MNZ) or {-4,-1,+1,+4} (PoT).
 *            Passing levels rather than codes keeps this boundary independent
 *            of the code assignment.
 *   scales   fp16 s_w[N], nullable; not read, recorded in *out.
 *   fmt      QIFT_W2_MNZ or QIFT_W2_POT; or QIFT_W2_LUT, where the "levels"
 *            are the codes 0..3 (table indices) themselves.
 *   packed   out: uint32 [N][K/16].
 *   out      host, out, nullable: filled with the view of the result.
 * An offline call: it validates every level and SYNCHRONIZES the stream to
 * read the count back.  A level outside the set returns QIFT_ERR_CODE (the
 * words are then written with code 0 in its place and must not be used).
 * The count lives in a 4-byte device word that the library allocates on the
 * first pack call on a device and keeps until the process ends; pack calls
 * are serialized by a lock.  Not capturable in a HIP graph.
 */
int qift_pack_w2(const int8_t *levels, const uint16_t *scales, int64_t N, int64_t K,
                 int32_t fmt, uint32_t *packed, qift_packed_w *out, qift_stream_t stream);

/*
 * Pack W4 levels q in -7..7 (int8 [N][K]) into QW4v1 words uint32 [N][K/8].
 * Same conventions, validation and synchronization as qift_pack_w2.
 */
int qift_pack_w4(const int8_t *levels, const uint16_t *scales, int64_t N, int64_t K,
                 uint32_t *packed, qift_packed_w *out, qift_stream_t stream);

/*
 * Offline weight quantization, the step before packing (Sec. 3.1 rotation;
 * Sec. 3.3, Sec. 3.5 and Sec. 4.5.1 per-channel scales; Eq. (1) for W4).
 * For each row n of W:
 *   w      = (I_{K/b} (x) H_b) W[n, :] / sqrt(b)   in fp64 (the orthonormal
 *            rotation that the online activation rotation undoes);
 *   MNZ    s_w = fp16(RMS(w) / 2); level +3 if w/s_w > 2, +1 if 0 <= w/s_w
 *          <= 2, -1 if -2 <= w/s_w < 0, -3 below (Eqs. (13)-(14));
 *   PoT    s_w = fp16(c* max|w| / 4) with c* the first minimiser over the 64
 *          candidates c_j = 0.2 + 0.8 j / 63 of sum (w - s level)^2; level
 *          sign(w) * (4 if |w/s| > 5/2 else 1), sign(0) = + (Eq. (17));
 *   W4     s_w = fp16(max|w| / 7), q = clip(rne(w / s_w), -7, 7) (Eq. (1)).
 * fp16 means round to nearest, ties to even; levels are assigned against the
 * stored fp16 scale; a row whose stored scale is 0 gets level +1 (W2) or 0
 * (W4).  The rotation of fp32 rows is not exact: its last bits depend on the
 * order of the sums, which can move a value that lies within rounding of a
 * threshold, or a near-tie of two PoT candidates, to the other side.
 * Arguments:
 *   W       fp32 [N][spec.K], finite.
 *   spec    K (multiple of 64, at most 16384), block b (power of two,
 *           2..4096, dividing K); flags 0.
 *   fmt     QIFT_W2_MNZ, QIFT_W2_POT or QIFT_W4_SYM.
 *   levels  out: int8 [N][K], the input of qift_pack_w2 / qift_pack_w4.
 *   scales  out: fp16 s_w[N].
 * Limits: N * K < 2^31.
 */
int qift_quantize_weights(const float *W, int64_t N, qift_hadamard_spec spec,
                          int32_t fmt, int8_t *levels, uint16_t *scales,
                          qift_stream_t stream);

/*
 * The same quantization onto any set of the mirror family
 *   G(r) = {-1, -r, +r, +1},  0 < r < 1   (Sec. 3.4 Eq. (18); r = 1/3 is the
 * MNZ grid, r = 1/4 the PoT grid, r near 0.30 the Lloyd-Max optimum of the
 * ratio study of Sec. 4.5.3), with the PoT scale rule: the outer level is 1,
 * s_w = fp16(c* max|w|) with c* the first minimiser over the 64 candidates
 * c_j = 0.2 + 0.8 j / 63 of sum (w - s level)^2, and against the stored
 * scale the level is sign(w) * (1 if |w/s_w| > (1 + r)/2 else r), sign(0) = +.
 * The result is written as codes, the indices of the ascending levels
 * (0: -1, 1: -r, 2: +r, 3: +1); a row whose stored scale is 0 gets code 2.
 * The codes are the input of qift_pack_w2 with QIFT_W2_LUT, and the table of
 * qift_w2a4_lut_linear is then {-1, -r, +r, +1} in fp16 (r rounded to fp16
 * there, the scale unchanged).  At r = 1/4 the codes are those of the PoT
 * levels and s_w is 4 times the PoT scale.  Same rotation, arguments, limits
 * and caveat on the rotation's rounding as qift_quantize_weights; r outside
 * (0, 1) (or NaN) returns QIFT_ERR_SPEC.
 */
int qift_quantize_weights_mirror(const float *W, int64_t N, qift_hadamard_spec spec,
                                 double r, int8_t *codes, uint16_t *scales,
                                 qift_stream_t stream);

/*
 * Ratio scan of the mirror family (the sensitivity study of Sec. 4.5.3):
 * for fp64 samples x[0..n) (e.g. pooled rotated weights), every ratio
 * ratios[i] and every clip candidate cands[j]:
 *   s         = cands[j] * max|x|;
 *   level     = sign(x) * (1 if |x / s| > (1 + r)/2 else r), sign(0) = +;
 *   sse[i][j] = sum over x of (x - s level)^2   (0 for all-zero x);
 *   best[i]   = the first j minimising sse[i][j];
 *   nmse[i]   = sse[i][best[i]] / sum x^2        (0 where sum x^2 is 0);
 *   stats     = {max|x|, sum x^2}.
 * Each term is formed with correctly rounded fp64 operations in that order
 * (quotient, compare, product, difference, square; no fused multiply-add);
 * the n-term sums are taken in a fixed order of the library's, so sse, nmse
 * and stats agree with any other summation order to within n ulps of the sum
 * (and best, where two candidates' errors lie closer than that, may name
 * either).
 * Arguments:
 *   x        fp64 [n], finite; 1 <= n < 2^40.
 *   ratios   host: n_ratios values in (0, 1); 1 <= n_ratios <= 1024.
 *   cands    host: n_cands positive finite values; 1 <= n_cands <= 256.
 *   sse      out: fp64 [n_ratios][n_cands].
 *   nmse     out: fp64 [n_ratios].
 *   best     out: int32 [n_ratios].
 *   stats    out: fp64 [2].
 * A ratio outside (0, 1) or a candidate that is not positive and finite
 * returns QIFT_ERR_SPEC; counts outside their ranges QIFT_ERR_SHAPE.  The
 * host arrays are read before the call returns.  Three launches on the stream.
 */
int qift_ratio_scan(const double *x, int64_t n, const double *ratios, int32_t n_ratios,
                    const double *cands, int32_t n_cands, double *sse, double *nmse,
                    int32_t *best, double *stats, qift_stream_t stream);

/*
 * Online Hadamard rotation + per-token symmetric INT4 quantization
 * (Sec. 3.1; Sec. 4.1 "Quantization configuration").  For each token m:
 *   X      = (I_{K/b} (x) H_b) x[m]   computed exactly (each fp16 input is an
 *            integer multiple of 2^-24, and the sums stay below 2^53 units);
 *   A      = max_k |X_k|;
 *   q[m,k] = sign(X_k) * min(7, rne(7 |X_k| / (c A)))  (round half to even,
 *            decided in exact integer arithmetic; A = 0 gives q = 0);
 *   s_x[m] = fp32( (A * num) / ((den * 7) * sqrt(b)) ), i.e. c * max|X| / 7
 *            for the orthonormal rotation H_b / sqrt(b), c = num / den from
 *            spec.flags;
 *   sum[m] = sum_k q[m, k].
 * Arguments:
 *   x          fp16 [M][spec.K], finite values (non-finite input is outside
 *              the contract).
 *   act_q      out: int8 [M][K].
 *   act_scale  out: fp32 [M].
 *   act_sum    out, nullable: int32 [M] (the linear calls compute this sum
 *              themselves; qift_w2a4_linear_ex may take it to skip that).
 * Limits: spec.K <= 32768.
 */
int qift_rotate_quant_act(const uint16_t *x, int64_t M, qift_hadamard_spec spec,
                          int8_t *act_q, float *act_scale, int32_t *act_sum,
                          qift_stream_t stream);

/*
 * qift_rotate_quant_act for bf16 activations (x: bf16 bits [M][spec.K]), for
 * callers whose models run in bf16 (the paper's full-precision reference is
 * fp16); the same as qift_rotate_quant_act with QIFT_SPEC_BF16 in spec.flags.
 * Any finite bf16 value is accepted.  Each is widened exactly to fp64 and X is
 * the fp64 result of the butterfly stages over the index bits in ascending
 * order, each sum and difference rounded to fp64; A, the codes (decided
 * exactly on those fp64 values, ties to even), s_x and the code sums follow
 * from X as for fp16.  On the fp16 grid (zero, or a magnitude in [2^-17, 2^16):
 * multiples of 2^-24) every partial sum is exact, so the result is the exact
 * rotation's, identical to the fp16 call on the same values.
 */
int qift_rotate_quant_act_bf16(const uint16_t *x, int64_t M, qift_hadamard_spec spec,
                               int8_t *act_q, float *act_scale, int32_t *act_sum,
                               qift_stream_t stream);

/*
 * Quantized linear with 2-bit weights (Sec. 1; Sec. 3.6):
 *   acc[m][n] = sum_k level[n][k] * act_q[m][k]   exact int32
 *   y[m][n]   = fp16( fp32( fp32(acc) * act_scale[m] ) * fp32(s_w[n]) )
 * with each fp32 product and the fp16 conversion rounded to nearest even.
 *   w          host: packed weights with fmt QIFT_W2_MNZ or QIFT_W2_POT.
 *   act_q, act_scale   the codes and scales of qift_rotate_quant_act for M
 *              tokens of width w->K (codes in -7..7).
 *   out        out: fp16 y [M][N].
 * The kernels run the MFMA on the raw 2-bit codes and add the exact level
 * correction from the per-token sum of the codes, which they compute from
 * the act_q tiles they stage.  M <= 64 runs the skinny decode kernel; larger
 * M runs the tiled prefill kernel; both give identical results.
 */
int qift_w2a4_linear(const qift_packed_w *w, const int8_t *act_q, const float *act_scale,
                     int64_t M, uint16_t *out, qift_stream_t stream);

/*
 * Same as qift_w2a4_linear, and additionally:
 *   act_sum    nullable: int32 [M], sum_k act_q[m][k] as written by
 *              qift_rotate_quant_act for these codes; when given the kernels
 *              use it instead of summing the codes (a wrong sum shifts every
 *              output: it is taken as is).  NULL: summed in the kernel.
 *   acc_out    out, nullable: int32 [M][N], the exact accumulators.
 *   workspace, workspace_bytes   optional device scratch (16-byte aligned).
 *              NULL / 0 runs the int8 MFMA kernels.  With at least
 *              qift_workspace_bytes(w, M) bytes, where that is not 0 (MNZ
 *              and PoT weights):
 *                M > 64 (and from M = 33 on N >= 16384, or N >= 4096 with
 *                K > 4096), where the prefill
 *                GEMM's 256-row x 64-token tiles are few (about 65-1024
 *                tokens, by N): the int8 GEMM split
 *                over K, int32 partial sums of each K-range in the
 *                workspace, then added and the epilogue applied;
 *                M > 64 otherwise: the activations are re-coded to FP6 E2M3
 *                in it and the prefill contraction runs on the FP4 x FP6
 *                scaled MFMA: the MNZ code c read as FP4 E2M1 is c / 2, the
 *                PoT levels +-1, +-4 are E2M1 values, and every partial sum
 *                stays exact in fp32 (split over K too where its tiles are
 *                few);
 *                M <= 64 otherwise (K > 4096, few 16-row tiles; up to 16 tokens only
 *                where the codes exceed the decode kernel's LDS): the decode
 *                linear is split over K, int32 partial sums of each K-range in
 *                the workspace, then added and the epilogue applied.
 *              Either way the results are bit-identical.  A non-zero size
 *              below the query is QIFT_ERR_WORKSPACE.  The workspace is
 *              overwritten.
 */
int qift_w2a4_linear_ex(const qift_packed_w *w, const int8_t *act_q, const float *act_scale,
                        const int32_t *act_sum, int64_t M, uint16_t *out, int32_t *acc_out,
                        void *workspace, size_t workspace_bytes, qift_stream_t stream);

/*
 * Quantized linear over a four-level fp16 table (fmt QIFT_W2_LUT), for the
 * non-integer reference grids of Sec. 3.3 (Lloyd-Max, NF2):
 *   t[m][n] = sum_k lut[code[n][k]] * act_q[m][k]        exact
 *   y[m][n] = fp16( fp32( fp32(t) * act_scale[m] ) * fp32(s_w[n]) )
 * i.e. the epilogue of qift_w2a4_linear with t in place of the accumulator.
 *   w        host: packed code words (qift_pack_w2 with QIFT_W2_LUT).
 *   lut      host: 4 fp16 bit patterns, the level of codes 0..3; each finite
 *            with magnitude <= 256 (QIFT_ERR_SPEC otherwise).
 *   act_q, act_scale   as for qift_w2a4_linear.
 *   out      out: fp16 y [M][N].
 * t is computed as L0 sum q + (L1 - L0) sum c q + (L2 - 2 L1 + L0) sum b1 q
 * + (L3 - L2 - L1 + L0) sum b0 b1 q over the code bits c = b0 + 2 b1, with the
 * three sums on the int8 MFMA: every term is then an exact fp64 multiple of
 * 2^-24 below 2^53, so the results are bit-exact.
 * Limits: K a multiple of 256 and at most 16384; M <= 1048560.  One kernel for
 * all M (workgroups of 16 rows x 16 tokens); no tiled prefill form.
 */
int qift_w2a4_lut_linear(const qift_packed_w *w, const uint16_t *lut, const int8_t *act_q,
                         const float *act_scale, int64_t M, uint16_t *out, qift_stream_t stream);

/* The W4 sibling (fmt QIFT_W4_SYM); same arguments and results.  The workspace of the _ex call is
 * used where qift_workspace_bytes is not 0: the int8 prefill GEMM split over K, as for W2 but from 24
 * tokens on for the wide and long linears (no FP4 form). */
int qift_w4a4_linear(const qift_packed_w *w, const int8_t *act_q, const float *act_scale,
                     int64_t M, uint16_t *out, qift_stream_t stream);
int qift_w4a4_linear_ex(const qift_packed_w *w, const int8_t *act_q, const float *act_scale,
                        const int32_t *act_sum, int64_t M, uint16_t *out, int32_t *acc_out,
                        void *workspace, size_t workspace_bytes, qift_stream_t stream);

/*
 * Fused decode form of qift_rotate_quant_act followed by qift_w2a4_linear or
 * qift_w4a4_linear (any w->fmt), for a few tokens: every workgroup rotates and
 * quantizes the tokens itself on chip while its first weight tiles stream
 * in, so the activations never make a round trip through HBM.  Results are
 * bit-identical to the two-call form.
 *   x          fp16 [M][w->K] (finite values), or bf16 with QIFT_SPEC_BF16 in
 *              spec.flags (the reading of qift_rotate_quant_act_bf16).
 *   spec       as for qift_rotate_quant_act; spec.K must equal w->K.
 *   out        out: fp16 y [M][N].
 *   acc_out    out, nullable: int32 [M][N].
 *   act_q, act_scale, act_sum   out, nullable (all three or none): the
 *              quantized activations, identical to qift_rotate_quant_act's.
 * Limits: 1 <= M <= 4, w->K <= 16384, spec.block <= 4096 (QIFT_ERR_SHAPE /
 * QIFT_ERR_SPEC otherwise).
 */
int qift_rotate_quant_linear(const qift_packed_w *w, const uint16_t *x, int64_t M, qift_hadamard_spec spec,
                             uint16_t *out, int32_t *acc_out, int8_t *act_q, float *act_scale,
                             int32_t *act_sum, qift_stream_t stream);

/*
 * Decode chain: a whole decode step of a layer stack (Sec. 1: at decode the step streams every
 * quantized weight once per token) as ONE launch of a persistent kernel.  Each link is the fused
 * rotate + quantize + linear of qift_rotate_quant_linear (Sec. 3.1 rotation and per-token INT4
 * quantizer, Sec. 3.3 / 3.6 integer dot product, scales in the epilogue) whose input is either the
 * chain input x or a slice of an earlier link's output; the kernel honours those dependencies
 * through exchange copies of the outputs in the workspace (a consumer reads its input there until
 * no value is the not-written pattern), while the weight stream of the next link runs ahead of
 * them.  Results are bit-identical to calling qift_rotate_quant_linear link by link.
 *
 *   qift_chain_link   (host) one linear:
 *     w          the weights (fmt MNZ, PoT or W4; one format for the whole chain).
 *     block      Hadamard block of the link's input: 64, 256, 2048 or 4096 (the blocks of the
 *                LLaMA-shaped stacks, compiled in), dividing w.K.
 *     flags      clip flags of the input's quantizer, as qift_hadamard_spec.flags.
 *     in_link    index of the link whose output is this link's input (lower than this link's
 *                index), or -1 for the chain input x (then w.K must equal the chain's K0).
 *     in_offset  first element taken from each token's row of that output: the input is
 *                elements [in_offset, in_offset + w.K) (a multiple of 8; 0 for the chain input).
 *     out        device, out: fp16 y [M][w.N]; the outputs of all links must be disjoint.
 *     acc_out    device, out, nullable: int32 [M][w.N] accumulators.
 *   qift_chain        (host) the prepared chain, filled by qift_chain_prepare: a view of the
 *                workspace plus the launch geometry.  The caller keeps the workspace alive, and
 *                the weights and output buffers the links name, while it uses the chain.
 */
typedef struct {
  qift_packed_w w;
  int32_t block;
  int32_t flags;
  int32_t in_link;
  int32_t reserved;          /* 0 */
  int64_t in_offset;
  uint16_t *out;
  int32_t *acc_out;
} qift_chain_link;

typedef struct {
  int32_t fmt, n_links;
  int32_t M, K0;             /* tokens per call, width of the chain input */
  int32_t grid, kmax;        /* workgroups (one per CU), largest K of the links */
  int32_t region0, reserved; /* LDS bytes of the activation group's work region */
  const void *table;         /* device: the link table (in the workspace) */
  uint32_t *counters;        /* device: finished-workgroup count and run number (in the workspace) */
} qift_chain;

/*
 * Workspace bytes of a chain (host links, n_links of them, M tokens): the link table, two counters,
 * and for every link whose output another link reads, two exchange copies of that output
 * (2 x M x N8 fp16 values, N8 = N rounded up to a multiple of 8), each buffer 256-byte aligned.
 * 0 for a chain that qift_chain_prepare would reject.
 */
size_t qift_chain_workspace_bytes(const qift_chain_link *links, int32_t n_links, int64_t M);

/*
 * Validate the links, write the link table, the counters and the exchange copies (every value
 * marked not written, 0xFFFF) into the workspace and fill *chain.  An offline call: it SYNCHRONIZES the stream (the table is copied
 * from host memory); not capturable in a HIP graph.
 *   links      host: n_links links (1 <= n_links <= 4096).
 *   M          tokens per call, 1..4, as far as one workgroup's LDS holds M tokens' codes next to
 *              the rotation buffers (three of them for a chain with a link of K > 4096: with a
 *              K = 14336 link, M <= 3).
 *   K0         width of the chain input x.
 *   workspace  device, 16-byte aligned, at least qift_chain_workspace_bytes(links, n_links, M).
 *   chain      host, out.
 * Errors: QIFT_ERR_NULL, QIFT_ERR_FORMAT (mixed or unknown formats), QIFT_ERR_SHAPE (K above
 * 16384, an input slice past the producer's row, overlapping outputs, M outside 1..4, or LDS
 * beyond 160 KiB), QIFT_ERR_SPEC (block not one of 64, 256, 2048, 4096, or bad flags),
 * QIFT_ERR_ALIGN, QIFT_ERR_WORKSPACE.
 */
int qift_chain_prepare(const qift_chain_link *links, int32_t n_links, int64_t M, int64_t K0, void *workspace,
                       size_t workspace_bytes, qift_chain *chain, qift_stream_t stream);

/*
 * Run one decode step of a prepared chain on the tokens x (device, fp16 [M][K0], 16-byte
 * aligned, not overlapping any link's output).  Asynchronous; capturable in a HIP graph (one
 * kernel launch).  The grid is one workgroup per CU and relies on all of them running at once:
 * calls must not overlap one another on a device (they share the chain's counters and exchange
 * buffers, and a concurrent kernel that holds CUs delays the grid).  Call r (counted from 1 by the
 * chain) writes copy r mod 2 of each exchange buffer and marks the other copy not written; a link
 * waits until none of its input values in copy r mod 2 is 0xFFFF (a NaN output reaches the next
 * link as the quiet NaN 0xFE00).  A wait that gives up (the call not done
 * within about a second) sets QIFT_DEVERR_CHAIN_WAIT in the device error word
 * (qift_device_error) and the results of that call are not to be trusted.
 */
int qift_decode_chain(const qift_chain *chain, const uint16_t *x, qift_stream_t stream);

/*
 * Measurement helper, not part of the method: the achievable HBM read
 * bandwidth, the floor of the decode kernels' weight streams.  Reads the
 * device buffer buf[0 .. bytes) once with 16-byte loads spread over every CU;
 * workgroup b XORs the 32-bit words of the 64 KiB segment b of the buffer
 * into partials[b] (device, uint32[(bytes + 65535) / 65536], every slot
 * written), so the XOR of all partials is the XOR of the buffer's words.
 *   bytes      a positive multiple of 16 (QIFT_ERR_SHAPE); buf 16-byte
 *              aligned, partials 4-byte aligned (QIFT_ERR_ALIGN).
 *   Asynchronous on stream.
 */
int qift_hbm_read_probe(const void *buf, size_t bytes, uint32_t *partials, qift_stream_t stream);

/*
 * KV4: the four-bit key/value cache of the W2A4/KV4 setting (Sec. 4.1
 * "Quantization configuration": asymmetric key and value quantization with
 * clipping ratio 0.95) with the conventional asymmetric quantizer of
 * Sec. 3.3 Eq. (15), q = clip(round(x / s) + z, 0, 15), x_hat = s (q - z).
 * One group per token and KV head (head_dim = 128 values).  In fp32, in this
 * order, rounding half to even:
 *   x_max = c * max(max x, 0), x_min = c * min(min x, 0), c = fp32(0.95);
 *   s = (x_max - x_min) / 15 (1 for a group of zeros); z = round(-x_min / s);
 *   q = clip(round(x / s) + z, 0, 15).
 *   x        fp16 [groups][128], 16-byte aligned.
 *   codes    out: uint8 [groups][64], value 2i in the low nibble of byte i;
 *            4-byte aligned.
 *   scales   out: fp32 s [groups], 4-byte aligned.
 *   zeros    out: uint8 z [groups], any alignment (so a view of a cache at
 *            any token position, e.g. one appended decode token, is valid).
 */
int qift_kv4_quant(const uint16_t *x, int64_t groups, int32_t head_dim, uint8_t *codes,
                   float *scales, uint8_t *zeros, qift_stream_t stream);

/* Workspace bytes of qift_kv4_attention_decode (0 for an unsupported shape). */
size_t qift_kv4_attention_workspace_bytes(int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim,
                                          int64_t T);

/* Cache row orders of qift_kv4_attention_decode (a row is one token's key or value vector of
 * one KV head: 64 code bytes, one scale, one zero-point).  Token-major [B][T][Hkv] is the order
 * of a [B, T, Hkv, 128] tensor, as one decode step appends a token; head-major [B][Hkv][T] keeps
 * each KV head's tokens contiguous, which the attention reads as one stream per workgroup
 * (measured faster: the token-major order interleaves KV heads at 64-byte granularity). */
enum { QIFT_KV4_TOKEN_MAJOR = 0, QIFT_KV4_HEAD_MAJOR = 1 };

/*
 * One decode step of grouped-query attention over a KV4 cache (Sec. 1: the
 * decode stream is weights plus KV cache).  For batch b and query head h,
 * with KV head kv = h / (Hq / Hkv):
 *   out[b][h] = sum_t softmax_t( q[b][h] . k_hat[b, t, kv] / sqrt(128) )
 *               * v_hat[b, t, kv],   x_hat = s (code - z) per group,
 * with an fp16 result.  Scores: exact fp16 operands (code - z, the queries)
 * summed in fp32 on the f16 MFMA; exponentials and statistics in fp32; value
 * sums: p * s split into two fp16 parts (2^-21 relative) times the codes,
 * summed in fp32.  Per query head the result is within (2^-11 + 1.1e-4) of
 * the head's largest output of the exact softmax over the reconstructed
 * cache (the fp16 rounding of the output being the 2^-11).
 *   q        fp16 [B][Hq][128], the new token's queries.
 *   layout   QIFT_KV4_TOKEN_MAJOR or QIFT_KV4_HEAD_MAJOR (QIFT_ERR_SPEC otherwise).
 *   k_*, v_* the cache as written by qift_kv4_quant for groups in that row
 *            order: codes uint8 [rows][64], scales fp32 and zeros uint8
 *            [rows], rows = [B][T][Hkv] or [B][Hkv][T].
 *   out      out: fp16 [B][Hq][128].
 *   workspace  device scratch of qift_kv4_attention_workspace_bytes bytes
 *            (per 256 cached tokens and query head: 128 partial sums, the
 *            chunk's maximum score and sum of exponentials).
 * Limits: head_dim = 128, Hq / Hkv in {1, 2, 4, 8}, B and Hkv <= 65535,
 * T * Hkv * 64 < 2^31.
 */
int qift_kv4_attention_decode(const uint16_t *q, int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim,
                              int64_t T, int32_t layout, const uint8_t *k_codes, const float *k_scales,
                              const uint8_t *k_zeros, const uint8_t *v_codes, const float *v_scales,
                              const uint8_t *v_zeros, uint16_t *out, void *workspace,
                              size_t workspace_bytes, qift_stream_t stream);

/* Size of the device array behind qift_kv4_attention_decode_noalloc: 8 MiB per GPU, i.e. calls with
 * qift_kv4_attention_workspace_bytes(B, Hq, Hkv, 128, T) up to that, B * Hq * ceil(T / 256) <= 16131
 * partial records of 520 bytes (for example B = 1, Hq = 32 up to T = 129024). */
#define QIFT_KV4_SCRATCH_BYTES (8u << 20)

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): qift_kv4_attention_decode without a workspace argument.  The
 * partial records live in a library-owned device array of QIFT_KV4_SCRATCH_BYTES on each GPU, held
 * until the process ends; the call allocates nothing (no hipMalloc, hipFree or allocating library
 * routine).  The first call on a device resolves that device's address of the array (a symbol
 * query, not an allocation), so make one call before capturing a graph if the runtime forbids such
 * queries during capture.  Arguments, results and errors are those of qift_kv4_attention_decode,
 * plus QIFT_ERR_WORKSPACE when the call needs more than QIFT_KV4_SCRATCH_BYTES.  Every call on a GPU
 * shares that GPU's array and the array keeps the last call's records: calls that overlap on one
 * GPU (several streams or threads) race, so the caller serializes them.  Nothing in the array has
 * to start at zero: a call writes every record its merge reads.
 */
int qift_kv4_attention_decode_noalloc(const uint16_t *q, int64_t B, int32_t Hq, int32_t Hkv, int32_t head_dim,
                                      int64_t T, int32_t layout, const uint8_t *k_codes, const float *k_scales,
                                      const uint8_t *k_zeros, const uint8_t *v_codes, const float *v_scales,
                                      const uint8_t *v_zeros, uint16_t *out, qift_stream_t stream);

/* Workspace bytes that the _ex calls use for this weight and M, 0 where none is used (host
 * query).  N4 = N rounded up to 4; T = ceil(N / 256) * ceil(M / 64) prefill tiles; a count S of
 * K-ranges is recounted once the ranges are sized (ranges of ceil(steps / S) steps).
 *   M > 64, and from M = 33 (W4: 24) on N >= 16384 or N >= 4096 with K > 4096: the int8 GEMM split
 *     over S = min(ceil(512 / T), floor(512 / T), floor(steps / s0)) K-ranges when that is at least S0
 *     (W2: 256-k steps, s0 = 4, S0 = 2; W4: 128-k steps, s0 = 8, S0 = 3): S * M * N4 int32 partial
 *     sums (256-byte aligned), then S * M int32 code sums.
 *   M > 64 otherwise, MNZ and PoT: the FP4 x FP6 prefill kernel's M * 3K/4 bytes of FP6 codes and
 *     M * ceil(K / 8192) int32 code sums, split over S = min(ceil(512 / T), floor(768 / T),
 *     floor(ceil(K / 256) / 4)) K-ranges when that is at least 2, the S * M * N4 int32 partial sums
 *     following at the next multiple of 256 bytes; W4: 0.
 *   M <= 64 otherwise, MNZ and PoT: the decode linear split over K, where it applies (K > 4096 and at most 680
 *     16-row tiles, N <= 10880; up to 16 tokens only where the codes exceed the decode kernel's LDS):
 *     S * M * N4 int32 partial sums (256-byte aligned) and S * M int32 code sums; W4: 0. */
size_t qift_workspace_bytes(const qift_packed_w *w, int64_t M);

/* Static text for a status code. */
const char *qift_status_string(int status);

/* The hipError_t value behind the calling thread's last QIFT_ERR_HIP. */
int qift_last_hip_error(void);

/*
 * Device-side error report.  Every wait inside a kernel is bounded: the
 * waves of a workgroup that wait for each other (the fused decode) and the
 * workgroups that wait for another workgroup's result (qift_decode_chain)
 * give up after a limit, set a bit in a per-device error word and carry on,
 * so every kernel exits; the results of the affected call are then not to be
 * trusted.  Bits: QIFT_DEVERR_GROUP_WAIT (a wave barrier inside a
 * workgroup), QIFT_DEVERR_CHAIN_WAIT (a wait for another workgroup).
 * qift_device_error synchronizes the stream, writes the word of the current
 * device to *bits (host) and, if clear is non-zero, resets it.  Not
 * capturable in a HIP graph.
 */
enum { QIFT_DEVERR_GROUP_WAIT = 1, QIFT_DEVERR_CHAIN_WAIT = 2 };
int qift_device_error(uint32_t *bits, int32_t clear, qift_stream_t stream);

/*
 * Test hook: the spin limit (iterations) of the in-workgroup wave barriers
 * for launches made after the call, process-wide; 0 restores the default
 * (2^22).  A tiny limit makes those waits give up, which the error word then
 * reports.  QIFT_ERR_SHAPE for a negative value.
 */
int qift_set_wait_limit(int32_t spins);

/* Library version string, e.g. "qift 0.1 gfx950". */
const char *qift_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QIFT_H */
