// Prefill linear for W2 weights on the CDNA4 scaled MFMA with FP4 (E2M1) weights and FP6 (E2M3)
// activations, v_mfma_scale_f32_16x16x128_f8f6f4 with unit scales (E8M0 127).
//
// Exactness, MNZ: a code c in 0..3 read as the E2M1 nibble 0b00cc is c / 2 (0, 0.5, 1, 1.5) and
// the INT4 codes -7..7 are exact in E2M3, so every product is c q / 2 and every partial sum a
// multiple of 1/2 below 2^23: the fp32 accumulator holds D = sum c q / 2 exactly, and the integer
// accumulator of the method is acc = 2 (2 D) - 3 sum q (Sec. 3.3: level = 2 c - 3).
// PoT-MNZ: the levels -4, -1, +1, +4 (Sec. 3.3, Eq. (17)) are themselves E2M1 values (0b1110,
// 0b1010, 0b0010, 0b0110): for the code c = 2 b1 + b0 the nibble has sign bit !b1, exponent bits
// (!(b1 ^ b0), 1) and mantissa 0, built from the masked code nibbles by a few bitwise operations
// per word; every product level q and every partial sum (|sum| <= 28 K < 2^24) is an integer, so
// the accumulator holds acc = sum level q exactly.  Results are bit-identical to the int8 path.
//
// Operand layouts (measured on gfx950): A lane (row r, group g) nibble i <-> k = 32 g + i of the
// MFMA's 128; B lane (column m, group g) element i at bits 6 i .. 6 i + 5 of its 192 bits <-> the
// same k; D as for the int8 MFMA.  A lane takes its 32 weights from two packed words with two masks
// per word (w & 0x33333333, (w >> 2) & 0x33333333): nibble 8 D + i of the operand then holds the
// code of word k-offset kperm(8 D + i) = 16 (D >> 1) + 4 (D & 1) + 8 (i & 1) + (i >> 1), and the
// FP6 activations are stored in that order inside each 32-k group (k_act_fp6).
#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"
#include "qift_split.h"

namespace qift {
namespace {

using namespace mma;

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kF6GroupBytes = 24;   // 32 FP6 codes
constexpr int kF6StepBytes = 192;   // 256 k of one token

__host__ __device__ constexpr int kperm(int n) {
  return 16 * ((n >> 3) >> 1) + 4 * ((n >> 3) & 1) + 8 * (n & 1) + ((n & 7) >> 1);
}

// act_q int8 [M][K] -> FP6 E2M3 codes [M][K / 32][24 bytes], element n of group G = code of
// k = 32 G + kperm(n).  One thread per group.  With psum (non-null), workgroup x also writes the sum
// of the codes of its 256 groups of token m to psum[m * gridDim.x + x].
__global__ __launch_bounds__(256) void k_act_fp6(const int8_t* __restrict__ act_q, int M, int K,
                                                 uint8_t* __restrict__ act6, int32_t* __restrict__ psum) {
  __shared__ int red[4];
  const int groups = K >> 5;
  const int G = blockIdx.x * 256 + threadIdx.x;
  const bool valid = G < groups;
  for (int m = blockIdx.y; m < M; m += gridDim.y) {
    if (psum) {   // uniform over the workgroup: every thread takes part in the reduction
      int sq = 0;
      if (valid) {
        const uint4* src = reinterpret_cast<const uint4*>(act_q + (int64_t)m * K + 32 * G);
        sq = sum16_i8(src[1], sum16_i8(src[0], 0));
      }
      sq = dev::wave_sum(sq);
      if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sq;
      __syncthreads();
      if (threadIdx.x == 0) psum[(int64_t)m * gridDim.x + blockIdx.x] = red[0] + red[1] + red[2] + red[3];
      __syncthreads();
    }
    if (!valid) continue;
    const uint4* src = reinterpret_cast<const uint4*>(act_q + (int64_t)m * K + 32 * G);
    const uint4 lo = src[0], hi = src[1];
    const uint32_t wq[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    uint32_t out[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int n = 0; n < 32; ++n) {
      const int k = kperm(n);
      const int q = (int)(int8_t)(wq[k >> 2] >> (8 * (k & 3)));
      const int a = q < 0 ? -q : q;
      // E2M3 (bias 1) of 0..7: 0, 1.0, 2.0, 1.5 * 2, 4.0, 1.25 * 4, 1.5 * 4, 1.75 * 4
      const uint32_t mag = a == 0 ? 0u : a == 1 ? 0x08u : a == 2 ? 0x10u : a == 3 ? 0x14u
                         : 0x18u + 2u * (uint32_t)(a - 4);
      const uint32_t code = mag | (q < 0 ? 0x20u : 0u);
      const int bit = 6 * n;
      out[bit >> 5] |= code << (bit & 31);
      if ((bit & 31) > 26) out[(bit >> 5) + 1] |= code >> (32 - (bit & 31));
    }
    uint2* dst = reinterpret_cast<uint2*>(act6 + (int64_t)m * (3 * (K >> 2)) + kF6GroupBytes * G);
    dst[0] = make_uint2(out[0], out[1]);
    dst[1] = make_uint2(out[2], out[3]);
    dst[2] = make_uint2(out[4], out[5]);
  }
}

// Tiles of 256 weight rows x 64 tokens x 256 k, 4 waves (64 rows x 64 tokens each), three
// workgroups per CU: the structure of the int8 prefill kernel (weights one step ahead in
// alternating register sets, activations by direct-to-LDS loads into two distinct buffers) with
// two 16x16x128 MFMAs per row tile and step instead of four 16x16x64 ones.  The step's FP6 row is
// 192 bytes: twelve 16-byte chunks in a 256-byte LDS row, chunk c of row r in slot c ^ (r mod 16)
// (the four spare slots receive zeros).
// FP4 operand nibbles of eight PoT codes from their masked code nibbles 0b00cc (see above)
__device__ __forceinline__ uint32_t pot_f4(uint32_t x) {
  const uint32_t b0 = x & 0x11111111u, b1 = (x >> 1) & 0x11111111u;
  return ((b1 ^ 0x11111111u) << 3) | ((b1 ^ b0 ^ 0x11111111u) << 2) | 0x22222222u;
}

// SPLIT: workgroup z of the grid's third dimension takes the steps [z us, (z + 1) us) of K and writes
// its exact partial sums (int32) to part [z][M][N rounded up to 4] instead of the outputs.
template <int FMT, int OCC, bool SPLIT>
__global__ __launch_bounds__(256, OCC) void k_gemm_f4(const uint32_t* __restrict__ P, const uint16_t* __restrict__ sw,
                                                      int N, int K, const uint8_t* __restrict__ act6,
                                                      const float* __restrict__ sx, const int32_t* __restrict__ asum,
                                                      const int32_t* __restrict__ psum, int npsum,
                                                      int M, uint16_t* __restrict__ y, int32_t* __restrict__ acc_out,
                                                      int us, int32_t* __restrict__ part) {
  constexpr int BM = 64, BK = 256;
  __shared__ __align__(16) uint8_t lds0[BM * 256];
  __shared__ __align__(16) uint8_t lds1[BM * 256];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int n_base = blockIdx.x * 256 + wave * 64;
  const int m_base = blockIdx.y * BM;
  const int rowbytes = K / 4, row6 = 3 * (K / 4);
  const int KA = (K + BK - 1) / BK;
  const int kt0 = SPLIT ? (int)blockIdx.z * us : 0;
  const int KT = SPLIT ? (kt0 + us < KA ? kt0 + us : KA) : KA;   // steps past this workgroup's range

  // weights: as in the int8 kernel (lanes past K in a last partial step meet zero activations)
  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(P, (uint32_t)N * (uint32_t)rowbytes);
  uint32_t wbase[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n_base + 16 * j + r16;
    wbase[j] = n < N ? (uint32_t)n * (uint32_t)rowbytes + 16u * g : dev::kOutOfRange;
  }
  auto load_w = [&](uint4 (&w)[4], int kt) {
    const uint32_t ko = 64u * (uint32_t)kt;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = dev::bload16(wrs, wbase[j] + ko);
  };
  // activations: load q moves 1 KB = rows 4 (4 wave + q) .. + 3; lane l fills slot l mod 16 of row
  // 4 (4 wave + q) + l / 16 with the row's chunk (l mod 16) ^ (row mod 16), zeros for chunks >= 12
  const int mrows = M - m_base < BM ? M - m_base : BM;
  const __amdgpu_buffer_rsrc_t ars = dev::make_rsrc(act6 + (int64_t)m_base * row6, (uint32_t)(mrows * row6));
  uint32_t abase[4];
  int acol[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = 4 * (4 * wave + q) + (lane >> 4);
    const int c = (lane & 15) ^ (row & 15);
    acol[q] = 16 * c;
    abase[q] = row < mrows && c < 12 ? (uint32_t)(row * row6 + 16 * c) : dev::kOutOfRange;
  }
  auto issue_a = [&](int kt, uint8_t* dst) {
    const int ko = kt * kF6StepBytes;
    const bool tail = ko + kF6StepBytes > row6;   // the last step of a K that is not a multiple of 256
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int chunk = 4 * wave + q;
      uint32_t off = abase[q] + (uint32_t)ko;
      if (tail && acol[q] + ko >= row6) off = dev::kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ars, (__attribute__((address_space(3))) void*)(dst + 1024 * chunk), 16, off, 0, 0, 0);
    }
  };

  v4f acc[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[j][t] = v4f{0.f, 0.f, 0.f, 0.f};

  // MFMA kb of lane group g covers k = kt 256 + 64 g + 32 kb + kperm(0 .. 31): words 2 kb, 2 kb + 1
  // of the lane's 16 bytes, and FP6 group 2 g + kb of the step
  auto step = [&](int kt, const uint8_t* tileb, uint8_t* nextb, const uint4 (&wc)[4], uint4 (&wn)[4]) {
    if (kt + 1 < KT) {
      issue_a(kt + 1, nextb);
      load_w(wn, kt + 1);
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      v8i a[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t w0 = kb ? wc[j].z : wc[j].x, w1 = kb ? wc[j].w : wc[j].y;
        uint32_t n0 = w0 & 0x33333333u, n1 = (w0 >> 2) & 0x33333333u, n2 = w1 & 0x33333333u,
                 n3 = (w1 >> 2) & 0x33333333u;
        if constexpr (FMT == FMT_POT) {
          n0 = pot_f4(n0);
          n1 = pot_f4(n1);
          n2 = pot_f4(n2);
          n3 = pot_f4(n3);
        }
        a[j] = v8i{(int)n0, (int)n1, (int)n2, (int)n3, 0, 0, 0, 0};
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int row = 16 * t + r16;
        const uint8_t* rp = tileb + row * 256;
        uint2 pc[3];
#pragma unroll
        for (int p = 0; p < 3; ++p) {
          const int off = kF6GroupBytes * (2 * g + kb) + 8 * p;   // never crosses a 16-byte chunk
          pc[p] = *reinterpret_cast<const uint2*>(rp + 16 * ((off >> 4) ^ r16) + (off & 15));
        }
        const v8i b = v8i{(int)pc[0].x, (int)pc[0].y, (int)pc[1].x, (int)pc[1].y, (int)pc[2].x, (int)pc[2].y, 0, 0};
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[j][t] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a[j], b, acc[j][t], 4, 2, 0, 127, 0, 127);
      }
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // this wave's loads of step kt+1 have landed
    __syncthreads();
  };

  uint4 wa[4], wb[4];
  issue_a(kt0, lds0);
  load_w(wa, kt0);
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  for (int kt = kt0; kt < KT; kt += 2) {
    step(kt, lds0, lds1, wa, wb);
    if (kt + 1 < KT) step(kt + 1, lds1, lds0, wb, wa);
  }

  if constexpr (SPLIT) {
    const int np = (N + 3) & ~3;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int m = m_base + 16 * t + r16;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n0 = n_base + 16 * j + 4 * g;
        const float f = FMT == FMT_MNZ ? 2.f : 1.f;
        if (m < M && n0 < N)
          *reinterpret_cast<int4*>(part + ((size_t)blockIdx.z * M + m) * np + n0) =
              make_int4((int)(f * acc[j][t][0]), (int)(f * acc[j][t][1]), (int)(f * acc[j][t][2]),
                        (int)(f * acc[j][t][3]));
      }
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int m = m_base + 16 * t + r16;
    if (m < M) {
      const float s_x = sx[m];
      int sq = 0;
      if (asum) {
        sq = asum[m];
      } else {
        for (int p = 0; p < npsum; ++p) sq += psum[(int64_t)m * npsum + p];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // MNZ: 2 D = sum c q exactly (an integer below 2^24); PoT: D = sum level q exactly
        const float f = FMT == FMT_MNZ ? 2.f : 1.f;
        const v4i D = v4i{(int)(f * acc[j][t][0]), (int)(f * acc[j][t][1]), (int)(f * acc[j][t][2]),
                          (int)(f * acc[j][t][3])};
        store4<FMT>(D, m, n_base + 16 * j + 4 * g, N, s_x, sq, sw, y, acc_out);
      }
    }
  }
}

}  // namespace

// workgroups of the FP6 re-coding per token (256 groups of 32 k each)
inline int64_t act_fp6_blocks(int64_t K) { return (K / 32 + 255) / 256; }

// Split over K where the 256 x 64 tiles leave most of the chip idle (down at 65-512 tokens: 16 x
// ceil(M / 64) tiles of 56 steps): S ranges of at least kF4MinSteps steps, S the smallest count that
// gives about kF4SplitTarget workgroups, and no more than kF4Resident (three workgroups on each of
// the 256 CUs) so that the split grid is resident at once: with more, the partial sums' traffic (S M N
// int32, written and read back) outweighs what the split hides (gate|up at 256 tokens, 448 tiles:
// 47 -> 56 us at S = 2).  Down at 65-128 tokens: 78-81 -> 26-29 us.
constexpr int64_t kF4SplitTarget = 512, kF4Resident = 768, kF4MinSteps = 4;
struct F4Split {
  int S = 1, us = 0;
};
inline F4Split f4_split_plan(int64_t N, int64_t M, int64_t K) {
  F4Split p;
  const int64_t tiles = ((N + 255) / 256) * ((M + 63) / 64), KT = (K + 255) / 256;
  p.us = (int)KT;
  int64_t S = (kF4SplitTarget + tiles - 1) / tiles;
  if (S > kF4Resident / tiles) S = kF4Resident / tiles;
  if (S > KT / kF4MinSteps) S = KT / kF4MinSteps;
  if (S < 2) return p;
  p.us = (int)((KT + S - 1) / S);
  p.S = (int)((KT + p.us - 1) / p.us);
  return p;
}

// FP6 codes (M 3K/4 bytes, a multiple of 16), then the per-workgroup code sums int32 [M][blocks];
// split over K, the partial sums follow at the next multiple of 256 bytes.
inline size_t f4_codes_bytes(int64_t M, int64_t K) {
  return (size_t)M * (size_t)(3 * (K / 4)) + (size_t)M * (size_t)act_fp6_blocks(K) * 4;
}
size_t gemm_f4_workspace(int64_t N, int64_t M, int64_t K) {
  const F4Split p = f4_split_plan(N, M, K);
  const size_t base = f4_codes_bytes(M, K);
  return p.S > 1 ? (base + 255) / 256 * 256 + split::part_bytes(p.S, M, N) : base;
}

hipError_t launch_gemm_f4(int fmt, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K,
                          const int8_t* act_q, const float* sx, const int32_t* asum, int64_t M, uint16_t* y,
                          int32_t* acc_out, void* ws, hipStream_t s) {
  if (fmt != FMT_POT && fmt != FMT_MNZ) return hipErrorInvalidValue;
  uint8_t* act6 = static_cast<uint8_t*>(ws);
  int32_t* psum = asum ? nullptr : reinterpret_cast<int32_t*>(act6 + (size_t)M * (size_t)(3 * (K / 4)));
  const int gx = (int)act_fp6_blocks(K);
  const unsigned gy = (unsigned)(M < 65535 ? M : 65535);
  hipLaunchKernelGGL(k_act_fp6, dim3((unsigned)gx, gy), dim3(256), 0, s, act_q, (int)M, (int)K, act6, psum);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const F4Split p = f4_split_plan(N, M, K);
  const dim3 grid((unsigned)((N + 255) / 256), (unsigned)((M + 63) / 64), (unsigned)p.S);
  if (p.S > 1) {
    int32_t* part = reinterpret_cast<int32_t*>(act6 + (f4_codes_bytes(M, K) + 255) / 256 * 256);
    if (fmt == FMT_POT)
      hipLaunchKernelGGL((k_gemm_f4<FMT_POT, 3, true>), grid, dim3(256), 0, s, P, sw, (int)N, (int)K, act6, sx, asum,
                         psum, gx, (int)M, y, acc_out, p.us, part);
    else
      hipLaunchKernelGGL((k_gemm_f4<FMT_MNZ, 3, true>), grid, dim3(256), 0, s, P, sw, (int)N, (int)K, act6, sx, asum,
                         psum, gx, (int)M, y, acc_out, p.us, part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // code sums of token m at psum[m gx + p]
    return fmt == FMT_POT
               ? split::launch_sum<FMT_POT>(part, p.S, M, N, sx, asum, psum, gx, gx, 1, sw, y, acc_out, s)
               : split::launch_sum<FMT_MNZ>(part, p.S, M, N, sx, asum, psum, gx, gx, 1, sw, y, acc_out, s);
  }
  if (fmt == FMT_POT)
    hipLaunchKernelGGL((k_gemm_f4<FMT_POT, 3, false>), grid, dim3(256), 0, s, P, sw, (int)N, (int)K, act6, sx, asum,
                       psum, gx, (int)M, y, acc_out, 0, nullptr);
  else
    hipLaunchKernelGGL((k_gemm_f4<FMT_MNZ, 3, false>), grid, dim3(256), 0, s, P, sw, (int)N, (int)K, act6, sx, asum,
                       psum, gx, (int)M, y, acc_out, 0, nullptr);
  return hipGetLastError();
}

}  // namespace qift
