// Quantized linear over a four-level grid read through an fp16 level table: the reference grids
// of Sec. 3.3 (Lloyd-Max Eq. (9), NF2 Eq. (10)), whose levels are not integers.
//
//   t[m][n] = sum_k lut[c[n][k]] q[m][k]                 exact
//   y[m][n] = fp16(fp32(fp32(t) * s_x[m]) * fp32(s_w[n]))  (the epilogue of the integer formats)
//
// The table lookup is written over the bits of the code c = b0 + 2 b1:
//   lut[c] = L0 + e1 c + e2 b1 + e3 b0 b1,  e1 = L1 - L0, e2 = L2 - 2 L1 + L0, e3 = L3 - L2 - L1 + L0,
// so t = L0 sum q + e1 sum c q + e2 sum b1 q + e3 sum b0 b1 q, three exact int32 sums on the int8
// MFMA (operands: the codes, the high bits, the products of the bits, one byte per weight) plus
// the per-token sum of q, added up from the activation operands the lanes already hold (dot
// products with 1).  Every table entry is a multiple of 2^-24 of magnitude at most 256 and
// K <= 16384, so every term and partial sum of the fp64 combination is an integer number of
// 2^-24 units below 2^53: t is exact, and y is bit-exact.
//
// Workgroup (16 rows, 16 tokens), NW waves over interleaved 256-k blocks of K.  Where the row tiles
// alone would leave the chip with about one wave per SIMD, NW = 8 and each wave keeps the next
// block's loads in flight while it computes the current one (measured: with many row tiles that
// costs occupancy and is slower, so NW = 4 loads block by block there): lane (i, g) =
// (lane mod 16, lane / 16) loads 16 bytes of packed words of row i (words 16 S + 4 g .. + 3 of
// block S); MFMA j uses word 16 S + 4 g + j, i.e. k = 256 S + 64 g + 16 j .. + 15, and the
// activation bytes of token i at the same k (A and B lanes of a lane group meet element by
// element, so the k-slot assignment cancels).  The waves' sums are added through LDS.
#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"

namespace qift {
namespace {

using mma::v4i;

struct LutCoef {
  double L0, e1, e2, e3;
};

template <int NW, bool PREFETCH>
__global__ __launch_bounds__(64 * NW) void k_lut_linear(const uint32_t* __restrict__ W, const uint16_t* __restrict__ s_w,
                                                    const int8_t* __restrict__ act_q, const float* __restrict__ s_x,
                                                    int M, int64_t N, int64_t K, LutCoef cf, uint16_t* __restrict__ y) {
  __shared__ int red[NW][3][16][16];   // [wave][sum][row][token]
  __shared__ int redq[NW][4][16];      // [wave][k-group][token]: partial sums of q
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, kg = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int m0 = (int)blockIdx.y * 16;
  const int nrows = N - n0 < 16 ? (int)(N - n0) : 16;
  const int mrows = M - m0 < 16 ? M - m0 : 16;
  const uint32_t rowbytes = (uint32_t)(K / 4);
  // packed bytes of the tile and activation bytes of the token block stay below 2^31 (host check)
  const __amdgpu_buffer_rsrc_t wr = dev::make_rsrc(W + n0 * (K / 16), (uint32_t)nrows * rowbytes);
  const __amdgpu_buffer_rsrc_t ar = dev::make_rsrc(act_q + (int64_t)m0 * K, (uint32_t)mrows * (uint32_t)K);
  // rows and tokens past the tile read as zeros (range-checked loads); k offsets below add < 2^15
  const uint32_t wbase = li < nrows ? (uint32_t)li * rowbytes : dev::kOutOfRange;
  const uint32_t abase = li < mrows ? (uint32_t)li * (uint32_t)K : dev::kOutOfRange;
  v4i dc = {0, 0, 0, 0}, d1 = dc, d01 = dc;
  int sq = 0;
  const int nblk = (int)(K / 256);
  // block S's loads; a block past the end reads zeros (its offsets are past both buffers)
  auto load = [&](int S, uint4& wq, uint4 (&aq)[4]) {
    const uint32_t o = S < nblk ? 0u : dev::kOutOfRange;
    wq = dev::bload16(wr, (wbase | o) + 64u * S + 16u * kg);
#pragma unroll
    for (int j = 0; j < 4; ++j) aq[j] = dev::bload16(ar, (abase | o) + 256u * S + 64u * kg + 16u * j);
  };
  uint4 wn, an[4];
  if (PREFETCH) load(wave, wn, an);
  for (int S = wave; S < nblk; S += NW) {
    uint4 wq, aq[4];
    if (PREFETCH) {
      wq = wn;
#pragma unroll
      for (int j = 0; j < 4; ++j) aq[j] = an[j];
      load(S + NW, wn, an);
    } else {
      load(S, wq, aq);
    }
    const uint32_t ww[4] = {wq.x, wq.y, wq.z, wq.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v4i c, hb, both;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        // byte lanes: the codes of k = 16 word + 4 t .. + 3 (bits 8 beta + 2 t of the word)
        const uint32_t ct = (ww[j] >> (2 * t)) & 0x03030303u;
        const uint32_t h = (ct >> 1) & 0x01010101u;
        c[t] = (int)ct;
        hb[t] = (int)h;
        both[t] = (int)(ct & h);
      }
      const v4i b = __builtin_bit_cast(v4i, aq[j]);
      sq = mma::sum16_i8(aq[j], sq);
      dc = mma::mfma_i8(c, b, dc);
      d1 = mma::mfma_i8(hb, b, d1);
      d01 = mma::mfma_i8(both, b, d01);
    }
  }
  // D lane (token li, group kg) holds rows 4 kg + r
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    red[wave][0][4 * kg + r][li] = dc[r];
    red[wave][1][4 * kg + r][li] = d1[r];
    red[wave][2][4 * kg + r][li] = d01[r];
  }
  redq[wave][kg][li] = sq;
  __syncthreads();
  const int m = tid >> 4, n = tid & 15;
  if (m < mrows && n < nrows) {
    int s[3];
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      s[p] = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) s[p] += red[w][p][n][m];
    }
    int sum_q = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) sum_q += redq[w][0][m] + redq[w][1][m] + redq[w][2][m] + redq[w][3][m];
    const double t = cf.L0 * (double)sum_q + cf.e1 * (double)s[0] + cf.e2 * (double)s[1] + cf.e3 * (double)s[2];
    // fp32 intermediates pinned to registers: otherwise the backend fuses the second product with the
    // fp16 conversion (one rounding instead of two), as in the integer formats' epilogue
    float a = (float)t * s_x[m0 + m];
    float w = __half2float(__ushort_as_half(s_w[n0 + n]));
    asm volatile("" : "+v"(a), "+v"(w));
    float v = a * w;
    asm volatile("" : "+v"(v));
    y[(int64_t)(m0 + m) * N + n0 + n] = __half_as_ushort(__float2half_rn(v));
  }
}

}  // namespace

hipError_t launch_lut_linear(const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K, const double lut[4],
                             const int8_t* act_q, const float* act_scale, int64_t M, uint16_t* out, hipStream_t s) {
  const LutCoef cf{lut[0], lut[1] - lut[0], lut[2] - 2.0 * lut[1] + lut[0], lut[3] - lut[2] - lut[1] + lut[0]};
  const dim3 grid((unsigned)((N + 15) / 16), (unsigned)((M + 15) / 16));
  if ((int64_t)grid.x * grid.y < 512)
    hipLaunchKernelGGL((k_lut_linear<8, true>), grid, dim3(512), 0, s, packed, scales, act_q, act_scale, (int)M, N, K,
                       cf, out);
  else
    hipLaunchKernelGGL((k_lut_linear<4, false>), grid, dim3(256), 0, s, packed, scales, act_q, act_scale, (int)M, N, K,
                       cf, out);
  return hipGetLastError();
}

}  // namespace qift
