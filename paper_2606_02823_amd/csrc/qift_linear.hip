// Quantized linear y = s_w[n] s_x[m] sum_k level[n,k] q[m,k] on int8 MFMA.
//
// Decoded levels are small fixed signed integers (Sec. 3.6), so the integer
// dot product runs on CDNA4's v_mfma_i32_16x16x64_i8 with exact int32
// accumulation, and the per-channel and per-token scales are applied once in
// the epilogue (Sec. 1).
//
// One packed QW2v1 word holds 16 weights k = 16j .. 16j+15 and
// (word >> 2t) & 0x03030303 puts the codes of k = 16j+4t .. +3 in byte lanes,
// so one word decodes with 3 shifts + 4 ands into exactly one lane's 16-byte
// MFMA operand, in natural k order.  The level is an affine function of the
// code for MNZ (level = 2c - 3, the fractional-midpoint form of Sec. 3.3) and
// of the nibble for W4 (q = u - 8), so the MFMA runs on the raw codes and the
// epilogue adds the exact correction from the per-token sum of q:
//     MNZ: acc = 2 D - 3 sum_q        W4: acc = D - 8 sum_q
// For PoT-MNZ the code picks its level through a byte permute (v_perm_b32
// with the table {-4,-1,+1,+4}): the sign-and-shift magnitudes of
// Sec. 3.3/3.6 become a one-instruction lookup per four weights.
//
// Operand mapping for one MFMA (A = weights, B = activations):
//   lane l: row/column l & 15, k-group g = l >> 4 (16 k-slots each).
//   A lane (n, g) carries 16 decoded weights of row n; B lane (m, g) carries
//   the 16 activation bytes of token m at the same 16 k, so the k-slot
//   assignment inside the instruction is the same for both and cancels.
//   Result: lane l, register r holds D[n = 4 (l >> 4) + r][m = l & 15].
#include <hip/hip_fp16.h>

#include "qift_internal.h"

namespace qift {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int FMT_MNZ = 0, FMT_POT = 1, FMT_W4 = 2;

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// One packed 2-bit word -> 16 int8 operand bytes (natural k order).
template <int FMT>
__device__ __forceinline__ v4i decode_w2(uint32_t w) {
  const uint32_t c0 = w & 0x03030303u, c1 = (w >> 2) & 0x03030303u;
  const uint32_t c2 = (w >> 4) & 0x03030303u, c3 = (w >> 6) & 0x03030303u;
  if constexpr (FMT == FMT_POT) {
    // byte table {-4, -1, +1, +4} indexed by the code
    constexpr uint32_t lut = 0x0401FFFCu;
    v4i r;
    r[0] = (int)__builtin_amdgcn_perm(0u, lut, c0);
    r[1] = (int)__builtin_amdgcn_perm(0u, lut, c1);
    r[2] = (int)__builtin_amdgcn_perm(0u, lut, c2);
    r[3] = (int)__builtin_amdgcn_perm(0u, lut, c3);
    return r;
  } else {
    v4i r;
    r[0] = (int)c0; r[1] = (int)c1; r[2] = (int)c2; r[3] = (int)c3;
    return r;
  }
}

// Two packed 4-bit words (16 weights) -> 16 unsigned nibbles u = q + 8 as bytes.
__device__ __forceinline__ v4i decode_w4(uint32_t w0, uint32_t w1) {
  v4i r;
  r[0] = (int)(w0 & 0x0F0F0F0Fu);
  r[1] = (int)((w0 >> 4) & 0x0F0F0F0Fu);
  r[2] = (int)(w1 & 0x0F0F0F0Fu);
  r[3] = (int)((w1 >> 4) & 0x0F0F0F0Fu);
  return r;
}

template <int FMT>
__device__ __forceinline__ int finish_acc(int D, int sum_q) {
  if constexpr (FMT == FMT_MNZ) return 2 * D - 3 * sum_q;
  else if constexpr (FMT == FMT_W4) return D - 8 * sum_q;
  else return D;
}

// y = fp16(fp32(fp32(acc) * s_x) * fp32(s_w)), each product rounded to fp32.
// The empty asm statements keep the fp32 intermediates in registers: without
// them the backend fuses the second product with the fp16 conversion
// (v_fma_mixlo_f16, one rounding instead of two, and +0 for a -0 product).
__device__ __forceinline__ uint16_t epilogue(int acc, float s_x, uint16_t s_w_bits) {
  float t1 = (float)acc * s_x;
  float w = __half2float(__ushort_as_half(s_w_bits));
  asm volatile("" : "+v"(t1), "+v"(w));
  float t2 = t1 * w;
  asm volatile("" : "+v"(t2));
  return __half_as_ushort(__float2half_rn(t2));
}

// ---------------------------------------------------------------------------
// Skinny kernel for M <= 16 * MT tokens per workgroup column.
// Workgroup = 4 waves on one 16-row tile; wave w takes the 1024-k chunks
// w, w+4, ...; inside a chunk, lane group g covers k0 = 1024c + 256u + 64g,
// u = 0..3 (64 weights per lane per unit, 16 B of W2 words).  Partial
// accumulators are summed across the waves through LDS.
// ---------------------------------------------------------------------------
template <int FMT, int MT>
__global__ __launch_bounds__(256) void k_linear_skinny(
    const uint32_t* __restrict__ P, const uint16_t* __restrict__ sw, int N, int K,
    const int8_t* __restrict__ act, const float* __restrict__ sx, const int32_t* __restrict__ asum,
    int M, uint16_t* __restrict__ y, int32_t* __restrict__ acc_out) {
  constexpr bool W4 = FMT == FMT_W4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const int mbase = blockIdx.y * 16 * MT;
  const int n = n0 + r16;
  const bool nvalid = n < N;
  const int64_t rowbytes = W4 ? (int64_t)K / 2 : (int64_t)K / 4;
  const char* prow = reinterpret_cast<const char*>(P) + (int64_t)(nvalid ? n : 0) * rowbytes;

  v4i acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = v4i{0, 0, 0, 0};

  const int nchunks = (K + 1023) >> 10;
  for (int c = wave; c < nchunks; c += 4) {
    uint4 wq[4][W4 ? 2 : 1];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k0 = (c << 10) + (u << 8) + (g << 6);
      const bool ok = nvalid && k0 < K;
#pragma unroll
      for (int h = 0; h < (W4 ? 2 : 1); ++h) {
        const uint4* src = reinterpret_cast<const uint4*>(prow + (W4 ? k0 / 2 : k0 / 4)) + h;
        wq[u][h] = ok ? *src : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if ((c << 10) + (u << 8) >= K) break;   // wave-uniform tail
      const int k0 = (c << 10) + (u << 8) + (g << 6);
      const bool kok = k0 < K;
      uint32_t wd[W4 ? 8 : 4];
      wd[0] = wq[u][0].x; wd[1] = wq[u][0].y; wd[2] = wq[u][0].z; wd[3] = wq[u][0].w;
      if constexpr (W4) {
        wd[4] = wq[u][1].x; wd[5] = wq[u][1].y; wd[6] = wq[u][1].z; wd[7] = wq[u][1].w;
      }
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        v4i a;
        if constexpr (W4) a = decode_w4(wd[2 * d], wd[2 * d + 1]);
        else a = decode_w2<FMT>(wd[d]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = mbase + mt * 16 + r16;
          v4i b = v4i{0, 0, 0, 0};
          if (kok && m < M) {
            const uint4 bb = *reinterpret_cast<const uint4*>(act + (int64_t)m * K + k0 + 16 * d);
            b = v4i{(int)bb.x, (int)bb.y, (int)bb.z, (int)bb.w};
          }
          acc[mt] = mfma_i8(a, b, acc[mt]);
        }
      }
    }
  }

  __shared__ v4i red[4][MT][64];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) red[wave][mt][lane] = acc[mt];
  __syncthreads();
  // wave w finishes token tiles mt = w, w+4, ... (only mt < MT exist)
  for (int mt = wave; mt < MT; mt += 4) {
    v4i D = red[0][mt][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) D += red[w][mt][lane];
    const int m = mbase + mt * 16 + r16;
    if (m < M) {
      const float s_x = sx[m];
      const int sq = asum[m];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int nn = n0 + 4 * g + r;
        if (nn < N) {
          const int a = finish_acc<FMT>(D[r], sq);
          y[(int64_t)m * N + nn] = epilogue(a, s_x, sw[nn]);
          if (acc_out) acc_out[(int64_t)m * N + nn] = a;
        }
      }
    }
  }
}

template <int FMT>
hipError_t launch_fmt(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                      const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                      hipStream_t s) {
  const unsigned gx = (unsigned)((N + 15) / 16);
  const int Ni = (int)N, Ki = (int)K, Mi = (int)M;
  if (M <= 16) {
    hipLaunchKernelGGL((k_linear_skinny<FMT, 1>), dim3(gx, 1), dim3(256), 0, s, P, sw, Ni, Ki, act, sx,
                       asum, Mi, y, acc_out);
  } else if (M <= 32) {
    hipLaunchKernelGGL((k_linear_skinny<FMT, 2>), dim3(gx, 1), dim3(256), 0, s, P, sw, Ni, Ki, act, sx,
                       asum, Mi, y, acc_out);
  } else {
    // 64 tokens per workgroup column; larger M tiles the grid in y
    const unsigned gy = (unsigned)((M + 63) / 64);
    hipLaunchKernelGGL((k_linear_skinny<FMT, 4>), dim3(gx, gy), dim3(256), 0, s, P, sw, Ni, Ki, act, sx,
                       asum, Mi, y, acc_out);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_linear(int fmt, const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K,
                         const int8_t* act_q, const float* act_scale, const int32_t* act_sum, int64_t M,
                         uint16_t* out, int32_t* acc_out, hipStream_t s) {
  switch (fmt) {
    case FMT_MNZ: return launch_fmt<FMT_MNZ>(packed, scales, N, K, act_q, act_scale, act_sum, M, out, acc_out, s);
    case FMT_POT: return launch_fmt<FMT_POT>(packed, scales, N, K, act_q, act_scale, act_sum, M, out, acc_out, s);
    case FMT_W4: return launch_fmt<FMT_W4>(packed, scales, N, K, act_q, act_scale, act_sum, M, out, acc_out, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qift
