// int8-MFMA building blocks shared by the linear kernels: the packed-word
// decoders, the MFMA wrapper, the exact accumulator correction and the fp16
// epilogue of y = s_w[n] s_x[m] sum_k level[n,k] q[m,k].
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
//
// A lane's 16-byte load of packed words covers 4 MFMAs: lane group g of a
// 256-k block reads words [4g, 4g + 4) of that block for each of its rows,
// and MFMA s uses word 4g + s, i.e. k = 64g + 16s .. +15 within the block.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qift {
namespace mma {

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
  v4i r;
  if constexpr (FMT == FMT_POT) {
    // byte table {-4, -1, +1, +4} indexed by the code
    constexpr uint32_t lut = 0x0401FFFCu;
    r[0] = (int)__builtin_amdgcn_perm(0u, lut, c0);
    r[1] = (int)__builtin_amdgcn_perm(0u, lut, c1);
    r[2] = (int)__builtin_amdgcn_perm(0u, lut, c2);
    r[3] = (int)__builtin_amdgcn_perm(0u, lut, c3);
  } else {
    r[0] = (int)c0; r[1] = (int)c1; r[2] = (int)c2; r[3] = (int)c3;
  }
  return r;
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

// Operand s (0..3) of a lane's 64-weight unit: W2 uses one 16-byte load, W4 two.
template <int FMT>
__device__ __forceinline__ v4i decode_unit(const uint4 (&u)[FMT == FMT_W4 ? 2 : 1], int s) {
  if constexpr (FMT == FMT_W4) {
    const uint4 h = u[s >> 1];
    return (s & 1) ? decode_w4(h.z, h.w) : decode_w4(h.x, h.y);
  } else {
    const uint32_t w = s == 0 ? u[0].x : s == 1 ? u[0].y : s == 2 ? u[0].z : u[0].w;
    return decode_w2<FMT>(w);
  }
}

// Bit-plane decode of a lane's four packed MNZ words (u.x .. u.w, 64 weights):
// operand t takes the 2-bit field t of every byte of the four words, i.e. the
// codes of k = 16i + 4t + b (word i, byte b), left in place (scaled by 4^t)
// for t < 3, which costs one AND per word, and shifted down for t = 3.  With
// the codes of the same k as B operand (the planar code layout) and one
// accumulator per plane, the unit's code dot product is
//     D = acc0 + acc1 / 4 + acc2 / 16 + acc3,
// where every division is exact (acc_t is 4^t times an integer sum).  Planes
// 0 and 3 carry the same factor, so they may share one accumulator.
__device__ __forceinline__ v4i decode_plane(const uint4& u, int t) {
  if (t == 3)
    return v4i{(int)((u.x >> 6) & 0x03030303u), (int)((u.y >> 6) & 0x03030303u),
               (int)((u.z >> 6) & 0x03030303u), (int)((u.w >> 6) & 0x03030303u)};
  const uint32_t mk = 0x03030303u << (2 * t);
  return v4i{(int)(u.x & mk), (int)(u.y & mk), (int)(u.z & mk), (int)(u.w & mk)};
}

__device__ __forceinline__ v4i combine_planes(const v4i& a0, const v4i& a1, const v4i& a2, const v4i& a3) {
  v4i d;
#pragma unroll
  for (int r = 0; r < 4; ++r) d[r] = a0[r] + (a1[r] >> 2) + (a2[r] >> 4) + a3[r];
  return d;
}

// The same with planes 0 and 3 accumulated together in a03.
__device__ __forceinline__ v4i combine_planes(const v4i& a03, const v4i& a1, const v4i& a2) {
  v4i d;
#pragma unroll
  for (int r = 0; r < 4; ++r) d[r] = a03[r] + (a1[r] >> 2) + (a2[r] >> 4);
  return d;
}

// Bit planes of a lane's four packed MNZ words with two accumulators: planes 0 and 3 as codes (factor
// 1), planes 1 and 2 as codes times 4 (plane 2 shifted down by one field), so that
//   D = acc03 + acc12 / 4,
// exact since acc12 is 4 times an integer sum.  One more shift per word than
// decode_plane, half the accumulators (for kernels that hold many tiles' accumulators).
__device__ __forceinline__ v4i decode_plane2(const uint4& u, int t) {
  if (t == 0) return v4i{(int)(u.x & 0x03030303u), (int)(u.y & 0x03030303u), (int)(u.z & 0x03030303u), (int)(u.w & 0x03030303u)};
  if (t == 1) return v4i{(int)(u.x & 0x0C0C0C0Cu), (int)(u.y & 0x0C0C0C0Cu), (int)(u.z & 0x0C0C0C0Cu), (int)(u.w & 0x0C0C0C0Cu)};
  if (t == 2)
    return v4i{(int)((u.x >> 2) & 0x0C0C0C0Cu), (int)((u.y >> 2) & 0x0C0C0C0Cu), (int)((u.z >> 2) & 0x0C0C0C0Cu),
               (int)((u.w >> 2) & 0x0C0C0C0Cu)};
  return v4i{(int)((u.x >> 6) & 0x03030303u), (int)((u.y >> 6) & 0x03030303u), (int)((u.z >> 6) & 0x03030303u),
             (int)((u.w >> 6) & 0x03030303u)};
}

// Sum of the 16 signed bytes of a 16-byte group of activation codes (four dot products with 1).
__device__ __forceinline__ int sum16_i8(const uint4& b, int acc) {
  acc = __builtin_amdgcn_sdot4((int)b.x, 0x01010101, acc, false);
  acc = __builtin_amdgcn_sdot4((int)b.y, 0x01010101, acc, false);
  acc = __builtin_amdgcn_sdot4((int)b.z, 0x01010101, acc, false);
  return __builtin_amdgcn_sdot4((int)b.w, 0x01010101, acc, false);
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

// Store the 4 consecutive outputs n0..n0+3 of token m held in D (and their accumulators).
template <int FMT>
__device__ __forceinline__ void store4(const v4i& D, int m, int n0, int N, float s_x, int sum_q,
                                       const uint16_t* __restrict__ sw, uint16_t* __restrict__ y,
                                       int32_t* __restrict__ acc_out) {
  int a[4];
  uint16_t h[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int n = n0 + r;
    a[r] = finish_acc<FMT>(D[r], sum_q);
    h[r] = n < N ? epilogue(a[r], s_x, sw[n]) : 0;
  }
  const int64_t o = (int64_t)m * N + n0;
  if (n0 + 3 < N && (o & 3) == 0) {
    *reinterpret_cast<uint2*>(y + o) =
        make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
    if (acc_out) *reinterpret_cast<int4*>(acc_out + o) = make_int4(a[0], a[1], a[2], a[3]);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (n0 + r < N) {
        y[o + r] = h[r];
        if (acc_out) acc_out[o + r] = a[r];
      }
    }
  }
}

// store4 with the four fp16 scales s_w[n0..n0+3] already in registers (swq,
// low half first; zeros past N).
template <int FMT>
__device__ __forceinline__ void store4_sw(const v4i& D, int m, int n0, int N, float s_x, int sum_q, uint2 swq,
                                          uint16_t* __restrict__ y, int32_t* __restrict__ acc_out) {
  const uint16_t swv[4] = {(uint16_t)(swq.x & 0xFFFFu), (uint16_t)(swq.x >> 16), (uint16_t)(swq.y & 0xFFFFu),
                           (uint16_t)(swq.y >> 16)};
  int a[4];
  uint16_t h[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    a[r] = finish_acc<FMT>(D[r], sum_q);
    h[r] = n0 + r < N ? epilogue(a[r], s_x, swv[r]) : 0;
  }
  const int64_t o = (int64_t)m * N + n0;
  if (n0 + 3 < N && (o & 3) == 0) {
    *reinterpret_cast<uint2*>(y + o) =
        make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
    if (acc_out) *reinterpret_cast<int4*>(acc_out + o) = make_int4(a[0], a[1], a[2], a[3]);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (n0 + r < N) {
        y[o + r] = h[r];
        if (acc_out) acc_out[o + r] = a[r];
      }
    }
  }
}

}  // namespace mma
}  // namespace qift
