// Packing of decoded weight levels into the QW2v1 / QW4v1 words.
//
// The paper fixes a four-level set per format and leaves the 2-bit code
// assignment free (Sec. 3.3); here code = ascending index of the level.  The
// packer is an offline, bandwidth-bound elementwise pass: one thread per
// output word, a 16-byte (W2) or 8-byte (W4) coalesced read of levels.
#include "qift_internal.h"

namespace qift {
namespace {

__global__ void k_zero_i32(int32_t* p) { *p = 0; }

// Level -> 2-bit code for the set {l0 < l1 < l2 < l3}; -1 when not a member.
__device__ __forceinline__ int level_code(int v, int l0, int l1, int l2, int l3) {
  return v == l0 ? 0 : v == l1 ? 1 : v == l2 ? 2 : v == l3 ? 3 : -1;
}

__global__ __launch_bounds__(256) void k_pack_w2(const int8_t* __restrict__ levels, int64_t words,
                                                 uint32_t* __restrict__ packed, int32_t* invalid_count,
                                                 int l0, int l1, int l2, int l3) {
  int bad = 0;
  for (int64_t w = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; w < words;
       w += (int64_t)gridDim.x * blockDim.x) {
    // 16 consecutive levels k = 16j .. 16j+15 of one row (rows are K/16 words long).
    const uint4 raw = reinterpret_cast<const uint4*>(levels)[w];
    const uint32_t d[4] = {raw.x, raw.y, raw.z, raw.w};
    uint32_t word = 0;
#pragma unroll
    for (int p = 0; p < 16; ++p) {
      const int v = (int)(int8_t)((d[p >> 2] >> (8 * (p & 3))) & 0xFF);
      int c = level_code(v, l0, l1, l2, l3);
      bad += (c < 0);
      c = c < 0 ? 0 : c;
      const int t = p >> 2, b = p & 3;  // k = 16j + 4t + b
      word |= (uint32_t)c << (8 * b + 2 * t);
    }
    packed[w] = word;
  }
  if (invalid_count && bad) atomicAdd(invalid_count, bad);
}

__global__ __launch_bounds__(256) void k_pack_w4(const int8_t* __restrict__ levels, int64_t words,
                                                 uint32_t* __restrict__ packed, int32_t* invalid_count) {
  int bad = 0;
  for (int64_t w = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; w < words;
       w += (int64_t)gridDim.x * blockDim.x) {
    // 8 consecutive levels k = 8j .. 8j+7 of one row (rows are K/8 words long).
    const uint2 raw = reinterpret_cast<const uint2*>(levels)[w];
    const uint32_t d[2] = {raw.x, raw.y};
    uint32_t word = 0;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      int v = (int)(int8_t)((d[p >> 2] >> (8 * (p & 3))) & 0xFF);
      const bool ok = v >= -7 && v <= 7;
      bad += !ok;
      v = ok ? v : 0;
      const int t = p >> 2, b = p & 3;  // k = 8j + 4t + b
      word |= (uint32_t)(v + 8) << (8 * b + 4 * t);
    }
    packed[w] = word;
  }
  if (invalid_count && bad) atomicAdd(invalid_count, bad);
}

int grid_for(int64_t items) {
  int64_t g = (items + 255) / 256;
  return (int)(g < 8192 ? (g < 1 ? 1 : g) : 8192);
}

}  // namespace

hipError_t launch_pack_w2(const int8_t* levels, int64_t N, int64_t K, int fmt, uint32_t* packed,
                          int32_t* invalid_count, hipStream_t s) {
  // ascending level lists: MNZ at half scale, PoT-MNZ, and the codes themselves (level table)
  const int l[3][4] = {{-3, -1, 1, 3}, {-4, -1, 1, 4}, {0, 1, 2, 3}};
  const int* L = l[fmt == 1 ? 1 : fmt == 3 ? 2 : 0];
  const int64_t words = N * (K / 16);
  if (invalid_count) hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(1), 0, s, invalid_count);
  hipLaunchKernelGGL(k_pack_w2, dim3(grid_for(words)), dim3(256), 0, s, levels, words, packed,
                     invalid_count, L[0], L[1], L[2], L[3]);
  return hipGetLastError();
}

hipError_t launch_pack_w4(const int8_t* levels, int64_t N, int64_t K, uint32_t* packed,
                          int32_t* invalid_count, hipStream_t s) {
  const int64_t words = N * (K / 8);
  if (invalid_count) hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(1), 0, s, invalid_count);
  hipLaunchKernelGGL(k_pack_w4, dim3(grid_for(words)), dim3(256), 0, s, levels, words, packed,
                     invalid_count);
  return hipGetLastError();
}

}  // namespace qift
