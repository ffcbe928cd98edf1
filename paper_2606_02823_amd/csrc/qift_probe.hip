// Streaming-read probe: the read bandwidth this GPU achieves on a buffer, the
// floor against which the decode kernels' weight streams are measured.  A
// measurement helper, not part of the method.
//
// One-shot grid: workgroup b reads the 64 KiB segment b of the buffer, every
// thread keeping 16 coalesced 16-byte loads in flight, and folds the words
// into an XOR that it writes to partials[b] (no atomics, so no serialization
// on one address); the host XORs the partials.
#include "qift_internal.h"

namespace qift {
namespace {

constexpr int kProbeLoads = 16;    // 16-byte loads per thread

__global__ __launch_bounds__(256) void k_read_probe(const uint4* __restrict__ buf, size_t n16,
                                                    uint32_t* __restrict__ partials) {
  __shared__ uint32_t red[4];
  const size_t base = (size_t)blockIdx.x * (256 * kProbeLoads) + threadIdx.x;
  uint4 v[kProbeLoads];
#pragma unroll
  for (int i = 0; i < kProbeLoads; ++i) {
    const size_t idx = base + (size_t)i * 256;
    v[i] = idx < n16 ? buf[idx] : make_uint4(0u, 0u, 0u, 0u);
  }
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < kProbeLoads; ++i) acc ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) partials[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace

size_t read_probe_slots(size_t bytes) { return (bytes + kReadProbeSegment - 1) / kReadProbeSegment; }

hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* partials, hipStream_t s) {
  static_assert(kReadProbeSegment == 256 * kProbeLoads * 16, "segment of one workgroup");
  hipLaunchKernelGGL(k_read_probe, dim3((unsigned)read_probe_slots(bytes)), dim3(256), 0, s,
                     reinterpret_cast<const uint4*>(buf), bytes / 16, partials);
  return hipGetLastError();
}

}  // namespace qift
