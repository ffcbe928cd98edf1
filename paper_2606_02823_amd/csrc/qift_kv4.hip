// KV4: the asymmetric 4-bit key/value cache of the W2A4/KV4 setting (Sec. 3.3 Eq. (15) with the
// Sec. 4.1 configuration: clipping ratio 0.95 for keys and values) and one decode step of
// grouped-query attention that reads it.
//
// Quantizer (k_kv4_quant): one 64-lane wave per group of 128 values (one token's key or value
// vector of one KV head), lane l holding values 2l and 2l + 1.  In fp32, in this order, rounding
// half to even:
//   x_max = c max(max x, 0), x_min = c min(min x, 0) with c = fp32(0.95),
//   s = (x_max - x_min) / 15 (1 for a group of zeros), z = round(-x_min / s),
//   q = clip(round(x / s) + z, 0, 15),   reconstruction s (q - z).
// Codes are packed two per byte, value 2i in the low nibble of byte i: the cache holds 64 bytes
// of codes, an fp32 scale and a zero-point byte per token and KV head.
//
// Decode attention (k_kv4_attn, k_kv4_merge): for query head h and KV head h / G (G = Hq / Hkv),
//   out_h = sum_t softmax_t(q_h . k_t / sqrt(d)) v_t.
// Workgroup (chunk, kv, b) covers 256 cached tokens for the G query heads of one KV head and
// writes its unnormalized partial output with the chunk's maximum score and sum of exponentials;
// k_kv4_merge combines the chunks.  The reconstruction is folded into the sums:
//   q . k_t = s_t (sum_i code_{t,i} q_i - z_t sum_i q_i),
//   sum_t p_t v_t = sum_t (p_t s_t) code_t - sum_t p_t s_t z_t,
// so the key phase (one cached token per lane: a dot product without cross-lane reductions)
// converts codes to fp32 and multiplies, and the value phase (lanes over dimensions, four token
// streams per wave) accumulates with one multiply-add per code.
#include "qift_fwht.h"
#include "qift_internal.h"

namespace qift {
namespace {

constexpr int kD = 128;         // head dimension
constexpr int kChunk = 256;     // cached tokens per workgroup

__global__ __launch_bounds__(256) void k_kv4_quant(const uint16_t* __restrict__ x, int64_t groups,
                                                   uint8_t* __restrict__ codes, float* __restrict__ scales,
                                                   uint8_t* __restrict__ zeros) {
  const int lane = threadIdx.x & 63;
  const int64_t grp = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (grp >= groups) return;   // whole waves leave together; no barrier follows
  const uint32_t pair = reinterpret_cast<const uint32_t*>(x + grp * kD)[lane];
  const float a = __half2float(__ushort_as_half((uint16_t)(pair & 0xFFFFu)));
  const float b = __half2float(__ushort_as_half((uint16_t)(pair >> 16)));
  float mx = fmaxf(a, b), mn = fminf(a, b);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o));
    mn = fminf(mn, __shfl_xor(mn, o));
  }
  const float c = 0.95f;
  const float x_max = fmaxf(mx, 0.f) * c, x_min = fminf(mn, 0.f) * c;
  float s = (x_max - x_min) / 15.f;
  if (s == 0.f) s = 1.f;
  const float z = fminf(fmaxf(rintf(-x_min / s), 0.f), 15.f);
  const int qa = (int)fminf(fmaxf(rintf(a / s) + z, 0.f), 15.f);
  const int qb = (int)fminf(fmaxf(rintf(b / s) + z, 0.f), 15.f);
  codes[grp * (kD / 2) + lane] = (uint8_t)(qa | (qb << 4));
  if (lane == 0) {
    scales[grp] = s;
    zeros[grp] = (uint8_t)z;
  }
}

// partial record of one (b, kv, chunk, g): kD unnormalized output sums, then the chunk's maximum
// score m and sum of exp(score - m)
constexpr int kPart = kD + 2;

template <int G>
__global__ __launch_bounds__(256) void k_kv4_attn(const uint16_t* __restrict__ q, int Hq, int Hkv, int64_t T,
                                                  const uint8_t* __restrict__ kc, const float* __restrict__ ks,
                                                  const uint8_t* __restrict__ kz, const uint8_t* __restrict__ vc,
                                                  const float* __restrict__ vs, const uint8_t* __restrict__ vz,
                                                  float* __restrict__ part, int nchunks) {
  __shared__ float qs[kD][G];            // the group's queries / sqrt(d), dimension-major
  __shared__ float qsum[G];
  __shared__ float pr[G][kChunk];        // scores, then exp(score - m)
  __shared__ float stat[G][2];
  __shared__ float red[4][G][kD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int chunk = blockIdx.x, kv = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int64_t t0 = (int64_t)chunk * kChunk;

  const float rsd = 1.0f / sqrtf((float)kD);
  for (int i = tid; i < kD * G; i += 256) {
    const int g = i / kD, dd = i % kD;
    qs[dd][g] = __half2float(__ushort_as_half(q[(b * Hq + (int64_t)kv * G + g) * kD + dd])) * rsd;
  }
  __syncthreads();
  if (tid < G) {
    float sum = 0.f;
    for (int dd = 0; dd < kD; ++dd) sum += qs[dd][tid];
    qsum[tid] = sum;
  }
  __syncthreads();

  // ---- scores: one cached token per lane
  {
    const int64_t t = t0 + 64 * wave + lane;
    float sc[G];
    if (t < T) {
      const int64_t row = (b * T + t) * Hkv + kv;
      const uint4* src = reinterpret_cast<const uint4*>(kc + row * (kD / 2));
      float acc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] = 0.f;
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) {
        const uint4 w = src[c4];
        const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t lo = ww[k] & 0x0F0F0F0Fu, hi = (ww[k] >> 4) & 0x0F0F0F0Fu;
#pragma unroll
          for (int by = 0; by < 4; ++by) {
            const int j = 16 * c4 + 4 * k + by;   // byte j holds values 2j (low) and 2j + 1 (high)
            const float ce = (float)((lo >> (8 * by)) & 0xFFu), co = (float)((hi >> (8 * by)) & 0xFFu);
#pragma unroll
            for (int g = 0; g < G; ++g) acc[g] = fmaf(co, qs[2 * j + 1][g], fmaf(ce, qs[2 * j][g], acc[g]));
          }
        }
      }
      const float s = ks[row], z = (float)kz[row];
#pragma unroll
      for (int g = 0; g < G; ++g) sc[g] = s * (acc[g] - z * qsum[g]);
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g) sc[g] = -INFINITY;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) pr[g][64 * wave + lane] = sc[g];
  }
  __syncthreads();

  // ---- the chunk's softmax statistics, one wave per head
  for (int g = wave; g < G; g += 4) {
    float v[kChunk / 64];
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kChunk / 64; ++i) {
      v[i] = pr[g][64 * i + lane];
      m = fmaxf(m, v[i]);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float l = 0.f;
#pragma unroll
    for (int i = 0; i < kChunk / 64; ++i) {
      const float e = v[i] == -INFINITY ? 0.f : expf(v[i] - m);
      pr[g][64 * i + lane] = e;
      l += e;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o);
    if (lane == 0) {
      stat[g][0] = m;
      stat[g][1] = l;
    }
  }
  __syncthreads();

  // ---- values: lane l covers dimensions 8 (l mod 16) .. + 7 of tokens 64 wave + 4 j + l / 16.  All
  // sixteen tokens' codes, scales and zero-points are loaded first (range-checked buffer loads: zeros
  // past T, where the weights are 0 as well), then accumulated.
  {
    const int dq = lane & 15, ts = lane >> 4;
    const int64_t row0 = (b * T) * Hkv + kv;   // cache row of token 0; token t is row0 + t Hkv
    const uint32_t rows = (uint32_t)(T * Hkv);   // T Hkv 64 < 2^31: checked by the host
    const __amdgpu_buffer_rsrc_t crs = dev::make_rsrc(vc + row0 * (kD / 2), rows * (kD / 2));
    const __amdgpu_buffer_rsrc_t srs = dev::make_rsrc(vs + row0, rows * 4u);
    const __amdgpu_buffer_rsrc_t zrs = dev::make_rsrc(vz + row0, rows);
    uint32_t vw[16];
    float vsc[16], vzz[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int64_t t = t0 + 64 * wave + 4 * j + ts;
      const bool ok = t < T;
      const uint32_t r = (uint32_t)(t * Hkv);   // rows from row0
      vw[j] = __builtin_amdgcn_raw_buffer_load_b32(crs, ok ? r * (kD / 2) + 4u * dq : dev::kOutOfRange, 0, 0);
      vsc[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(srs, ok ? 4u * r : dev::kOutOfRange, 0, 0));
      vzz[j] = (float)__builtin_amdgcn_raw_buffer_load_b8(zrs, ok ? r : dev::kOutOfRange, 0, 0);
    }
    float acc[G][8], accz[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      accz[g] = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[g][i] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int tl = 64 * wave + 4 * j + ts;
      const uint32_t lo = vw[j] & 0x0F0F0F0Fu, hi = (vw[j] >> 4) & 0x0F0F0F0Fu;
      float cv[8];
#pragma unroll
      for (int by = 0; by < 4; ++by) {
        cv[2 * by] = (float)((lo >> (8 * by)) & 0xFFu);
        cv[2 * by + 1] = (float)((hi >> (8 * by)) & 0xFFu);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float ps = pr[g][tl] * vsc[j];
        accz[g] = fmaf(ps, vzz[j], accz[g]);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[g][i] = fmaf(ps, cv[i], acc[g][i]);
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float v = acc[g][i] - accz[g];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        acc[g][i] = v;
      }
    if (lane < 16) {
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < 8; ++i) red[wave][g][8 * dq + i] = acc[g][i];
    }
  }
  __syncthreads();
  float* out = part + ((((int64_t)b * Hkv + kv) * nchunks + chunk) * G) * kPart;
  for (int i = tid; i < G * kD; i += 256) {
    const int g = i / kD, dd = i % kD;
    out[g * kPart + dd] = (red[0][g][dd] + red[1][g][dd]) + (red[2][g][dd] + red[3][g][dd]);
  }
  if (tid < G) {
    out[tid * kPart + kD] = stat[tid][0];
    out[tid * kPart + kD + 1] = stat[tid][1];
  }
}

// out[b][kv G + g][:] = sum_c e^(m_c - M) part_c / sum_c e^(m_c - M) l_c,  M = max_c m_c.
// Workgroup (kv G + g, b), thread dd: the maximum by a block reduction, then per tile of 128 chunks
// the chunk weights once into LDS and the sum over the tile (independent, coalesced loads).
template <int G>
__global__ __launch_bounds__(kD) void k_kv4_merge(const float* __restrict__ part, int Hq, int Hkv, int nchunks,
                                                  uint16_t* __restrict__ y) {
  __shared__ float red[kD / 64];
  __shared__ float ew[kD], lw[kD];
  const int dd = threadIdx.x, lane = dd & 63, wave = dd >> 6;
  const int kv = blockIdx.x / G, g = blockIdx.x % G;
  const int64_t b = blockIdx.y;
  const float* base = part + (((int64_t)b * Hkv + kv) * nchunks) * G * kPart + g * kPart;
  const int64_t cstride = (int64_t)G * kPart;
  float M = -INFINITY;
  for (int c = dd; c < nchunks; c += kD) M = fmaxf(M, base[c * cstride + kD]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  if (lane == 0) red[wave] = M;
  __syncthreads();
  M = fmaxf(red[0], red[1]);
  float acc = 0.f, L = 0.f;
  for (int c0 = 0; c0 < nchunks; c0 += kD) {
    __syncthreads();   // the previous tile's weights have been read
    if (c0 + dd < nchunks) {
      const float* r = base + (c0 + dd) * cstride;
      const float e = expf(r[kD] - M);
      ew[dd] = e;
      lw[dd] = r[kD + 1] * e;
    }
    __syncthreads();
    const int n = nchunks - c0 < kD ? nchunks - c0 : kD;
#pragma unroll 8
    for (int i = 0; i < n; ++i) {
      acc = fmaf(base[(c0 + i) * cstride + dd], ew[i], acc);
      L += lw[i];
    }
  }
  y[(b * Hq + (int64_t)kv * G + g) * kD + dd] = __half_as_ushort(__float2half_rn(acc / L));
}

template <int G>
hipError_t launch_attn_g(const uint16_t* q, int64_t B, int Hq, int Hkv, int64_t T, const uint8_t* kc,
                         const float* ks, const uint8_t* kz, const uint8_t* vc, const float* vs,
                         const uint8_t* vz, uint16_t* y, float* part, hipStream_t s) {
  const int nchunks = (int)((T + kChunk - 1) / kChunk);
  hipLaunchKernelGGL((k_kv4_attn<G>), dim3((unsigned)nchunks, (unsigned)Hkv, (unsigned)B), dim3(256), 0, s, q, Hq,
                     Hkv, T, kc, ks, kz, vc, vs, vz, part, nchunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_kv4_merge<G>), dim3((unsigned)(Hkv * G), (unsigned)B), dim3(kD), 0, s, part, Hq, Hkv, nchunks,
                     y);
  return hipGetLastError();
}

}  // namespace

size_t kv4_attention_workspace(int64_t B, int64_t Hq, int64_t T) {
  const int64_t nchunks = (T + kChunk - 1) / kChunk;
  return (size_t)(B * Hq * nchunks * kPart) * sizeof(float);
}

hipError_t launch_kv4_quant(const uint16_t* x, int64_t groups, uint8_t* codes, float* scales, uint8_t* zeros,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_kv4_quant, dim3((unsigned)((groups + 3) / 4)), dim3(256), 0, s, x, groups, codes, scales, zeros);
  return hipGetLastError();
}

hipError_t launch_kv4_attention(const uint16_t* q, int64_t B, int Hq, int Hkv, int64_t T, const uint8_t* kc,
                                const float* ks, const uint8_t* kz, const uint8_t* vc, const float* vs,
                                const uint8_t* vz, uint16_t* y, void* ws, hipStream_t s) {
  float* part = static_cast<float*>(ws);
  switch (Hq / Hkv) {
    case 1: return launch_attn_g<1>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, s);
    case 2: return launch_attn_g<2>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, s);
    case 4: return launch_attn_g<4>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, s);
    case 8: return launch_attn_g<8>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qift
