// KV4: the asymmetric 4-bit key/value cache of the W2A4/KV4 setting (Sec. 3.3 Eq. (15) with the
// Sec. 4.1 configuration: clipping ratio 0.95 for keys and values) and one decode step of
// grouped-query attention that reads it.
//
// Quantizer (k_kv4_quant): 16 lanes per group of 128 values (one token's key or value vector of
// one KV head), lane j holding values 8j .. 8j + 7 (one 16-byte load, one 4-byte store of their
// codes), 4 groups per wave and step of a grid-stride loop.  In fp32, in this order, rounding
// half to even:
//   x_max = c max(max x, 0), x_min = c min(min x, 0) with c = fp32(0.95),
//   s = (x_max - x_min) / 15 (1 for a group of zeros), z = round(-x_min / s),
//   q = clip(round(x / s) + z, 0, 15),   reconstruction s (q - z).
// Codes are packed two per byte, value 2i in the low nibble of byte i: the cache holds 64 bytes
// of codes, an fp32 scale and a zero-point byte per token and KV head.
//
// Decode attention (k_kv4_attn, then a merge kernel: k_kv4_merge_regs or k_kv4_merge): for query head h and KV head h / G (G = Hq / Hkv),
//   out_h = sum_t softmax_t(q_h . k_t / sqrt(d)) v_t.
// Workgroup (chunk, kv, b) covers 256 cached tokens for the G query heads of one KV head and
// writes its unnormalized partial output with the chunk's maximum score and sum of exponentials;
// the merge kernel combines the chunks.  The reconstruction is folded into the sums:
//   q . k_t = s_t sum_i (code_{t,i} - z_t) q_i,
//   sum_t p_t v_t = sum_t (p_t s_t) code_t - sum_t p_t s_t z_t,
// so both phases run on the f16 MFMA with the codes as exact fp16 operands: the key phase codes x
// queries (16 tokens x 32 dimensions per instruction), the value phase P = p s (split into two fp16
// parts) x codes (16 heads x 32 tokens x 16 dimensions), its operands read from LDS with the 4-bit
// transposing read.  A workgroup issues all its loads first and waits on HBM once.
#include "qift_fwht.h"
#include "qift_internal.h"

namespace qift {
namespace {

constexpr int kD = 128;         // head dimension
constexpr int kChunk = 256;     // cached tokens per workgroup

typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));

// Eight 4-bit codes of a word (nibble n at bits 4n) as MFMA fp16 operands without conversion: a code
// masked in place within a 16-bit half is an exact fp16 subnormal, code 2^-24 (bits 0-3 of the half)
// or code 2^-20 (bits 4-7).  Element e is nibble kNib[e]; elements with e & 2 carry the 2^-20 kind,
// so the other operand's element e takes a factor 1/16 there and the product sums are 2^-24 times
// the code sums.  The f16 MFMA sums products of subnormal inputs less precisely than those of
// normal ones (measured on gfx950: about 9e-7 against 6e-8 of the sum of |products|), which the
// value phase can afford (its error is linear in the output) and the scores cannot.
constexpr int kNib[8] = {0, 4, 1, 5, 2, 6, 3, 7};
__device__ __forceinline__ v8h codes_f16(uint32_t w) {
  const uint32_t w8 = w >> 8;
  const uint4 h = {w & 0x000F000Fu, w & 0x00F000F0u, w8 & 0x000F000Fu, w8 & 0x00F000F0u};
  return __builtin_bit_cast(v8h, h);
}

// Eight 4-bit codes of one group minus its zero-point z, as exact normal fp16 values: a byte
// permute puts each code below an 0x64 byte (the fp16 value 1024 + code) and a packed subtraction
// of 1024 + z leaves code - z.  Element e is nibble kNibK[e] of the word.
constexpr int kNibK[8] = {0, 2, 4, 6, 1, 3, 5, 7};
__device__ __forceinline__ v8h codes_minus_z(uint32_t w, v2h base) {
  const uint32_t lo = w & 0x0F0F0F0Fu, hi = (w >> 4) & 0x0F0F0F0Fu;   // byte m: nibble 2m / 2m + 1
  const uint32_t k64 = 0x64646464u;
  // selector bytes 0-3 pick from the second operand, 4-7 from the first (all 0x64)
  const uint32_t s01 = 0x04010400u, s23 = 0x04030402u;
  const v2h h0 = __builtin_bit_cast(v2h, __builtin_amdgcn_perm(k64, lo, s01)) - base;   // nibbles 0, 2
  const v2h h1 = __builtin_bit_cast(v2h, __builtin_amdgcn_perm(k64, lo, s23)) - base;   // nibbles 4, 6
  const v2h h2 = __builtin_bit_cast(v2h, __builtin_amdgcn_perm(k64, hi, s01)) - base;   // nibbles 1, 3
  const v2h h3 = __builtin_bit_cast(v2h, __builtin_amdgcn_perm(k64, hi, s23)) - base;   // nibbles 5, 7
  return v8h{h0[0], h0[1], h1[0], h1[1], h2[0], h2[1], h3[0], h3[1]};
}

__global__ __launch_bounds__(256) void k_kv4_quant(const uint16_t* __restrict__ x, int64_t groups,
                                                   uint8_t* __restrict__ codes, float* __restrict__ scales,
                                                   uint8_t* __restrict__ zeros) {
  const int lane = threadIdx.x & 63, j = lane & 15;
  const int64_t quads = (groups + 3) / 4;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  for (int64_t wq = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wq < quads; wq += nwaves) {
    const int64_t grp = wq * 4 + (lane >> 4);
    const bool ok = grp < groups;   // lanes of a missing group run along with zeros (the shuffles need them)
    uint4 u = {0u, 0u, 0u, 0u};
    if (ok) u = reinterpret_cast<const uint4*>(x + grp * kD)[j];
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = __half2float(__ushort_as_half((uint16_t)(w[e >> 1] >> (16 * (e & 1)))));
    float mx = v[0], mn = v[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) {
      mx = fmaxf(mx, v[e]);
      mn = fminf(mn, v[e]);
    }
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) {   // within the 16 lanes of the group
      mx = fmaxf(mx, __shfl_xor(mx, o));
      mn = fminf(mn, __shfl_xor(mn, o));
    }
    const float c = 0.95f;
    const float x_max = fmaxf(mx, 0.f) * c, x_min = fminf(mn, 0.f) * c;
    float s = (x_max - x_min) / 15.f;
    if (s == 0.f) s = 1.f;
    const float z = fminf(fmaxf(rintf(-x_min / s), 0.f), 15.f);
    // rint of the rounded quotient v / s without the division where it is clear: q0 = rint(v (1/s))
    // is that value when the residual v - q0 s lies inside half a step by more than the quotient's
    // rounding (|v / s| < 32 here); the others (a wave-uniform branch, rarely taken) divide
    const float inv = 1.0f / s;
    float qf[8];
    bool nr = false;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      qf[e] = rintf(v[e] * inv);
      nr |= fabsf(fmaf(-qf[e], s, v[e])) >= (0.5f - 0x1p-16f) * s;
    }
    if (__any(nr)) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (fabsf(fmaf(-qf[e], s, v[e])) >= (0.5f - 0x1p-16f) * s) qf[e] = rintf(v[e] / s);
    }
    uint32_t packed = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) packed |= (uint32_t)(int)fminf(fmaxf(qf[e] + z, 0.f), 15.f) << (4 * e);
    if (ok) {
      reinterpret_cast<uint32_t*>(codes + grp * (kD / 2))[j] = packed;   // values 8j .. 8j + 7
      if (j == 0) {
        scales[grp] = s;
        zeros[grp] = (uint8_t)z;
      }
    }
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
                                                  float* __restrict__ part, int nchunks, int head_major) {
  constexpr int Gp = G < 4 ? 4 : G;      // heads per value-phase output row, padded to a float4
  __shared__ float pr[G][kChunk];        // scores, then P_t f_g (below)
  __shared__ float sz[4][kChunk];        // key scale, key zero-point, value scale, value zero-point
  __shared__ float stat[G][4];           // m, l, Z, 2^24 / f_g
  // value codes, 64 bytes per token with the 16-byte slots of row r XOR-swizzled by (r / 4) mod 4
  // (the transposed reads below then hit 32 distinct banks per 16 lanes); once a wave has read its
  // 64 rows it reuses them for its partial sums [dimension][Gp]
  __shared__ __attribute__((aligned(16))) uint32_t vl[kChunk * (kD / 8)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int chunk = blockIdx.x, kv = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int64_t t0 = (int64_t)chunk * kChunk;
  const int nt = (int)(T - t0 < kChunk ? T - t0 : kChunk);   // tokens of this chunk
  // cache row of token t: row0 + t rs, rows ordered [B][T][Hkv] (token-major) or [B][Hkv][T]
  const uint32_t rs = head_major ? 1u : (uint32_t)Hkv;
  const int64_t row0 = head_major ? ((int64_t)b * Hkv + kv) * T : (b * T) * Hkv + kv;
  const uint32_t rows = (uint32_t)(T * rs);    // T Hkv 64 < 2^31: checked by the host, so 32-bit
  const uint32_t rc = (uint32_t)t0 * rs;       // offsets below cannot wrap
  const __amdgpu_buffer_rsrc_t kcr = dev::make_rsrc(kc + row0 * (kD / 2), rows * (kD / 2));
  const __amdgpu_buffer_rsrc_t vcr = dev::make_rsrc(vc + row0 * (kD / 2), rows * (kD / 2));
  const __amdgpu_buffer_rsrc_t ksr = dev::make_rsrc(ks + row0, rows * 4u);
  const __amdgpu_buffer_rsrc_t vsr = dev::make_rsrc(vs + row0, rows * 4u);
  const __amdgpu_buffer_rsrc_t kzr = dev::make_rsrc(kz + row0, rows);
  const __amdgpu_buffer_rsrc_t vzr = dev::make_rsrc(vz + row0, rows);

  // ---- every load of the chunk is issued before any is used, so a workgroup waits on HBM once.
  // Range-checked buffer loads return zeros for tokens past T (their weights are zeroed below).
  // Thread tid: scale and zero-point of token t0 + tid, key and value.
  float own[4];
  {
    const bool ok = tid < nt;
    const uint32_t r = rc + (uint32_t)tid * rs;
    own[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ksr, ok ? 4u * r : dev::kOutOfRange, 0, 0));
    own[1] = (float)__builtin_amdgcn_raw_buffer_load_b8(kzr, ok ? r : dev::kOutOfRange, 0, 0);
    own[2] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(vsr, ok ? 4u * r : dev::kOutOfRange, 0, 0));
    own[3] = (float)__builtin_amdgcn_raw_buffer_load_b8(vzr, ok ? r : dev::kOutOfRange, 0, 0);
  }
  // Key phase operands, lane (c, kg) = (lane mod 16, lane / 16): the A operand of tile i is 16
  // tokens' codes, a lane loading the 16 bytes of dimensions 32 kg .. + 31 of token 64 wave + 16 i + c,
  // word st holding dimensions 32 kg + 8 st + n in nibble n; the B operand holds the G queries
  // (columns >= G zero) with element e of k-step st = dimension 32 kg + 8 st + kNibK[e] (the MFMA
  // pairs A and B element by element within a lane group).
  // (branch-free range-checked loads: a branch here would make the compiler wait for every load
  // issued so far before the code loads below are issued)
  const int c = lane & 15, kg = lane >> 4;
  const __amdgpu_buffer_rsrc_t qr = dev::make_rsrc(q + (b * Hq + (int64_t)kv * G) * kD, G * kD * 2u);
  uint4 qu[4];
#pragma unroll
  for (int st = 0; st < 4; ++st)
    qu[st] = dev::bload16(qr, c < G ? 2u * (c * kD + 32 * kg + 8 * st) : dev::kOutOfRange);
  uint4 kw[4];
#pragma unroll
  for (int tile = 0; tile < 4; ++tile) {
    const int tl = 64 * wave + 16 * tile + c;
    kw[tile] = dev::bload16(kcr, tl < nt ? (rc + (uint32_t)tl * rs) * (kD / 2) + 16u * kg : dev::kOutOfRange);
  }
  // Value codes of the wave's 64 tokens: load u, lane l takes 16-byte slot l mod 4 of token
  // 64 wave + 16 u + l / 4 (it goes to LDS before the value phase).
  uint4 vq[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int tl = 64 * wave + 16 * u + (lane >> 2);
    vq[u] = dev::bload16(vcr, tl < nt ? (rc + (uint32_t)tl * rs) * (kD / 2) + 16u * (lane & 3) : dev::kOutOfRange);
  }

  v8h qb[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const v8h qraw = __builtin_bit_cast(v8h, qu[st]);
#pragma unroll
    for (int e = 0; e < 8; ++e) qb[st][e] = qraw[kNibK[e]];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) sz[i][tid] = own[i];
  __syncthreads();

  // ---- scores on the f16 MFMA: per 16 tokens, D[token][head] = sum over the 128 dimensions of
  // (code - z_t) x query (4 MFMAs of 32 dimensions, every operand exact); q . k_t = s_t D.
  {
    const float rsd = 1.0f / sqrtf((float)kD);
#pragma unroll
    for (int tile = 0; tile < 4; ++tile) {
      const uint32_t ww[4] = {kw[tile].x, kw[tile].y, kw[tile].z, kw[tile].w};
      const _Float16 zb = (_Float16)(1024.0f + sz[1][64 * wave + 16 * tile + c]);   // exact: z <= 15
      const v2h base = {zb, zb};
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 4; ++st)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(codes_minus_z(ww[st], base), qb[st], acc, 0, 0, 0);
      // D: lane (c, kg) holds tokens 16 tile + 4 kg + i of head c
      if (c < G) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tl = 64 * wave + 16 * tile + 4 * kg + i;
          pr[c][tl] = tl < nt ? sz[0][tl] * acc[i] * rsd : -INFINITY;
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int row = 64 * wave + 16 * u + (lane >> 2);   // (row / 4) mod 4 = (lane / 16) mod 4
    *reinterpret_cast<uint4*>(&vl[row * (kD / 8) + 4 * ((lane & 3) ^ ((lane >> 4) & 3))]) = vq[u];
  }
  __syncthreads();

  // ---- the chunk's softmax statistics, one wave per head: m, l = sum_t e_t with e_t = exp(score_t
  // - m), and for the value phase P_t = e_t s_t and Z = sum_t P_t z_t.  pr receives P_t f_g with f_g
  // the power of two that puts the chunk's largest P in [2^14, 2^15): the value phase splits it into
  // two fp16 parts without overflow and with the small terms far above the fp16 subnormal range.
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
    float l = 0.f, zs = 0.f, pm = __FLT_MIN__;
#pragma unroll
    for (int i = 0; i < kChunk / 64; ++i) {
      const int tl = 64 * i + lane;
      const float e = v[i] == -INFINITY ? 0.f : expf(v[i] - m);
      const float P = e * sz[2][tl];
      v[i] = P;
      pm = fmaxf(pm, P);
      l += e;
      zs = fmaf(P, sz[3][tl], zs);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      l += __shfl_xor(l, o);
      zs += __shfl_xor(zs, o);
      pm = fmaxf(pm, __shfl_xor(pm, o));
    }
    const int ex = ilogbf(pm);   // pm normal: P of the top token is its scale s > 0
    const float f = ldexpf(1.0f, 14 - ex);
#pragma unroll
    for (int i = 0; i < kChunk / 64; ++i) pr[g][64 * i + lane] = v[i] * f;
    if (lane == 0) {
      stat[g][0] = m;
      stat[g][1] = l;
      stat[g][2] = zs;
      stat[g][3] = ldexpf(1.0f, 10 + ex);   // 2^24 / f
    }
  }
  __syncthreads();

  // ---- values on the f16 MFMA: D[head][dim] = sum over the wave's 64 tokens of A[head][token]
  // B[token][dim], A = P f (rows >= G zero) as an fp16 high part plus an fp16 low part (two MFMAs,
  // 2^-22 relative), B = the codes.  The transposing LDS read gives lane (i, kg) = (lane mod 16,
  // lane / 16) the 16 codes of dimension 16 dt + i for tokens 64 wave + 16 kg + 0 .. 15 (the rows
  // that the 16 lanes of its group address), nibble n for token n.  B element e is the code of
  // token kNib[e] of the word (codes_f16), and the A element it meets carries 1/16 where e & 2:
  // D = 2^-24 sum_t P_t f code_t.  Z is subtracted when the partial is written.
  {
    const int i16 = lane & 15, kg = lane >> 4;
    v8h ahi[2], alo[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      float pv[8];
      if (i16 < G) {
        const float4 x0 = *reinterpret_cast<const float4*>(&pr[i16][64 * wave + 16 * kg + 8 * st]);
        const float4 x1 = *reinterpret_cast<const float4*>(&pr[i16][64 * wave + 16 * kg + 8 * st + 4]);
        pv[0] = x0.x; pv[1] = x0.y; pv[2] = x0.z; pv[3] = x0.w;
        pv[4] = x1.x; pv[5] = x1.y; pv[6] = x1.z; pv[7] = x1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float x = (e & 2) ? pv[kNib[e]] * 0.0625f : pv[kNib[e]];
        const float y = (e & 2) ? pv[kNib[e + 1]] * 0.0625f : pv[kNib[e + 1]];
        const v2h h = __builtin_bit_cast(v2h, __builtin_amdgcn_cvt_pkrtz(x, y));
        const v2h r = __builtin_bit_cast(v2h, __builtin_amdgcn_cvt_pkrtz(x - (float)h[0], y - (float)h[1]));
        ahi[st][e] = h[0];
        ahi[st][e + 1] = h[1];
        alo[st][e] = r[0];
        alo[st][e + 1] = r[1];
      }
    }
    const int row = 64 * wave + 16 * kg + i16;   // the row this lane addresses
    v4f acc[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const uint32_t off = row * (kD / 8) + 4 * ((dt >> 1) ^ ((row >> 2) & 3)) + 2 * (dt & 1);
      const v2i t = __builtin_amdgcn_ds_read_tr4_b64_v2i32((__attribute__((address_space(3))) v2i*)(vl + off));
      acc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const v8h bv = codes_f16(st ? (uint32_t)t.y : (uint32_t)t.x);
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ahi[st], bv, acc[dt], 0, 0, 0);
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(alo[st], bv, acc[dt], 0, 0, 0);
      }
    }
    // D lane (i16, kg) holds heads 4 kg .. 4 kg + 3 of dimension 16 dt + i16; the wave's own rows
    // take them (its transposed reads above are done: a wave's LDS operations complete in order)
    if (4 * kg < G) {
      float* red = reinterpret_cast<float*>(vl) + 64 * wave * (kD / 8);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        *reinterpret_cast<v4f*>(&red[(16 * dt + i16) * Gp + 4 * kg]) = acc[dt];
    }
  }
  __syncthreads();
  float* out = part + ((((int64_t)b * Hkv + kv) * nchunks + chunk) * G) * kPart;
  const float* red = reinterpret_cast<const float*>(vl);
  constexpr int kWaveRed = 64 * (kD / 8);   // floats per wave's region
  for (int i = tid; i < G * kD; i += 256) {
    const int g = i / kD, dd = i % kD, o = dd * Gp + g;
    const float sum = (red[o] + red[kWaveRed + o]) + (red[2 * kWaveRed + o] + red[3 * kWaveRed + o]);
    out[g * kPart + dd] = sum * stat[g][3] - stat[g][2];
  }
  if (tid < G) {
    out[tid * kPart + kD] = stat[tid][0];
    out[tid * kPart + kD + 1] = stat[tid][1];
  }
}

// out[b][kv G + g][:] = sum_c e^(m_c - M) part_c / sum_c e^(m_c - M) l_c,  M = max_c m_c.
// Up to NC chunks: thread dd loads its value and every chunk's m and l at once (independent loads,
// one wait on memory), then reduces in registers.
template <int G, int NC>
__global__ __launch_bounds__(kD) void k_kv4_merge_regs(const float* __restrict__ part, int Hq, int Hkv, int nchunks,
                                                       uint16_t* __restrict__ y) {
  const int dd = threadIdx.x;
  const int kv = blockIdx.x / G, g = blockIdx.x % G;
  const int64_t b = blockIdx.y;
  const float* base = part + (((int64_t)b * Hkv + kv) * nchunks) * G * kPart + g * kPart;
  const int64_t cstride = (int64_t)G * kPart;
  float pv[NC], mv[NC], lv[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const bool ok = c < nchunks;   // chunks past the count: weight 0
    const float* r = base + (ok ? c : 0) * cstride;
    pv[c] = r[dd];
    mv[c] = ok ? r[kD] : -INFINITY;
    lv[c] = r[kD + 1];
  }
  float M = mv[0];
#pragma unroll
  for (int c = 1; c < NC; ++c) M = fmaxf(M, mv[c]);
  float acc = 0.f, L = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const float e = c < nchunks ? expf(mv[c] - M) : 0.f;
    acc = fmaf(pv[c], e, acc);
    L = fmaf(lv[c], e, L);
  }
  y[(b * Hq + (int64_t)kv * G + g) * kD + dd] = __half_as_ushort(__float2half_rn(acc / L));
}

// More chunks: workgroup (kv G + g, b) of S x 128 threads (S = blockDim.x / 128 <= kMergeSlices).
// Slice j takes batches of kMergeBatch chunks (chunks j kMergeBatch + i, then S kMergeBatch further
// on, ...), each batch's values and statistics loaded at once (one wait on memory per batch) and
// folded into the slice's running maximum and sums; the slices' results are rescaled to the common
// maximum through LDS.
constexpr int kMergeSlices = 8;
constexpr int kMergeBatch = 16;
template <int G>
__global__ __launch_bounds__(kMergeSlices * kD) void k_kv4_merge(const float* __restrict__ part, int Hq, int Hkv,
                                                                 int nchunks, uint16_t* __restrict__ y) {
  __shared__ float sacc[kMergeSlices][kD];
  __shared__ float sm[kMergeSlices], sl[kMergeSlices];
  const int S = blockDim.x / kD;
  const int tid = threadIdx.x, dd = tid % kD, slice = tid / kD;
  const int kv = blockIdx.x / G, g = blockIdx.x % G;
  const int64_t b = blockIdx.y;
  const float* base = part + (((int64_t)b * Hkv + kv) * nchunks) * G * kPart + g * kPart;
  const int64_t cstride = (int64_t)G * kPart;
  float m = -INFINITY, acc = 0.f, L = 0.f;
  for (int c0 = slice * kMergeBatch; c0 < nchunks; c0 += S * kMergeBatch) {
    float pv[kMergeBatch], mv[kMergeBatch], lv[kMergeBatch];
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const bool ok = c0 + i < nchunks;      // chunks past the count: weight 0
      const float* r = base + (ok ? c0 + i : c0) * cstride;
      pv[i] = r[dd];
      mv[i] = ok ? r[kD] : -INFINITY;
      lv[i] = r[kD + 1];
    }
    float mb = mv[0];                        // chunk c0 exists: mb and the new maximum are finite
#pragma unroll
    for (int i = 1; i < kMergeBatch; ++i) mb = fmaxf(mb, mv[i]);
    const float mn = fmaxf(m, mb);
    const float sc = expf(m - mn);           // 0 for the first batch (m = -inf)
    acc *= sc;
    L *= sc;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const float e = c0 + i < nchunks ? expf(mv[i] - mn) : 0.f;
      acc = fmaf(pv[i], e, acc);
      L = fmaf(lv[i], e, L);
    }
    m = mn;
  }
  sacc[slice][dd] = acc;
  if (dd == 0) {
    sm[slice] = m;
    sl[slice] = L;
  }
  __syncthreads();
  if (tid < kD) {
    float M = sm[0];
    for (int j = 1; j < S; ++j) M = fmaxf(M, sm[j]);
    float a = 0.f, l = 0.f;
    for (int j = 0; j < S; ++j) {
      const float e = expf(sm[j] - M);       // 0 for a slice without chunks (sm = -inf, M finite)
      a = fmaf(sacc[j][tid], e, a);
      l = fmaf(sl[j], e, l);
    }
    y[(b * Hq + (int64_t)kv * G + g) * kD + tid] = __half_as_ushort(__float2half_rn(a / l));
  }
}

template <int G>
hipError_t launch_attn_g(const uint16_t* q, int64_t B, int Hq, int Hkv, int64_t T, const uint8_t* kc,
                         const float* ks, const uint8_t* kz, const uint8_t* vc, const float* vs,
                         const uint8_t* vz, uint16_t* y, float* part, int head_major, hipStream_t s) {
  const int nchunks = (int)((T + kChunk - 1) / kChunk);
  hipLaunchKernelGGL((k_kv4_attn<G>), dim3((unsigned)nchunks, (unsigned)Hkv, (unsigned)B), dim3(256), 0, s, q, Hq,
                     Hkv, T, kc, ks, kz, vc, vs, vz, part, nchunks, head_major);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 mgrid((unsigned)(Hkv * G), (unsigned)B);
  if (nchunks <= 8) {
    hipLaunchKernelGGL((k_kv4_merge_regs<G, 8>), mgrid, dim3(kD), 0, s, part, Hq, Hkv, nchunks, y);
  } else if (nchunks <= 16) {
    hipLaunchKernelGGL((k_kv4_merge_regs<G, 16>), mgrid, dim3(kD), 0, s, part, Hq, Hkv, nchunks, y);
  } else if (nchunks <= 32) {
    hipLaunchKernelGGL((k_kv4_merge_regs<G, 32>), mgrid, dim3(kD), 0, s, part, Hq, Hkv, nchunks, y);
  } else {
    // slices of kMergeBatch chunks, at most kMergeSlices
    const int want = (nchunks + kMergeBatch - 1) / kMergeBatch;
    const int slices = want > kMergeSlices ? kMergeSlices : want;
    hipLaunchKernelGGL((k_kv4_merge<G>), dim3((unsigned)(Hkv * G), (unsigned)B), dim3(slices * kD), 0, s, part, Hq,
                       Hkv, nchunks, y);
  }
  return hipGetLastError();
}

}  // namespace

size_t kv4_attention_workspace(int64_t B, int64_t Hq, int64_t T) {
  const int64_t nchunks = (T + kChunk - 1) / kChunk;
  return (size_t)(B * Hq * nchunks * kPart) * sizeof(float);
}

hipError_t launch_kv4_quant(const uint16_t* x, int64_t groups, uint8_t* codes, float* scales, uint8_t* zeros,
                            hipStream_t s) {
  // 16 groups per workgroup step; a grid-stride loop beyond 8 workgroups per CU
  const int64_t wgs = (groups + 15) / 16;
  hipLaunchKernelGGL(k_kv4_quant, dim3((unsigned)(wgs < 2048 ? wgs : 2048)), dim3(256), 0, s, x, groups, codes, scales,
                     zeros);
  return hipGetLastError();
}

hipError_t launch_kv4_attention(const uint16_t* q, int64_t B, int Hq, int Hkv, int64_t T, int head_major,
                                const uint8_t* kc, const float* ks, const uint8_t* kz, const uint8_t* vc,
                                const float* vs, const uint8_t* vz, uint16_t* y, void* ws, hipStream_t s) {
  float* part = static_cast<float*>(ws);
  switch (Hq / Hkv) {
    case 1: return launch_attn_g<1>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, head_major, s);
    case 2: return launch_attn_g<2>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, head_major, s);
    case 4: return launch_attn_g<4>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, head_major, s);
    case 8: return launch_attn_g<8>(q, B, Hq, Hkv, T, kc, ks, kz, vc, vs, vz, y, part, head_major, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qift
