// Fused online rotation + INT4 quantization + quantized linear for decode
// (M <= 4 tokens): y = s_w[n] s_x[m] sum_k level[n,k] q[m,k] with q, s_x
// computed in the kernel from the fp16 tokens (Sec. 3.1 for the rotation and
// the per-token quantizer, Sec. 3.6 for the integer dot product).
//
// The workgroup owns T consecutive 16-row tiles.  Waves 0-3 (activation
// waves) load the tokens, rotate them exactly in fp64 registers
// (qift_fwht.h), find the absmax, quantize and write the int8 codes to LDS;
// they synchronize only among themselves (an LDS counter), so their
// arithmetic never waits for the other waves, and they issue no weight loads
// (a wave that issues loads into a full memory pipeline stalls until they are
// accepted).  The NS weight waves that follow cut K into NS slices, one per
// wave, of every tile: 8 for tokens of one rotation tile (12 waves, 3 per
// SIMD), else 4 (the activation waves of longer tokens need the registers of
// 2 waves per SIMD).  They issue their weight loads at once (for long tokens
// just after the token loads have gone out, so x is not queued behind the
// weight stream) and wait at one barrier for the codes, so the weight stream
// overlaps the whole activation phase.  After the barrier they run the MFMAs
// of their slices; with NS = 8 two per SIMD, so one wave's decode arithmetic
// overlaps the other's MFMAs.
// The MFMAs read the codes from LDS once per 64-k group and reuse them across
// the T tiles; consecutive MFMAs go to independent accumulators, so they
// pipeline instead of waiting on each other.  MNZ weights are decoded by bit
// plane (one AND per packed word and plane, qift_mma.h), with the codes stored
// in the matching planar order in LDS and one accumulator per plane.
// The K-slices of each tile meet in LDS and wave j < T stores tile j
// (4 consecutive outputs per lane, epilogue in qift_mma.h); the storing lanes
// load their four s_w values at kernel start.
//
// The block exponent L of the rotation is a template parameter (LC) for the
// block sizes in common use, which makes the transform straight-line code;
// LC = 0 covers any other block size with L read at run time.
//
// Included once per weight format (qift_fused_<fmt>.hip), so the instances
// of the three formats compile in parallel.
#pragma once

#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"

namespace qift {
namespace {

using namespace mma;

constexpr int kXchBytes = dev::Tile<256, 16>::LDS_DOUBLES * 8;   // one exchange buffer

template <int NTILES>
constexpr int xch_count() { return NTILES > 1 ? 2 : 1; }

// Weight waves, one per K-slice: 8 for tokens of one rotation tile (whose activation waves fit in
// the registers of 3 waves per SIMD) and whenever the codes come precomputed, else 4.
template <int NTILES, bool CODES>
constexpr int k_slices() { return CODES || NTILES == 1 ? 8 : 4; }

template <int NTILES, bool CODES>
constexpr int fused_threads() { return 64 * (4 + k_slices<NTILES, CODES>()); }

// 256-k units per wave and tile loaded in one batch: every unit of a slice (2 or 4 per rotation
// tile with 8 or 4 slices), except W4 at K > 8192 with the rotation in the kernel (8 units per
// batch: its units take twice the registers).
template <int FMT, int NTILES, bool CODES>
constexpr int units_per_batch() {
  return NTILES == 1 ? 2 : CODES ? 2 * NTILES : FMT == mma::FMT_W4 && NTILES > 2 ? 8 : 4 * NTILES;
}

// The exchange buffers of the rotation, reused after the MFMAs for the K-slice partial sums of T
// tiles (with precomputed codes only the latter).
template <int NTILES, int T, bool CODES>
constexpr int xch_region() {
  return (CODES ? 0 : xch_count<NTILES>() * kXchBytes) > k_slices<NTILES, CODES>() * T * 1024
             ? xch_count<NTILES>() * kXchBytes
             : k_slices<NTILES, CODES>() * T * 1024;
}

// LDS bytes after the codes: exchange region, then s_scale[16] f32, red_d[16] f64, red_i[16] i32, 2 counters,
// and 64 zero bytes (the activation operand of k-groups past K).
template <int NTILES, int T, bool CODES>
constexpr int tail_bytes() { return xch_region<NTILES, T, CODES>() + 64 + 128 + 64 + 16 + 64; }

// CODES = false: the tokens x are rotated and quantized in the kernel (M <= 4; the codes, scales and
// sums may be written to act_q_out / scale_out / sum_out).  CODES = true: the linear on precomputed
// codes aq_in [M][K] and scales sx_in [M] (M <= 16), staged into LDS by waves 0-3, which also add up
// each token's codes unless the sums come in sum_in [M] (nullable).
template <int FMT, int NTILES, int T, int LC, bool CODES>
__global__ __launch_bounds__((fused_threads<NTILES, CODES>())) void k_fused_decode(
    const uint32_t* __restrict__ P, const uint16_t* __restrict__ sw, int N, int K,
    const uint16_t* __restrict__ x, int L, int num, int den, double denom, int xbf16,
    int8_t* __restrict__ act_q_out, float* __restrict__ scale_out, int32_t* __restrict__ sum_out,
    const int8_t* __restrict__ aq_in, const float* __restrict__ sx_in, const int32_t* __restrict__ sum_in,
    int M, int Kpad, uint16_t* __restrict__ y, int32_t* __restrict__ acc_out, int wait_limit,
    uint32_t* __restrict__ err) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr bool PLANAR = FMT == FMT_MNZ;                   // plane decode, codes in planar layout
  // accumulators per tile (MNZ: one per bit plane, planes 0 and 3 sharing one from 4 tiles on, where
  // registers are scarce and the MFMA chains are long enough)
  constexpr int NA = PLANAR ? (T >= 4 ? 3 : 4) : T >= 3 ? 1 : 4 / T;
  constexpr int NS = k_slices<NTILES, CODES>();
  constexpr int UPT = units_per_batch<FMT, NTILES, CODES>();
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: role branches stay scalar
  const int r16 = lane & 15, g = lane >> 4;

  const int act_bytes = (M * Kpad + 15) & ~15;
  int8_t* act_l = reinterpret_cast<int8_t*>(smem);
  double* xch0 = reinterpret_cast<double*>(smem + act_bytes);
  double* xch1 = xch0 + (xch_count<NTILES>() - 1) * (kXchBytes / 8);
  unsigned char* tl = smem + act_bytes + xch_region<NTILES, T, CODES>();
  float* s_scale = reinterpret_cast<float*>(tl);
  double* red_d = reinterpret_cast<double*>(tl + 64);
  int* red_i = reinterpret_cast<int*>(tl + 64 + 128);
  unsigned* ctr = reinterpret_cast<unsigned*>(tl + 64 + 128 + 64);
  int8_t* zero64 = reinterpret_cast<int8_t*>(tl + 64 + 128 + 64 + 16);

  unsigned* xflag = ctr + 1;   // activation waves whose token loads have gone out
  if (tid == 0) {
    ctr[0] = 0u;
    xflag[0] = 0u;
  }
  if (tid < 4) reinterpret_cast<uint4*>(zero64)[tid] = make_uint4(0u, 0u, 0u, 0u);
  if (CODES && tid < 16) red_i[tid] = 0;   // sums of q accumulated while the codes are staged
  __syncthreads();   // nothing is in flight yet: this costs only the launch skew of the waves

  const int tile0 = blockIdx.x * T;
  const int64_t rowbytes = FMT == FMT_W4 ? (int64_t)K / 2 : (int64_t)K / 4;
  const int NC = (K + NS * 256 - 1) / (NS * 256);   // 256-k units per K-slice
  const int slice = wave - 4;                        // K-slice of this wave (negative: none)
  const int kq0 = slice * NC * 256;                  // first k of the slice
  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(P, (uint32_t)(N * rowbytes));
  uint32_t rowoff[T];
  bool rowok[T];
#pragma unroll
  for (int j = 0; j < T; ++j) {
    const int n = (tile0 + j) * 16 + r16;
    rowok[j] = n < N;
    rowoff[j] = (uint32_t)(n * rowbytes);
  }
  uint4 w[T][UPT][NH];
  auto load_batch = [&](int b) {   // in the order the MFMAs consume them (unit-major)
#pragma unroll
    for (int u = 0; u < UPT; ++u)
#pragma unroll
      for (int j = 0; j < T; ++j) {
        const int uu = b * UPT + u;
        const int k0 = kq0 + (uu << 8) + (g << 6);
        const bool ok = rowok[j] && uu < NC && k0 < K;
        const uint32_t off = ok ? rowoff[j] + (uint32_t)(FMT == FMT_W4 ? k0 / 2 : k0 / 4) : dev::kOutOfRange;
#pragma unroll
        for (int h = 0; h < NH; ++h) w[j][u][h] = dev::bload16(wrs, off + 16 * h);
      }
  };
  // s_w of the 4 outputs this lane stores (wave j stores tile j)
  const int n_st = (tile0 + wave) * 16 + 4 * g;
  const __amdgpu_buffer_rsrc_t srs = dev::make_rsrc(sw, (uint32_t)(N * 2));
  uint2 swq = make_uint2(0u, 0u);

  if (wave < 4 && CODES) {
    // ---- staging waves: the precomputed codes of the M tokens into LDS (planar order for MNZ),
    // their scales and sums
    const int per_row = K >> 4;   // 16-byte pieces per token (K is a multiple of 64)
    const int npieces = M * per_row;
    const __amdgpu_buffer_rsrc_t ars = dev::make_rsrc(aq_in, (uint32_t)(M * K));
    for (int i0 = 0; i0 < npieces; i0 += 256 * 8) {
      uint4 c[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int i = i0 + tid + 256 * q;
        c[q] = dev::bload16(ars, i < npieces ? (uint32_t)(16 * i) : dev::kOutOfRange);
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int i = i0 + tid + 256 * q;
        if (!sum_in) {
          // sum_k q of each token: the piece sums go to red_i[m] by LDS atomics, one per wave when
          // all 64 pieces of the wave belong to one token (the common case: K >= 1024)
          const bool ok = i < npieces;
          const int m = ok ? i / per_row : -1;
          const int s = ok ? sum16_i8(c[q], 0) : 0;
          const int m0 = __builtin_amdgcn_readfirstlane(m);
          if (__all(m == m0)) {
            const int ws = dev::wave_sum(s);
            if (lane == 0 && m0 >= 0) atomicAdd(&red_i[m0], ws);
          } else if (ok) {
            atomicAdd(&red_i[m], s);
          }
        }
        if (i < npieces) {
          const int m = i / per_row, j = i - m * per_row;
          if constexpr (PLANAR) {
            // word a of natural piece j (k = 16j + 4a + b) goes to 16a + 4 (j mod 4) + b of its 64-k chunk
            uint32_t* d = reinterpret_cast<uint32_t*>(act_l + m * Kpad + 64 * (j >> 2) + 4 * (j & 3));
            d[0] = c[q].x;
            d[4] = c[q].y;
            d[8] = c[q].z;
            d[12] = c[q].w;
          } else {
            *reinterpret_cast<uint4*>(act_l + m * Kpad + 16 * j) = c[q];
          }
        }
      }
    }
    if (tid < M) {
      s_scale[tid] = sx_in[tid];
      if (sum_in) red_i[tid] = sum_in[tid];
    }
    swq = dev::bload8(srs, wave < T && n_st < N ? (uint32_t)(2 * n_st) : dev::kOutOfRange);
  } else if (wave < 4) {
    // ---- activation waves: rotate and quantize every token into LDS
    dev::GroupSync<4> sync{ctr, 0u, wait_limit, err};
    dev::TokenRaw<NTILES> raw;
    dev::load_token_raw<256, NTILES>(raw, x, K);
    swq = dev::bload8(srs, wave < T && n_st < N ? (uint32_t)(2 * n_st) : dev::kOutOfRange);
    if constexpr (NTILES > 1 && !CODES) {
      // long tokens: the weight waves wait for this before issuing, so the token's loads reach the
      // memory pipeline ahead of the weight stream (which has time to spare until the codes are in)
      asm volatile("" ::: "memory");
      if (lane == 0) __hip_atomic_fetch_add(xflag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    for (int m = 0; m < M; ++m) {
      dev::TokenRaw<NTILES> cur = raw;
      if constexpr (NTILES <= 2) {
        if (m + 1 < M) dev::load_token_raw<256, NTILES>(raw, x + (int64_t)(m + 1) * K, K);   // next token in flight
      } else {
        if (m > 0) dev::load_token_raw<256, NTILES>(cur, x + (int64_t)m * K, K);
      }
      const double A = dev::quant_token_group<NTILES, LC, PLANAR>(cur, K, L, num, den, xch0, xch1, red_d + 4 * m,
                                                          red_i + 4 * m, sync, act_l + m * Kpad, xbf16 != 0);
      if (tid == 0) s_scale[m] = (float)((A * (double)num) / denom);
    }
  } else {
    // ---- weight waves: the first batch of weights (zeros for rows past N and k past K)
    if constexpr (NTILES > 1 && !CODES) {
      for (int spin = 0; spin < (1 << 20); ++spin)   // bounded: a lost flag costs time, never a hang
        if (__builtin_amdgcn_readfirstlane(__hip_atomic_load(xflag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) >= 4u)
          break;
      asm volatile("" ::: "memory");
    }
    swq = dev::bload8(srs, wave < T && n_st < N ? (uint32_t)(2 * n_st) : dev::kOutOfRange);
    load_batch(0);
  }
  dev::lds_barrier();   // codes, scales and partial sums are in LDS; weight loads stay in flight

  v4i acc[T][NA];
#pragma unroll
  for (int j = 0; j < T; ++j)
#pragma unroll
    for (int a = 0; a < NA; ++a) acc[j][a] = v4i{0, 0, 0, 0};
  if (slice >= 0) {
    const int m = r16;
    const bool mok = m < M;
    // lanes of absent tokens read row 0: their MFMA output columns are never stored
    const int8_t* arow = act_l + (mok ? m : 0) * Kpad;
    // activation operands of unit uu (k-groups past K take zero codes: a zero PoT word decodes to -4)
    auto load_b = [&](int uu, v4i (&bq)[4]) {
      const int k0 = kq0 + (uu << 8) + (g << 6);
      const int8_t* bp = uu < NC && k0 < K ? arow + k0 : zero64;
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) {
        const uint4 bb = *reinterpret_cast<const uint4*>(bp + 16 * s2);
        bq[s2] = v4i{(int)bb.x, (int)bb.y, (int)bb.z, (int)bb.w};
      }
    };
    auto unit_mfmas = [&](int u, const v4i (&cur)[4]) {
      if constexpr (PLANAR && T <= 3) {
        // every operand of the unit decoded before its MFMAs (distinct registers, so the decode of
        // the next operand never waits for an MFMA still reading the previous one): measured 12 %
        // fewer cycles per MFMA than decoding each operand just before its MFMA
        v4i A[4][T];
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
          for (int j = 0; j < T; ++j) A[s2][j] = decode_plane(w[j][u][0], s2);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
          for (int j = 0; j < T; ++j) acc[j][s2] = mfma_i8(A[s2][j], cur[s2], acc[j][s2]);
        __builtin_amdgcn_sched_barrier(0);
      } else {
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
          for (int j = 0; j < T; ++j) {
            // MNZ: operand s2 is bit-plane s2 of the unit's four words; else word s2
            if constexpr (PLANAR) {
              const int a = NA == 3 && s2 == 3 ? 0 : s2;
              acc[j][a] = mfma_i8(decode_plane(w[j][u][0], s2), cur[s2], acc[j][a]);
            }
            else acc[j][s2 % NA] = mfma_i8(decode_unit<FMT>(w[j][u], s2), cur[s2], acc[j][s2 % NA]);
          }
      }
    };
    if constexpr (NTILES == 1) {
      // one batch; every operand of the slice is read up front, and units past the slice or past
      // K run on zero weights and zero codes instead of branching (no block boundary between them)
      v4i bq[UPT][4];
#pragma unroll
      for (int u = 0; u < UPT; ++u) load_b(u, bq[u]);
#pragma unroll
      for (int u = 0; u < UPT; ++u) unit_mfmas(u, bq[u]);
    } else if constexpr (UPT * NS == 16 * NTILES) {
      // one batch of every unit a slice can have; units past the slice or past K run on zeros
      v4i bq[2][4];   // double buffer: the next unit's operands are read during this unit's MFMAs
      load_b(0, bq[0]);
#pragma unroll
      for (int u = 0; u < UPT; ++u) {
        if (u + 1 < UPT) load_b(u + 1, bq[(u + 1) & 1]);
        unit_mfmas(u, bq[u & 1]);
      }
    } else {
      for (int b = 0; b * UPT < NC; ++b) {
        if (b > 0) load_batch(b);
        v4i bq[2][4];   // double buffer: the next unit's operands are read during this unit's MFMAs
        load_b(b * UPT, bq[0]);
#pragma unroll
        for (int u = 0; u < UPT; ++u) {
          const int uu = b * UPT + u;
          if (uu >= NC || kq0 + (uu << 8) >= K) break;     // wave-uniform
          if (u + 1 < UPT) load_b(uu + 1, bq[(u + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);   // the next unit's reads go out before these MFMAs
          unit_mfmas(u, bq[u & 1]);
        }
      }
    }
  }
  if (!CODES && wave < 4 && blockIdx.x == 0 && act_q_out) {
    // the codes of the first workgroup double as the stand-alone quantizer's outputs
    const int per_row = K >> 4;
    for (int i = tid; i < M * per_row; i += 256) {
      const int m = i / per_row, j = i - m * per_row;
      uint4 c;
      if constexpr (PLANAR) {
        // bytes 4t..4t+3 of natural chunk j sit at 16t + 4 (j mod 4) of its 64-k chunk
        const int8_t* src = act_l + m * Kpad + 64 * (j >> 2) + 4 * (j & 3);
        c = make_uint4(*reinterpret_cast<const uint32_t*>(src), *reinterpret_cast<const uint32_t*>(src + 16),
                       *reinterpret_cast<const uint32_t*>(src + 32), *reinterpret_cast<const uint32_t*>(src + 48));
      } else {
        c = *reinterpret_cast<const uint4*>(act_l + m * Kpad + 16 * j);
      }
      *reinterpret_cast<uint4*>(act_q_out + (int64_t)m * K + 16 * j) = c;
    }
    if (tid < M) {
      scale_out[tid] = s_scale[tid];
      sum_out[tid] = red_i[4 * tid] + red_i[4 * tid + 1] + red_i[4 * tid + 2] + red_i[4 * tid + 3];
    }
  }

  // the K-slices of each tile meet in LDS (the exchange region is free again)
  v4i* red = reinterpret_cast<v4i*>(xch0);
  if (slice >= 0) {
#pragma unroll
    for (int j = 0; j < T; ++j) {
      v4i s;
      if constexpr (PLANAR) {
        if constexpr (NA == 3) s = combine_planes(acc[j][0], acc[j][1], acc[j][2]);
        else s = combine_planes(acc[j][0], acc[j][1], acc[j][2], acc[j][NA - 1]);
      } else {
        s = acc[j][0];
#pragma unroll
        for (int a = 1; a < NA; ++a) s += acc[j][a];
      }
      red[(j * NS + slice) * 64 + lane] = s;
    }
  }
  __syncthreads();
  if (wave < T) {
    const int j = wave;
    v4i D = red[(j * NS) * 64 + lane];
#pragma unroll
    for (int q = 1; q < NS; ++q) D += red[(j * NS + q) * 64 + lane];
    const int m = r16;
    if (m < M && n_st < N) {
      const int sq = CODES ? red_i[m] : red_i[4 * m] + red_i[4 * m + 1] + red_i[4 * m + 2] + red_i[4 * m + 3];
      store4_sw<FMT>(D, m, n_st, N, s_scale[m], sq, swq, y, acc_out);
    }
  }
}

inline int kpad_of(int64_t K) { return (int)K + 16; }

struct FusedArgs {
  const uint32_t* P;
  const uint16_t* sw;
  int64_t N, K;
  const uint16_t* x;              // rotation in the kernel: fp16 (or, with bf16, bf16) tokens [M][K]
  int L, num, den;
  double denom;
  int8_t* aq_out;                 // optional outputs of the rotation
  float* sc_out;
  int32_t* sm_out;
  const int8_t* aq_in;            // precomputed codes [M][K], scales [M], sums [M]
  const float* sx_in;
  const int32_t* sum_in;
  int64_t M;
  uint16_t* y;
  int32_t* acc_out;
  bool bf16 = false;              // x holds bf16 values
};

// Tiles per workgroup: for K <= 4096 (one rotation tile) as many as keep the grid within one
// workgroup per CU (at most 7; W4, whose units take twice the registers, at most 3); longer K one.
template <int FMT>
inline int64_t fused_tiles(int64_t N, int64_t K) {
  if (K > 4096) return 1;
  const int64_t t = ((N + 15) / 16 + 255) / 256;
  const int64_t cap = FMT == FMT_W4 ? 3 : 7;
  return t < 1 ? 1 : t > cap ? cap : t;
}

template <int NTILES, int T, bool CODES>
inline size_t fused_shmem(int64_t M, int64_t K) {
  return (size_t)((((int)M * kpad_of(K)) + 15) & ~15) + tail_bytes<NTILES, T, CODES>();
}

template <int FMT, int NTILES, int T, int LC, bool CODES>
hipError_t launch_t(const FusedArgs& a, hipStream_t s) {
  const int ntiles = (int)((a.N + 15) / 16);
  const int grid = (ntiles + T - 1) / T;
  const size_t shmem = fused_shmem<NTILES, T, CODES>(a.M, a.K);
  if (shmem > 160 * 1024) return hipErrorInvalidValue;
  if (shmem > 65536) {
    // opt in to more than 64 KiB of dynamic LDS (gfx950 has 160 KiB per workgroup)
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&k_fused_decode<FMT, NTILES, T, LC, CODES>),
        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
  }
  hipLaunchKernelGGL((k_fused_decode<FMT, NTILES, T, LC, CODES>), dim3(grid), dim3(fused_threads<NTILES, CODES>()),
                     shmem, s, a.P, a.sw, (int)a.N, (int)a.K, a.x, a.L, a.num, a.den, a.denom, a.bf16 ? 1 : 0,
                     a.aq_out, a.sc_out,
                     a.sm_out, a.aq_in, a.sx_in, a.sum_in, (int)a.M, kpad_of(a.K), a.y, a.acc_out, wait_limit(),
                     device_error_word());
  return hipGetLastError();
}

// Block exponents compiled as constants: 12 and 8 for tokens of one rotation
// tile (K <= 4096), 12, 11 and 6 for longer tokens; anything else at run time.
// Precomputed codes need no rotation: one instance.
template <int FMT, int NTILES, int T, bool CODES>
hipError_t launch_l(const FusedArgs& a, hipStream_t s) {
  if constexpr (CODES) {
    return launch_t<FMT, NTILES, T, 0, true>(a, s);
  } else {
    if constexpr (NTILES == 1) {
      if (a.L == 12) return launch_t<FMT, NTILES, T, 12, false>(a, s);
      if (a.L == 8) return launch_t<FMT, NTILES, T, 8, false>(a, s);
    } else {
      if (a.L == 12) return launch_t<FMT, NTILES, T, 12, false>(a, s);
      if (a.L == 11) return launch_t<FMT, NTILES, T, 11, false>(a, s);
      if (a.L == 6) return launch_t<FMT, NTILES, T, 6, false>(a, s);
    }
    return launch_t<FMT, NTILES, T, 0, false>(a, s);
  }
}

template <int FMT, int NTILES, bool CODES>
hipError_t launch_nt(const FusedArgs& a, hipStream_t s) {
  if constexpr (NTILES == 1) {
    switch (fused_tiles<FMT>(a.N, a.K)) {
      case 1: return launch_l<FMT, NTILES, 1, CODES>(a, s);
      case 2: return launch_l<FMT, NTILES, 2, CODES>(a, s);
      case 3: return launch_l<FMT, NTILES, 3, CODES>(a, s);
      default: break;
    }
    if constexpr (FMT != FMT_W4) {
      switch (fused_tiles<FMT>(a.N, a.K)) {
        case 4: return launch_l<FMT, NTILES, 4, CODES>(a, s);
        case 5: return launch_l<FMT, NTILES, 5, CODES>(a, s);
        case 6: return launch_l<FMT, NTILES, 6, CODES>(a, s);
        default: return launch_l<FMT, NTILES, 7, CODES>(a, s);
      }
    }
    return hipErrorInvalidValue;
  } else {
    return launch_l<FMT, NTILES, 1, CODES>(a, s);
  }
}

template <int FMT, bool CODES>
hipError_t launch_ntiles(const FusedArgs& a, hipStream_t s) {
  switch ((a.K + 4095) / 4096) {
    case 1: return launch_nt<FMT, 1, CODES>(a, s);
    case 2: return launch_nt<FMT, 2, CODES>(a, s);
    case 3: return launch_nt<FMT, 3, CODES>(a, s);
    case 4: return launch_nt<FMT, 4, CODES>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int FMT>
hipError_t launch_fused_fmt(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const uint16_t* x,
                            int block, int num, int den, int64_t M, uint16_t* y, int32_t* acc_out, int8_t* aq,
                            float* sc, int32_t* sm, bool bf16, hipStream_t s) {
  if (M < 1 || M > kFusedMaxM || K > kFusedMaxK || block > kFusedMaxBlock) return hipErrorInvalidValue;
  FusedArgs a{P, sw, N, K, x, dev::ilog2c(block), num, den, act_denominator(block, den), aq, sc, sm,
              nullptr, nullptr, nullptr, M, y, acc_out, bf16};
  return launch_ntiles<FMT, false>(a, s);
}

// LDS bytes of the linear on precomputed codes (0 when the shape is outside its limits).
template <int FMT>
size_t codes_shmem_fmt(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || M > kCodesMaxM || K > kFusedMaxK || N < 1) return 0;
  const int64_t T = fused_tiles<FMT>(N, K);
  switch ((K + 4095) / 4096) {
    case 1:
      switch (T) {
        case 1: return fused_shmem<1, 1, true>(M, K);
        case 2: return fused_shmem<1, 2, true>(M, K);
        case 3: return fused_shmem<1, 3, true>(M, K);
        case 4: return fused_shmem<1, 4, true>(M, K);
        case 5: return fused_shmem<1, 5, true>(M, K);
        case 6: return fused_shmem<1, 6, true>(M, K);
        default: return fused_shmem<1, 7, true>(M, K);
      }
    case 2: return fused_shmem<2, 1, true>(M, K);
    case 3: return fused_shmem<3, 1, true>(M, K);
    case 4: return fused_shmem<4, 1, true>(M, K);
    default: return 0;
  }
}

template <int FMT>
hipError_t launch_codes_fmt(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* aq,
                            const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                            hipStream_t s) {
  const size_t shmem = codes_shmem_fmt<FMT>(M, N, K);
  if (shmem == 0 || shmem > 160 * 1024) return hipErrorInvalidValue;
  FusedArgs a{P, sw, N, K, nullptr, 0, 1, 1, 1.0, nullptr, nullptr, nullptr, aq, sx, asum, M, y, acc_out};
  return launch_ntiles<FMT, true>(a, s);
}

}  // namespace
}  // namespace qift
