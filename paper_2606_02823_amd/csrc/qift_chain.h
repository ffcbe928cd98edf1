// Persistent decode step: one co-resident grid walks a chain of quantized linears (a layer stack at
// decode), each taking its input from an earlier linear's output, so that the weight stream of the
// next linear is already in flight while the current one's dependency resolves.  Every linear is
// the fused form of the method (Sec. 3.1 online rotation and per-token INT4 quantizer, Sec. 3.3 /
// Sec. 3.6 integer dot product on the fixed level set, scales in the epilogue, Sec. 1) with results
// bit-identical to qift_rotate_quant_linear on the same input.
//
// Grid: one workgroup per CU, 12 waves each.  Linear ("link") i of the chain is cut into 16-row
// tiles; workgroup g owns tiles [g T / G, (g + 1) T / G) of it.  Per link:
//   * activation waves (0-3; 0-7 for K > 4096, two groups of four sharing the rotation tiles)
//     wait until every workgroup has published the link's input (an arrival counter per link in
//     device memory, polled by wave 0 with agent-coherent loads, then handed on through LDS), load
//     the token(s) with agent-coherent loads, rotate exactly in fp64, quantize and write the codes
//     to LDS (the routines of qift_fwht.h);
//   * weight waves (4-11, K-slices of 512 k; 8-11 for K > 4096, slices of K/4) issued their
//     weight loads at the end of the previous link, so those bytes stream during the wait, the
//     token load and the rotation; after the codes barrier they run the MFMAs (qift_mma.h) and
//     write per-slice partial sums to LDS;
//   * waves 0-3 add the slices, apply the epilogue and store y with agent-coherent (sc1) stores,
//     wait for the stores to complete and bump the link's arrival counter.
// Cross-XCD visibility: y is stored with sc1 (coherent at device scope) and read back by the
// consumers with sc1 loads, and the counter is incremented only after the stores have completed,
// so no L2 writeback or invalidation of the whole cache is needed.  Every wait is bounded (by
// time); a wait that gives up sets a bit in the device error word and the workgroup carries on, so
// the grid always drains.  The last workgroup to finish resets the counters for the next call.
#pragma once

#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"

namespace qift {

constexpr int kChainWaves = 12;
constexpr int kChainThreads = 64 * kChainWaves;
constexpr int kChainShortK = 4096;   // one rotation tile: 4 activation waves, 8 K-slices
// LDS after the codes and the exchange / partial-sum region (kChainTailBytes): s_scale[4] f32,
// red_d[4][8] f64, red_i[4][8] i32, ctr[4] u32, 64 zero bytes
static_assert(kChainTailBytes == 16 + 256 + 128 + 16 + 64, "tail layout");

template <int FMT>
constexpr int chain_tmax() { return FMT == mma::FMT_W4 ? 3 : 7; }   // tiles per chunk, K <= 4096

namespace chain {

using namespace mma;

constexpr int kXchBytes = dev::Tile<256, 16>::LDS_DOUBLES * 8;   // one rotation exchange buffer
static_assert(kXchBytes == kChainXchBytes, "exchange buffer size");

struct Geom {
  int t0, T, tmax, nchunks;
  bool lng;
};

__device__ __forceinline__ Geom geom(const ChainDesc& d, int wg, int G, int tmax_short) {
  Geom r;
  const int a = (int)((int64_t)wg * d.tiles / G), b = (int)((int64_t)(wg + 1) * d.tiles / G);
  r.t0 = a;
  r.T = b - a;
  r.lng = d.K > kChainShortK;
  r.tmax = r.lng ? 1 : tmax_short;
  r.nchunks = (r.T + r.tmax - 1) / r.tmax;
  return r;
}

// ---------------------------------------------------------------------------------------------
// weight waves

// Loads of one chunk of T tiles into wr (unit-major, the order the MFMAs consume them).  Short
// links: 8 slices of NC <= 2 units of 256 k; long links: 4 slices of NC <= 16 units (W4: batch b
// of 8).  Rows past N and k past K read zeros (out-of-range offsets).
template <int FMT, int T, bool LONG>
__device__ __forceinline__ void load_chunk(uint4 (&wr)[16], const ChainDesc& d, int tile0, int slice, int batch) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr int NS = LONG ? 4 : 8;
  constexpr int UPT = LONG ? (FMT == FMT_W4 ? 8 : 16) : 2;
  static_assert(T * UPT * NH <= 16, "weight registers");
  const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
  const int K = d.K, N = d.N;
  const int64_t rowbytes = FMT == FMT_W4 ? (int64_t)K / 2 : (int64_t)K / 4;
  const int NC = (K + NS * 256 - 1) / (NS * 256);
  const int kq0 = slice * NC * 256;
  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(d.P, (uint32_t)(N * rowbytes));
#pragma unroll
  for (int u = 0; u < UPT; ++u)
#pragma unroll
    for (int j = 0; j < T; ++j) {
      const int n = (tile0 + j) * 16 + r16;
      const int uu = batch * UPT + u;
      const int k0 = kq0 + (uu << 8) + (g << 6);
      const bool ok = n < N && uu < NC && k0 < K;
      const uint32_t off = ok ? (uint32_t)(n * rowbytes) + (uint32_t)(FMT == FMT_W4 ? k0 / 2 : k0 / 4) : dev::kOutOfRange;
#pragma unroll
      for (int h = 0; h < NH; ++h) wr[(u * T + j) * NH + h] = dev::bload16(wrs, off + 16 * h);
    }
}

template <int FMT, bool LONG>
__device__ __forceinline__ void load_chunk_rt(uint4 (&wr)[16], const ChainDesc& d, int tile0, int T, int slice) {
  if constexpr (LONG) {
    load_chunk<FMT, 1, true>(wr, d, tile0, slice, 0);
  } else {
    switch (T) {
      case 1: load_chunk<FMT, 1, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=1"); break;
      case 2: load_chunk<FMT, 2, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=2"); break;
      case 3: load_chunk<FMT, 3, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=3"); break;
      default:
        if constexpr (FMT != FMT_W4) {
          switch (T) {
            case 4: load_chunk<FMT, 4, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=4"); break;
            case 5: load_chunk<FMT, 5, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=5"); break;
            case 6: load_chunk<FMT, 6, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=6"); break;
            default: load_chunk<FMT, 7, false>(wr, d, tile0, slice, 0); asm volatile("; chain load_chunk T=7"); break;
          }
        }
        break;
    }
  }
}

// Bit planes of a lane's four packed MNZ words with two accumulators: planes 0 and 3 as codes (factor
// 1), planes 1 and 2 as codes times 4 (plane 2 shifted down by one field), so that
//   D = acc03 + acc12 / 4,
// exact since acc12 is 4 times an integer sum.  One more shift per word than qift_mma.h's
// decode_plane, half the accumulators: the registers that a workgroup of seven 16-row tiles needs.
__device__ __forceinline__ v4i decode_plane2(const uint4& u, int t) {
  if (t == 0) return v4i{(int)(u.x & 0x03030303u), (int)(u.y & 0x03030303u), (int)(u.z & 0x03030303u), (int)(u.w & 0x03030303u)};
  if (t == 1) return v4i{(int)(u.x & 0x0C0C0C0Cu), (int)(u.y & 0x0C0C0C0Cu), (int)(u.z & 0x0C0C0C0Cu), (int)(u.w & 0x0C0C0C0Cu)};
  if (t == 2)
    return v4i{(int)((u.x >> 2) & 0x0C0C0C0Cu), (int)((u.y >> 2) & 0x0C0C0C0Cu), (int)((u.z >> 2) & 0x0C0C0C0Cu),
               (int)((u.w >> 2) & 0x0C0C0C0Cu)};
  return v4i{(int)((u.x >> 6) & 0x03030303u), (int)((u.y >> 6) & 0x03030303u), (int)((u.z >> 6) & 0x03030303u),
             (int)((u.w >> 6) & 0x03030303u)};
}

// MFMAs of one chunk; the slice's partial sums of tile j go to red[(j * NS + slice) * 64 + lane].
template <int FMT, int T, bool LONG>
__device__ __forceinline__ void mfma_chunk(uint4 (&wr)[16], const ChainDesc& d, int tile0, int slice,
                                           const int8_t* act_l, int Kpad, int M, const int8_t* zero64,
                                           v4i* red) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr int NS = LONG ? 4 : 8;
  constexpr int UPT = LONG ? (FMT == FMT_W4 ? 8 : 16) : 2;
  constexpr bool PLANAR = FMT == FMT_MNZ;
  // accumulators per tile: MNZ one per bit plane up to 3 tiles, from 4 tiles on two (decode_plane2)
  constexpr bool TWO = PLANAR && T >= 4;
  constexpr int NA = PLANAR ? (TWO ? 2 : 4) : T >= 3 ? 1 : 4 / T;
  const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
  const int K = d.K;
  const int NC = (K + NS * 256 - 1) / (NS * 256);
  const int kq0 = slice * NC * 256;
  const int8_t* arow = act_l + (r16 < M ? r16 : 0) * Kpad;   // absent tokens read row 0 (never stored)
  v4i acc[T][NA];
#pragma unroll
  for (int j = 0; j < T; ++j)
#pragma unroll
    for (int a = 0; a < NA; ++a) acc[j][a] = v4i{0, 0, 0, 0};
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
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
      for (int j = 0; j < T; ++j) {
        if constexpr (TWO) {
          const uint4 w4 = wr[(u * T + j) * NH];
          const int a = s2 == 0 || s2 == 3 ? 0 : 1;
          acc[j][a] = mfma_i8(decode_plane2(w4, s2), cur[s2], acc[j][a]);
        } else if constexpr (PLANAR) {
          const uint4 w4 = wr[(u * T + j) * NH];
          acc[j][s2] = mfma_i8(decode_plane(w4, s2), cur[s2], acc[j][s2]);
        } else {
          uint4 uw[NH];
#pragma unroll
          for (int h = 0; h < NH; ++h) uw[h] = wr[(u * T + j) * NH + h];
          acc[j][s2 % NA] = mfma_i8(decode_unit<FMT>(uw, s2), cur[s2], acc[j][s2 % NA]);
        }
      }
  };
  if constexpr (!LONG) {
    // one batch; every operand of the slice read up front, units past the slice or K on zeros
    v4i bq[UPT][4];
#pragma unroll
    for (int u = 0; u < UPT; ++u) load_b(u, bq[u]);
#pragma unroll
    for (int u = 0; u < UPT; ++u) unit_mfmas(u, bq[u]);
  } else {
    constexpr int NB = FMT == FMT_W4 ? 2 : 1;   // batches of UPT units (W4 holds 8 units at a time)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b > 0) {
        if (b * UPT >= NC) break;   // wave-uniform
        load_chunk<FMT, 1, true>(wr, d, tile0, slice, b);
      }
      v4i bq[2][4];   // the next unit's operands are read during this unit's MFMAs
      load_b(b * UPT, bq[0]);
#pragma unroll
      for (int u = 0; u < UPT; ++u) {
        if (u + 1 < UPT) load_b(b * UPT + u + 1, bq[(u + 1) & 1]);
        unit_mfmas(u, bq[u & 1]);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < T; ++j) {
    v4i s;
    if constexpr (TWO) {
#pragma unroll
      for (int r = 0; r < 4; ++r) s[r] = acc[j][0][r] + (acc[j][1][r] >> 2);
    } else if constexpr (PLANAR) {
      s = combine_planes(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
    } else {
      s = acc[j][0];
#pragma unroll
      for (int a = 1; a < NA; ++a) s += acc[j][a];
    }
    red[(j * NS + slice) * 64 + lane] = s;
  }
}

template <int FMT, bool LONG>
__device__ __forceinline__ void mfma_chunk_rt(uint4 (&wr)[16], const ChainDesc& d, int tile0, int T, int slice,
                                              const int8_t* act_l, int Kpad, int M, const int8_t* zero64, v4i* red) {
  if constexpr (LONG) {
    mfma_chunk<FMT, 1, true>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red);
  } else {
    switch (T) {
      case 1: mfma_chunk<FMT, 1, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=1"); break;
      case 2: mfma_chunk<FMT, 2, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=2"); break;
      case 3: mfma_chunk<FMT, 3, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=3"); break;
      default:
        if constexpr (FMT != FMT_W4) {
          switch (T) {
            case 4: mfma_chunk<FMT, 4, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=4"); break;
            case 5: mfma_chunk<FMT, 5, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=5"); break;
            case 6: mfma_chunk<FMT, 6, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=6"); break;
            default: mfma_chunk<FMT, 7, false>(wr, d, tile0, slice, act_l, Kpad, M, zero64, red); asm volatile("; chain mfma_chunk T=7"); break;
          }
        }
        break;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// activation waves

// Raw fp16 bits of tiles [tau0, tau0 + ntg) of one token, 16 consecutive elements per thread of
// the group (t = 0..255), read with agent-coherent loads (the producer may sit on another XCD).
template <int NTG>
__device__ __forceinline__ void load_tiles_sc1(dev::TokenRaw<NTG>& raw, const uint16_t* xr, int K, int tau0, int ntg,
                                               int t) {
  const __amdgpu_buffer_rsrc_t r = dev::make_rsrc(xr, (uint32_t)(K * 2));
#pragma unroll
  for (int tau = 0; tau < NTG; ++tau) {
    const int base = (tau0 + tau) * 4096 + 16 * t;   // elements past K (or past the group's tiles) read zeros
    const uint32_t off = tau < ntg && base < K ? (uint32_t)(base * 2) : dev::kOutOfRange;
    const auto a = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16);
    const auto b = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, 16);
    raw.d[tau][0] = make_uint4(a[0], a[1], a[2], a[3]);
    raw.d[tau][1] = make_uint4(b[0], b[1], b[2], b[3]);
  }
}

// Rotation + quantization of the group's tiles [tau0, tau0 + ntg) of one token (the steps of
// dev::quant_token_group, for a group of four waves that may own only part of the token).  The
// group's waves synchronize through gsync; the absmax of all ngroups groups meets in red_d through
// gall.  Codes go to dst at code_pos<PLANAR>; the group's code sums to red_i[4 gi + w].
template <int NTG, int LC, bool PLANAR, typename GS, typename GA>
__device__ __forceinline__ double quant_tiles(const dev::TokenRaw<NTG>& raw, int ntg, int tau0, int K, int L_rt,
                                              int num, int den, double* xch, double* red_d, int* red_i, int gi,
                                              int ngroups, GS& gsync, GA& gall, int8_t* dst) {
  using S = dev::Tile<256, 16>;
  const int L = LC > 0 ? LC : L_rt;
  const int t = threadIdx.x & 255, lane = t & 63, w = t >> 6;
  double v[NTG][16];
  double amax = 0.0;
  int wend = 0;
#pragma unroll
  for (int tau = 0; tau < NTG; ++tau) {
    if (tau < ntg) {
      dev::unpack16<false>(v[tau], raw.d[tau]);
      if (tau > 0 && L > 6) gsync();   // one exchange buffer per group: the previous tile's reads are done
      wend = dev::fwht_tile_s<256, 16, false>(v[tau], xch, t, L, gsync);
#pragma unroll
      for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[tau][e]));
    }
  }
  amax = dev::wave_max(amax);
  if (lane == 0) red_d[4 * gi + w] = amax;
  gall();
  double A = red_d[0];
  for (int q = 1; q < 4 * ngroups; ++q) A = fmax(A, red_d[q]);
  const dev::QuantParams p = dev::make_qparams(A, num, den);
  int qs = 0;
#pragma unroll
  for (int tau = 0; tau < NTG; ++tau) {
    if (tau < ntg) {
      int q[16];
      dev::quant16(v[tau], p, q);
#pragma unroll
      for (int e = 0; e < 16; ++e) qs += q[e];
      const int tg = tau0 + tau;
      int8_t* tile_dst = dst + tg * S::T;
      if ((tg + 1) * S::T <= K) {
        if (wend == 0) dev::store_codes<0, PLANAR>(tile_dst, q, t);
        else if (wend == 4) dev::store_codes<4, PLANAR>(tile_dst, q, t);
        else dev::store_codes<8, PLANAR>(tile_dst, q, t);
      } else if (wend == 0) {
        if (tg * S::T + 16 * t < K) dev::store_codes<0, PLANAR>(tile_dst, q, t);   // K is a multiple of 64
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int i = wend == 4 ? dev::win_elem<4>(t) + (e << 4) : dev::win_elem<8>(t) + (e << 8);
          if (tg * S::T + i < K) tile_dst[dev::code_pos<PLANAR>(i)] = (int8_t)q[e];
        }
      }
    }
  }
  qs = dev::wave_sum(qs);
  if (lane == 0) red_i[4 * gi + w] = qs;
  return A;
}

// The activation phase of one link for one group: every token of the link.
template <int NTG, int LC, bool PLANAR, typename GS, typename GA>
__device__ __forceinline__ void act_phase(const ChainDesc& d, const uint16_t* xin, int xstride, int M, int ntg, int tau0,
                                          int gi, int ngroups, GS& gsync, GA& gall, double* xch, int8_t* act_l,
                                          int Kpad, double* red_d, int* red_i, float* s_scale) {
  const int t = threadIdx.x & 255;
  for (int m = 0; m < M; ++m) {
    dev::TokenRaw<NTG> cur;
    load_tiles_sc1<NTG>(cur, xin + (int64_t)m * xstride, d.K, tau0, ntg, t);
    const double A = quant_tiles<NTG, LC, PLANAR>(cur, ntg, tau0, d.K, d.L, d.num, d.den, xch, red_d + 8 * m,
                                                  red_i + 8 * m, gi, ngroups, gsync, gall, act_l + m * Kpad);
    if (threadIdx.x == 0) s_scale[m] = (float)((A * (double)d.num) / d.denom);
  }
}

// y[m][n0 .. n0 + 3] (and the accumulators) with agent-coherent stores: the consumers of this link
// may run on other XCDs.
template <int FMT>
__device__ __forceinline__ void store4_sc1(const v4i& D, int m, int n0, int N, float s_x, int sum_q, uint2 swq,
                                           __amdgpu_buffer_rsrc_t yr, int32_t* __restrict__ acc_out) {
  typedef unsigned v2u __attribute__((ext_vector_type(2)));
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
    __builtin_amdgcn_raw_buffer_store_b64(
        v2u{(uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16)}, yr, (int)(2 * o), 0, 16);
    if (acc_out) *reinterpret_cast<int4*>(acc_out + o) = make_int4(a[0], a[1], a[2], a[3]);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (n0 + r < N) {
        __builtin_amdgcn_raw_buffer_store_b16(h[r], yr, (int)(2 * (o + r)), 0, 16);
        if (acc_out) acc_out[o + r] = a[r];
      }
    }
  }
}

}  // namespace chain

// ---------------------------------------------------------------------------------------------
// the kernel
//
// The waves run one of three loops over the links, each taking the same sequence of workgroup
// barriers (per link: codes ready, then per chunk of tiles: partial sums ready, and between chunks:
// partial sums read), so that a wave's registers hold only what its own roles need:
//   waves 0-3   activation group 0, then the K-slice reduction, epilogue, stores and publishing;
//   waves 4-7   activation group 1 on links with K > 4096, else weight slices 0-3 of 8;
//   waves 8-11  weight slices: 0-3 of 4 on links with K > 4096, else 4-7 of 8.
namespace chain {

// Input of link i: wave 0 waits until every workgroup has stored its share of the producing link,
// then releases the other activation waves of the workgroup through LDS (in_ready = i + 1).  Wave 0
// gets here only after the previous link's publishing barrier of waves 0-3, i.e. after their last
// reads of the partial sums, scales and code sums that this link's activation phase overwrites.
__device__ __forceinline__ void wait_input(const ChainDesc& d, int i, int wave, unsigned* counters, unsigned G,
                                           unsigned* in_ready, long long wait_ticks, uint32_t* err) {
  const int lane = threadIdx.x & 63;
  const long long t_start = wall_clock64();
  if (wave == 0) {
    if (d.in_link >= 0) {
      unsigned* c = counters + d.in_link;
      for (;;) {
        const unsigned v = __builtin_amdgcn_readfirstlane(__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        if (v >= G) break;
        if (wall_clock64() - t_start > wait_ticks) {
          if (lane == 0) dev::flag_error(err, dev::kErrChainWait);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (lane == 0) __hip_atomic_store(in_ready, (unsigned)(i + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  } else {
    for (;;) {
      const unsigned v =
          __builtin_amdgcn_readfirstlane(__hip_atomic_load(in_ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
      if (v >= (unsigned)(i + 1)) break;
      if (wall_clock64() - t_start > 2 * wait_ticks) {
        if (lane == 0) dev::flag_error(err, dev::kErrChainWait);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  asm volatile("" ::: "memory");
}

// The activation phase of link i for group gi (0: waves 0-3, 1: waves 4-7, links with K > 4096).
template <bool PLANAR, typename GS>
__device__ __forceinline__ void link_act(const ChainDesc& d, bool lng, int gi, const uint16_t* x0, int M, GS& gsync,
                                         dev::GroupSync<8>& gs8, double* xch, int8_t* act_l, int Kpad, double* red_d,
                                         int* red_i, float* s_scale) {
  const uint16_t* xin = d.in_link < 0 ? x0 : d.x;
  const int xstride = d.in_link < 0 ? d.K : d.xstride;
  // the block sizes compiled in (chain_block_ok): every butterfly stage is straight-line code
  if (!lng) {
    switch (d.L) {
      case 12: act_phase<1, 12, PLANAR>(d, xin, xstride, M, 1, 0, 0, 1, gsync, gsync, xch, act_l, Kpad, red_d, red_i, s_scale); break;
      case 11: act_phase<1, 11, PLANAR>(d, xin, xstride, M, 1, 0, 0, 1, gsync, gsync, xch, act_l, Kpad, red_d, red_i, s_scale); break;
      case 8: act_phase<1, 8, PLANAR>(d, xin, xstride, M, 1, 0, 0, 1, gsync, gsync, xch, act_l, Kpad, red_d, red_i, s_scale); break;
      default: act_phase<1, 6, PLANAR>(d, xin, xstride, M, 1, 0, 0, 1, gsync, gsync, xch, act_l, Kpad, red_d, red_i, s_scale); break;
    }
    return;
  }
  // group 0 takes the first ceil(NT / 2) rotation tiles, group 1 the rest
  const int NT = (d.K + 4095) / 4096, h = (NT + 1) / 2;
  const int tau0 = gi ? h : 0, ntg = gi ? NT - h : h;
  double* xg = xch + gi * (kXchBytes / 8);
  switch (d.L) {
    case 12: act_phase<2, 12, PLANAR>(d, xin, xstride, M, ntg, tau0, gi, 2, gsync, gs8, xg, act_l, Kpad, red_d, red_i, s_scale); break;
    case 11: act_phase<2, 11, PLANAR>(d, xin, xstride, M, ntg, tau0, gi, 2, gsync, gs8, xg, act_l, Kpad, red_d, red_i, s_scale); break;
    case 8: act_phase<2, 8, PLANAR>(d, xin, xstride, M, ntg, tau0, gi, 2, gsync, gs8, xg, act_l, Kpad, red_d, red_i, s_scale); break;
    default: act_phase<2, 6, PLANAR>(d, xin, xstride, M, ntg, tau0, gi, 2, gsync, gs8, xg, act_l, Kpad, red_d, red_i, s_scale); break;
  }
}

}  // namespace chain

template <int FMT>
__global__ __launch_bounds__(kChainThreads) void k_decode_chain(const ChainDesc* __restrict__ links, int n_links,
                                                                const uint16_t* __restrict__ x0, int M, int Kpad,
                                                                int xch_bytes, unsigned* __restrict__ counters,
                                                                int wait_limit, long long wait_ticks,
                                                                uint32_t* __restrict__ err) {
  using namespace chain;
  constexpr bool PLANAR = FMT == FMT_MNZ;
  constexpr int TMAX = chain_tmax<FMT>();
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int G = gridDim.x, wg = blockIdx.x;

  const int act_bytes = (M * Kpad + 15) & ~15;
  int8_t* act_l = reinterpret_cast<int8_t*>(smem);
  double* xch = reinterpret_cast<double*>(smem + act_bytes);
  v4i* red = reinterpret_cast<v4i*>(xch);   // the K-slice partial sums reuse the exchange region
  unsigned char* tl = smem + act_bytes + xch_bytes;
  float* s_scale = reinterpret_cast<float*>(tl);
  double* red_d = reinterpret_cast<double*>(tl + 16);
  int* red_i = reinterpret_cast<int*>(tl + 16 + 256);
  unsigned* ctr = reinterpret_cast<unsigned*>(tl + 16 + 256 + 128);   // group 0, group 1, both, input-ready
  int8_t* zero64 = reinterpret_cast<int8_t*>(tl + 16 + 256 + 128 + 16);
  if (tid < 4) {
    ctr[tid] = 0u;
    reinterpret_cast<uint4*>(zero64)[tid] = make_uint4(0u, 0u, 0u, 0u);
  }
  __syncthreads();
  unsigned* in_ready = ctr + 3;   // 1 + the last link whose input is ready

  if (wave < 4) {
    // ================= waves 0-3: activation group 0, reduction, epilogue, publishing
    dev::GroupSync<4> gs0{ctr + 0, 0u, wait_limit, err};
    dev::GroupSync<8> gs8{ctr + 2, 0u, wait_limit, err};
    for (int i = 0; i < n_links; ++i) {
      const ChainDesc& d = links[i];
      const Geom gm = geom(d, wg, G, TMAX);
      uint2 swq[2] = {make_uint2(0u, 0u), make_uint2(0u, 0u)};
      if (gm.T > 0) {
        wait_input(d, i, wave, counters, (unsigned)G, in_ready, wait_ticks, err);
        link_act<PLANAR>(d, gm.lng, 0, x0, M, gs0, gs8, xch, act_l, Kpad, red_d, red_i, s_scale);
        // fp16 scales of the first chunk's tiles wave and wave + 4, in flight during the MFMAs
        const __amdgpu_buffer_rsrc_t srs = dev::make_rsrc(d.sw, (uint32_t)(d.N * 2));
        const int T0 = gm.T < gm.tmax ? gm.T : gm.tmax;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int j = wave + 4 * r, n = (gm.t0 + j) * 16 + 4 * g;
          swq[r] = dev::bload8(srs, j < T0 && n < d.N ? (uint32_t)(2 * n) : dev::kOutOfRange);
        }
      }
      dev::lds_barrier();   // codes, scales and code sums are in LDS
      const __amdgpu_buffer_rsrc_t yr = dev::make_rsrc(d.y, (uint32_t)(M * d.N * 2));
      const int NS = gm.lng ? 4 : 8, ngr = gm.lng ? 8 : 4;
      for (int c = 0; c < gm.nchunks; ++c) {
        const int tile0 = gm.t0 + c * gm.tmax;
        const int Tc = gm.T - c * gm.tmax < gm.tmax ? gm.T - c * gm.tmax : gm.tmax;
        dev::lds_barrier();   // the slices' partial sums are in LDS
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int j = wave + 4 * r;
          if (j < Tc) {
            v4i D = red[(j * NS) * 64 + lane];
            for (int q = 1; q < NS; ++q) D += red[(j * NS + q) * 64 + lane];
            const int m = r16, n0 = (tile0 + j) * 16 + 4 * g;
            if (c > 0) {
              const __amdgpu_buffer_rsrc_t srs = dev::make_rsrc(d.sw, (uint32_t)(d.N * 2));
              swq[r] = dev::bload8(srs, n0 < d.N ? (uint32_t)(2 * n0) : dev::kOutOfRange);
            }
            if (m < M && n0 < d.N) {
              int sq = 0;
              for (int q = 0; q < ngr; ++q) sq += red_i[8 * m + q];
              store4_sc1<FMT>(D, m, n0, d.N, s_scale[m], sq, swq[r], yr, d.acc);
            }
          }
        }
        if (c + 1 < gm.nchunks) dev::lds_barrier();   // the partial sums have been read
      }
      // publish: this workgroup's share of link i is stored (stores complete, then the counter)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      gs0();
      if (wave == 0 && lane == 0) __hip_atomic_fetch_add(counters + i, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  } else {
    // ================= waves 4-11: weight slices (and, waves 4-7, activation group 1 on long links)
    dev::GroupSync<4> gs1{ctr + 1, 0u, wait_limit, err};
    dev::GroupSync<8> gs8{ctr + 2, 0u, wait_limit, err};
    const bool mixed = wave < 8;
    auto slice_of = [&](bool lng) { return lng ? (mixed ? -1 : wave - 8) : wave - 4; };
    uint4 wr[16];
    auto prefetch = [&](const ChainDesc& dn) {   // the first chunk of a link, for this wave's slice
      const Geom gn = geom(dn, wg, G, TMAX);
      const int sn = slice_of(gn.lng);
      if (sn >= 0 && gn.T > 0) {
        const int T0 = gn.T < gn.tmax ? gn.T : gn.tmax;
        if (gn.lng) load_chunk_rt<FMT, true>(wr, dn, gn.t0, T0, sn);
        else load_chunk_rt<FMT, false>(wr, dn, gn.t0, T0, sn);
      }
    };
    prefetch(links[0]);
    for (int i = 0; i < n_links; ++i) {
      const ChainDesc& d = links[i];
      const Geom gm = geom(d, wg, G, TMAX);
      const int slice = slice_of(gm.lng);
      if (mixed && gm.lng) {
        if (gm.T > 0) {
          wait_input(d, i, wave, counters, (unsigned)G, in_ready, wait_ticks, err);
          link_act<PLANAR>(d, true, 1, x0, M, gs1, gs8, xch, act_l, Kpad, red_d, red_i, s_scale);
        }
        // the weight registers hold nothing on this path: let the compiler drop them
#pragma unroll
        for (int k = 0; k < 16; ++k) asm volatile("" : "=v"(wr[k]));
      }
      dev::lds_barrier();   // codes are in LDS; this wave's weight loads stay in flight
      for (int c = 0; c < gm.nchunks; ++c) {
        const int tile0 = gm.t0 + c * gm.tmax;
        const int Tc = gm.T - c * gm.tmax < gm.tmax ? gm.T - c * gm.tmax : gm.tmax;
        if (slice >= 0) {
          if (c > 0) {
            if (gm.lng) load_chunk_rt<FMT, true>(wr, d, tile0, Tc, slice);
            else load_chunk_rt<FMT, false>(wr, d, tile0, Tc, slice);
          }
          if (gm.lng) mfma_chunk_rt<FMT, true>(wr, d, tile0, Tc, slice, act_l, Kpad, M, zero64, red);
          else mfma_chunk_rt<FMT, false>(wr, d, tile0, Tc, slice, act_l, Kpad, M, zero64, red);
        }
        dev::lds_barrier();   // the slices' partial sums are in LDS
        if (c + 1 < gm.nchunks) dev::lds_barrier();   // the partial sums have been read
      }
      // every weight register has been consumed: no entry stays live into the next MFMA phase
#pragma unroll
      for (int k = 0; k < 16; ++k) asm volatile("" : "=v"(wr[k]));
      if (i + 1 < n_links) prefetch(links[i + 1]);   // the next link's weights stream during its wait
    }
  }

  // the last workgroup to finish returns the counters to zero for the next call (every workgroup has
  // passed all of its waits by then)
  __syncthreads();
  if (wave == 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this workgroup's counter increments have been performed
    unsigned prev = 0;
    if (lane == 0) prev = __hip_atomic_fetch_add(counters + n_links, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    prev = __builtin_amdgcn_readfirstlane(prev);
    if (prev == (unsigned)G - 1) {
      for (int k = lane; k <= n_links; k += 64) __hip_atomic_store(counters + k, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <int FMT>
hipError_t launch_chain_fmt(const ChainDesc* links, int n_links, const uint16_t* x0, int M, int Kmax, bool any_long,
                            int grid, unsigned* counters, hipStream_t s) {
  const int Kpad = Kmax + 16;
  const int xch = (int)chain_xch_bytes(any_long, FMT == mma::FMT_W4);
  const size_t shmem = chain_lds_bytes(M, Kmax, any_long, FMT == mma::FMT_W4);
  if (shmem > 160 * 1024) return hipErrorInvalidValue;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_decode_chain<FMT>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (attr != hipSuccess) return attr;
  const int limit = wait_limit();
  // bounded waits for other workgroups: wait_limit spins of the in-workgroup barriers correspond to
  // 25 ticks of the 100 MHz real-time clock each (about 1 s at the default)
  const long long ticks = (long long)limit * 25;
  hipLaunchKernelGGL((k_decode_chain<FMT>), dim3(grid), dim3(kChainThreads), shmem, s, links, n_links, x0, M, Kpad,
                     xch, counters, limit, ticks, device_error_word());
  return hipGetLastError();
}

}  // namespace qift
