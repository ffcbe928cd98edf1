// Persistent decode step: one co-resident grid walks a chain of quantized linears (a layer stack at
// decode), each taking its input from an earlier linear's output, so that the weight stream of the
// next linear is already in flight while the current one's dependency resolves.  Every linear is
// the fused form of the method (Sec. 3.1 online rotation and per-token INT4 quantizer, Sec. 3.3 /
// Sec. 3.6 integer dot product on the fixed level set, scales in the epilogue, Sec. 1) with results
// bit-identical to qift_rotate_quant_linear on the same input.
//
// Grid: one workgroup per CU, 12 waves each.  Linear ("link") i of the chain is cut into 16-row
// tiles; workgroup g owns tiles [g T / G, (g + 1) T / G) of it.  Per link:
//   * the activation group (waves 0-3) polls for the link's input in its producer's exchange copy
//     (agent-coherent loads until no value is the not-written pattern), rotates it exactly in fp64,
//     finds the token's absmax, quantizes and writes the codes and code sums to LDS (the routines of
//     qift_fwht.h); for K > 4096 the two halves of the weight waves rotate tiles 1 and 2 of the
//     token meanwhile (the activation group stages them in LDS);
//   * the weight waves (4-11, K-slices of 1/8 of K) issued their weight loads at the end of the
//     previous link, so those bytes stream during the wait and the rotation; after the codes
//     barrier they run the MFMAs (qift_mma.h) and write per-slice partial sums to LDS, and weight
//     wave 4 + j adds the slices of tile j, applies the epilogue and stores y, and the exchange copy
//     when another link reads this output, with agent-coherent (sc1) stores.
// Cross-XCD visibility: data and readiness travel in the same sc1 access (an exchange value is never
// the not-written pattern once written), so there is no flag, counter or L2 writeback per link.
// Every wait is bounded (by time); a wait that gives up sets a bit in the device error word and the
// workgroup carries on, so the grid always drains.  The last workgroup to finish advances the run
// number that selects the exchange copies of the next call.
#pragma once

#include "qift_fwht.h"
#include "qift_internal.h"
#include "qift_mma.h"

// Phase stamps (a diagnostic build, -DQIFT_CHAIN_STAMPS, libqift_stamps.so): the 100 MHz wall clock
// at marker k of link li in each workgroup, for the first 64 links of a call, kept per translation unit
// (qift_chain_stamps_read reads the MNZ instance's).  Markers: 0 the activation group passed its
// consumed wait, 1 its input is in, 2 its rotation is done, 3 the token's max is known, 4 its codes are
// in LDS; 5 wave 4 passed the codes barrier, 6 its MFMAs are done, 7 it passed the partial-sums
// barrier; 10 / 11 weight-wave group 1 starts / ends its rotation of a long link; 16 + s weight wave
// s has counted itself done with the link (its stores have completed).  The stamps are stores of
// their own: a stamped run is a little slower.
#ifdef QIFT_CHAIN_STAMPS
namespace qift {
static __device__ unsigned long long g_chain_stamps[256 * 64 * 32];
}
#define QIFT_STAMP(li, k)                                                                            \
  do {                                                                                              \
    if ((li) < 64 && blockIdx.x < 256)                                                              \
      qift::g_chain_stamps[((size_t)blockIdx.x * 64 + (li)) * 32 + (k)] = wall_clock64();          \
  } while (0)
#else
#define QIFT_STAMP(li, k) \
  do {                    \
  } while (0)
#endif

namespace qift {

constexpr int kChainWaves = 12;
constexpr int kChainThreads = 64 * kChainWaves;
constexpr int kChainShortK = 4096;   // one rotation tile: 4 activation waves, 8 K-slices
// LDS tail (kChainTailBytes): s_scale[2][4] f32, red_d[2][4][kChainSlots] f64, red_i[2][4][kChainSlots]
// i32, ctr[8] u32, 64 zero bytes, the weight waves' fp16 scale slots [8][64] u32
static_assert(kChainTailBytes == 32 + 64 * kChainSlots + 32 * kChainSlots + 32 + 64 + 8 * 256, "tail layout");

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

// Tiles of a link owned by workgroup wg of G: [wg T / G, (wg + 1) T / G) (32-bit arithmetic: the host
// keeps T (G + 1) below 2^32).
__device__ __forceinline__ Geom geom(const ChainDesc& d, int wg, int G, int tmax_short) {
  Geom r;
  const uint32_t tiles = (uint32_t)d.tiles;
  const int a = (int)(((uint32_t)wg * tiles) / (uint32_t)G), b = (int)(((uint32_t)(wg + 1) * tiles) / (uint32_t)G);
  r.t0 = a;
  r.T = b - a;
  r.lng = d.K > kChainShortK;
  r.tmax = r.lng ? 1 : tmax_short;
  r.nchunks = (r.T + r.tmax - 1) / r.tmax;
  return r;
}

// ---------------------------------------------------------------------------------------------
// weight waves

// Loads of one chunk of T tiles into wr (unit-major, the order the MFMAs consume them): 8 K-slices,
// of NC <= 2 units of 256 k (K <= 4096) or NC <= 8 units (K <= 16384, one tile).  Rows past N and
// k past K read zeros (out-of-range offsets).
template <int FMT, int T, bool LONG>
__device__ __forceinline__ void load_chunk(uint4 (&wr)[16], const ChainDesc& d, int tile0, int slice, int batch) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr int NS = 8;
  constexpr int UPT = LONG ? 8 : 2;
  static_assert(T * UPT * NH <= 16, "weight registers");
  // opaque lane index: the row offsets are computed per call rather than hoisted out of the link loop
  // (kept live across it they spill, and each spill reload's wait on the vector memory counter would
  // also wait for the loads just issued, one pair at a time)
  int lane = dev::lane_id();
  asm volatile("" : "+v"(lane));
  const int r16 = lane & 15, g = lane >> 4;
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

// MFMAs of one chunk; the slice's partial sums of tile j go to red[(j * NS + slice) * 64 + lane].
template <int FMT, int T, bool LONG>
__device__ __forceinline__ void mfma_chunk(uint4 (&wr)[16], const ChainDesc& d, int tile0, int slice,
                                           const int8_t* act_l, int Kpad, int M, const int8_t* zero64,
                                           v4i* red) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr int NS = 8;
  constexpr int UPT = LONG ? 8 : 2;
  constexpr bool PLANAR = FMT == FMT_MNZ;
  // accumulators per tile: MNZ one per bit plane up to 3 tiles, from 4 tiles on two (decode_plane2)
  constexpr bool TWO = PLANAR && T >= 4;
  constexpr int NA = PLANAR ? (TWO ? 2 : 4) : T >= 3 ? 1 : 4 / T;
  // opaque lane index (as in load_chunk): the operand addresses are made per call
  int lane = dev::lane_id();
  asm volatile("" : "+v"(lane));
  const int r16 = lane & 15, g = lane >> 4;
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
    v4i bq[2][4];   // the next unit's operands are read during this unit's MFMAs
    load_b(0, bq[0]);
#pragma unroll
    for (int u = 0; u < UPT; ++u) {
      if (u + 1 < UPT) load_b(u + 1, bq[(u + 1) & 1]);
      unit_mfmas(u, bq[u & 1]);
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

// One token's input for the activation group: 16 consecutive elements of each of the NT rotation
// tiles per thread (fp16 bits, 32 bytes per tile), element e = 4096 tau + 16 t + i.  The chain input
// x0 is read directly.  A link's output is read from its exchange copy of this call (the copy of the
// call's parity, written with agent-coherent stores) with agent-coherent loads, every tile's loads
// at once, until none of a wave's values is the not-written pattern kUnwritten: the data and its
// readiness arrive in the same access, so no flag or counter is needed.  Each lane reads its 16
// consecutive inputs as two 16-byte loads.  The wait is bounded by the deadline (100 MHz ticks); a
// wave that gives up sets kErrChainWait.
// 1 if a value of the 8 in a is kUnwritten (branch-free: the loads of a polling round stay in flight
// together)
__device__ __forceinline__ uint32_t unwritten8(const uint4& a) {
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
  uint32_t bad = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) bad |= (uint32_t)((w[k] & 0xFFFFu) == kUnwritten) | (uint32_t)(w[k] >= 0xFFFF0000u);
  return bad;
}

template <int NTMAX>
__device__ __forceinline__ void fetch_tiles(uint4 (&raw)[NTMAX][2], const ChainDesc& d, const uint16_t* x0, int M, int m,
                                            int NT, int t, int par, long long deadline, uint32_t* err) {
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  const bool from_x0 = d.in_link < 0;
  const uint16_t* src = from_x0 ? x0 + (int64_t)m * d.K : d.tx + ((int64_t)par * M + m) * d.xstride + d.xoff;
  const __amdgpu_buffer_rsrc_t r = dev::make_rsrc(src, (uint32_t)(d.K * 2));   // past K: zeros
  uint32_t off[NTMAX];
#pragma unroll
  for (int tau = 0; tau < NTMAX; ++tau) {
    const int e0 = tau * 4096 + 16 * t;
    off[tau] = tau < NT && e0 < d.K ? (uint32_t)(e0 * 2) : dev::kOutOfRange;
  }
  if (from_x0) {
#pragma unroll
    for (int tau = 0; tau < NTMAX; ++tau) {
      raw[tau][0] = dev::bload16(r, off[tau]);
      raw[tau][1] = dev::bload16(r, off[tau] + 16);
    }
    return;
  }
  for (;;) {
#pragma unroll
    for (int tau = 0; tau < NTMAX; ++tau)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, off[tau] + 16 * h, 0, 16);
        raw[tau][h] = make_uint4(v[0], v[1], v[2], v[3]);
      }
    uint32_t bad = 0;
#pragma unroll
    for (int tau = 0; tau < NTMAX; ++tau) bad |= unwritten8(raw[tau][0]) | unwritten8(raw[tau][1]);
    if (__all(bad == 0)) return;
    if (wall_clock64() > deadline) {
      if (dev::lane_id() == 0) dev::flag_error(err, dev::kErrChainWait);
      return;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Quantize 16 transformed values of tile tg and store their codes (the layout the transform ended
// in, at code_pos<PLANAR>); returns their sum.
template <bool PLANAR>
__device__ __forceinline__ int codes16(const double (&v)[16], const dev::QuantParams& p, int wend, int tg, int K, int t,
                                       int8_t* dst) {
  using S = dev::Tile<256, 16>;
  int q[16];
  dev::quant16(v, p, q);
  int qs = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) qs += q[e];
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
  return qs;
}

// Rotation + quantization of one token of a link with K <= 4096 (one rotation tile) by the four
// activation waves (the steps of dev::quant_token_group).  The waves synchronize through gsync; their
// maxima go to red_d[w] and their code sums to red_i[w].  Before it polls for its input the group waits
// (consumed) until the weight waves are done with the previous link: their stores are then issued
// ahead of the polling loads (polling that overlapped them was measured to starve them), and the
// previous link's partial sums, which share the group's LDS region, have been read.
// The thread's index within its group of four waves (gw: the wave's index in the group, uniform) as an
// opaque value: the per-thread LDS addresses derived from it are computed per call instead of being
// hoisted out of the link loop (where dozens of them would stay live across the whole loop and spill).
__device__ __forceinline__ int group_thread(int gw) {
  int t = 64 * gw + dev::lane_id();
  asm volatile("" : "+v"(t));
  return t;
}

__device__ __forceinline__ void wait_consumed(const unsigned* consumed, unsigned target, long long deadline,
                                              uint32_t* err) {
  for (;;) {
    const unsigned c = __builtin_amdgcn_readfirstlane(
        __hip_atomic_load(consumed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
    if (c >= target) break;
    if (wall_clock64() > deadline) {
      if (dev::lane_id() == 0) dev::flag_error(err, dev::kErrGroupWait);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  asm volatile("" ::: "memory");
}

template <int LC, bool PLANAR, typename GS>
__device__ __forceinline__ double quant_group(int gw, int li, const ChainDesc& d, const uint16_t* x0, int M, int m, int par,
                                              long long deadline, uint32_t* err, GS& gsync, double* xch,
                                              int8_t* dst, double* red_d, int* red_i, const unsigned* consumed,
                                              unsigned consumed_target) {
  const int t = group_thread(gw);
  const int lane = t & 63, w = t >> 6;
  if (consumed) wait_consumed(consumed, consumed_target, deadline, err);
  if (t == 0) QIFT_STAMP(li, 0);
  uint4 raw[1][2];
  fetch_tiles<1>(raw, d, x0, M, m, 1, t, par, deadline, err);
  if (t == 0) QIFT_STAMP(li, 1);
  double v[16];
  dev::unpack16<false>(v, raw[0]);
  const int wend = dev::fwht_tile_s<256, 16, false>(v, xch, t, LC, gsync);
  if (t == 0) QIFT_STAMP(li, 2);
  double amax = 0.0;
#pragma unroll
  for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[e]));
  amax = dev::wave_max(amax);
  if (lane == 0) red_d[w] = amax;
  gsync();
  if (t == 0) QIFT_STAMP(li, 3);
  const double A = fmax(fmax(red_d[0], red_d[1]), fmax(red_d[2], red_d[3]));
  const dev::QuantParams p = dev::make_qparams(A, d.num, d.den);
  int qs = codes16<PLANAR>(v, p, wend, 0, d.K, t, dst);
  qs = dev::wave_sum(qs);
  if (lane == 0) red_i[w] = qs;
  if (t == 0) QIFT_STAMP(li, 4);
  return A;
}

// Links with K > 4096 (NT = 2..4 rotation tiles): the tiles are rotated by three groups of four waves
// at once, the activation group (tiles 0 and 3, tile 0 kept in registers while it rotates tile 3) and
// the two halves of the weight waves (gi = 1: tile 1, gi = 2: tile 2 if NT > 2), whose weight loads for
// the link are in flight meanwhile.  Per token:
//   * the activation group polls for all tiles, puts tiles 1 and 2 (fp16 bits) into the exchange
//     buffers of groups 1 and 2 and counts them staged in LDS; the weight waves wait for that count
//     (a wave issuing weight loads stalls at the issue while its CU's memory queue is full: the
//     activation group does not wait for them);
//   * every group rotates its tile(s) in an exchange buffer of its own (its own wave barrier) and writes
//     the absmax of each wave to red_d[4 g + w]; a workgroup barrier;
//   * every group takes the token's max over the twelve slots and quantizes its tile(s) into the
//     codes; code sums go to red_i[4 g + w].
template <int LC, bool PLANAR, typename GS>
__device__ __forceinline__ double long_group_a(int gw, int li, const ChainDesc& d, const uint16_t* x0, int M, int m, int NT,
                                               int par, long long deadline, uint32_t* err, GS& gsync,
                                               double* xch, double* xch_b, double* xch_c, int8_t* dst,
                                               double* red_d, int* red_i, const unsigned* consumed,
                                               unsigned consumed_target, unsigned* staged) {
  const int t = group_thread(gw);
  const int lane = t & 63, w = t >> 6;
  if (consumed) wait_consumed(consumed, consumed_target, deadline, err);
  if (t == 0) QIFT_STAMP(li, 0);
  uint4 raw[4][2];
  fetch_tiles<4>(raw, d, x0, M, m, NT, t, par, deadline, err);
  if (t == 0) QIFT_STAMP(li, 1);
  // the other groups' input: 32 bytes per thread at the start of their exchange buffers (their
  // exchanges of the previous token ended before the previous token's second barrier)
  uint4* sb = reinterpret_cast<uint4*>(xch_b);
  sb[2 * t] = raw[1][0];
  sb[2 * t + 1] = raw[1][1];
  if (NT > 2) {
    uint4* sc = reinterpret_cast<uint4*>(xch_c);
    sc[2 * t] = raw[2][0];
    sc[2 * t + 1] = raw[2][1];
  }
  // the other groups' tiles are in LDS: each wave counts itself (no workgroup barrier, so a weight
  // wave still issuing its loads for this link does not hold the group up)
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  if (lane == 0) __hip_atomic_fetch_add(staged, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  double v[16];
  dev::unpack16<false>(v, raw[0]);
  const int wend = dev::fwht_tile_s<256, 16, false>(v, xch, t, LC, gsync);
  double amax = 0.0;
#pragma unroll
  for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[e]));
  double v3[16];
  if (NT > 3) {
    if (LC > 6) gsync();   // one exchange buffer: tile 0's exchange reads are done
    dev::unpack16<false>(v3, raw[3]);
    dev::fwht_tile_s<256, 16, false>(v3, xch, t, LC, gsync);
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v3[e]));
  }
  if (t == 0) QIFT_STAMP(li, 2);
  amax = dev::wave_max(amax);
  if (lane == 0) red_d[w] = amax;
  dev::lds_barrier();   // every group's maxima are in LDS
  if (t == 0) QIFT_STAMP(li, 3);
  double A = red_d[0];
#pragma unroll
  for (int k = 1; k < 12; ++k) A = fmax(A, red_d[k]);
  const dev::QuantParams p = dev::make_qparams(A, d.num, d.den);
  int qs = codes16<PLANAR>(v, p, wend, 0, d.K, t, dst);
  if (NT > 3) qs += codes16<PLANAR>(v3, p, wend, 3, d.K, t, dst);
  qs = dev::wave_sum(qs);
  if (lane == 0) red_i[w] = qs;
  if (t == 0) QIFT_STAMP(li, 4);
  return A;
}

// The weight waves' part of a long link (group gi = 1: tile 1, gi = 2: tile 2 if NT > 2): they wait
// until the four activation waves have counted their staging writes (staged reaches stage_target),
// then meet the activation group at the workgroup barrier after the maxima.
template <int LC, bool PLANAR, typename GS>
__device__ __forceinline__ void long_group_w(int gw, int li, const ChainDesc& d, int NT, int gi, GS& gsync, double* xch_g,
                                             int8_t* dst, double* red_d, int* red_i, const unsigned* staged,
                                             unsigned stage_target, long long deadline, uint32_t* err) {
  const int t = group_thread(gw);
  const int lane = t & 63, w = t >> 6;
  const bool has = gi < NT;
  wait_consumed(staged, stage_target, deadline, err);   // the group's tile is in LDS
  double v[16];
  double amax = 0.0;
  int wend = 0;
  if (has) {
    const uint4* sg = reinterpret_cast<const uint4*>(xch_g);
    uint4 r[2] = {sg[2 * t], sg[2 * t + 1]};
    gsync();   // every wave of the group has its input before the exchanges overwrite it
    dev::unpack16<false>(v, r);
    if (t == 0 && gi == 1) QIFT_STAMP(li, 10);
    wend = dev::fwht_tile_s<256, 16, false>(v, xch_g, t, LC, gsync);
    if (t == 0 && gi == 1) QIFT_STAMP(li, 11);
#pragma unroll
    for (int e = 0; e < 16; ++e) amax = fmax(amax, fabs(v[e]));
  }
  amax = dev::wave_max(amax);
  if (lane == 0) red_d[4 * gi + w] = amax;
  dev::lds_barrier();   // every group's maxima are in LDS
  int qs = 0;
  if (has) {
    double A = red_d[0];
#pragma unroll
    for (int k = 1; k < 12; ++k) A = fmax(A, red_d[k]);
    const dev::QuantParams p = dev::make_qparams(A, d.num, d.den);
    qs = codes16<PLANAR>(v, p, wend, gi, d.K, t, dst);
    qs = dev::wave_sum(qs);
  }
  if (lane == 0) red_i[4 * gi + w] = qs;
}


// The activation group's part of one link: every token; the scale of token m goes to s_scale[m].
template <bool PLANAR, typename GS>
__device__ __forceinline__ void act_link(int gw, int li, const ChainDesc& d, const uint16_t* x0, int M, int par,
                                         long long deadline, uint32_t* err, GS& gsync, double* xch, double* xch_b,
                                         double* xch_c, int8_t* act_l, int Kpad, double* red_d, int* red_i,
                                         float* s_scale, const unsigned* consumed, unsigned consumed_target,
                                         unsigned* staged) {
  const int NT = (d.K + 4095) / 4096;
  for (int m = 0; m < M; ++m) {
    double A;
    const unsigned* cw = m == 0 ? consumed : nullptr;
    double* rd = red_d + kChainSlots * m;
    int* ri = red_i + kChainSlots * m;
    int8_t* dst = act_l + m * Kpad;
    // the block sizes compiled in (chain_block_ok): every butterfly stage is straight-line code
    if (NT > 1) {
      switch (d.L) {
        case 12: A = long_group_a<12, PLANAR>(gw, li, d, x0, M, m, NT, par, deadline, err, gsync, xch, xch_b, xch_c, dst, rd, ri, cw, consumed_target, staged); break;
        case 11: A = long_group_a<11, PLANAR>(gw, li, d, x0, M, m, NT, par, deadline, err, gsync, xch, xch_b, xch_c, dst, rd, ri, cw, consumed_target, staged); break;
        case 8: A = long_group_a<8, PLANAR>(gw, li, d, x0, M, m, NT, par, deadline, err, gsync, xch, xch_b, xch_c, dst, rd, ri, cw, consumed_target, staged); break;
        default: A = long_group_a<6, PLANAR>(gw, li, d, x0, M, m, NT, par, deadline, err, gsync, xch, xch_b, xch_c, dst, rd, ri, cw, consumed_target, staged); break;
      }
    } else {
      switch (d.L) {
        case 12: A = quant_group<12, PLANAR>(gw, li, d, x0, M, m, par, deadline, err, gsync, xch, dst, rd, ri, cw, consumed_target); break;
        case 11: A = quant_group<11, PLANAR>(gw, li, d, x0, M, m, par, deadline, err, gsync, xch, dst, rd, ri, cw, consumed_target); break;
        case 8: A = quant_group<8, PLANAR>(gw, li, d, x0, M, m, par, deadline, err, gsync, xch, dst, rd, ri, cw, consumed_target); break;
        default: A = quant_group<6, PLANAR>(gw, li, d, x0, M, m, par, deadline, err, gsync, xch, dst, rd, ri, cw, consumed_target); break;
      }
    }
    if (gw == 0 && dev::lane_id() == 0) s_scale[m] = (float)((A * (double)d.num) / d.denom);
  }
}

// The weight waves' part of a long link: every token.
// stage_count: the tokens of long links staged so far in this call (the same count in every wave).
template <bool PLANAR, typename GS>
__device__ __forceinline__ void act_link_w(int gw, int li, const ChainDesc& d, int M, int gi, GS& gsync, double* xch_g,
                                           int8_t* act_l, int Kpad, double* red_d, int* red_i,
                                           const unsigned* staged, unsigned& stage_count, long long deadline,
                                           uint32_t* err) {
  const int NT = (d.K + 4095) / 4096;
  for (int m = 0; m < M; ++m) {
    double* rd = red_d + kChainSlots * m;
    int* ri = red_i + kChainSlots * m;
    int8_t* dst = act_l + m * Kpad;
    const unsigned tg = 4u * ++stage_count;
    switch (d.L) {
      case 12: long_group_w<12, PLANAR>(gw, li, d, NT, gi, gsync, xch_g, dst, rd, ri, staged, tg, deadline, err); break;
      case 11: long_group_w<11, PLANAR>(gw, li, d, NT, gi, gsync, xch_g, dst, rd, ri, staged, tg, deadline, err); break;
      case 8: long_group_w<8, PLANAR>(gw, li, d, NT, gi, gsync, xch_g, dst, rd, ri, staged, tg, deadline, err); break;
      default: long_group_w<6, PLANAR>(gw, li, d, NT, gi, gsync, xch_g, dst, rd, ri, staged, tg, deadline, err); break;
    }
  }
}

// y[m][n0 .. n0 + 3] (fp16, and the accumulators) and, for the links whose output another link
// reads, the same four values into this call's exchange copy (a value equal to kUnwritten, a NaN,
// becomes the quiet NaN 0xFE00 there) and kUnwritten into the other copy (the one the next call
// writes; its readers of the previous call have finished), both with agent-coherent stores.
template <int FMT>
__device__ __forceinline__ void store4_chain(const v4i& D, const ChainDesc& d, int M, int m, int n0, float s_x,
                                             int sum_q, uint2 swq, __amdgpu_buffer_rsrc_t tyr, int par) {
  typedef unsigned v2u __attribute__((ext_vector_type(2)));
  const int N = d.N;
  const uint16_t swv[4] = {(uint16_t)(swq.x & 0xFFFFu), (uint16_t)(swq.x >> 16), (uint16_t)(swq.y & 0xFFFFu),
                           (uint16_t)(swq.y >> 16)};
  int a[4];
  uint16_t h[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    a[r] = finish_acc<FMT>(D[r], sum_q);
    h[r] = n0 + r < N ? epilogue(a[r], s_x, swv[r]) : 0;
  }
  const uint32_t lo = (uint32_t)h[0] | ((uint32_t)h[1] << 16), hi = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
  if (d.ty) {
    uint32_t e[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) e[r] = h[r] == kUnwritten ? 0xFE00u : h[r];
    const uint32_t row = (uint32_t)((par * M + m) * d.ystride), other = (uint32_t)(((1 - par) * M + m) * d.ystride);
    const bool in = n0 < N;   // rows past N (the rest of a 16-row tile) stay out of the copies
    __builtin_amdgcn_raw_buffer_store_b64(v2u{e[0] | (e[1] << 16), e[2] | (e[3] << 16)}, tyr,
                                          in ? (row + n0) * 2u : dev::kOutOfRange, 0, 16);
    uint32_t ones;   // the not-written pattern, made here (a constant kept from earlier would be spilled)
    asm volatile("v_mov_b32 %0, -1" : "=v"(ones));
    __builtin_amdgcn_raw_buffer_store_b64(v2u{ones, ones}, tyr, in ? (other + n0) * 2u : dev::kOutOfRange, 0, 16);
  }
  uint16_t* __restrict__ y = d.y;
  int32_t* __restrict__ acc_out = d.acc;
  const int64_t o = (int64_t)m * N + n0;
  if (n0 + 3 < N && (((uint32_t)m * (uint32_t)N + (uint32_t)n0) & 3u) == 0) {
    *reinterpret_cast<uint2*>(y + o) = make_uint2(lo, hi);
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

}  // namespace chain

// ---------------------------------------------------------------------------------------------
// the kernel
//
// Waves 0-3 (the activation group) and waves 4-11 (the weight waves, K-slices of 1/8 of K) run two
// loops over the links that take the same sequence of workgroup barriers (per link: codes ready,
// then per chunk of tiles: partial sums ready, and between chunks: partial sums read), so that a
// wave's registers hold only what its own role needs.  The activation group goes on to the next
// link's input as soon as this link's codes are in; after the MFMAs, weight wave 4 + j adds the
// K-slices of tile j of the chunk, applies the epilogue and stores it, and only then issues the next
// link's weight loads, so the stores are not queued behind them.
// Links with K > 4096 also use the weight waves for their rotation (long_group_a / long_group_w): one
// more workgroup barrier per token, taken by both loops, and an LDS count of the staged tiles.
// LDS: the codes [M][Kpad]; the rotation region (the activation group's exchange buffer, and for
// chains with K > 4096 those of the two weight-wave groups), aliased by the K-slice partial sums: the
// activation group writes it for the next link only once the 8 weight waves have counted themselves
// done with them; then the tail: s_scale, red_d and red_i double-buffered by link parity (the next
// link's activation phase runs while this link's are still read), the wave-barrier counters (the
// activation group's and the two weight-wave groups'), the weight waves' count and 64 zero bytes.
// Exchange copies: the call's run number r (read at the start; the last workgroup to finish advances
// it) selects copy r mod 2 of every exchange buffer.
template <int FMT>
__global__ __launch_bounds__(kChainThreads) void k_decode_chain(const ChainDesc* __restrict__ links, int n_links,
                                                                const uint16_t* __restrict__ x0, int M, int Kpad,
                                                                int region0, unsigned* __restrict__ counters,
                                                                int wait_limit, long long wait_ticks,
                                                                uint32_t* __restrict__ err) {
  using namespace chain;
  constexpr bool PLANAR = FMT == FMT_MNZ;
  constexpr int TMAX = chain_tmax<FMT>();
  extern __shared__ __align__(16) unsigned char smem[];
  // the work-item id is read here only (the loops below use dev::lane_id() and the uniform wave index)
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = gridDim.x, wg = blockIdx.x;

  const int act_bytes = (M * Kpad + 15) & ~15;
  int8_t* act_l = reinterpret_cast<int8_t*>(smem);
  double* xch = reinterpret_cast<double*>(smem + act_bytes);
  double* xch_b = xch + kXchBytes / 8;   // the weight-wave groups' exchange buffers (chains with K > 4096)
  double* xch_c = xch_b + kXchBytes / 8;
  v4i* red = reinterpret_cast<v4i*>(xch);   // the K-slice partial sums reuse the rotation region
  unsigned char* tl = smem + act_bytes + region0;
  constexpr int RS = 4 * kChainSlots;   // red_d / red_i entries per link parity
  float* s_scale = reinterpret_cast<float*>(tl);                      // [2][4]
  double* red_d = reinterpret_cast<double*>(tl + 32);                 // [2][4][kChainSlots]
  int* red_i = reinterpret_cast<int*>(tl + 32 + 16 * RS);             // [2][4][kChainSlots]
  // ctr: [0..2] group barriers, [3] weight waves done, [4] long-link tiles staged
  unsigned* ctr = reinterpret_cast<unsigned*>(tl + 32 + 24 * RS);
  int8_t* zero64 = reinterpret_cast<int8_t*>(tl + 32 + 24 * RS + 32);
  uint32_t* sw_slots = reinterpret_cast<uint32_t*>(tl + 32 + 24 * RS + 96);   // [weight wave][64]
  if (tid < 8) ctr[tid] = 0u;
  if (tid < 4) reinterpret_cast<uint4*>(zero64)[tid] = make_uint4(0u, 0u, 0u, 0u);
  const unsigned run = __builtin_amdgcn_readfirstlane(
      __hip_atomic_load(counters + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  const int rpar = (int)(run & 1u);
  const long long deadline = wall_clock64() + wait_ticks;   // every wait of this call ends by then
  __syncthreads();
  unsigned* consumed = ctr + 3;   // bumped by each weight wave once it is done with a link's partial sums

  if (wave < 4) {
    // ================= waves 0-3: the activation group
    dev::GroupSync<4> gs{ctr + 0, 0u, wait_limit, err};
    for (int i = 0; i < n_links; ++i) {
      const ChainDesc& d = links[i];
      const Geom gm = geom(d, wg, G, TMAX);
      const int par = i & 1;
      if (gm.T > 0)
        act_link<PLANAR>(wave, i, d, x0, M, rpar, deadline, err, gs, xch, xch_b, xch_c, act_l, Kpad, red_d + RS * par,
                         red_i + RS * par, s_scale + 4 * par, consumed, 8u * (unsigned)i, ctr + 4);
      dev::lds_barrier();   // codes, scales and code sums are in LDS
      for (int c = 0; c < gm.nchunks; ++c) {
        dev::lds_barrier();                           // partial sums are in LDS
        if (c + 1 < gm.nchunks) dev::lds_barrier();   // partial sums have been read
      }
    }
  } else {
    // ================= waves 4-11: weight slices, then the reduction, epilogue and stores
    const int slice = wave - 4;
    const int gi = slice < 4 ? 1 : 2;   // rotation group of long links: tile 1 or tile 2
    dev::GroupSync<4> gsw{ctr + gi, 0u, wait_limit, err};
    unsigned stage_count = 0;
    uint4 wr[16];
    // this wave's fp16 scales: the 16 of the tile it stores (tile `slice` of a link's first chunk) go
    // straight into its LDS slot with the prefetch (a direct-to-LDS load: no register is held across
    // the link loop), lanes 0-7 one dword each
    uint32_t* my_sw = sw_slots + 64 * slice;
    auto prefetch = [&](const ChainDesc& dn) {   // the first chunk of a link, for this wave's slice
      const Geom gn = geom(dn, wg, G, TMAX);
      if (gn.T > 0) {
        const int T0 = gn.T < gn.tmax ? gn.T : gn.tmax;
        if (gn.lng) load_chunk_rt<FMT, true>(wr, dn, gn.t0, T0, slice);
        else load_chunk_rt<FMT, false>(wr, dn, gn.t0, T0, slice);
        int ln = dev::lane_id();
        asm volatile("" : "+v"(ln));
        const int n = (gn.t0 + slice) * 16 + 2 * ln;   // rows n, n + 1 in dword ln of the slot
        const __amdgpu_buffer_rsrc_t srs = dev::make_rsrc(dn.sw, (uint32_t)(dn.N * 2));
        const uint32_t off = slice < T0 && ln < 8 && n < dn.N ? (uint32_t)(2 * n) : dev::kOutOfRange;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (__attribute__((address_space(3))) void*)my_sw, 4, off, 0, 0, 0);
      }
    };
    prefetch(links[0]);
    for (int i = 0; i < n_links; ++i) {
      const ChainDesc& d = links[i];
      const Geom gm = geom(d, wg, G, TMAX);
      const int par = i & 1;
      if (gm.lng && gm.T > 0)
        act_link_w<PLANAR>(slice & 3, i, d, M, gi, gsw, gi == 1 ? xch_b : xch_c, act_l, Kpad, red_d + RS * par,
                           red_i + RS * par, ctr + 4, stage_count, deadline, err);
      dev::lds_barrier();   // codes are in LDS; this wave's weight loads stay in flight
      if (wave == 4 && dev::lane_id() == 0) QIFT_STAMP(i, 5);
      const __amdgpu_buffer_rsrc_t tyr = dev::make_rsrc(d.ty, (uint32_t)(2 * M * d.ystride * 2));
      for (int c = 0; c < gm.nchunks; ++c) {
        const int tile0 = gm.t0 + c * gm.tmax;
        const int Tc = gm.T - c * gm.tmax < gm.tmax ? gm.T - c * gm.tmax : gm.tmax;
        if (c > 0) {
          if (gm.lng) load_chunk_rt<FMT, true>(wr, d, tile0, Tc, slice);
          else load_chunk_rt<FMT, false>(wr, d, tile0, Tc, slice);
        }
        if (gm.lng) mfma_chunk_rt<FMT, true>(wr, d, tile0, Tc, slice, act_l, Kpad, M, zero64, red);
        else mfma_chunk_rt<FMT, false>(wr, d, tile0, Tc, slice, act_l, Kpad, M, zero64, red);
        if (wave == 4 && c == 0 && dev::lane_id() == 0) QIFT_STAMP(i, 6);
        dev::lds_barrier();   // the slices' partial sums are in LDS
        if (wave == 4 && c == 0 && dev::lane_id() == 0) QIFT_STAMP(i, 7);
        if (slice < Tc) {
          // this wave's tile: add the K-slices, apply the epilogue and store.  The lane index is
          // opaque here, so the per-lane addresses are computed in place rather than hoisted out of
          // the link loop: kept live across it they spill, and a spill reload's wait on the vector
          // memory counter would also wait for the agent-coherent stores issued before it.
          int ln = dev::lane_id();
          asm volatile("" : "+v"(ln));
          const int n0 = (tile0 + slice) * 16 + 4 * (ln >> 4), m = ln & 15;
          uint2 swq;
          if (c > 0) {
            const __amdgpu_buffer_rsrc_t srs = dev::make_rsrc(d.sw, (uint32_t)(d.N * 2));
            swq = dev::bload8(srs, n0 < d.N ? (uint32_t)(2 * n0) : dev::kOutOfRange);
          } else {
            // the direct-to-LDS scale load of the prefetch (issued after this wave's weight loads, which
            // the MFMAs have consumed) has landed; rows 4 g .. 4 g + 3 are dwords 2 g, 2 g + 1
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            swq = *reinterpret_cast<const uint2*>(my_sw + 2 * (ln >> 4));
          }
          v4i D = red[(slice * 8) * 64 + ln];
#pragma unroll
          for (int q = 1; q < 8; ++q) D += red[(slice * 8 + q) * 64 + ln];
          if (m < M && n0 < d.N) {
            const int* ri = red_i + RS * par + kChainSlots * m;
            int sq = ri[0] + ri[1] + ri[2] + ri[3];
            if (gm.lng) {
#pragma unroll
              for (int k = 4; k < 12; ++k) sq += ri[k];
            }
            store4_chain<FMT>(D, d, M, m, n0, s_scale[4 * par + m], sq, swq, tyr, rpar);
          }
        }
        if (c + 1 < gm.nchunks) dev::lds_barrier();   // the partial sums have been read
      }
      // done with this link's partial sums (the LDS reads have returned) and with its stores: the
      // activation group starts polling for the next link's input on this count, and polls that
      // overlapped this CU's stores in flight were measured to slow the step by 5 %
      __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0)
      if (dev::lane_id() == 0) __hip_atomic_fetch_add(consumed, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (dev::lane_id() == 0) QIFT_STAMP(i, 16 + slice);
      // every weight register has been consumed: no entry stays live into the next MFMA phase
#pragma unroll
      for (int k = 0; k < 16; ++k) asm volatile("" : "=v"(wr[k]));
      if (i + 1 < n_links) prefetch(links[i + 1]);   // behind this wave's stores: the next link's weights
    }
  }

  // the last workgroup to finish resets the arrival count and advances the run number (every
  // workgroup has read the run number at its start and passed all of its waits by then)
  __syncthreads();
  if (wave == 0) {
    unsigned prev = 0;
    const int lane = dev::lane_id();
    if (lane == 0) prev = __hip_atomic_fetch_add(counters, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    prev = __builtin_amdgcn_readfirstlane(prev);
    if (prev == (unsigned)G - 1 && lane == 0) {
      __hip_atomic_store(counters, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(counters + 1, run + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <int FMT>
hipError_t launch_chain_fmt(const ChainDesc* links, int n_links, const uint16_t* x0, int M, int Kmax, int region0,
                            int grid, unsigned* counters, hipStream_t s) {
  const int Kpad = Kmax + 16;
  const size_t shmem = chain_lds_bytes(M, Kmax, region0);
  if (shmem > 160 * 1024) return hipErrorInvalidValue;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_decode_chain<FMT>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (attr != hipSuccess) return attr;
  const int limit = wait_limit();
  // bounded waits for other workgroups: wait_limit spins of the in-workgroup barriers correspond to
  // 25 ticks of the 100 MHz real-time clock each (about 1 s for the whole call at the default)
  const long long ticks = (long long)limit * 25;
  hipLaunchKernelGGL((k_decode_chain<FMT>), dim3(grid), dim3(kChainThreads), shmem, s, links, n_links, x0, M, Kpad,
                     region0, counters, limit, ticks, device_error_word());
  return hipGetLastError();
}

}  // namespace qift
