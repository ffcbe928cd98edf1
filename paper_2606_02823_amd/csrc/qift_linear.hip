// Quantized linear kernels on int8 MFMA (operand layout and decoding:
// qift_mma.h): the decode kernels for up to 16 tokens and the tiled prefill
// GEMM.
#include "qift_fwht.h"   // buffer-load helpers
#include "qift_internal.h"
#include "qift_mma.h"
#include "qift_split.h"

namespace qift {
namespace {

using namespace mma;

// ===========================================================================
// Decode kernel for act_q in global memory: M <= 16 tokens (one 16-token
// MFMA column) whose codes do not fit in LDS.
//
// Workgroup = 4 waves on one 16-row tile at a time; wave w takes the 1024-k
// chunks w, w+4, ... of the tile; inside a chunk, lane group g covers
// k0 = 1024c + 256u + 64g, u = 0..3 (one 16-byte W2 load per unit).  The
// workgroup walks row tiles blockIdx.x, +gridDim.x, ...; each wave issues
// the loads of its next chunk (possibly of the next tile) before computing
// the current one, so weight traffic stays in flight across tiles and during
// the cross-wave reduction.  B operands come straight from act_q; partial
// accumulators meet in LDS.
// ===========================================================================

template <int FMT>
struct WChunk {
  uint4 v[4][FMT == FMT_W4 ? 2 : 1];
};

template <int FMT>
__device__ __forceinline__ void load_chunk(WChunk<FMT>& ck, const char* prow, bool rowok, int K, int c,
                                           int g) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int k0 = (c << 10) + (u << 8) + (g << 6);
    const bool ok = rowok && k0 < K;
    const uint4* src = reinterpret_cast<const uint4*>(prow + (FMT == FMT_W4 ? k0 / 2 : k0 / 4));
#pragma unroll
    for (int h = 0; h < NH; ++h) ck.v[u][h] = ok ? src[h] : make_uint4(0, 0, 0, 0);
  }
}

// With sumq the codes of the chunk are also added to sq (the first tile of a workgroup visits every
// k of every token once across its lanes and waves).
template <int FMT>
__device__ __forceinline__ void mma_chunk(const WChunk<FMT>& ck, v4i& acc, int K, int c, int g, int m, int M,
                                          const int8_t* __restrict__ act, bool sumq, int& sq) {
  const bool mok = m < M;
  // B operands of the whole chunk first (independent loads, one wait)
  v4i b[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int k0 = (c << 10) + (u << 8) + (g << 6);
    const bool ok = mok && k0 < K;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 bb = make_uint4(0, 0, 0, 0);
      if (ok) bb = *reinterpret_cast<const uint4*>(act + (int64_t)m * K + k0 + 16 * s);
      b[u][s] = v4i{(int)bb.x, (int)bb.y, (int)bb.z, (int)bb.w};
    }
  }
  if (sumq) {   // wave-uniform
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int s = 0; s < 4; ++s)
        sq = sum16_i8(make_uint4((uint32_t)b[u][s][0], (uint32_t)b[u][s][1], (uint32_t)b[u][s][2],
                                 (uint32_t)b[u][s][3]), sq);
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if ((c << 10) + (u << 8) >= K) break;   // wave-uniform tail
#pragma unroll
    for (int s = 0; s < 4; ++s) acc = mfma_i8(decode_unit<FMT>(ck.v[u], s), b[u][s], acc);
  }
}

template <int FMT>
__global__ __launch_bounds__(256) void k_decode(
    const uint32_t* __restrict__ P, const uint16_t* __restrict__ sw, int N, int K,
    const int8_t* __restrict__ act, const float* __restrict__ sx, const int32_t* __restrict__ asum,
    int M, uint16_t* __restrict__ y, int32_t* __restrict__ acc_out) {
  __shared__ v4i red[4 * 64];
  __shared__ float s_scale[16];
  __shared__ int s_sum[16];
  __shared__ int s_part[4][16];   // per-wave sums of q (no asum given)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ntiles = (N + 15) >> 4;
  const int NC = (K + 1023) >> 10;
  const int64_t rowbytes = FMT == FMT_W4 ? (int64_t)K / 2 : (int64_t)K / 4;

  // first chunk of this wave's first tile
  int tile = blockIdx.x;
  WChunk<FMT> cur;
  {
    const int n = tile * 16 + r16;
    const bool rowok = tile < ntiles && n < N && wave < NC;
    const char* prow = reinterpret_cast<const char*>(P) + (int64_t)(rowok ? n : 0) * rowbytes;
    load_chunk<FMT>(cur, prow, rowok, K, wave, g);
  }
  if (tid < M) {
    s_scale[tid] = sx[tid];
    if (asum) s_sum[tid] = asum[tid];
  }
  __syncthreads();

  const int m = r16;   // token of this lane's B operand and outputs
  bool first = asum == nullptr;   // sum the codes of the first tile's B operands
  for (; tile < ntiles; tile += gridDim.x) {
    v4i acc = v4i{0, 0, 0, 0};
    int sq = 0;
    for (int c = wave; c < NC; c += 4) {
      // prefetch the wave's next chunk: same tile, or the first chunk of the next tile
      int nc = c + 4, nt = tile;
      if (nc >= NC) {
        nc = wave;
        nt = tile + gridDim.x;
      }
      WChunk<FMT> nxt;
      {
        const int n = nt * 16 + r16;
        const bool rowok = nt < ntiles && n < N;
        const char* prow = reinterpret_cast<const char*>(P) + (int64_t)(rowok ? n : 0) * rowbytes;
        load_chunk<FMT>(nxt, prow, rowok, K, nc, g);
      }
      mma_chunk<FMT>(cur, acc, K, c, g, m, M, act, first, sq);
      cur = nxt;
    }
    red[wave * 64 + lane] = acc;
    if (first) {
      // lanes m, m + 16, m + 32, m + 48 hold the four k-groups of token m
      sq += __shfl_xor(sq, 16);
      sq += __shfl_xor(sq, 32);
      if (lane < 16) s_part[wave][lane] = sq;
    }
    __syncthreads();
    if (first) {
      if (tid < 16) s_sum[tid] = s_part[0][tid] + s_part[1][tid] + s_part[2][tid] + s_part[3][tid];
      __syncthreads();
      first = false;
    }
    if (wave == 0) {
      v4i D = red[lane];
#pragma unroll
      for (int w = 1; w < 4; ++w) D += red[w * 64 + lane];
      if (m < M) store4<FMT>(D, m, tile * 16 + 4 * g, N, s_scale[m], s_sum[m], sw, y, acc_out);
    }
    __syncthreads();
  }
}

// ===========================================================================
// Decode kernel with deep loads: M <= 16 tokens whose int8 activation codes
// fit in LDS (the unfused path; the fused rotation has its own kernel in
// qift_fused.h).
//
// A workgroup (4 waves) owns T consecutive 16-row tiles; wave w owns the
// w-th quarter of K of each of them: NC = ceil(K/1024) units of 256 k, in
// each of which lane group g reads 64 weights (one 16-byte W2 load).  A wave
// holds UPT units per tile in registers and issues all of them before it
// waits, so a workgroup keeps 4*T*UPT KB (W2) of packed weights in flight.
// The first activation loads are issued before the weight loads: the
// vector-memory counter retires loads in order, so staging the codes into
// LDS overlaps the weight stream.  T is chosen per launch so that the grid
// covers every CU with one workgroup each (up to 6 tiles).  The four
// quarters of a tile meet in LDS and wave j mod 4 stores tile j (4
// consecutive outputs per lane).
// ===========================================================================
template <int FMT, int T, int UPT>
__global__ __launch_bounds__(256) void k_decode_deep(
    const uint32_t* __restrict__ P, const uint16_t* __restrict__ sw, int N, int K,
    const int8_t* __restrict__ act, const float* __restrict__ sx, const int32_t* __restrict__ asum,
    int M, int Kpad, uint16_t* __restrict__ y, int32_t* __restrict__ acc_out) {
  constexpr int NH = FMT == FMT_W4 ? 2 : 1;
  constexpr int kRed = 4 * T * 64 * 16;
  constexpr int kPre = 4;                   // activation pieces per thread loaded ahead of the weights
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int64_t rowbytes = FMT == FMT_W4 ? (int64_t)K / 2 : (int64_t)K / 4;
  const int NC = (K + 1023) >> 10;          // 256-k units per quarter of K
  const int kq0 = wave * NC * 256;          // first k of this wave's quarter

  const int act_bytes = (M * Kpad + 15) & ~15;
  int8_t* act_l = reinterpret_cast<int8_t*>(smem);
  unsigned char* scratch = smem + act_bytes;
  float* s_scale = reinterpret_cast<float*>(scratch + kRed);
  int* s_sum = reinterpret_cast<int*>(s_scale + 16);

  const int tile0 = blockIdx.x * T;
  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(P, (uint32_t)(N * rowbytes));
  uint32_t rowoff[T];
  bool rowok[T];
#pragma unroll
  for (int j = 0; j < T; ++j) {
    const int n = (tile0 + j) * 16 + r16;
    rowok[j] = n < N;
    rowoff[j] = (uint32_t)(n * rowbytes);
  }

  // (1) activation loads first
  const int per_row = K >> 4;               // 16-byte pieces per activation row
  uint4 apre[kPre];
  {
    const __amdgpu_buffer_rsrc_t ars = dev::make_rsrc(act, (uint32_t)(M * K));
#pragma unroll
    for (int q = 0; q < kPre; ++q) {
      const int i = tid + 256 * q;
      apre[q] = dev::bload16(ars, i < M * per_row ? (uint32_t)(16 * i) : dev::kOutOfRange);
    }
  }
  const int mm = tid < M ? tid : 0;
  const float sx_pre = sx[mm];
  const int sum_pre = asum ? asum[mm] : 0;
  if (!asum && tid < 16) s_sum[tid] = 0;
  // keep every activation load ahead of the weight loads in the instruction stream
  __builtin_amdgcn_sched_barrier(0);

  // (2) the first batch of weights (zeros for rows past N and k past K)
  uint4 w[T][UPT][NH];
  auto load_batch = [&](int b) {
#pragma unroll
    for (int j = 0; j < T; ++j)
#pragma unroll
      for (int u = 0; u < UPT; ++u) {
        const int uu = b * UPT + u;
        const int k0 = kq0 + (uu << 8) + (g << 6);
        const bool ok = rowok[j] && uu < NC && k0 < K;
        const uint32_t off = ok ? rowoff[j] + (uint32_t)(FMT == FMT_W4 ? k0 / 2 : k0 / 4) : dev::kOutOfRange;
#pragma unroll
        for (int h = 0; h < NH; ++h) w[j][u][h] = dev::bload16(wrs, off + 16 * h);
      }
  };
  load_batch(0);

  // (3) activations into LDS
  if (!asum) dev::lds_barrier();   // the zeroed sums before any wave adds to them (weights stay in flight)
#pragma unroll
  for (int q = 0; q < kPre; ++q) {
    const int i = tid + 256 * q;
    const int m = i / per_row, j = i - m * per_row;
    if (i < M * per_row) *reinterpret_cast<uint4*>(act_l + m * Kpad + 16 * j) = apre[q];
  }
  for (int i = tid + 256 * kPre; i < M * per_row; i += 256) {
    const int m = i / per_row, j = i - m * per_row;
    *reinterpret_cast<uint4*>(act_l + m * Kpad + 16 * j) =
        *reinterpret_cast<const uint4*>(act + (int64_t)m * K + 16 * j);
  }
  if (asum == nullptr) {
    // sum_k q per token from the staged codes (each thread re-reads the pieces it staged itself; LDS
    // atomics into s_sum, zeroed before the barrier above)
    for (int i = tid; i < M * per_row; i += 256) {
      const int mm2 = i / per_row, j = i - mm2 * per_row;
      atomicAdd(&s_sum[mm2], sum16_i8(*reinterpret_cast<const uint4*>(act_l + mm2 * Kpad + 16 * j), 0));
    }
  }
  if (tid < M) {
    s_scale[tid] = sx_pre;
    if (asum) s_sum[tid] = sum_pre;
  }
  __syncthreads();

  // (4) MFMAs, batch by batch (one batch unless K > 4096 * UPT)
  v4i acc[T];
#pragma unroll
  for (int j = 0; j < T; ++j) acc[j] = v4i{0, 0, 0, 0};
  const int m = r16;
  const bool mok = m < M;
  const int8_t* arow = act_l + m * Kpad;
  for (int b = 0; b * UPT < NC; ++b) {
    if (b > 0) load_batch(b);
#pragma unroll
    for (int j = 0; j < T; ++j) {
#pragma unroll
      for (int u = 0; u < UPT; ++u) {
        const int uu = b * UPT + u;
        const int kb = kq0 + (uu << 8);
        if (uu >= NC || kb >= K) break;       // wave-uniform
        const int k0 = kb + (g << 6);
        const bool ok = mok && k0 < K;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
          uint4 bb = make_uint4(0, 0, 0, 0);
          if (ok) bb = *reinterpret_cast<const uint4*>(arow + k0 + 16 * s2);
          acc[j] = mfma_i8(decode_unit<FMT>(w[j][u], s2), v4i{(int)bb.x, (int)bb.y, (int)bb.z, (int)bb.w},
                           acc[j]);
        }
      }
    }
  }

  // (5) quarters of each tile meet in LDS; wave j mod 4 stores tile j
  v4i* red = reinterpret_cast<v4i*>(scratch);
#pragma unroll
  for (int j = 0; j < T; ++j) red[(j * 4 + wave) * 64 + lane] = acc[j];
  __syncthreads();
  for (int j = wave; j < T; j += 4) {
    v4i D = red[(j * 4) * 64 + lane];
#pragma unroll
    for (int q = 1; q < 4; ++q) D += red[(j * 4 + q) * 64 + lane];
    const int tile = tile0 + j;
    if (mok && tile * 16 < N) store4<FMT>(D, m, tile * 16 + 4 * g, N, s_scale[m], s_sum[m], sw, y, acc_out);
  }
}

// k per step of the prefill GEMM: every lane loads one 16-byte group of each of its weight rows per
// step (64 W2 or 32 W4 weights), i.e. S MFMA operands of 16 k per lane group
template <int FMT>
constexpr int gemm_ops() { return FMT == FMT_W4 ? 2 : 4; }
template <int FMT>
constexpr int gemm_bk() { return 64 * gemm_ops<FMT>(); }

// MFMA operand s of a lane's 16-byte weight group: 16 weights as int8 bytes in natural k order
template <int FMT>
__device__ __forceinline__ v4i gemm_operand(const uint4& u, int s) {
  if constexpr (FMT == FMT_W4) return s ? decode_w4(u.z, u.w) : decode_w4(u.x, u.y);
  else return decode_w2<FMT>(s == 0 ? u.x : s == 1 ? u.y : s == 2 ? u.z : u.w);
}

// ===========================================================================
// Prefill kernel: tiles of 256 weight rows x 16 TT tokens, BK-k steps (BK = 256 for W2, 128 for W4).
//
// Workgroup = 4 waves; wave w owns weight rows [64 w, +64) of the tile (4
// MFMA row tiles) and all tokens (TT column tiles): 4 TT int32 accumulator
// tiles.  Each wave reads its own packed weights straight into registers
// (one 16-byte load per lane per row tile and step: S MFMAs' worth of A
// operands) one step ahead, alternating between two register sets (the k
// loop is unrolled by two).  W4 steps over half as many k as W2, so both
// formats hold the same weight registers and a wave fits 3 per SIMD (OCC =
// 3: three workgroups per CU hide each other's load latency and barriers).
// The activation tile [16 TT][BK] int8 is double-buffered in LDS and filled
// one step ahead by direct-to-LDS buffer loads (no staging registers).  The
// tile has no row padding: the 16-byte column c of row r sits in slot
// c ^ (r mod SL) of the row (SL = BK / 16 slots), which spreads the rows an
// MFMA operand read touches over the banks.  The two buffers are distinct
// arrays, so the compiler can tell that the loads into one never alias the
// operand reads from the other and waits for them only at the end of the
// step.
// ===========================================================================
// With SUMQ (no per-token sums given) wave w also adds up the codes of token tiles t = w (mod 4): one
// more 16-byte LDS read and four dot products per MFMA operand step of its own tile(s).
// SPLIT (three stages only): workgroup z of the grid's third dimension takes the steps [z us, (z + 1) us)
// and writes its int32 accumulators to part [z][M][N rounded up to 4] (and, with SUMQ, workgroup column
// 0 its range's code sums to psum [z][M]) instead of the outputs.
template <int FMT, int OCC, int TT, bool SUMQ, int NS, bool SPLIT = false>
__global__ __launch_bounds__(256, OCC) void k_gemm(const uint32_t* __restrict__ P, const uint16_t* __restrict__ sw,
                                                   int N, int K, const int8_t* __restrict__ act,
                                                   const float* __restrict__ sx, const int32_t* __restrict__ asum,
                                                   int M, uint16_t* __restrict__ y, int32_t* __restrict__ acc_out,
                                                   int us = 0, int32_t* __restrict__ part = nullptr,
                                                   int32_t* __restrict__ psum = nullptr) {
  constexpr int S = gemm_ops<FMT>();
  constexpr int BK = gemm_bk<FMT>();
  constexpr int SL = BK / 16;            // 16-byte slots per activation row
  constexpr int RPC = 1024 / BK;         // activation rows per direct-to-LDS load (1 KB)
  constexpr int BM = 16 * TT;            // tokens per workgroup: every wave covers all of them
  constexpr int NQ = BM * BK / 4096;     // direct-to-LDS loads per wave and step
  static_assert(NQ >= 1 && RPC * SL == 64, "tile geometry");
  // two distinct arrays (not one indexed by the step's parity), so that the compiler can tell that
  // the direct-to-LDS loads into one never alias the operand reads from the other
  __shared__ __align__(16) int8_t lds0[BM * BK];
  __shared__ __align__(16) int8_t lds1[BM * BK];
  __shared__ __align__(16) int8_t lds2[NS == 3 ? BM * BK : 16];
  static_assert(NS == 2 || NS == 3, "pipeline depth");
  static_assert(!SPLIT || NS == 3, "a split runs three stages");
  constexpr int NL = NQ + 4;   // vector-memory loads a wave issues per step

  // the wave index as a scalar, so that the LDS destinations of the direct-to-LDS loads are scalar too
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int n_base = blockIdx.x * 256 + wave * 64;
  const int m_base = blockIdx.y * BM;
  const int64_t rowbytes = FMT == FMT_W4 ? (int64_t)K / 2 : (int64_t)K / 4;
  const int KA = (K + BK - 1) / BK;
  const int kt0 = SPLIT ? (int)blockIdx.z * us : 0;
  const int KT = SPLIT ? (kt0 + us < KA ? kt0 + us : KA) : KA;   // steps past this workgroup's range

  const __amdgpu_buffer_rsrc_t wrs = dev::make_rsrc(P, (uint32_t)(N * rowbytes));
  // Load offsets are a per-lane base (the out-of-range offset for rows past N, which stays out of
  // range with any step's k added) plus the step's k offset.  Lane group g of step kt covers
  // k = kt BK + (BK / 4) g .. + BK / 4 - 1: bytes 64 kt + 16 g .. + 15 of the row in either format.
  // In a last step past K the lanes beyond K read the next row (or zeros): their activations are
  // zero, so those weights add nothing.
  uint32_t wbase[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n_base + 16 * j + r16;
    wbase[j] = n < N ? (uint32_t)(n * rowbytes) + 16u * g : dev::kOutOfRange;
  }
  auto load_w = [&](uint4 (&w)[4], int kt) {
    const uint32_t ko = 64u * (uint32_t)kt;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = dev::bload16(wrs, wbase[j] + ko);
  };
  // activation tile of step kt into lds[buf]: wave w moves rows RPC NQ w .. RPC NQ (w + 1) - 1 (NQ loads
  // of 1 KB, RPC rows each; lane l of a load fills slot l of the kilobyte, i.e. row RPC q + l / SL,
  // slot l mod SL)
  const int mrows = M - m_base < BM ? M - m_base : BM;
  const __amdgpu_buffer_rsrc_t ars = dev::make_rsrc(act + (int64_t)m_base * K, (uint32_t)(mrows * K));
  uint32_t abase[NQ];   // row K + 16 col, or out of range for rows past M
  int acol[NQ];         // 16 col: the lane's k inside a step
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int row = RPC * (NQ * wave + q) + lane / SL;
    acol[q] = 16 * ((lane % SL) ^ (row % SL));
    abase[q] = row < mrows ? (uint32_t)(row * K + acol[q]) : dev::kOutOfRange;
  }
  auto issue_a = [&](int kt, int8_t* dst) {
    const int ko = kt * BK;
    const bool tail = ko + BK > K;   // the last step of a K that is not a multiple of BK
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int chunk = NQ * wave + q;
      uint32_t off = abase[q] + (uint32_t)ko;
      if (tail && acol[q] + ko >= K) off = dev::kOutOfRange;   // columns past K read as zeros
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ars, (__attribute__((address_space(3))) void*)(dst + 1024 * chunk), 16, off, 0, 0, 0);
    }
  };

  v4i acc[4][TT];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int t = 0; t < TT; ++t) acc[j][t] = v4i{0, 0, 0, 0};
  static_assert(TT % 4 == 0, "token tiles per wave for the sums");
  int sq[TT / 4];
#pragma unroll
  for (int t4 = 0; t4 < TT / 4; ++t4) sq[t4] = 0;

  // one step: prefetch step kt + NS - 1 (activations into pfb, weights into wpf), MFMAs of step kt from
  // tileb and wc; the k loop is unrolled by NS so the weight registers rotate instead of being copied.
  // MFMA s of lane group g covers k = kt BK + 16 (S g + s) .. + 15 (slot S g + s).
  // With three stages the prefetch is issued on every step, past K too (activation loads out of range,
  // weight loads of bytes no MFMA uses), so that every path issues the same loads and the compiler's
  // wait counts stay exact across the loop.
  auto step = [&](int kt, const int8_t* tileb, int8_t* pfb, const uint4 (&wc)[4], uint4 (&wpf)[4]) {
    const bool more = NS == 3 || kt + 1 < KT;
    if (more) {
      issue_a(kt + NS - 1, pfb);   // a buffer every wave finished reading before the last barrier
      load_w(wpf, kt + NS - 1);
    }
    // the loads stay ahead of the step's MFMAs (unguarded, the scheduler sinks them to the barrier)
    if constexpr (NS == 3) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < S; ++s) {
      v4i a[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) a[j] = gemm_operand<FMT>(wc[j], s);
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        const int row = 16 * t + r16;
        const uint4 bb = *reinterpret_cast<const uint4*>(&tileb[row * BK + 16 * ((S * g + s) ^ (row % SL))]);
        const v4i b = v4i{(int)bb.x, (int)bb.y, (int)bb.z, (int)bb.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j][t] = mfma_i8(a[j], b, acc[j][t]);
      }
      if constexpr (SUMQ) {
#pragma unroll
        for (int t4 = 0; t4 < TT / 4; ++t4) {
          const int row = 16 * (4 * t4 + wave) + r16;
          sq[t4] = sum16_i8(*reinterpret_cast<const uint4*>(&tileb[row * BK + 16 * ((S * g + s) ^ (row % SL))]),
                            sq[t4]);
        }
      }
    }
    // this wave's loads of step kt+1 have landed (vmcnt with lgkmcnt and expcnt untouched): with three
    // stages the NL loads of step kt+2 just issued may still be in flight
    if constexpr (NS == 3) {
      // a bare barrier (a workgroup fence would also wait for the loads of step kt+2 into LDS), after
      // this wave's operand reads of step kt have returned: the buffer is refilled from the next step on
      __builtin_amdgcn_s_waitcnt(0x0070 | NL);   // vmcnt(NL) lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
    } else {
      __builtin_amdgcn_s_waitcnt(0x0F70);
      __syncthreads();
    }
  };

  if constexpr (NS == 2) {
    uint4 wa[4], wb[4];
    issue_a(0, lds0);
    load_w(wa, 0);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
    for (int kt = 0; kt < KT; kt += 2) {
      step(kt, lds0, lds1, wa, wb);
      if (kt + 1 < KT) step(kt + 1, lds1, lds0, wb, wa);
    }
  } else {
    uint4 w0[4], w1[4], w2[4];
    issue_a(kt0, lds0);
    load_w(w0, kt0);
    issue_a(kt0 + 1, lds1);
    load_w(w1, kt0 + 1);
    __builtin_amdgcn_s_waitcnt(0x0F70 | NL);   // step 0's loads
    __syncthreads();
    // a loop body without conditions (the wait counts carried round the loop stay exact), then the
    // last one or two steps
    int kt = kt0;
    for (; kt + 3 <= KT; kt += 3) {
      step(kt, lds0, lds2, w0, w2);
      step(kt + 1, lds1, lds0, w1, w0);
      step(kt + 2, lds2, lds1, w2, w1);
    }
    if (kt < KT) step(kt, lds0, lds2, w0, w2);
    if (kt + 1 < KT) step(kt + 1, lds1, lds0, w1, w0);
    // the prefetches past K have landed before any buffer is reused
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
  }

  // per-token sums: the four lane groups of a token add up, then the waves exchange them through
  // the (now idle) first activation buffer
  int* s_q = reinterpret_cast<int*>(lds0);
  if constexpr (SUMQ) {
#pragma unroll
    for (int t4 = 0; t4 < TT / 4; ++t4) {
      int v = sq[t4];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) s_q[16 * (4 * t4 + wave) + lane] = v;
    }
    __syncthreads();
  }
  if constexpr (SPLIT) {
    const int np = (N + 3) & ~3;
#pragma unroll
    for (int t = 0; t < TT; ++t) {
      const int m = m_base + 16 * t + r16;
      if (m < M) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n0 = n_base + 16 * j + 4 * g;
          if (n0 < N)
            *reinterpret_cast<int4*>(part + ((size_t)blockIdx.z * M + m) * np + n0) =
                make_int4(acc[j][t][0], acc[j][t][1], acc[j][t][2], acc[j][t][3]);
        }
        if (SUMQ && blockIdx.x == 0 && wave == 0 && g == 0) psum[(size_t)blockIdx.z * M + m] = s_q[16 * t + r16];
      }
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < TT; ++t) {
    const int m = m_base + 16 * t + r16;
    if (m < M) {
      const float s_x = sx[m];
      const int sqm = SUMQ ? s_q[16 * t + r16] : asum[m];
#pragma unroll
      for (int j = 0; j < 4; ++j) store4<FMT>(acc[j][t], m, n_base + 16 * j + 4 * g, N, s_x, sqm, sw, y, acc_out);
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
// GEMM pipeline depth and workgroups per CU of the 256 x 64 tiles, per weight format.  W4 steps over
// 128 k (half the MFMAs of a W2 step), so one step ahead does not cover its loads: three stages at two
// workgroups per CU (M = 512: down 111 -> 72 us, gate|up 104 -> 90, q|k|v 36 -> 30; M = 2048 within
// 3 %).  W2 at three stages needs two workgroups per CU too, and loses more to that than it gains
// (gate|up at M = 2048 254 -> 285 us).
template <int FMT>
constexpr int gemm_stages() { return FMT == FMT_W4 ? 3 : 2; }
template <int FMT>
constexpr int gemm_occ() { return FMT == FMT_W4 ? 2 : 3; }
// Above 64 tokens with a workspace, where the 256 x 64 tiles are few (down at 65-512 tokens: 16 x
// ceil(M / 64) tiles, each a chain of 56 W2 or 112 W4 steps whose loads are not hidden), the GEMM is
// split over K at three stages and two workgroups per CU: S ranges of at least 4 W2 or 8 W4 steps
// (1024 k), about 512 workgroups and no more than are resident at once.  W2 (at 65 / 128 / 1024
// tokens): down 78.3 / 81.0 / 98.7 -> 19.6 / 23.8 / 63.1 us, q|k|v 35.1 -> 11.6 at 65, o 35.3 -> 11.1;
// it replaces the FP4 x FP6 kernel split the same way (down 25.4 / 29.4 / 80.3 us: the FP6 re-coding
// is a launch of its own).  W4 takes at least three ranges (two measured no faster: gate|up at 128
// tokens 31.1 -> 33.4 us, q|k|v at 512 30.0 -> 32.4): down at 65 / 128 / 512 tokens 71.9 / 72.5 /
// 74.8 -> 22.1 / 25.0 / 46.6 us, q|k|v and o at 65 26.6 -> 11.3 / 10.9.
// From 33 tokens on, a wide linear (N >= 16384: gate|up) or a long one (N >= 4096, K > 4096: down)
// takes the split GEMM instead of the skinny kernel, whose workgroups each read all M x K codes
// (gate|up at 33 / 64 tokens, W2 22.9 / 27.6 -> 18.6 / 24.3 us, W4 35.3 / 45.2 -> 22.4 / 27.0; down,
// W2 12.7 / 16.1 -> 11.6 / 15.3, W4 21.6 / 30.5 -> 14.8 / 17.6).  Smaller linears lose: W2 q|k|v at 33
// tokens 8.2 -> 10.1, 1000 x 14336 at 64 11.0 -> 12.8.  W4, whose skinny kernel reads twice the weight
// bytes, from 24 tokens on (at 32: down 18.3 -> 14.4, gate|up 25.9 -> 22.0; at 24 a 22016-row gate|up
// loses 17.8 -> 18.6 while the others gain 1.2-2.7 us).
constexpr int64_t kSplitTarget = 512, kSplitResident = 512, kSplitWideMinM = 33, kSplitWideMinMW4 = 24,
                  kSplitWideMinN = 16384,
                  kSplitLongMinN = 4096, kSplitLongMinK = 4097;
struct GemmSplit {
  int S = 1, us = 0;
};
inline GemmSplit gemm_split_plan(int fmt, int64_t N, int64_t M, int64_t K) {
  GemmSplit p;
  const int64_t bk = fmt == FMT_W4 ? 128 : 256, min_steps = fmt == FMT_W4 ? 8 : 4, min_s = fmt == FMT_W4 ? 3 : 2;
  const int64_t tiles = ((N + 255) / 256) * ((M + 63) / 64), KT = (K + bk - 1) / bk;
  p.us = (int)KT;
  const bool wide = M >= (fmt == FMT_W4 ? kSplitWideMinMW4 : kSplitWideMinM) &&
                    (N >= kSplitWideMinN || (N >= kSplitLongMinN && K >= kSplitLongMinK));
  if (M < kGemmF4MinM && !wide) return p;
  int64_t S = (kSplitTarget + tiles - 1) / tiles;
  if (S > kSplitResident / tiles) S = kSplitResident / tiles;
  if (S > KT / min_steps) S = KT / min_steps;
  if (S < min_s) return p;
  p.us = (int)((KT + S - 1) / S);
  p.S = (int)((KT + p.us - 1) / p.us);
  return p;
}

template <int FMT, bool SUMQ>
hipError_t launch_gemm_split(const GemmSplit& p, const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K,
                           const int8_t* act, const float* sx, const int32_t* asum, int64_t M, uint16_t* y,
                           int32_t* acc_out, void* ws, hipStream_t s) {
  int32_t* part = static_cast<int32_t*>(ws);
  int32_t* psum = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(ws) + split::part_bytes(p.S, M, N));
  const dim3 grid((unsigned)((N + 255) / 256), (unsigned)((M + 63) / 64), (unsigned)p.S);
  hipLaunchKernelGGL((k_gemm<FMT, 2, 4, SUMQ, 3, true>), grid, dim3(256), 0, s, P, sw, (int)N,
                     (int)K, act, sx, asum, (int)M, y, acc_out, p.us, part, psum);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // code sums of range z at psum[z M + m]
  return split::launch_sum<FMT>(part, p.S, M, N, sx, asum, psum, p.S, 1, (int)M, sw, y, acc_out, s);
}

constexpr int kDecodeMaxLds = 96 * 1024;   // activation bytes staged in LDS by the decode kernel
constexpr int kDecodeGrid = 512;           // workgroups of the decode kernel (2 per CU)

inline int kpad_of(int64_t K) { return (int)K + 16; }

template <int FMT>
hipError_t launch_decode(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                         const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                         hipStream_t s) {
  const int ntiles = (int)((N + 15) / 16);
  const int grid = ntiles < kDecodeGrid ? ntiles : kDecodeGrid;
  hipLaunchKernelGGL((k_decode<FMT>), dim3(grid), dim3(256), 0, s, P, sw, (int)N, (int)K, act, sx, asum, (int)M,
                     y, acc_out);
  return hipGetLastError();
}

template <int FMT, int T, int UPT>
hipError_t launch_deep_t(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                         const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                         hipStream_t s) {
  const int Kpad = kpad_of(K);
  const int ntiles = (int)((N + 15) / 16);
  const int grid = (ntiles + T - 1) / T;
  constexpr int kRed = 4 * T * 64 * 16;
  const size_t shmem = (size_t)((((int)M * Kpad) + 15) & ~15) + kRed + 16 * 4 + 16 * 4;
  if (shmem > 65536) {
    // opt in to more than 64 KiB of dynamic LDS (gfx950 has 160 KiB per workgroup)
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_decode_deep<FMT, T, UPT>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
  }
  hipLaunchKernelGGL((k_decode_deep<FMT, T, UPT>), dim3(grid), dim3(256), shmem, s, P, sw, (int)N, (int)K, act,
                     sx, asum, (int)M, Kpad, y, acc_out);
  return hipGetLastError();
}

// K <= 4096: 4 units per wave and tile, T tiles per workgroup (as many as keep the grid within one
// workgroup per CU, up to 6).  Longer K: one tile per workgroup and up to 16 (W4: 8) units per batch.
template <int FMT>
hipError_t launch_deep(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                       const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out,
                       hipStream_t s) {
#define QIFT_DEEP(TT, UU) launch_deep_t<FMT, TT, UU>(P, sw, N, K, act, sx, asum, M, y, acc_out, s)
  if (K <= 4096) {
    const int64_t ntiles = (N + 15) / 16;
    const int64_t t = (ntiles + 255) / 256;
    if (t <= 1) return QIFT_DEEP(1, 4);
    if (t == 2) return QIFT_DEEP(2, 4);
    if (t == 3) return QIFT_DEEP(3, 4);
    if (t == 4) return QIFT_DEEP(4, 4);
    if (t == 5) return QIFT_DEEP(5, 4);
    return QIFT_DEEP(6, 4);
  }
  if constexpr (FMT == FMT_W4) return QIFT_DEEP(1, 8);
  else return QIFT_DEEP(1, 16);
#undef QIFT_DEEP
}

template <int FMT>
hipError_t launch_fmt(const uint32_t* P, const uint16_t* sw, int64_t N, int64_t K, const int8_t* act,
                      const float* sx, const int32_t* asum, int64_t M, uint16_t* y, int32_t* acc_out, void* ws,
                      hipStream_t s) {
  // with a workspace the GEMM split over K where that applies (above 64 tokens, or a wide or long linear
  // from 33 on), else above 64 tokens for W2 the FP4 x FP6 kernel
  if (ws) {
    const GemmSplit p = gemm_split_plan(FMT, N, M, K);
    if (p.S > 1)
      return asum ? launch_gemm_split<FMT, false>(p, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s)
                  : launch_gemm_split<FMT, true>(p, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s);
    if constexpr (FMT != FMT_W4) {
      if (M >= kGemmF4MinM) return launch_gemm_f4(FMT, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s);
    }
  }
  // 17..64 tokens: the skinny kernel, one pass over the weights (the codes of that many tokens do not
  // fit the decode kernel's LDS, and the GEMM's grid of N/256 workgroups would leave most CUs idle)
  if (M > kCodesMaxM && M <= kSkinnyMaxM && K <= kSkinnyMaxK)
    return launch_skinny_ws(FMT, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s);
  if (M <= kCodesMaxM) {
    // the decode kernel on precomputed codes (K-slice weight waves, the codes staged in LDS)
    const size_t cs = FMT == FMT_MNZ ? codes_shmem_mnz(M, N, K) : FMT == FMT_POT ? codes_shmem_pot(M, N, K)
                                                                                  : codes_shmem_w4(M, N, K);
    if (cs != 0 && cs <= 160 * 1024) {
      if constexpr (FMT == FMT_MNZ) return launch_codes_mnz(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
      else if constexpr (FMT == FMT_POT) return launch_codes_pot(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
      else return launch_codes_w4(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
    }
    // codes beyond LDS (e.g. 16 tokens of K = 14336): with a workspace the skinny linear split over K;
    // else the decode kernels that read them from memory (measured faster there than the skinny
    // kernel unsplit with one token tile: 16 tokens at K = 14336)
    if constexpr (FMT != FMT_W4) {
      if (ws && skinny_workspace(FMT, N, K, M) != 0)
        return launch_skinny_ws(FMT, P, sw, N, K, act, sx, asum, M, y, acc_out, ws, s);
    }
    if (M * kpad_of(K) <= kDecodeMaxLds) return launch_deep<FMT>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
    return launch_decode<FMT>(P, sw, N, K, act, sx, asum, M, y, acc_out, s);
  }
  const unsigned gx = (unsigned)((N + 255) / 256);
  // 256 x 64 tiles (gemm_occ, gemm_stages).  W4 on grids that fill the chip at least twice over with
  // 256 x 128 tiles (two per CU) takes those instead: half the weight loads and decode per MFMA
  // (stacked gate|up at M = 2048: 318 -> 264 us).  W2 does not gain from them (222 -> 225 us), and
  // smaller grids lose to the idle CUs (q,k,v W4 74 -> 78 us).  Also measured slower at M = 2048: 256 x 32 tiles and activations staged through
  // registers.
  if constexpr (FMT == FMT_W4) {
    const unsigned gy8 = (unsigned)((M + 127) / 128);
    if ((uint64_t)gx * gy8 >= 1024) {
      if (asum)
        hipLaunchKernelGGL((k_gemm<FMT, 2, 8, false, 2>), dim3(gx, gy8), dim3(256), 0, s, P, sw, (int)N, (int)K, act, sx,
                           asum, (int)M, y, acc_out);
      else
        hipLaunchKernelGGL((k_gemm<FMT, 2, 8, true, 2>), dim3(gx, gy8), dim3(256), 0, s, P, sw, (int)N, (int)K, act, sx,
                           asum, (int)M, y, acc_out);
      return hipGetLastError();
    }
  }
  const dim3 grid(gx, (unsigned)((M + 63) / 64));
  if (asum)
    hipLaunchKernelGGL((k_gemm<FMT, gemm_occ<FMT>(), 4, false, gemm_stages<FMT>()>), grid, dim3(256), 0, s, P, sw, (int)N, (int)K, act, sx, asum, (int)M,
                       y, acc_out);
  else
    hipLaunchKernelGGL((k_gemm<FMT, gemm_occ<FMT>(), 4, true, gemm_stages<FMT>()>), grid, dim3(256), 0, s, P, sw, (int)N, (int)K, act, sx, asum, (int)M,
                       y, acc_out);
  return hipGetLastError();
}

}  // namespace

size_t gemm_split_workspace(int fmt, int64_t N, int64_t M, int64_t K) {
  const GemmSplit p = gemm_split_plan(fmt, N, M, K);
  return p.S > 1 ? split::part_bytes(p.S, M, N) + (size_t)p.S * (size_t)M * 4 : 0;
}

hipError_t launch_linear(int fmt, const uint32_t* packed, const uint16_t* scales, int64_t N, int64_t K,
                         const int8_t* act_q, const float* act_scale, const int32_t* act_sum, int64_t M,
                         uint16_t* out, int32_t* acc_out, void* ws, hipStream_t s) {
  switch (fmt) {
    case FMT_MNZ:
      return launch_fmt<FMT_MNZ>(packed, scales, N, K, act_q, act_scale, act_sum, M, out, acc_out, ws, s);
    case FMT_POT:
      return launch_fmt<FMT_POT>(packed, scales, N, K, act_q, act_scale, act_sum, M, out, acc_out, ws, s);
    case FMT_W4:
      return launch_fmt<FMT_W4>(packed, scales, N, K, act_q, act_scale, act_sum, M, out, acc_out, ws, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qift
