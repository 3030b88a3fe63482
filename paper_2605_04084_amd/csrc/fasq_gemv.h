// Decode GEMV for M <= 16 tokens: y[m, n] = sum_s dot(x[m, s*d:(s+1)*d], codebook[u(n, s)]).
//
// Design (gfx950, wave64, v_mfma_f32_16x16x32_f16):
//   * A wave computes 16 output rows at a time.  Lane l owns output row
//     n = l % 16 and K group g = l / 16: it streams the packed ids of row n
//     in 16-byte chunks (12 bytes for 12-bit ids), gathers the codewords of
//     eight consecutive K values straight into the MFMA B operand, and the
//     matrix core does the dot products with x (A operand, read from LDS)
//     and the sum over the four K groups.  No VALU work is spent on
//     products; the per-id VALU cost is the id decode and the LDS address.
//   * The four groups of a row read four consecutive chunks, so one
//     wave-wide load reads 16 rows x 64 contiguous bytes.  Inside a chunk the
//     K order is permuted identically for A and B (the contraction is a sum
//     over K), which is what lets a lane consume its ids in stream order.
//   * A row's chunks are split into P parts, one per wave of the workgroup
//     (split-K inside the workgroup); each wave covers T chunk columns per
//     lane.  Partials go to LDS and are summed over the P waves in a fixed
//     order after one barrier: deterministic, no atomics, no workspace.
//   * Every wave runs a software pipeline that keeps kGemvPipe - 1 chunk
//     loads in flight, so the index stream keeps HBM busy while earlier
//     chunks are decoded.  Loads are unconditional (clamped addresses) so
//     the compiler can count outstanding loads exactly.
//   * The codebook (replicated per lane slot when small) and x are staged in
//     LDS once per workgroup before any index load is issued: the vector L1
//     returns data in order, so L2-resident loads queued behind HBM loads
//     would wait for them.
#pragma once

#include <type_traits>

#include "fasq_codebook.h"
#include "fasq_device.h"
#include "fasq_internal.h"

namespace fasq {

// One part of a k_gemv launch: a range of rows of one matrix.  Grid row
// blockIdx.y works on part blockIdx.y; every part has gridDim.x workgroups.
struct GemvPart {
  const uint8_t* idx;  // id row of the part's first row
  const half_t* cb;
  half_t* y;           // output of the part's first row, token 0
  int64_t N;           // rows of the part
  int64_t ldy;         // elements between the outputs of consecutive tokens
  int C;
  int nsl;             // codebook slices; k_gemv takes one (the whole codebook)
  int64_t ws_row;      // K split: the partials of the part's first row are at ws + ws_row
};

constexpr int kGemvMaxParts = 8;  // parts one k_gemv launch can take

struct GemvArgs {
  const half_t* x;
  int64_t M, K;
  int64_t R;   // bytes per row (= CH * chunk bytes)
  int64_t CH;  // chunks per row
  int CHS;       // chunks per x slab (a multiple of 4; CH when x is staged whole)
  int nslab;     // x slabs: ceil(CH / CHS)
  int P;         // waves per row (K split inside the workgroup)
  int TW;        // 16-row tiles per workgroup, a multiple of waves / P
  int cb_bytes;  // LDS bytes of the codebook (x follows)
  int xs;        // LDS bytes between rows of x
  int x_bytes;   // LDS bytes of x (partials follow)
  int sl_shift;  // CB_SLICE: log2 of the entries of the one LDS slice (at least C)
  int head;      // CB_SPLIT: entries staged in LDS (the rest are read from global memory)
  // K split over workgroups (gridDim.z segments of seg_slabs slabs each):
  // segment z writes its fp32 partial of (token m, row n) to
  // ws[(z * M + m) * ld_ws + part.ws_row + n]; one segment writes y itself.
  int seg_slabs;
  float* ws;
  int64_t ld_ws;
  // 1 (K split with one slab per segment and many tokens, or a codebook head
  // in LDS): the partials of each round of tiles (tile j of every row group)
  // are summed and written as soon as the round is done, so LDS holds one
  // round's partials instead of every tile's
  int round_sum;
  GemvPart part[kGemvMaxParts];
};

constexpr int kGemvPipe = 8;      // load units per wave in the software pipeline
// Floats between the partial sums of consecutive (row, token) pairs in the
// 16-row-tile kernel's LDS buffer, which holds P per pair (one per wave of a
// row).  An odd stride for P > 1: with a stride of P = 16 floats the 64
// lanes of a wave that write one MFMA result (16 rows x 4 tokens) hit one
// or two banks when M is even, and the final sum's reads hit one.
__host__ __device__ constexpr int gemv_red_stride(int P) { return P > 1 ? P + 1 : 1; }
constexpr int kGemvSlabPipe = 4;  // the same with x in slabs
// Index loads each single-token wave keeps in flight.  Two per wave (32 KB
// per CU at 16 waves) already saturate a CU's share of HBM; more only make
// waves wait at the issue of loads that cannot enter the queue, where they
// cannot compute the data that has arrived.
constexpr int kM1Window = 2;
// Index loads a wave issues before the staging barrier (at least the window):
// the first ones keep the CU's memory queue busy while the codebook and x
// are staged.
constexpr int kM1EarlyLoads = 2;
static_assert(kM1Window <= kM1EarlyLoads && kM1EarlyLoads <= kGemvPipe, "early loads must cover the window");
constexpr int kXWordsPerThread = 8;  // first-round x words (16 B) per thread for M > 1
constexpr int kXSlabBatch = 4;       // x words (16 B) in flight per thread when a later slab is staged

// MR: token slots (16: one 16-row A tile of x per MFMA).
// x slabs: when M rows of x are too long for LDS, K is walked in slabs of
// CHS chunk columns; x is staged one slab at a time and every row's partial
// sums are carried across the slabs in LDS (added in slab order by the same
// lane, so the result stays deterministic).
// MASK: some lanes see chunk columns past the end of their slab or row; their
// operands are zeroed.  SLAB: x is staged in slabs (always with MASK); the
// slab loop keeps more state live, so these variants run a shallower
// pipeline (kGemvSlabPipe loads) to stay within the registers of 16 waves.
template <int BITS, int D, int T, int MODE, int MR, bool MASK, bool SLAB>
__global__ __launch_bounds__(1024) void k_gemv(GemvArgs a) {
  constexpr int G = Chunk<BITS>::G;      // ids per chunk
  constexpr int DW = Chunk<BITS>::DW;    // dwords per chunk
  constexpr int CBY = DW * 4;            // chunk bytes
  constexpr int SPC = G * D / 8;         // MFMA steps (8 K values each) per chunk
  constexpr int XCB = G * D * 2;         // bytes of x per chunk column and token
  constexpr int L = SLAB ? (T > kGemvSlabPipe ? T : kGemvSlabPipe) : kGemvPipe;
  static_assert(L % T == 0, "pipeline depth must be a multiple of T");
  static_assert(MR == 16, "16 token slots");
  static_assert(!SLAB || MASK, "slabs take the column checks");

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint8_t* xl = smem + a.cb_bytes;
  float* red = reinterpret_cast<float*>(smem + a.cb_bytes + a.x_bytes);  // [RW][M][PS], P used of each PS
  const GemvPart& pt = a.part[blockIdx.y];  // the rows this workgroup works on

  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int P = a.P;
  const int PS = gemv_red_stride(P);
  const int Q = (blockDim.x / kWave) / P;
  const int p = wave % P;
  const int q = wave / P;
  const int g = lane >> 4;    // K group
  const int nl = lane & 15;   // row within a 16-row tile
  const int M = (int)a.M;
  // Row tiles are dealt to workgroups round-robin (tile j of workgroup w is
  // global tile w + j * gridDim.x), so that at any moment the tiles being
  // streamed form one contiguous stretch of the table and load every HBM
  // channel; a block per workgroup would put all streams at the same
  // offset within equal-sized blocks.  Wave q takes local tiles q, q + Q, ...
  const int nrt = a.TW / Q;                // row tiles of this wave
  const int nunits = nrt * T;

  // chunk column of (t) within the slab: raw, and clamped for loads
  const int CH = (int)a.CH;
  auto ccol_raw = [&](int t) { return (p * T + t) * 4 + g; };

  // Units past the end of this wave's work, and rows past N, load the first
  // chunk of the table (one address for the whole wave: a single request) so
  // that every iteration issues exactly one load and the waits stay exact.
  // Byte offsets into the index table are 32-bit (the host checks that the
  // table is below 4 GiB) from one uniform base.
  auto tile_of = [&](int rt) { return (int64_t)blockIdx.x + (int64_t)(rt * Q + q) * gridDim.x; };
  const uint32_t lane_off0 = (uint32_t)(nl * a.R);
  const uint32_t tile_stride = (uint32_t)(16 * a.R);
  uint32_t buf[L][DW];
  // the slabs of this workgroup's K segment: [sb0, sb1)
  const int sb0 = SLAB ? (int)blockIdx.z * a.seg_slabs : 0;
  const int sb1 = SLAB ? (sb0 + a.seg_slabs < a.nslab ? sb0 + a.seg_slabs : a.nslab) : 1;
  int c0 = sb0 * a.CHS, chs = CH;  // the slab: chunk columns [c0, c0 + chs)
  // byte offset of the lane's chunk in column t of the slab within its row,
  // or ~0 for columns past the slab (set per slab)
  uint32_t col_off[T];
  auto set_cols = [&]() {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int c = ccol_raw(t);
      col_off[t] = (!MASK || c < chs) ? (uint32_t)(c0 + c) * CBY : ~0u;
    }
  };
  auto load_unit = [&](int slot, int u, int t) {
    const int64_t tile = tile_of(u / T);
    const bool live = u < nunits && tile * 16 + nl < pt.N && (!MASK || col_off[t] != ~0u);
    const uint32_t off = (uint32_t)tile * tile_stride + lane_off0 + col_off[t];
    load_chunk<BITS>(pt.idx + (live ? off : 0u), buf[slot]);
  };

  // ---- prologue.  The vector L1 returns loads in order, so an L2-resident
  // load queued behind HBM loads waits for them.  All waves of the
  // workgroup (the only one on its CU) issue their codebook and x loads,
  // meet at a barrier (which does not wait for memory), and only then issue
  // the first index loads: the codebook and x come back first while the
  // index stream is already in flight.
  const uint32_t lane_off = repl_lane_off<D>(lane);
  // A operands (x) live in registers when they fit (x staged whole, no
  // masked columns), loaded straight from global memory with the codebook
  // (x takes no LDS then); else x is staged in LDS, a slab at a time, and
  // read at every step.  Rows of A past M repeat a real row.
  constexpr bool kXInRegs = !MASK && T * SPC <= 8;
  const int mrow = nl < M ? nl : M - 1;  // x row this lane feeds to the A operand
  const uint8_t* xrow = xl + mrow * a.xs;
  half8_t xreg[kXInRegs ? T * SPC : 1];
  Slice sl;
  const half_t* scb = pt.cb;
  int sC = pt.C;
  if constexpr (MODE == CB_SLICE) {
    sl.base = 0;
    sl.mask = (1u << a.sl_shift) - 1u;
  } else if constexpr (MODE == CB_SPLIT) {
    sl.mask = (uint32_t)a.head - 1u;
    sC = a.head;
  }
  constexpr bool kStageSlice = MODE == CB_SLICE || MODE == CB_SPLIT;

  // x words (16 B) of the current slab: token m, slab-local word w of wpr
  auto x_word_src = [&](int w, int wpr) {
    const int m = w / wpr;
    return reinterpret_cast<const u32x4*>(a.x + (int64_t)m * a.K + (int64_t)c0 * (G * D)) + (w - m * wpr);
  };
  auto x_word_dst = [&](int w, int wpr) {
    const int m = w / wpr;
    return reinterpret_cast<u32x4*>(xl + m * a.xs + (w - m * wpr) * 16);
  };


  chs = CH - c0 < a.CHS ? CH - c0 : a.CHS;
  set_cols();
  {
    // codebook and the first slab of x (or x in registers)
    const int wpr = chs * XCB / 16;  // x words per token in this slab
    const int xw_total = wpr * M;
    CbStage cst;
    if constexpr (kStageSlice) slice_fetch(scb, sC * D * 2 / 16, cst);
    else cb_fetch<D, MODE>(pt.cb, pt.C, cst);
    u32x4 xst[kXInRegs ? 1 : kXWordsPerThread];
    if constexpr (kXInRegs) {
      const half_t* xg = a.x + (int64_t)mrow * a.K;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int c = ccol_raw(t) < CH ? ccol_raw(t) : CH - 1;
#pragma unroll
        for (int s = 0; s < SPC; ++s) xreg[t * SPC + s] = *reinterpret_cast<const half8_t*>(xg + c * (G * D) + s * 8);
      }
    } else {
#pragma unroll
      for (int k = 0; k < kXWordsPerThread; ++k) {
        int w = threadIdx.x + k * blockDim.x;
        w = w < xw_total ? w : xw_total - 1;
        xst[k] = *x_word_src(w, wpr);
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < L - 1; ++i) load_unit(i, i, i % T);

    if constexpr (kStageSlice) slice_store(smem, scb, sC * D * 2 / 16, cst);
    else cb_store<D, MODE>(smem, pt.cb, pt.C, cst);
    if constexpr (!kXInRegs) {
#pragma unroll
      for (int k = 0; k < kXWordsPerThread; ++k) {
        const int w = threadIdx.x + k * blockDim.x;
        if (w < xw_total) *x_word_dst(w, wpr) = xst[k];
      }
      for (int w = threadIdx.x + kXWordsPerThread * blockDim.x; w < xw_total; w += blockDim.x)
        *x_word_dst(w, wpr) = *x_word_src(w, wpr);
    }
    __syncthreads();
  }

  const bool rounds = (SLAB || MODE == CB_SPLIT) && a.round_sum != 0;
  // fixed-order sum over the P waves of the partials of the workgroup's
  // local rows [r0, r0 + nr) (LDS rows from lr0), one fp16 rounding, or one
  // fp32 partial of this K segment; consecutive threads take consecutive
  // (row, token) pairs, whose partials lie an odd stride apart in LDS
  auto sum_rows = [&](int r0, int lr0, int nr) {
    const int outs = nr * M;
    for (int o = threadIdx.x; o < outs; o += blockDim.x) {
      const int rr = o / M;
      const int m = o - rr * M;
      const int r = r0 + rr;
      const int64_t n = ((int64_t)blockIdx.x + (int64_t)(r / 16) * gridDim.x) * 16 + (r & 15);
      if (n < pt.N) {
        float sum = 0.f;
        const float* pr = red + ((lr0 + rr) * M + m) * PS;
        for (int pp = 0; pp < P; ++pp) sum += pr[pp];
        if (SLAB && gridDim.z > 1) a.ws[((int64_t)blockIdx.z * M + m) * a.ld_ws + pt.ws_row + n] = sum;
        else pt.y[(int64_t)m * pt.ldy + n] = static_cast<half_t>(sum);
      }
    }
  };

  for (int sb = sb0; sb < sb1; ++sb) {
    if (sb > sb0) {
      // the next slab: every wave is done with the previous slab's x; its
      // first index loads go out, then x is staged in batches of
      // kXSlabBatch words per thread
      c0 = sb * a.CHS;
      chs = CH - c0 < a.CHS ? CH - c0 : a.CHS;
      set_cols();
      const int wpr = chs * XCB / 16;
      const int xw_total = wpr * M;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < L - 1; ++i) load_unit(i, i, i % T);
      for (int base = threadIdx.x; base < xw_total; base += kXSlabBatch * blockDim.x) {
        u32x4 v[kXSlabBatch];
#pragma unroll
        for (int k = 0; k < kXSlabBatch; ++k) {
          const int w = base + k * blockDim.x;
          v[k] = *x_word_src(w < xw_total ? w : xw_total - 1, wpr);
        }
#pragma unroll
        for (int k = 0; k < kXSlabBatch; ++k) {
          const int w = base + k * blockDim.x;
          if (w < xw_total) *x_word_dst(w, wpr) = v[k];
        }
      }
      __syncthreads();
    }

    float4_t acc0 = {0.f, 0.f, 0.f, 0.f};
    float4_t acc1 = {0.f, 0.f, 0.f, 0.f};

    for (int base = 0; base < nunits; base += L) {
#pragma unroll
      for (int i = 0; i < L; ++i) {
        const int u = base + i;
        const int t = i % T;
        load_unit((i + L - 1) % L, u + L - 1, (i + L - 1) % T);
        if (u < nunits) {
          const uint32_t* w = buf[i];
          const int c = ccol_raw(t);
          const bool cval = !MASK || c < chs;
          const uint8_t* xa = xrow + (cval ? c : 0) * XCB;
#pragma unroll
          for (int s = 0; s < SPC; ++s) {
            half8_t bop = gather8<BITS, D, MODE>(pt.cb, lane_off, w, s * (8 / D), sl);
            half8_t aop;
            if constexpr (kXInRegs) aop = xreg[t * SPC + s];
            else aop = *reinterpret_cast<const half8_t*>(xa + s * 16);
            if (!cval) {
              bop = half8_t{};
              aop = half8_t{};
            }
            if (s & 1) acc1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, acc1, 0, 0, 0);
            else acc0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, acc0, 0, 0, 0);
          }
          if (t == T - 1) {
            // lane l holds rows m = 4g .. 4g + 3 of column nl of the 16 x 16
            // tile; the slabs of a row are summed in slab order by this lane
            const int lrow = ((rounds ? 0 : u / T) * Q + q) * 16 + nl;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int m = 4 * g + k;
              if (m < M) {
                float* r = &red[(lrow * M + m) * PS + p];
                *r = sb > sb0 ? *r + (acc0[k] + acc1[k]) : acc0[k] + acc1[k];
              }
            }
            acc0 = float4_t{0.f, 0.f, 0.f, 0.f};
            acc1 = float4_t{0.f, 0.f, 0.f, 0.f};
          }
        }
        // a round of tiles done (the condition is the same in every wave:
        // all waves have the same units): sum it while the next round's
        // loads are in flight
        if (rounds && t == T - 1 && u < nunits) {
          __syncthreads();
          sum_rows((u / T) * Q * 16, 0, Q * 16);
          __syncthreads();
        }
      }
    }
  }
  if (rounds) return;
  __syncthreads();
  sum_rows(0, 0, a.TW * 16);
}

}  // namespace fasq

namespace fasq {

// ---------------------------------------------------------------------------
// One or two tokens (M <= 2).  Reading 16 rows x 64 bytes per wave-wide load
// (the layout above) streams at well under half the rate of reading 1 KB of
// one row, so the row-streaming kernels map the MFMA differently: lane l of a
// wave-wide load holds chunk l of a 1 KB span of ONE weight row (lanes in
// address order, so every quarter-wave reads 256 contiguous bytes), and the
// A operand's "row" i is the set of chunks {i, i + 16, i + 32, i + 48} (K
// group g = chunk / 16).  B carries the x slice of each lane's own chunk, so
// the wanted partial sums are the diagonal of the 16 x 16 result (one MFMA
// per token).  The matrix core does 16x the useful MACs, which it has to
// spare at decode arithmetic intensity.
// ---------------------------------------------------------------------------
// One part of a row-streaming launch: a range of rows of one matrix (its ids,
// its codebook, its outputs).  Grid row blockIdx.y works on part blockIdx.y;
// every part has gridDim.x workgroups.
struct GemvM1Part {
  const uint8_t* idx;  // first id row of the part
  const half_t* cb;
  half_t* y;           // output of the part's first row (token 0)
  int64_t N;           // rows of the part
  int64_t ldy;         // elements between the outputs of consecutive tokens
  int C;
  int nsl;  // CB_SLICE: codebook slices (passes over the rows)
};

constexpr int kM1MaxParts = 8;   // parts one row-streaming launch can take
// x slices (16-byte words per lane) the one-token row-streaming kernel keeps
// in registers; more are read from LDS at every unit.  The two-token kernel
// keeps up to twice as many (it then has no other large state).
constexpr int kRowsXRegs = 8;
// Small one-token launches store each row sum from the wave that computed
// it (1), or all through LDS after a final barrier (0): a build-time switch
// for measuring the two against each other.
#ifndef FASQ_M1_DIRECT_STORE
#define FASQ_M1_DIRECT_STORE 1
#endif
constexpr bool kM1DirectStore = FASQ_M1_DIRECT_STORE != 0;

// Products of the row-streaming kernels: packed fp16 dot products on the
// vector ALU (1), or the diagonal of a 16 x 16 MFMA per token (0).
#ifndef FASQ_DECODE_DOT
#define FASQ_DECODE_DOT 1
#endif
constexpr bool kDecodeDot = FASQ_DECODE_DOT != 0;

struct GemvM1Args {
  const half_t* x;  // shared by every matrix of the launch
  int64_t K;
  int64_t R;     // bytes per row (= CH * chunk bytes)
  int64_t CH;    // chunks per row
  int P;         // waves per row (K split inside the workgroup)
  int NRW;       // rows per row group
  int cb_bytes;  // LDS bytes of the codebook (x follows)
  int x_bytes;   // LDS bytes of x (partials follow)
  int sl_shift;  // CB_SLICE: log2 of the entries per slice
  int wpp;       // workgroups per part (the grid's x size)
  int M;         // tokens (rows of x), at most the kernel's MT
  GemvM1Part part[kM1MaxParts];
};

// The body of the row-streaming decode kernel for MT token slots: x holds
// M <= MT rows (the others are zeros), and every codeword gathered feeds MT
// diagonal MFMAs, one per token.  k_gemv_m1 is the one-token kernel,
// k_gemv_mt the kernel for two tokens.
template <int BITS, int D, int T, int MODE, bool MASK, int MT>
__device__ __forceinline__ void gemv_rows_body(const GemvM1Args& a) {
  constexpr int G = Chunk<BITS>::G;
  constexpr int DW = Chunk<BITS>::DW;
  constexpr int CBY = DW * 4;
  constexpr int SPC = G * D / 8;     // MFMA steps per chunk
  static_assert(MT == 1 || MODE != CB_SLICE, "sliced codebooks take one token");
  // load slots: the sliced-codebook kernel keeps fewer (its extra state would
  // otherwise spill), the others a full pipeline's worth
  constexpr int L = MODE == CB_SLICE ? (T > 4 ? T : 4) : kGemvPipe;
  static_assert(L % T == 0, "pipeline depth must be a multiple of T");
  constexpr bool kXInRegs = MT * T * SPC <= kRowsXRegs * (MT > 1 ? 2 : 1);

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  // The part of this workgroup comes from the grid position alone, so its
  // arguments load in the same batch as the others: choosing it by the
  // value of an argument would cost one more memory round trip before the
  // first index load.
  const GemvM1Part& pt = a.part[blockIdx.y];
  const uint8_t* __restrict__ idx = pt.idx;
  const half_t* __restrict__ cb = pt.cb;
  half_t* __restrict__ y = pt.y;
  const int64_t N = pt.N;
  const int C = pt.C;
  const uint32_t wg = blockIdx.x;
  const uint32_t nwg = (uint32_t)a.wpp;

  uint8_t* xl = smem + a.cb_bytes;
  float* red = reinterpret_cast<float*>(smem + a.cb_bytes + a.x_bytes);  // [Q * NRW][MT][P]

  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int P = a.P;
  const int Q = (blockDim.x / kWave) / P;
  const int p = wave % P;
  const int q = wave / P;
  const int j = lane & 15;   // A row / B column of the lane's chunk
  const int g = lane >> 4;   // K group of the lane's chunk
  const int CH = (int)a.CH;
  const int nunits = a.NRW * T;
  // One token, one wave per row (P = 1), one pass and at most two rows per
  // wave (the small launches): the wave that sums a row stores it at once
  // (its lane 0) instead of meeting the slowest wave at a final barrier.
  // Otherwise the P waves' partials meet in LDS and are summed in a fixed
  // order at the end: with many rows per wave (lm_head) or two tokens the
  // scattered stores during the stream measured slower.
  const bool direct = kM1DirectStore && MODE != CB_SLICE && MT == 1 && P == 1 && a.NRW <= 2;

  // chunk of this lane in unit t of its row part
  auto ccol_raw = [&](int t) { return (p * T + t) * 64 + lane; };
  auto ccol = [&](int t) { const int c = ccol_raw(t); return c < CH ? c : CH - 1; };

  // Rows are dealt round-robin: local row rr of row group q of workgroup w is
  // row w + (rr * Q + q) * nwg.  The byte offset of the lane's chunk in
  // unit t of local row rr is row0 + rr * rstride + t * 64 * CBY.  Rows past N
  // (the pipeline reads up to L / T rows ahead) lie past the end of the
  // buffer resource and load zeros.
  const __amdgpu_buffer_rsrc_t rsrc = idx_rsrc(idx, (uint32_t)(N * a.R));
  const uint32_t rstride = (uint32_t)Q * nwg * (uint32_t)a.R;
  const uint32_t row0 = (wg + (uint32_t)q * nwg) * (uint32_t)a.R +
                        (uint32_t)ccol_raw(0) * CBY;

  uint32_t buf[L][DW];
  auto load_unit = [&](int slot, uint32_t roff, int t) {
    buffer_chunk<BITS>(rsrc, roff + (uint32_t)t * (64 * CBY), buf[slot]);
  };

  // ---- prologue (see k_gemv): codebook and x first, then the index stream.
  // CB_SLICE repeats everything from the codebook staging to the end of the
  // row loop once per slice; x is staged once.
  // x words each thread loads before the staging barrier: two per token
  // cover the longest rows here (K = 14336 on 14 waves).  Words past them are
  // loaded after the early index loads, one more round trip before the
  // barrier.
  constexpr int XWT = 2 * MT;
  const int xw_tok = (int)(a.K / 8);         // 16-byte words of x per token
  const int xw_total = xw_tok * a.M;          // 16-byte words of x
  const int xw_slots = xw_tok * MT;           // words of x staged (token slots past M hold zeros)
  // x in LDS: one unused word after every 16, so word r of a token sits at
  // LDS word r + r / 16.  The 16 lanes of one LDS cycle read word s of 16
  // consecutive chunks (SPC words each); without the padding, chunks of 4 or
  // more words put 4 or more of those lanes on the same banks.
  const int xw_tokp = xw_tok + (xw_tok + 15) / 16;  // LDS words per token
  auto xpos = [&](int w) {  // LDS word of x word w
    int r = w, m = 0;
    while (r >= xw_tok) { r -= xw_tok; ++m; }
    return m * xw_tokp + r + (r >> 4);
  };
  auto xword = [&](int m, int c, int s) {  // LDS address of word s of chunk c of token m
    const int r = c * SPC;
    return xl + (m * xw_tokp + r + (r >> 4)) * 16 + s * 16;
  };
  const uint32_t lane_off = repl_lane_off<D>(lane);
  half8_t xreg[kXInRegs ? MT * T * SPC : 1];
  // lane l holds D[4g + i][j]; the diagonal element D[j][j] sits in lane
  // j + 16 * (j / 4), register j % 4
  const bool on_diag = (j >> 2) == g;
  const int diag_reg = j & 3;
  const int nsl = MODE == CB_SLICE ? pt.nsl : 1;

  for (int si = 0; si < nsl; ++si) {
    Slice sl;
    const half_t* scb = cb;
    int sC = C;
    if constexpr (MODE == CB_SLICE) {
      sl.base = (uint32_t)si << a.sl_shift;
      sl.mask = (1u << a.sl_shift) - 1u;
      scb = cb + (size_t)sl.base * D;
      sC = C - (int)sl.base < (1 << a.sl_shift) ? C - (int)sl.base : (1 << a.sl_shift);
      if (si > 0) __syncthreads();  // every wave is done with the previous slice
    }
    CbStage cst;
    if constexpr (MODE == CB_SLICE) slice_fetch(scb, sC * D * 2 / 16, cst);
    else cb_fetch<D, MODE>(cb, C, cst);
    // x in 16-byte words: thread t stages words t and t + blockDim.x; waves
    // whose words all lie past the end of x issue no load for them.
    u32x4 xst[XWT];
    if (si == 0) {
#pragma unroll
      for (int k = 0; k < XWT; ++k) {
        xst[k] = u32x4{0u, 0u, 0u, 0u};
        if (wave * kWave + k * (int)blockDim.x < xw_total) {
          int w = threadIdx.x + k * blockDim.x;
          w = w < xw_total ? w : xw_total - 1;
          xst[k] = reinterpret_cast<const u32x4*>(a.x)[w];
        }
      }
    }
    // Every wave's codebook and x requests enter the CU's (in-order) memory
    // queue before any index load, and only the first kM1EarlyLoads index
    // loads of a wave go out before the staging barrier: the barrier then
    // waits for the small staging data alone, not for the whole workgroup to
    // get its loads accepted by a saturated memory queue.
    __syncthreads();
    // (issued whether or not the wave has that many units: these loads go
    // out first and return with the others, and a test here would make the
    // staging below wait for them)
#pragma unroll
    for (int i = 0; i < kM1EarlyLoads; ++i) load_unit(i, row0 + (uint32_t)(i / T) * rstride, i % T);

    if constexpr (MODE == CB_SLICE) slice_store(smem, scb, sC * D * 2 / 16, cst);
    else cb_store<D, MODE>(smem, cb, C, cst);
    if (si == 0) {
#pragma unroll
      for (int k = 0; k < XWT; ++k) {
        const int w = threadIdx.x + k * blockDim.x;
        if (w < xw_slots) reinterpret_cast<u32x4*>(xl)[xpos(w)] = w < xw_total ? xst[k] : u32x4{0u, 0u, 0u, 0u};
      }
      for (int w = threadIdx.x + XWT * blockDim.x; w < xw_slots; w += blockDim.x)
        reinterpret_cast<u32x4*>(xl)[xpos(w)] = w < xw_total ? reinterpret_cast<const u32x4*>(a.x)[w] : u32x4{0u, 0u, 0u, 0u};
    }
    __syncthreads();

    if (si == 0) {
      if constexpr (kXInRegs) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
#pragma unroll
          for (int t = 0; t < T; ++t) {
            const bool ok = !MASK || ccol_raw(t) < CH;
#pragma unroll
            for (int s = 0; s < SPC; ++s) {
              const half8_t v = *reinterpret_cast<const half8_t*>(xword(m, ccol(t), s));
              xreg[(m * T + t) * SPC + s] = ok ? v : half8_t{};
            }
          }
        }
      }
    }

    // per token: two fp32 partial sums of the lane's products (even and odd
    // steps), or the two diagonal-MFMA accumulators
    float dacc0[MT], dacc1[MT];
    float4_t acc0[kDecodeDot ? 1 : MT], acc1[kDecodeDot ? 1 : MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      dacc0[m] = dacc1[m] = 0.f;
      if constexpr (!kDecodeDot) acc0[m] = acc1[m] = float4_t{0.f, 0.f, 0.f, 0.f};
    }
    auto compute_unit = [&](int slot, int u, int t) {
      const uint32_t* w = buf[slot];
      const bool cval = !MASK || ccol_raw(t) < CH;
#pragma unroll
      for (int s = 0; s < SPC; ++s) {
        half8_t aop = gather8<BITS, D, MODE>(cb, lane_off, w, s * (8 / D), sl);
        if (MASK && !cval) aop = half8_t{};
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          half8_t bop;
          if constexpr (kXInRegs) bop = xreg[(m * T + t) * SPC + s];
          else bop = *reinterpret_cast<const half8_t*>(xword(m, ccol(t), s));
          if (MASK && !cval) bop = half8_t{};
          if constexpr (kDecodeDot) {
            // eight K values: four packed fp16 products-and-adds into fp32
            const u32x4 av = __builtin_bit_cast(u32x4, aop), bv = __builtin_bit_cast(u32x4, bop);
            float& d = (s & 1) ? dacc1[m] : dacc0[m];
            d = dot2(av[0], bv[0], d);
            d = dot2(av[1], bv[1], d);
            d = dot2(av[2], bv[2], d);
            d = dot2(av[3], bv[3], d);
          } else {
            if (s & 1) acc1[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, acc1[m], 0, 0, 0);
            else acc0[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, acc0[m], 0, 0, 0);
          }
        }
      }
      if (t == T - 1) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          float v;
          if constexpr (kDecodeDot) {
            v = dacc0[m] + dacc1[m];
          } else {
            const float4_t acc = acc0[m] + acc1[m];
            v = diag_reg == 0 ? acc[0] : diag_reg == 1 ? acc[1] : diag_reg == 2 ? acc[2] : acc[3];
            v = on_diag ? v : 0.f;
          }
          v = group_sum<16>(v);
          // the four rows of 16 lanes hold partial sums: combine in a fixed order
          const float sum = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)) +
                            __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16)) +
                            __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32)) +
                            __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
          // slices of a row are summed in slice order, each by the same lane
          if (lane == 0) {
            const int rl = (u / T) * Q + q;  // local row
            if (direct) {
              const int64_t n = (int64_t)wg + (int64_t)rl * nwg;
              if (n < N && m < a.M) y[(int64_t)m * pt.ldy + n] = static_cast<half_t>(sum);
            } else {
              float* r = &red[(rl * MT + m) * P + p];
              *r = (MODE == CB_SLICE && si > 0) ? *r + sum : sum;
            }
          }
          dacc0[m] = dacc1[m] = 0.f;
          if constexpr (!kDecodeDot) {
            acc0[m] = float4_t{0.f, 0.f, 0.f, 0.f};
            acc1[m] = float4_t{0.f, 0.f, 0.f, 0.f};
          }
        }
      }
    };

    // Unit k lives in slot k % L, and kM1Window loads stay in flight: once
    // unit k has arrived, the wave issues the load of unit k + W and then
    // computes unit k, so W loads stay in flight while it computes.  Units
    // below kM1EarlyLoads are already in flight.  Groups of L
    // units whose loads all lie within the wave's units run first; the last
    // R < L + W units run in code made for R, which issues no load past the
    // wave's last unit.  Such a load (it would read zeros) still holds the
    // wave, which ends only once all its loads are back, and it queues behind
    // the CU's real ones.  (A test around each load instead would make the
    // compiler wait for every load in flight before each unit.)
    constexpr int W = kM1Window;
    static_assert(W == kM1EarlyLoads, "the first group's loads start where the early loads end");
    constexpr uint32_t kGroupRows = L / T;  // local rows per group of L units
    int base = 0;
    uint32_t rbase = row0;  // offset of local row base / T
    for (; base + L + W <= nunits; base += L, rbase += kGroupRows * rstride) {
#pragma unroll
      for (int i = 0; i < L; ++i) {
        load_unit((i + W) % L, rbase + (uint32_t)((i + W) / T) * rstride, (i + W) % T);
        if (base + i < nunits) compute_unit(i, base + i, i % T);
      }
    }
    auto last = [&](auto rc) __attribute__((always_inline)) {
      constexpr int R = decltype(rc)::value;
#pragma unroll
      for (int i = 0; i < R; ++i) {
        if (i + W < R) load_unit((i + W) % L, rbase + (uint32_t)((i + W) / T) * rstride, (i + W) % T);
        compute_unit(i % L, base + i, i % T);
        // each load stays before the unit it overlaps (moved past later
        // units, it would leave the wave fewer loads in flight)
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    static_assert(L + W - 1 <= 10, "one case per possible remainder");
    switch (nunits - base) {  // 1 .. L + W - 1
      case 1: last(std::integral_constant<int, 1>{}); break;
      case 2: last(std::integral_constant<int, 2>{}); break;
      case 3: if constexpr (L + W > 3) last(std::integral_constant<int, 3>{}); break;
      case 4: if constexpr (L + W > 4) last(std::integral_constant<int, 4>{}); break;
      case 5: if constexpr (L + W > 5) last(std::integral_constant<int, 5>{}); break;
      case 6: if constexpr (L + W > 6) last(std::integral_constant<int, 6>{}); break;
      case 7: if constexpr (L + W > 7) last(std::integral_constant<int, 7>{}); break;
      case 8: if constexpr (L + W > 8) last(std::integral_constant<int, 8>{}); break;
      case 9: if constexpr (L + W > 9) last(std::integral_constant<int, 9>{}); break;
      default: break;
    }
  }
  if (direct) return;
  __syncthreads();

  // fixed-order sum over the P waves of each row, one fp16 rounding
  const int outs = Q * a.NRW * MT;
  for (int o = threadIdx.x; o < outs; o += blockDim.x) {
    const int r = o / MT;
    const int m = o - r * MT;
    const int64_t n = (int64_t)wg + (int64_t)r * nwg;
    if (n < N && m < a.M) {
      float sum = 0.f;
      for (int pp = 0; pp < P; ++pp) sum += red[o * P + pp];
      y[(int64_t)m * pt.ldy + n] = static_cast<half_t>(sum);
    }
  }
}

template <int BITS, int D, int T, int MODE, bool MASK>
__global__ __launch_bounds__(1024) void k_gemv_m1(GemvM1Args a) {
  gemv_rows_body<BITS, D, T, MODE, MASK, 1>(a);
}

template <int BITS, int D, int T, int MODE, bool MASK, int MT>
__global__ __launch_bounds__(1024) void k_gemv_mt(GemvM1Args a) {
  gemv_rows_body<BITS, D, T, MODE, MASK, MT>(a);
}

}  // namespace fasq
