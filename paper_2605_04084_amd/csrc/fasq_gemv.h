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

#include "fasq_codebook.h"
#include "fasq_device.h"

namespace fasq {

struct GemvArgs {
  const half_t* x;
  int64_t M, K, N;
  const uint8_t* idx;
  int64_t R;   // bytes per row (= CH * chunk bytes)
  int64_t CH;  // chunks per row
  const half_t* cb;
  int C;
  int P;         // waves per row (K split inside the workgroup)
  int RW;        // rows per workgroup, a multiple of 16 * (waves / P)
  int cb_bytes;  // LDS bytes of the codebook (x follows)
  int xs;        // LDS bytes between rows of x
  int x_bytes;   // LDS bytes of x (partials follow)
  half_t* y;
};

constexpr int kGemvPipe = 8;      // load units per wave in the software pipeline
constexpr int kXWordsPerThread = 8;  // first-round x words (16 B) per thread for M > 1

template <int BITS, int D, int T, int MODE, int MR>
__global__ __launch_bounds__(1024) void k_gemv(GemvArgs a) {
  constexpr int G = Chunk<BITS>::G;      // ids per chunk
  constexpr int DW = Chunk<BITS>::DW;    // dwords per chunk
  constexpr int CBY = DW * 4;            // chunk bytes
  constexpr int SPC = G * D / 8;         // MFMA steps (8 K values each) per chunk
  constexpr int L = kGemvPipe;
  static_assert(L % T == 0, "pipeline depth must be a multiple of T");

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint8_t* xl = smem + a.cb_bytes;
  float* red = reinterpret_cast<float*>(smem + a.cb_bytes + a.x_bytes);  // [RW][M][P]

  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int P = a.P;
  const int Q = (blockDim.x / kWave) / P;
  const int p = wave % P;
  const int q = wave / P;
  const int g = lane >> 4;    // K group
  const int nl = lane & 15;   // row within a 16-row tile
  const int M = (int)a.M;
  const int64_t r0 = (int64_t)blockIdx.x * a.RW;
  const int rows_q = a.RW / Q;
  const int nrt = rows_q / 16;             // row tiles of this wave
  const int nunits = nrt * T;
  const int64_t rowbase = r0 + (int64_t)q * rows_q + nl;
  // A chunk column is valid for every lane of the wave or for none but the
  // last few; `full` selects the unmasked path for the whole wave.
  const bool full = (int64_t)(p * T + T) * 4 <= a.CH;

  // chunk column of (t): raw value, and clamped into the row for loads
  const int CH = (int)a.CH;
  auto ccol_raw = [&](int t) { return (p * T + t) * 4 + g; };
  auto ccol = [&](int t) { const int c = ccol_raw(t); return c < CH ? c : CH - 1; };

  // Units past the end of this wave's work load the first chunk of the table
  // (one address for the whole wave: a single request) so that every
  // iteration issues exactly one load and the waits stay exact.
  // Rows past N read row N - 1 (computed, never stored).
  const int64_t row0 = rowbase < a.N ? rowbase : a.N - 1;
  int rtmax = 0;
  if (rowbase < a.N) {
    const int64_t last = (a.N - 1 - rowbase) / 16;
    rtmax = (int)(last < nrt - 1 ? last : nrt - 1);
  }
  const uint8_t* lp = a.idx + row0 * a.R;
  const int64_t tile_stride = 16 * a.R;
  uint32_t buf[L][DW];
  auto load_unit = [&](int slot, int u, int t) {
    int rt = u / T;
    rt = rt < rtmax ? rt : rtmax;
    const uint8_t* src = u < nunits ? lp + rt * tile_stride + ccol(t) * CBY : a.idx;
    load_chunk<BITS>(src, buf[slot]);
  };

  // ---- prologue.  The vector L1 returns loads in order, so an L2-resident
  // load queued behind HBM loads waits for them: the codebook and x are
  // fetched and written to LDS first, and the index stream starts after the
  // barrier.
  CbStage cst;
  cb_fetch<D, MODE>(a.cb, a.C, cst);
  constexpr int XWT = MR == 1 ? 2 : kXWordsPerThread;
  const int xw_row = (int)(a.K / 8);        // 16-byte words per row of x
  const int xw_total = xw_row * M;
  u32x4 xst[XWT];
#pragma unroll
  for (int k = 0; k < XWT; ++k) {
    int w = threadIdx.x + k * blockDim.x;
    w = w < xw_total ? w : xw_total - 1;
    xst[k] = reinterpret_cast<const u32x4*>(a.x)[w];
  }
  cb_store<D, MODE>(smem, a.cb, a.C, cst);
#pragma unroll
  for (int k = 0; k < XWT; ++k) {
    const int w = threadIdx.x + k * blockDim.x;
    if (w < xw_total) {
      const int m = w / xw_row;
      *reinterpret_cast<u32x4*>(xl + m * a.xs + (w - m * xw_row) * 16) = xst[k];
    }
  }
  for (int w = threadIdx.x + XWT * blockDim.x; w < xw_total; w += blockDim.x) {
    const int m = w / xw_row;
    *reinterpret_cast<u32x4*>(xl + m * a.xs + (w - m * xw_row) * 16) = reinterpret_cast<const u32x4*>(a.x)[w];
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < L - 1; ++i) load_unit(i, i, i % T);

  const uint32_t lane_off = repl_lane_off<D>(lane);
  const int mrow = MR == 1 ? 0 : (nl < M ? nl : M - 1);  // x row this lane feeds to the A operand
  const uint8_t* xrow = xl + mrow * a.xs;

  float4_t acc0 = {0.f, 0.f, 0.f, 0.f};
  float4_t acc1 = {0.f, 0.f, 0.f, 0.f};

  // One chunk: SPC MFMA steps.  MASKED zeroes both operands of lanes whose
  // chunk column lies past the end of the row (only the last wave of a
  // ragged row needs it).
  auto chunk_steps = [&](const uint32_t* w, int t, bool masked) {
    const uint8_t* xa = xrow + ccol(t) * (G * D * 2);
    const bool cval = ccol_raw(t) < CH;
#pragma unroll
    for (int s = 0; s < SPC; ++s) {
      half8_t bop = gather8<BITS, D, MODE>(smem, a.cb, lane_off, w, s * (8 / D));
      half8_t aop = *reinterpret_cast<const half8_t*>(xa + s * 16);
      if (masked && !cval) {
        bop = half8_t{};
        aop = half8_t{};
      }
      if (s & 1) acc1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, acc1, 0, 0, 0);
      else acc0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, acc0, 0, 0, 0);
    }
  };
  const bool full_wave = __builtin_amdgcn_readfirstlane((int)full) != 0;

  for (int base = 0; base < nunits; base += L) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int u = base + i;
      const int t = i % T;
      load_unit((i + L - 1) % L, u + L - 1, (i + L - 1) % T);
      if (u < nunits) {
        if (full_wave) chunk_steps(buf[i], t, false);
        else chunk_steps(buf[i], t, true);
        if (t == T - 1) {
          // lane l holds rows m = 4g .. 4g + 3 of column nl of the 16 x 16 tile
          const int lrow = q * rows_q + (u / T) * 16 + nl;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int m = 4 * g + k;
            if (m < M) red[(lrow * M + m) * P + p] = acc0[k] + acc1[k];
          }
          acc0 = float4_t{0.f, 0.f, 0.f, 0.f};
          acc1 = float4_t{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
  }
  __syncthreads();

  // fixed-order sum over the P waves, one fp16 rounding, row-contiguous stores
  const int outs = a.RW * M;
  for (int o = threadIdx.x; o < outs; o += blockDim.x) {
    const int m = o / a.RW;
    const int r = o - m * a.RW;
    const int64_t n = r0 + r;
    if (n < a.N) {
      float sum = 0.f;
      const float* pr = red + (r * M + m) * P;
      for (int pp = 0; pp < P; ++pp) sum += pr[pp];
      a.y[(int64_t)m * a.N + n] = static_cast<half_t>(sum);
    }
  }
}

}  // namespace fasq
