// Decode GEMV for one token (M = 1): y[n] = sum_s dot(x[s*d:(s+1)*d], codebook[u(n, s)]).
//
// Work decomposition (gfx950, wave64):
//   * The packed index table is streamed once from HBM in 16-byte (8/16-bit
//     ids) or 12-byte (12-bit ids) chunks per lane.  LPR lanes cover LPR
//     consecutive chunks of one row, so one wave-wide load reads 64 / LPR rows
//     of LPR*16 contiguous bytes each.
//   * A row's chunks are split into P equal parts, one per wave of a
//     workgroup (split-K inside the workgroup); each lane owns T chunk
//     columns of its part.  Because a lane always sees the same chunk
//     columns, its slice of x is loaded into registers once per workgroup.
//   * Codewords are gathered from LDS.  When C is small the codebook is
//     replicated per lane slot so that the random gathers of one LDS cycle
//     hit distinct banks (CB_REPL); otherwise it is stored once (CB_LDS); a
//     codebook larger than the LDS budget is gathered from global memory
//     (L2/MALL resident, CB_GLOBAL).
//   * Partial sums: in registers (fp32) -> across the LPR lanes of a row with
//     DPP -> across the P waves through LDS, in a fixed order, so results are
//     deterministic.  Each output is rounded to fp16 once and written by a
//     contiguous store per batch of rows.
//   * Rows are processed in batches; the index chunks of the next batch are
//     loaded before the current batch is computed (register double buffer).
#pragma once

#include "fasq_device.h"
#include "fasq_internal.h"

namespace fasq {

enum CbMode { CB_REPL = 0, CB_LDS = 1, CB_GLOBAL = 2 };

template <int BITS>
struct Chunk;
template <>
struct Chunk<8> {
  static constexpr int G = 16;  // ids per chunk
  static constexpr int DW = 4;  // dwords per chunk
};
template <>
struct Chunk<16> {
  static constexpr int G = 8;
  static constexpr int DW = 4;
};
template <>
struct Chunk<12> {
  static constexpr int G = 8;
  static constexpr int DW = 3;
};

// Replicated codebook layout: entry e occupies one LDS row of STRIDE bytes
// holding COPIES copies of ESZ bytes; lane slot c reads copy c.  With 32
// lanes per cycle for 4/8-byte reads and 16 lanes per cycle for 16-byte
// reads, the lanes of one cycle always address distinct banks.
template <int D>
struct Repl {
  static constexpr int ESZ = (D == 1) ? 4 : 2 * D;
  static constexpr int STRIDE = (ESZ <= 4) ? 128 : 256;
  static constexpr int COPIES = STRIDE / ESZ;
};

template <int D>
constexpr int repl_bytes_per_entry() { return Repl<D>::STRIDE; }

// Copy the codebook into LDS in the requested layout.
template <int D, int MODE>
__device__ __forceinline__ void stage_codebook(uint8_t* __restrict__ lds, const half_t* __restrict__ cb, int C) {
  if constexpr (MODE == CB_REPL) {
    constexpr int WPE = Repl<D>::STRIDE / 16;  // 16-byte words per entry row
    const int total = C * WPE;
    for (int w = threadIdx.x; w < total; w += blockDim.x) {
      const int e = w / WPE;
      uint4 v;
      if constexpr (D == 1) {
        const uint32_t c = reinterpret_cast<const uint16_t*>(cb)[e];
        v = make_uint4(c, c, c, c);
      } else if constexpr (D == 2) {
        const uint32_t c = reinterpret_cast<const uint32_t*>(cb)[e];
        v = make_uint4(c, c, c, c);
      } else if constexpr (D == 4) {
        const uint2 c = reinterpret_cast<const uint2*>(cb)[e];
        v = make_uint4(c.x, c.y, c.x, c.y);
      } else {
        v = reinterpret_cast<const uint4*>(cb)[e];
      }
      *reinterpret_cast<uint4*>(lds + (size_t)w * 16) = v;
    }
  } else if constexpr (MODE == CB_LDS) {
    const int bytes = C * D * 2;
    if ((bytes & 15) == 0) {
      for (int w = threadIdx.x; w < bytes / 16; w += blockDim.x)
        reinterpret_cast<uint4*>(lds)[w] = reinterpret_cast<const uint4*>(cb)[w];
    } else {
      for (int w = threadIdx.x; w < bytes / 2; w += blockDim.x)
        reinterpret_cast<uint16_t*>(lds)[w] = reinterpret_cast<const uint16_t*>(cb)[w];
    }
  }
}

// Gather codeword u into `out` (D == 1: one fp16 in the low half of out[0];
// D >= 2: D / 2 dwords of packed fp16 pairs).
template <int D, int MODE>
__device__ __forceinline__ void gather(const uint8_t* __restrict__ lds, const half_t* __restrict__ gcb,
                                       uint32_t lane_off, uint32_t u, uint32_t* out) {
  if constexpr (MODE == CB_REPL) {
    const uint8_t* p = lds + u * Repl<D>::STRIDE + lane_off;
    if constexpr (D == 1) out[0] = *reinterpret_cast<const uint16_t*>(p);
    else if constexpr (D == 2) out[0] = *reinterpret_cast<const uint32_t*>(p);
    else if constexpr (D == 4) { const uint2 v = *reinterpret_cast<const uint2*>(p); out[0] = v.x; out[1] = v.y; }
    else { const uint4 v = *reinterpret_cast<const uint4*>(p); out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w; }
  } else {
    const uint8_t* p = (MODE == CB_LDS) ? lds + u * (2 * D) : reinterpret_cast<const uint8_t*>(gcb) + (size_t)u * (2 * D);
    if constexpr (D == 1) out[0] = *reinterpret_cast<const uint16_t*>(p);
    else if constexpr (D == 2) out[0] = *reinterpret_cast<const uint32_t*>(p);
    else if constexpr (D == 4) { const uint2 v = *reinterpret_cast<const uint2*>(p); out[0] = v.x; out[1] = v.y; }
    else { const uint4 v = *reinterpret_cast<const uint4*>(p); out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w; }
  }
}

template <int BITS>
__device__ __forceinline__ void load_chunk(const uint8_t* __restrict__ p, uint32_t* w) {
  if constexpr (Chunk<BITS>::DW == 4) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  } else {
    const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
    w[0] = q[0]; w[1] = q[1]; w[2] = q[2];
  }
}

struct GemvM1Args {
  const half_t* x;
  int64_t K, N;
  const uint8_t* idx;
  int64_t R;   // bytes per row (= CH * chunk bytes)
  int64_t CH;  // chunks per row
  const half_t* cb;
  int C;
  int P;       // waves per row (K split inside the workgroup)
  int cb_lds_bytes;
  half_t* y;
};

template <int BITS, int D, int LPR, int T, int MODE>
__global__ __launch_bounds__(512) void k_gemv_m1(GemvM1Args a) {
  constexpr int G = Chunk<BITS>::G;
  constexpr int DW = Chunk<BITS>::DW;
  constexpr int CB = DW * 4;       // chunk bytes
  constexpr int RPI = kWave / LPR; // rows per wave-wide load
  constexpr int U = (T >= 4) ? 1 : 4 / T;
  constexpr int XW = G * D / 2;    // x dwords per chunk
  constexpr int CW = (D == 1) ? 1 : D / 2;

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int P = a.P;
  const int Q = (blockDim.x / kWave) / P;
  const int p = wave % P;
  const int q = wave / P;
  const int seg = lane / LPR;
  const int j = lane % LPR;
  const int BR = RPI * U * Q;
  const int64_t nb = (a.N + BR - 1) / BR;
  float* red = reinterpret_cast<float*>(smem + a.cb_lds_bytes);  // 2 x [BR][P]

  // chunk column of (t) for this lane; columns are contiguous across lanes
  int64_t ccol[T];
  bool cval[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    ccol[t] = (int64_t)p * LPR * T + t * LPR + j;
    cval[t] = ccol[t] < a.CH;
  }

  uint32_t bufA[U][T][DW], bufB[U][T][DW];

  auto load_batch = [&](uint32_t (&buf)[U][T][DW], int64_t b) {
    const int64_t row0 = b * BR + (int64_t)q * (RPI * U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t n = row0 + u * RPI + seg;
      const uint8_t* rp = a.idx + n * a.R;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (n < a.N && cval[t]) {
          load_chunk<BITS>(rp + ccol[t] * CB, buf[u][t]);
        } else {
#pragma unroll
          for (int w = 0; w < DW; ++w) buf[u][t][w] = 0u;
        }
      }
    }
  };

  int64_t b = blockIdx.x;
  if (b < nb) load_batch(bufA, b);

  if constexpr (MODE != CB_GLOBAL) stage_codebook<D, MODE>(smem, a.cb, a.C);

  // this lane's slice of x, kept in registers for the whole kernel
  uint32_t xr[T][XW];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const uint4* xs = reinterpret_cast<const uint4*>(a.x) + ccol[t] * (XW / 4);
#pragma unroll
    for (int w4 = 0; w4 < XW / 4; ++w4) {
      uint4 v = cval[t] ? xs[w4] : make_uint4(0, 0, 0, 0);
      xr[t][4 * w4 + 0] = v.x; xr[t][4 * w4 + 1] = v.y; xr[t][4 * w4 + 2] = v.z; xr[t][4 * w4 + 3] = v.w;
    }
  }
  __syncthreads();

  const uint32_t lane_off = (uint32_t)(lane % Repl<D>::COPIES) * Repl<D>::ESZ;
  int parity = 0;

  auto compute_batch = [&](uint32_t (&buf)[U][T][DW], int64_t bb) {
    float* rb = red + parity * (BR * P);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        if (cval[t]) {
          if constexpr (D == 1) {
#pragma unroll
            for (int g = 0; g < G; g += 2) {
              uint32_t c0[1], c1[1];
              gather<D, MODE>(smem, a.cb, lane_off, chunk_id<BITS>(buf[u][t], g), c0);
              gather<D, MODE>(smem, a.cb, lane_off, chunk_id<BITS>(buf[u][t], g + 1), c1);
              const uint32_t pair = (c0[0] & 0xFFFFu) | (c1[0] << 16);
              if ((g & 2) == 0) acc0 = dot2(pair, xr[t][g / 2], acc0);
              else acc1 = dot2(pair, xr[t][g / 2], acc1);
            }
          } else {
#pragma unroll
            for (int g = 0; g < G; ++g) {
              uint32_t c[CW];
              gather<D, MODE>(smem, a.cb, lane_off, chunk_id<BITS>(buf[u][t], g), c);
#pragma unroll
              for (int w = 0; w < CW; ++w) {
                if (((g * CW + w) & 1) == 0) acc0 = dot2(c[w], xr[t][g * CW + w], acc0);
                else acc1 = dot2(c[w], xr[t][g * CW + w], acc1);
              }
            }
          }
        }
      }
      float s = group_sum<LPR>(acc0 + acc1);
      if (j == 0) rb[(q * (RPI * U) + u * RPI + seg) * P + p] = s;
    }
    __syncthreads();
    if ((int)threadIdx.x < BR) {
      const int64_t n = bb * BR + threadIdx.x;
      if (n < a.N) {
        float s = 0.f;
        for (int pp = 0; pp < P; ++pp) s += rb[threadIdx.x * P + pp];
        a.y[n] = static_cast<half_t>(s);
      }
    }
    parity ^= 1;
  };

  while (b < nb) {
    int64_t bn = b + gridDim.x;
    if (bn < nb) load_batch(bufB, bn);
    compute_batch(bufA, b);
    b = bn;
    if (b >= nb) break;
    bn = b + gridDim.x;
    if (bn < nb) load_batch(bufA, bn);
    compute_batch(bufB, b);
    b = bn;
  }
}

}  // namespace fasq
