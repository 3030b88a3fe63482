// Prefill GEMM: Y[M x N] = X[M x K] . W_hat^T with W_hat decoded tile by tile.
//
// Design (gfx950, wave64, v_mfma_f32_32x32x16_f16):
//   * A workgroup of 4 waves owns a BM x BN output tile; the waves form a
//     2 x 2 grid, each wave owning (BM/2) x (BN/2) = FM x FN MFMA tiles of
//     32 x 32 with fp32 accumulators in registers.
//   * K is walked in chunks of 64.  The X chunk (BM x 64 fp16) is staged in
//     LDS (row stride padded to 144 B so that the 16-byte operand reads of one
//     LDS cycle hit distinct banks), double-buffered, with the next chunk held
//     in registers while the current one is consumed.
//   * W_hat is never written to memory, not even to LDS: each lane decodes
//     the ids of its own B-operand column straight from the packed index row
//     and gathers the codewords from the LDS codebook into the MFMA B
//     registers.  The order of K inside a chunk is permuted identically for
//     A and B (allowed: the contraction is a sum over K), so that lane half h
//     reads one contiguous run of 32/d ids per chunk.
//   * Epilogue: fp32 -> fp16 once, direct stores.
#pragma once

#include "fasq_device.h"
#include "fasq_codebook.h"
#include "fasq_internal.h"

namespace fasq {

constexpr int kGemmKC = 64;          // K per chunk
constexpr int kXRowBytes = 144;      // padded LDS row of one X chunk (128 B of data)

struct GemmArgs {
  const half_t* x;
  int64_t M, K, N;
  const uint8_t* idx;
  int64_t R;
  const half_t* cb;
  int C;
  int cb_lds_bytes;
  half_t* y;
};

template <int BITS, int D, int MODE, int BM, int BN>
__global__ __launch_bounds__(256) void k_gemm_mfma(GemmArgs a) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int IDS_HALF = 32 / D;                 // ids per lane half per chunk
  constexpr int HB = IDS_HALF * BITS / 8;          // bytes per lane half per chunk
  constexpr int HW = HB / 4;                       // dwords per lane half per chunk
  constexpr int IPS = 8 / D;                       // ids per k-step per lane
  constexpr int XPASS = BM * 128 / (256 * 16);     // 16-byte X loads per thread per chunk
  static_assert(HB % 4 == 0, "index run must be whole dwords");
  static_assert(XPASS >= 1, "tile too small");

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint8_t* xs = smem + a.cb_lds_bytes;  // 2 x [BM][144 B]

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int wm = wave >> 1, wn = wave & 1;
  const int h = lane >> 5, l32 = lane & 31;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const int64_t n0 = (int64_t)blockIdx.x * BN;
  const int64_t nchunks = a.K / kGemmKC;

  // ---- index pointers for this lane's B columns
  const uint8_t* irow[FN];
  bool nval[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int64_t n = n0 + wn * WN + fn * 32 + l32;
    nval[fn] = n < a.N;
    irow[fn] = a.idx + (nval[fn] ? n : 0) * a.R + h * HB;
  }
  auto load_ids = [&](uint32_t (&buf)[FN][HW], int64_t c) {
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const uint32_t* p = reinterpret_cast<const uint32_t*>(irow[fn] + c * (2 * HB));
      if constexpr (HW % 4 == 0) {
#pragma unroll
        for (int w = 0; w < HW; w += 4) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(p + w);
          buf[fn][w] = v[0]; buf[fn][w + 1] = v[1]; buf[fn][w + 2] = v[2]; buf[fn][w + 3] = v[3];
        }
      } else if constexpr (HW % 2 == 0) {
#pragma unroll
        for (int w = 0; w < HW; w += 2) {
          const u32x2 v = *reinterpret_cast<const u32x2*>(p + w);
          buf[fn][w] = v[0]; buf[fn][w + 1] = v[1];
        }
      } else {
#pragma unroll
        for (int w = 0; w < HW; ++w) buf[fn][w] = p[w];
      }
    }
  };

  // ---- X chunk loads: thread -> (row, 16-byte column)
  // rows >= M read row M - 1: they are computed but never stored
  const half_t* xrow[XPASS];
#pragma unroll
  for (int ps = 0; ps < XPASS; ++ps) {
    const int64_t m = m0 + ps * 32 + tid / 8;
    xrow[ps] = a.x + (m < a.M ? m : a.M - 1) * a.K + (tid % 8) * 8;
  }
  u32x4 xreg[XPASS];
  auto load_x = [&](int64_t c) {
#pragma unroll
    for (int ps = 0; ps < XPASS; ++ps)
      xreg[ps] = *reinterpret_cast<const u32x4*>(xrow[ps] + c * kGemmKC);
  };
  auto store_x = [&](int buf) {
    uint8_t* base = xs + buf * (BM * kXRowBytes);
#pragma unroll
    for (int ps = 0; ps < XPASS; ++ps) {
      const int r = ps * 32 + tid / 8;
      *reinterpret_cast<u32x4*>(base + r * kXRowBytes + (tid % 8) * 16) = xreg[ps];
    }
  };

  // The codebook (L2-resident) is staged before the first index / X loads:
  // the vector L1 returns loads in order, so it would otherwise wait for them.
  CbStage cst;
  cb_fetch<D, MODE>(a.cb, a.C, cst);
  cb_store<D, MODE>(smem, a.cb, a.C, cst);
  uint32_t idsA[FN][HW], idsB[FN][HW];
  load_ids(idsA, 0);
  load_x(0);
  store_x(0);
  __syncthreads();

  float16_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[fm][fn][i] = 0.f;

  const uint32_t lane_off = repl_lane_off<D>(lane);

  auto compute_chunk = [&](const uint32_t (&ids)[FN][HW], int buf) {
    const uint8_t* xb = xs + buf * (BM * kXRowBytes);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      half8_t bop[FN];
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) bop[fn] = gather8<BITS, D, MODE>(a.cb, lane_off, ids[fn], t * IPS);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        const int r = wm * WM + fm * 32 + l32;
        const half8_t aop = *reinterpret_cast<const half8_t*>(xb + r * kXRowBytes + (h * 32 + t * 8) * 2);
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(aop, bop[fn], acc[fm][fn], 0, 0, 0);
      }
    }
  };

  // Chunk c lives in one register set / LDS buffer while chunk c + 1 is
  // loaded into the other.  The next-chunk loads are unconditional (the last
  // chunk is re-read) so that the number of loads in flight is static.
  int64_t c = 0;
  int buf = 0;
  while (c < nchunks) {
    int64_t cn = (c + 1) < nchunks ? c + 1 : c;
    load_ids(idsB, cn);
    load_x(cn);
    compute_chunk(idsA, buf);
    store_x(buf ^ 1);
    __syncthreads();
    ++c; buf ^= 1;
    if (c >= nchunks) break;
    cn = (c + 1) < nchunks ? c + 1 : c;
    load_ids(idsA, cn);
    load_x(cn);
    compute_chunk(idsB, buf);
    store_x(buf ^ 1);
    __syncthreads();
    ++c; buf ^= 1;
  }

  // ---- epilogue: lane l holds rows (i/4)*8 + h*4 + i%4, column l32 of each 32x32 tile
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t n = n0 + wn * WN + fn * 32 + l32;
      if (n >= a.N) continue;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t m = m0 + wm * WM + fm * 32 + (i / 4) * 8 + h * 4 + (i % 4);
        if (m < a.M) a.y[m * a.N + n] = static_cast<half_t>(acc[fm][fn][i]);
      }
    }
  }
}

}  // namespace fasq
