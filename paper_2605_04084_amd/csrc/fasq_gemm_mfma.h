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
#include "fasq_gemv_m1.h"
#include "fasq_internal.h"

namespace fasq {

// Id i of an LSB-first stream held in dwords w[] (i is a compile-time constant
// after unrolling).
template <int BITS>
__device__ __forceinline__ uint32_t stream_id(const uint32_t* w, int i) {
  const int bit = i * BITS;
  const int word = bit >> 5;
  const int sh = bit & 31;
  if (sh + BITS <= 32) return __builtin_amdgcn_ubfe(w[word], sh, BITS);
  return __builtin_amdgcn_alignbit(w[word + 1], w[word], sh) & ((1u << BITS) - 1u);
}

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
          const uint4 v = *reinterpret_cast<const uint4*>(p + w);
          buf[fn][w] = v.x; buf[fn][w + 1] = v.y; buf[fn][w + 2] = v.z; buf[fn][w + 3] = v.w;
        }
      } else if constexpr (HW % 2 == 0) {
#pragma unroll
        for (int w = 0; w < HW; w += 2) {
          const uint2 v = *reinterpret_cast<const uint2*>(p + w);
          buf[fn][w] = v.x; buf[fn][w + 1] = v.y;
        }
      } else {
#pragma unroll
        for (int w = 0; w < HW; ++w) buf[fn][w] = p[w];
      }
    }
  };

  // ---- X chunk loads: thread -> (row, 16-byte column)
  uint4 xreg[XPASS];
  auto load_x = [&](int64_t c) {
#pragma unroll
    for (int ps = 0; ps < XPASS; ++ps) {
      const int r = ps * 32 + tid / 8;
      const int64_t m = m0 + r;
      if (m < a.M) xreg[ps] = *reinterpret_cast<const uint4*>(a.x + m * a.K + c * kGemmKC + (tid % 8) * 8);
      else xreg[ps] = make_uint4(0, 0, 0, 0);
    }
  };
  auto store_x = [&](int buf) {
    uint8_t* base = xs + buf * (BM * kXRowBytes);
#pragma unroll
    for (int ps = 0; ps < XPASS; ++ps) {
      const int r = ps * 32 + tid / 8;
      *reinterpret_cast<uint4*>(base + r * kXRowBytes + (tid % 8) * 16) = xreg[ps];
    }
  };

  uint32_t idsA[FN][HW], idsB[FN][HW];
  load_ids(idsA, 0);
  load_x(0);
  if constexpr (MODE != CB_GLOBAL) stage_codebook<D, MODE>(smem, a.cb, a.C);
  store_x(0);
  __syncthreads();

  float16_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[fm][fn][i] = 0.f;

  const uint32_t lane_off = (uint32_t)(lane % Repl<D>::COPIES) * Repl<D>::ESZ;

  auto compute_chunk = [&](const uint32_t (&ids)[FN][HW], int buf) {
    const uint8_t* xb = xs + buf * (BM * kXRowBytes);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      half8_t bop[FN];
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        uint32_t w4[4];
        if constexpr (D == 1) {
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            uint32_t c0[1], c1[1];
            gather<D, MODE>(smem, a.cb, lane_off, stream_id<BITS>(ids[fn], t * IPS + e), c0);
            gather<D, MODE>(smem, a.cb, lane_off, stream_id<BITS>(ids[fn], t * IPS + e + 1), c1);
            w4[e / 2] = (c0[0] & 0xFFFFu) | (c1[0] << 16);
          }
        } else {
          constexpr int CW = D / 2;
#pragma unroll
          for (int e = 0; e < IPS; ++e) {
            uint32_t c[CW];
            gather<D, MODE>(smem, a.cb, lane_off, stream_id<BITS>(ids[fn], t * IPS + e), c);
#pragma unroll
            for (int w = 0; w < CW; ++w) w4[e * CW + w] = c[w];
          }
        }
        bop[fn] = __builtin_bit_cast(half8_t, make_uint4(w4[0], w4[1], w4[2], w4[3]));
      }
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

  int64_t c = 0;
  int buf = 0;
  while (c < nchunks) {
    // chunk c lives in idsA / LDS buffer `buf`
    const bool more = (c + 1) < nchunks;
    if (more) { load_ids(idsB, c + 1); load_x(c + 1); }
    compute_chunk(idsA, buf);
    if (more) store_x(buf ^ 1);
    __syncthreads();
    ++c; buf ^= 1;
    if (c >= nchunks) break;
    const bool more2 = (c + 1) < nchunks;
    if (more2) { load_ids(idsA, c + 1); load_x(c + 1); }
    compute_chunk(idsB, buf);
    if (more2) store_x(buf ^ 1);
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
