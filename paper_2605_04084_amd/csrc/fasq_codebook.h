// Packed-index chunks, codebook placement in LDS, and codeword gathers.
#pragma once

#include "fasq_device.h"

namespace fasq {

// Where the kernels read codewords from.
//   CB_REPL  : LDS, each entry replicated once per lane slot of an LDS cycle,
//              so that random gathers never collide in a bank.
//   CB_LDS   : LDS, one copy (larger codebooks; gathers may collide).
//   CB_GLOBAL: global memory (L2 / Infinity Cache resident), for codebooks
//              larger than the LDS budget.
enum CbMode { CB_REPL = 0, CB_LDS = 1, CB_GLOBAL = 2 };

// One lane's unit of the packed index stream.
template <int BITS>
struct Chunk;
template <>
struct Chunk<8> {
  static constexpr int G = 16;  // ids per chunk
  static constexpr int DW = 4;  // dwords per chunk (16 bytes)
};
template <>
struct Chunk<16> {
  static constexpr int G = 8;
  static constexpr int DW = 4;
};
template <>
struct Chunk<12> {
  static constexpr int G = 8;
  static constexpr int DW = 3;  // 12 bytes: two ids per three bytes
};

// Id i of an LSB-first stream of BITS-bit fields held in dwords w[] (i is a
// compile-time constant after unrolling).
template <int BITS>
__device__ __forceinline__ uint32_t stream_id(const uint32_t* w, int i) {
  const int bit = i * BITS;
  const int word = bit >> 5;
  const int sh = bit & 31;
  if (sh + BITS <= 32) return __builtin_amdgcn_ubfe(w[word], sh, BITS);
  return __builtin_amdgcn_alignbit(w[word + 1], w[word], sh) & ((1u << BITS) - 1u);
}

template <int BITS>
__device__ __forceinline__ void load_chunk(const uint8_t* __restrict__ p, uint32_t* w) {
  if constexpr (Chunk<BITS>::DW == 4) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
    w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
  } else {
    const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
    w[0] = q[0]; w[1] = q[1]; w[2] = q[2];
  }
}

// Replicated layout: entry e owns one LDS row of STRIDE bytes holding COPIES
// copies of ESZ bytes, and lane slot c reads copy c.  gfx950 serves 32 lanes
// per cycle for 4- and 8-byte LDS reads and 16 lanes per cycle for 16-byte
// reads, so the lanes of one cycle always address distinct banks.
template <int D>
struct Repl {
  static constexpr int ESZ = (D == 1) ? 4 : 2 * D;
  static constexpr int STRIDE = (ESZ <= 4) ? 128 : 256;
  static constexpr int COPIES = STRIDE / ESZ;
  static constexpr int WPE = STRIDE / 16;                  // 16-byte words per replicated row
};

// LDS bytes a codebook of C entries takes in a given placement.
__host__ __device__ constexpr int64_t cb_lds_bytes(int mode, int64_t C, int d) {
  return mode == CB_REPL ? C * (d <= 2 ? 128 : 256) : mode == CB_LDS ? C * d * 2 : 0;
}

// ---------------------------------------------------------------------------
// Staging.  The unit is one 16-byte LDS word; consecutive threads write
// consecutive words, so the stores are conflict-free.
//   CB_LDS : word w is source word w (C * d * 2 must be a multiple of 16).
//   CB_REPL: word w of the replicated table holds copies of entry
//            w / Repl::WPE, which the thread loads on its own (the loads of
//            one wave touch one or two cache lines).
// The fetch phase issues the global loads and the store phase writes LDS, so
// that a kernel can issue its index-stream loads in between without waiting
// on them here.
// ---------------------------------------------------------------------------
constexpr int kCbWordsPerThread = 4;  // first-round words per thread (64 KB at 1024 threads)

struct CbStage {
  u32x4 w[kCbWordsPerThread];
};

template <int D, int MODE>
__device__ __forceinline__ int cb_words(int C) {
  return MODE == CB_REPL ? C * Repl<D>::WPE : C * D * 2 / 16;
}

template <int D, int MODE>
__device__ __forceinline__ u32x4 cb_word(const half_t* __restrict__ cb, int w) {
  if constexpr (MODE == CB_LDS) {
    return reinterpret_cast<const u32x4*>(cb)[w];
  } else {
    const int e = w / Repl<D>::WPE;
    if constexpr (D == 1) {
      const uint32_t h = reinterpret_cast<const uint16_t*>(cb)[e];
      return u32x4{h, h, h, h};
    } else if constexpr (D == 2) {
      const uint32_t c = reinterpret_cast<const uint32_t*>(cb)[e];
      return u32x4{c, c, c, c};
    } else if constexpr (D == 4) {
      const u32x2 c = reinterpret_cast<const u32x2*>(cb)[e];
      return u32x4{c[0], c[1], c[0], c[1]};
    } else {
      return reinterpret_cast<const u32x4*>(cb)[e];
    }
  }
}

template <int D, int MODE>
__device__ __forceinline__ void cb_fetch(const half_t* __restrict__ cb, int C, CbStage& st) {
  if constexpr (MODE != CB_GLOBAL) {
    const int n = cb_words<D, MODE>(C);
#pragma unroll
    for (int k = 0; k < kCbWordsPerThread; ++k) {
      const int w = threadIdx.x + k * blockDim.x;
      st.w[k] = cb_word<D, MODE>(cb, w < n ? w : n - 1);
    }
  }
}

template <int D, int MODE>
__device__ __forceinline__ void cb_store(uint8_t* __restrict__ lds, const half_t* __restrict__ cb, int C,
                                         const CbStage& st) {
  if constexpr (MODE != CB_GLOBAL) {
    const int n = cb_words<D, MODE>(C);
    u32x4* dst = reinterpret_cast<u32x4*>(lds);
#pragma unroll
    for (int k = 0; k < kCbWordsPerThread; ++k) {
      const int w = threadIdx.x + k * blockDim.x;
      if (w < n) dst[w] = st.w[k];
    }
    for (int w = threadIdx.x + kCbWordsPerThread * blockDim.x; w < n; w += blockDim.x) dst[w] = cb_word<D, MODE>(cb, w);
  }
}

// Gather codeword u into `out` (D == 1: one fp16 in the low half of out[0];
// D >= 2: D / 2 dwords of packed fp16 pairs).
template <int D, int MODE>
__device__ __forceinline__ void gather(const uint8_t* __restrict__ lds, const half_t* __restrict__ gcb,
                                       uint32_t lane_off, uint32_t u, uint32_t* out) {
  const uint8_t* p;
  if constexpr (MODE == CB_REPL) p = lds + u * Repl<D>::STRIDE + lane_off;
  else if constexpr (MODE == CB_LDS) p = lds + u * (2 * D);
  else p = reinterpret_cast<const uint8_t*>(gcb) + (size_t)u * (2 * D);
  if constexpr (D == 1) {
    out[0] = *reinterpret_cast<const uint16_t*>(p);
  } else if constexpr (D == 2) {
    out[0] = *reinterpret_cast<const uint32_t*>(p);
  } else if constexpr (D == 4) {
    const u32x2 v = *reinterpret_cast<const u32x2*>(p);
    out[0] = v[0]; out[1] = v[1];
  } else {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
    out[0] = v[0]; out[1] = v[1]; out[2] = v[2]; out[3] = v[3];
  }
}

template <int D>
__device__ __forceinline__ uint32_t repl_lane_off(int lane) {
  return (uint32_t)(lane % Repl<D>::COPIES) * Repl<D>::ESZ;
}

// Eight consecutive K values of W_hat for one lane, as an MFMA operand:
// ids first .. first + 8/D - 1 of the lane's chunk w[], gathered and packed.
template <int BITS, int D, int MODE>
__device__ __forceinline__ half8_t gather8(const uint8_t* __restrict__ lds, const half_t* __restrict__ gcb,
                                           uint32_t lane_off, const uint32_t* w, int first) {
  uint32_t o[4];
  if constexpr (D == 1) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      uint32_t c0[1], c1[1];
      gather<D, MODE>(lds, gcb, lane_off, stream_id<BITS>(w, first + e), c0);
      gather<D, MODE>(lds, gcb, lane_off, stream_id<BITS>(w, first + e + 1), c1);
      o[e / 2] = (c0[0] & 0xFFFFu) | (c1[0] << 16);
    }
  } else {
    constexpr int CW = D / 2;
#pragma unroll
    for (int e = 0; e < 8 / D; ++e) {
      uint32_t c[CW];
      gather<D, MODE>(lds, gcb, lane_off, stream_id<BITS>(w, first + e), c);
#pragma unroll
      for (int k = 0; k < CW; ++k) o[e * CW + k] = c[k];
    }
  }
  return __builtin_bit_cast(half8_t, u32x4{o[0], o[1], o[2], o[3]});
}

}  // namespace fasq
