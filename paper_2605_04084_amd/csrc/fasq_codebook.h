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
//   CB_SLICE : LDS, one slice of 2^k entries at a time (codebooks larger than
//              LDS): the kernel makes one pass over its rows per slice, and
//              an id contributes only in the pass of its own slice.
//   CB_SPLIT : the first entries in LDS, as many as fit, the rest gathered
//              from global memory (codebooks larger than LDS, one pass).
//   CB_HALF  : LDS, each entry replicated over a 128-byte row (half of
//              CB_REPL's), for a tile whose ring leaves no room for the full
//              table: with 8-byte codewords two lanes of an LDS cycle share
//              each copy, so a gather costs at most two cycles.
enum CbMode { CB_REPL = 0, CB_LDS = 1, CB_GLOBAL = 2, CB_SLICE = 3, CB_SPLIT = 4, CB_HALF = 5 };

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

// Replicated layout: entry e owns one 256-byte LDS row (address e << 8)
// holding COPIES copies of its ESZ bytes from the start of the row, and lane
// l reads copy l % COPIES.  gfx950 serves 32 lanes per cycle for 4- and
// 8-byte LDS reads and 16 lanes per cycle for 16-byte reads, so the lanes of
// one cycle always address distinct banks.  With 256-byte rows the address of
// id u is (u << 8) | lane_off: for 8-bit ids one byte permute builds it
// straight from the packed id bytes.  (For ESZ = 4 only the first 128 bytes
// of a row are used.)
template <int D>
struct Repl {
  static constexpr int ESZ = (D <= 2) ? 4 : 2 * D;
  static constexpr int STRIDE = 256;
  static constexpr int COPIES = (ESZ == 4) ? 32 : STRIDE / ESZ;
  static constexpr int WPE = COPIES * ESZ / 16;  // 16-byte words staged per row
};

// The half-row layout (CB_HALF): entry e owns the 128-byte row at e << 7,
// filled with 128 / ESZ copies; lane l reads copy l % HCOPIES.
template <int D>
struct ReplHalf {
  static constexpr int ESZ = Repl<D>::ESZ;
  static constexpr int STRIDE = 128;
  static constexpr int COPIES = STRIDE / ESZ;
  static constexpr int WPE = STRIDE / 16;
};

// LDS bytes a codebook of C entries takes in a given placement.
// (CB_SLICE: the slice size is chosen by the launcher, not given by C.)
__host__ __device__ constexpr int64_t cb_lds_bytes(int mode, int64_t C, int d) {
  return mode == CB_REPL ? C * 256 : mode == CB_HALF ? C * 128 : mode == CB_LDS ? C * d * 2 : 0;
}

// ---------------------------------------------------------------------------
// Staging.  The unit is one 16-byte LDS word; consecutive threads write
// consecutive words, so the stores are conflict-free.
//   CB_LDS : word w is source word w, stored at LDS byte 16 w (C * d * 2 must
//            be a multiple of 16).
//   CB_REPL: word w holds copies of entry e = w / WPE and is stored at
//            (e << 8) + 16 (w % WPE); the thread loads the entry itself (the
//            loads of one wave touch one or two cache lines).
//   CB_HALF: as CB_REPL with 128-byte rows: (e << 7) + 16 (w % 8).
// The fetch phase issues the global loads and the store phase writes LDS, so
// that a kernel can issue its index-stream loads in between without waiting
// on them here.
// ---------------------------------------------------------------------------
constexpr int kCbWordsPerThread = 8;  // first-round words per thread

// Replicated two-fp16 codewords (d = 2, C <= 256) take a shorter route: every
// wave loads the whole raw codebook (one 16-byte load per lane, 4 entries per
// lane) and the replicated rows are written from registers, each entry's
// codeword fetched from the lane that holds it with a cross-lane permute.
template <int D, int MODE>
constexpr bool cb_fast_stage() { return MODE == CB_REPL && D == 2; }

struct CbStage {
  u32x4 w[kCbWordsPerThread];
};

template <int D, int MODE>
__device__ __forceinline__ int cb_words(int C) {
  return MODE == CB_REPL ? C * Repl<D>::WPE : MODE == CB_HALF ? C * ReplHalf<D>::WPE : C * D * 2 / 16;
}

template <int D, int MODE>
__device__ __forceinline__ uint32_t cb_word_addr(int w) {
  if constexpr (MODE == CB_REPL) return ((uint32_t)(w / Repl<D>::WPE) << 8) + (uint32_t)(w % Repl<D>::WPE) * 16;
  else if constexpr (MODE == CB_HALF)
    return ((uint32_t)(w / ReplHalf<D>::WPE) << 7) + (uint32_t)(w % ReplHalf<D>::WPE) * 16;
  else return (uint32_t)w * 16;
}

template <int D, int MODE>
__device__ __forceinline__ u32x4 cb_word(const half_t* __restrict__ cb, int w) {
  if constexpr (MODE == CB_LDS) {
    return reinterpret_cast<const u32x4*>(cb)[w];
  } else {
    const int e = w / (MODE == CB_HALF ? ReplHalf<D>::WPE : Repl<D>::WPE);
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
  if constexpr (cb_fast_stage<D, MODE>()) {
    const int chunks = C / 4;  // 16-byte chunks of the raw codebook (C * 4 % 16 == 0)
    const int l = threadIdx.x % kWave;
    st.w[0] = reinterpret_cast<const u32x4*>(cb)[l < chunks ? l : chunks - 1];
  } else if constexpr (MODE != CB_GLOBAL) {
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
  if constexpr (cb_fast_stage<D, MODE>()) {
    // Wave v writes entry blocks v, v + waves, ... of 32 entries; in step k,
    // lane l writes 16 bytes of row e = 32 b + 4 (l / 8) + k, whose codeword
    // is dword k of lane e / 4.
    const int l = threadIdx.x % kWave;
    const int waves = blockDim.x / kWave;
    for (int b = threadIdx.x / kWave; b * 32 < C; b += waves) {
      uint32_t c[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) c[k] = (uint32_t)__shfl((int)st.w[0][k], 8 * b + l / 8, kWave);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = 32 * b + 4 * (l / 8) + k;
        if (e < C) *reinterpret_cast<u32x4*>(lds + ((uint32_t)e << 8) + (uint32_t)(l % 8) * 16) = u32x4{c[k], c[k], c[k], c[k]};
      }
    }
  } else if constexpr (MODE != CB_GLOBAL) {
    const int n = cb_words<D, MODE>(C);
#pragma unroll
    for (int k = 0; k < kCbWordsPerThread; ++k) {
      const int w = threadIdx.x + k * blockDim.x;
      if (w < n) *reinterpret_cast<u32x4*>(lds + cb_word_addr<D, MODE>(w)) = st.w[k];
    }
    for (int w = threadIdx.x + kCbWordsPerThread * blockDim.x; w < n; w += blockDim.x)
      *reinterpret_cast<u32x4*>(lds + cb_word_addr<D, MODE>(w)) = cb_word<D, MODE>(cb, w);
  }
}

// CB_SLICE staging: the `words` 16-byte words of one slice (source `src`)
// go to LDS from address 0.  The first batch of loads is issued by
// slice_fetch (as cb_fetch), the rest by slice_store in batches of
// kCbWordsPerThread loads in flight per thread.
__device__ __forceinline__ void slice_fetch(const half_t* __restrict__ src, int words, CbStage& st) {
#pragma unroll
  for (int k = 0; k < kCbWordsPerThread; ++k) {
    const int w = threadIdx.x + k * blockDim.x;
    st.w[k] = reinterpret_cast<const u32x4*>(src)[w < words ? w : words - 1];
  }
}

__device__ __forceinline__ void slice_store(uint8_t* __restrict__ lds, const half_t* __restrict__ src, int words,
                                            const CbStage& st) {
#pragma unroll
  for (int k = 0; k < kCbWordsPerThread; ++k) {
    const int w = threadIdx.x + k * blockDim.x;
    if (w < words) *reinterpret_cast<u32x4*>(lds + (uint32_t)w * 16) = st.w[k];
  }
  for (int base = threadIdx.x + kCbWordsPerThread * blockDim.x; base < words;
       base += kCbWordsPerThread * blockDim.x) {
    u32x4 v[kCbWordsPerThread];
#pragma unroll
    for (int k = 0; k < kCbWordsPerThread; ++k) {
      const int w = base + k * blockDim.x;
      v[k] = reinterpret_cast<const u32x4*>(src)[w < words ? w : words - 1];
    }
#pragma unroll
    for (int k = 0; k < kCbWordsPerThread; ++k) {
      const int w = base + k * blockDim.x;
      if (w < words) *reinterpret_cast<u32x4*>(lds + (uint32_t)w * 16) = v[k];
    }
  }
}

// LDS-resident codebooks start at LDS address 0: the kernels that use them
// declare no static LDS (the launchers check this), so the dynamic segment
// begins at 0 and an LDS address can be formed as a plain integer.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(3))) T* lds_at(uint32_t addr) {
  return (const __attribute__((address_space(3))) T*)(size_t)addr;
}

// Codeword at LDS byte address addr (D == 1: one fp16 in the low half of
// out[0]; D >= 2: D / 2 dwords of packed fp16 pairs).
template <int D>
__device__ __forceinline__ void read_codeword_lds(uint32_t addr, uint32_t* out) {
  if constexpr (D == 1) {
    out[0] = *lds_at<uint16_t>(addr);
  } else if constexpr (D == 2) {
    out[0] = *lds_at<uint32_t>(addr);
  } else if constexpr (D == 4) {
    const u32x2 v = *lds_at<u32x2>(addr);
    out[0] = v[0]; out[1] = v[1];
  } else {
    const u32x4 v = *lds_at<u32x4>(addr);
    out[0] = v[0]; out[1] = v[1]; out[2] = v[2]; out[3] = v[3];
  }
}

// The codebook slice resident in LDS (CB_SLICE, CB_SPLIT): entries
// [base, base + mask].
struct Slice {
  uint32_t base = 0;
  uint32_t mask = 0;
};

// Gather codeword u into `out` (layout as for read_codeword_lds).  In
// CB_SLICE mode an id outside the resident slice reads nothing and yields
// a zero codeword.
// Codeword u read straight from the codebook in global memory.
template <int D>
__device__ __forceinline__ void read_codeword_global(const half_t* __restrict__ gcb, uint32_t u, uint32_t* out) {
  const uint8_t* p = reinterpret_cast<const uint8_t*>(gcb) + (size_t)u * (2 * D);
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

template <int D, int MODE>
__device__ __forceinline__ void gather(const half_t* __restrict__ gcb, uint32_t lane_off, uint32_t u,
                                       uint32_t* out, Slice sl = Slice()) {
  if constexpr (MODE == CB_REPL) {
    read_codeword_lds<D>((u << 8) | lane_off, out);
  } else if constexpr (MODE == CB_HALF) {
    read_codeword_lds<D>((u << 7) | lane_off, out);
  } else if constexpr (MODE == CB_LDS) {
    read_codeword_lds<D>(u * (2 * D), out);
  } else if constexpr (MODE == CB_SLICE) {
    const uint32_t loc = u - sl.base;
#pragma unroll
    for (int k = 0; k < (D + 1) / 2; ++k) out[k] = 0u;
    if (loc <= sl.mask) read_codeword_lds<D>(loc * (2 * D), out);
  } else if constexpr (MODE == CB_SPLIT) {
    if (u <= sl.mask) read_codeword_lds<D>(u * (2 * D), out);
    else read_codeword_global<D>(gcb, u, out);
  } else {
    read_codeword_global<D>(gcb, u, out);
  }
}

template <int D>
__device__ __forceinline__ uint32_t repl_lane_off(int lane) {
  return (uint32_t)(lane % Repl<D>::COPIES) * Repl<D>::ESZ;
}

// The lane's copy offset in the placement MODE (0 for a single copy).
template <int D, int MODE>
__device__ __forceinline__ uint32_t cb_lane_off(int lane) {
  if constexpr (MODE == CB_HALF) return (uint32_t)(lane % ReplHalf<D>::COPIES) * ReplHalf<D>::ESZ;
  else return repl_lane_off<D>(lane);
}

// Gather the codeword of id i of chunk w[].  For 8-bit ids in the replicated
// layout the LDS address is one byte permute: byte 0 = the lane's copy
// offset, byte 1 = the id byte, bytes 2 and 3 = 0.
template <int BITS, int D, int MODE>
__device__ __forceinline__ void gather_id(const half_t* __restrict__ gcb, uint32_t lane_off, const uint32_t* w,
                                          int i, uint32_t* out, Slice sl = Slice()) {
  if constexpr (BITS == 8 && MODE == CB_REPL) {
    const uint32_t sel = 0x0C0C0000u | ((4u + (uint32_t)(i & 3)) << 8);
    read_codeword_lds<D>(__builtin_amdgcn_perm(w[i >> 2], lane_off, sel), out);
  } else {
    gather<D, MODE>(gcb, lane_off, stream_id<BITS>(w, i), out, sl);
  }
}

// Eight consecutive K values of W_hat for one lane, as an MFMA operand:
// ids first .. first + 8/D - 1 of the lane's chunk w[], gathered and packed.
template <int BITS, int D, int MODE>
__device__ __forceinline__ half8_t gather8(const half_t* __restrict__ gcb, uint32_t lane_off, const uint32_t* w,
                                           int first, Slice sl = Slice()) {
  uint32_t o[4];
  if constexpr (D == 1) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      uint32_t c0[1], c1[1];
      gather_id<BITS, D, MODE>(gcb, lane_off, w, first + e, c0, sl);
      gather_id<BITS, D, MODE>(gcb, lane_off, w, first + e + 1, c1, sl);
      o[e / 2] = (c0[0] & 0xFFFFu) | (c1[0] << 16);
    }
  } else {
    constexpr int CW = D / 2;
#pragma unroll
    for (int e = 0; e < 8 / D; ++e) {
      uint32_t c[CW];
      gather_id<BITS, D, MODE>(gcb, lane_off, w, first + e, c, sl);
#pragma unroll
      for (int k = 0; k < CW; ++k) o[e * CW + k] = c[k];
    }
  }
  return __builtin_bit_cast(half8_t, u32x4{o[0], o[1], o[2], o[3]});
}

// ---------------------------------------------------------------------------
// Raw buffer loads of the index stream.  The resource covers exactly the
// index table, so a load whose offset lies past its end returns zeros and
// touches no memory; kernels use that for rows past N instead of clamping.
// Offsets are 32-bit: callers check N * R (plus the rows a pipeline reads
// ahead) against 2^32 on the host.
// ---------------------------------------------------------------------------
__device__ __forceinline__ __amdgpu_buffer_rsrc_t idx_rsrc(const uint8_t* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p), (short)0, (int)bytes, 0x00020000);
}

template <int BITS>
__device__ __forceinline__ void buffer_chunk(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t* w) {
  if constexpr (Chunk<BITS>::DW == 4) {
    const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
    w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
  } else {
    typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
    const u32x3 v = __builtin_bit_cast(u32x3, __builtin_amdgcn_raw_buffer_load_b96(r, (int)off, 0, 0));
    w[0] = v[0]; w[1] = v[1]; w[2] = v[2];
  }
}

}  // namespace fasq
