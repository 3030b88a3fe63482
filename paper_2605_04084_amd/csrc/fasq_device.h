// Device-side helpers shared by the libfasq kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fasq {

typedef _Float16 half_t;
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef float float16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// fp16 <-> bits without any arithmetic conversion
// ---------------------------------------------------------------------------
__device__ __forceinline__ half2_t as_half2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }
__device__ __forceinline__ uint32_t as_u32(half2_t v) { return __builtin_bit_cast(uint32_t, v); }

// fp32 -> fp16, round to nearest even (v_cvt_f16_f32 under the default mode).
__device__ __forceinline__ uint16_t f32_to_f16_bits(float v) {
  return __builtin_bit_cast(uint16_t, static_cast<half_t>(v));
}

// acc + a.x*b.x + a.y*b.y with fp16 inputs and an fp32 accumulator (v_dot2_f32_f16).
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2(as_half2(a), as_half2(b), acc, false);
}

// ---------------------------------------------------------------------------
// Packed-id decoding.  A row is an LSB-first stream of BITS-bit fields.
// ---------------------------------------------------------------------------

// Id `s` of a row starting at `row` (R bytes), decoded with byte loads only
// (any alignment).  Reads stay inside [row, row + R).
template <int BITS>
__device__ __forceinline__ uint32_t load_id_bytes(const uint8_t* __restrict__ row, int64_t s, int64_t R) {
  if constexpr (BITS == 8) {
    return row[s];
  } else if constexpr (BITS == 16) {
    return uint32_t(row[2 * s]) | (uint32_t(row[2 * s + 1]) << 8);
  } else {
    const int64_t bit = 12 * s;
    const int64_t byte = bit >> 3;
    uint32_t lo = row[byte];
    uint32_t hi = (byte + 1 < R) ? uint32_t(row[byte + 1]) : 0u;
    return ((lo | (hi << 8)) >> (bit & 7)) & 0xFFFu;
  }
}

// ---------------------------------------------------------------------------
// Reductions (DPP within rows of 16 lanes)
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of L lanes (L in {1, 2, 4, 8, 16}); every lane of a
// group ends with the group's sum.
template <int L>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (L >= 2) v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  if constexpr (L >= 4) v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  if constexpr (L >= 8) v += dpp_f<0x141>(v);  // row_half_mirror
  if constexpr (L >= 16) v += dpp_f<0x140>(v); // row_mirror
  return v;
}

// Full 64-lane sum, result valid in every lane.
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<16>(v);
  v += __shfl_xor(v, 16, kWave);
  v += __shfl_xor(v, 32, kWave);
  return v;
}

}  // namespace fasq
