// Host-side variant selection and launch for the M = 1 decode kernel.
#pragma once

#include <atomic>

#include "fasq_gemv_m1.h"

namespace fasq {

constexpr int kLdsCodebookBudget = 64 * 1024;  // bytes of LDS a codebook may take

// Raise a kernel's dynamic-LDS limit to the 160 KB the CU offers, once per
// device (one bit per device ordinal; ordinals >= 64 set it on every launch).
template <typename K>
hipError_t allow_lds(K kernel, int bytes) {
  static std::atomic<uint64_t> done{0};
  if (bytes <= 64 * 1024) return hipSuccess;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? (uint64_t(1) << dev) : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                          160 * 1024);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
  return e;
}

// x dwords one lane keeps per chunk column
template <int BITS, int D>
constexpr int gemv_xw() { return Chunk<BITS>::G * D / 2; }
constexpr int kMaxXRegs = 64;  // x registers (dwords) a lane may hold

template <int BITS, int D, int LPR, int T, int MODE>
hipError_t launch_gemv_m1_variant(const GemvM1Args& a, int threads, int blocks, int lds, hipStream_t stream) {
  if constexpr (T * gemv_xw<BITS, D>() > kMaxXRegs) {
    return hipErrorNotSupported;  // never selected: the host caps T * XW
  } else {
  auto kern = k_gemv_m1<BITS, D, LPR, T, MODE>;
  hipError_t e = allow_lds(kern, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(threads), lds, stream, a);
  return hipGetLastError();
  }
}

template <int BITS, int D, int MODE>
hipError_t launch_gemv_m1_shape(const GemvM1Args& a, int LPR, int T, int threads, int blocks, int lds,
                                hipStream_t stream) {
  if (LPR == 4) return launch_gemv_m1_variant<BITS, D, 4, 1, MODE>(a, threads, blocks, lds, stream);
  switch (T) {
    case 1: return launch_gemv_m1_variant<BITS, D, 16, 1, MODE>(a, threads, blocks, lds, stream);
    case 2: return launch_gemv_m1_variant<BITS, D, 16, 2, MODE>(a, threads, blocks, lds, stream);
    case 4: return launch_gemv_m1_variant<BITS, D, 16, 4, MODE>(a, threads, blocks, lds, stream);
    default: return launch_gemv_m1_variant<BITS, D, 16, 8, MODE>(a, threads, blocks, lds, stream);
  }
}

template <int BITS, int D>
hipError_t launch_gemv_m1_mode(const GemvM1Args& a, int mode, int LPR, int T, int threads, int blocks, int lds,
                               hipStream_t stream) {
  switch (mode) {
    case CB_REPL: return launch_gemv_m1_shape<BITS, D, CB_REPL>(a, LPR, T, threads, blocks, lds, stream);
    case CB_LDS: return launch_gemv_m1_shape<BITS, D, CB_LDS>(a, LPR, T, threads, blocks, lds, stream);
    default: return launch_gemv_m1_shape<BITS, D, CB_GLOBAL>(a, LPR, T, threads, blocks, lds, stream);
  }
}

// Pick (LPR, T, P, codebook placement, grid) for one call; hipErrorNotSupported
// when the call needs the general kernel.
template <int BITS>
hipError_t launch_gemv_m1_bits(const Problem& p, const DeviceInfo& dev, hipStream_t stream) {
  constexpr int G = Chunk<BITS>::G;
  constexpr int CB = Chunk<BITS>::DW * 4;
  const int d = p.d;
  if (p.M != 1) return hipErrorNotSupported;
  if (!(d == 1 || d == 2 || d == 4 || d == 8)) return hipErrorNotSupported;
  if (p.S % G) return hipErrorNotSupported;
  const int64_t CH = p.S / G;
  if (CH * CB != p.R || CH < 4) return hipErrorNotSupported;
  const uintptr_t ia = reinterpret_cast<uintptr_t>(p.idx);
  if ((CB == 16 && (ia & 15)) || (ia & 3)) return hipErrorNotSupported;
  if ((reinterpret_cast<uintptr_t>(p.x) & 15) || (reinterpret_cast<uintptr_t>(p.codebook) & 15))
    return hipErrorNotSupported;

  const int LPR = CH >= 16 ? 16 : 4;
  const int64_t CHL = (CH + LPR - 1) / LPR;
  const int XW = G * d / 2;  // x dwords per chunk column
  int T = 0;
  if (LPR == 4) {
    if (CHL <= 8) T = 1;
  } else {
    for (int t : {1, 2, 4, 8}) {
      if ((CHL + t - 1) / t <= 8 && t * XW <= kMaxXRegs) { T = t; break; }
    }
  }
  if (T == 0) return hipErrorNotSupported;
  const int P = (int)((CHL + T - 1) / T);
  const int Q = 8 / P;
  const int threads = P * Q * kWave;
  const int U = (T >= 4) ? 1 : 4 / T;
  const int BR = (kWave / LPR) * U * Q;

  int mode;
  int cb_bytes;
  const int64_t repl = p.C * (int64_t)(d <= 2 ? 128 : 256);  // Repl<d>::STRIDE
  if (repl <= kLdsCodebookBudget) {
    mode = CB_REPL;
    cb_bytes = (int)repl;
  } else if (p.C * d * 2 <= kLdsCodebookBudget) {
    mode = CB_LDS;
    cb_bytes = (int)((p.C * d * 2 + 15) / 16 * 16);
  } else {
    mode = CB_GLOBAL;
    cb_bytes = 0;
  }
  const int lds = cb_bytes + 2 * BR * P * 4;
  if (lds > dev.lds_per_block) return hipErrorNotSupported;

  const int64_t nb = (p.N + BR - 1) / BR;
  const int per_cu = (mode == CB_GLOBAL) ? 4 : 2;
  const int64_t maxb = (int64_t)dev.num_cus * per_cu;
  const int blocks = (int)(nb < maxb ? nb : maxb);

  GemvM1Args a;
  a.x = static_cast<const half_t*>(p.x);
  a.K = p.K;
  a.N = p.N;
  a.idx = static_cast<const uint8_t*>(p.idx);
  a.R = p.R;
  a.CH = CH;
  a.cb = static_cast<const half_t*>(p.codebook);
  a.C = (int)p.C;
  a.P = P;
  a.cb_lds_bytes = cb_bytes;
  a.y = static_cast<half_t*>(p.y);

  switch (d) {
    case 1: return launch_gemv_m1_mode<BITS, 1>(a, mode, LPR, T, threads, blocks, lds, stream);
    case 2: return launch_gemv_m1_mode<BITS, 2>(a, mode, LPR, T, threads, blocks, lds, stream);
    case 4: return launch_gemv_m1_mode<BITS, 4>(a, mode, LPR, T, threads, blocks, lds, stream);
    default: return launch_gemv_m1_mode<BITS, 8>(a, mode, LPR, T, threads, blocks, lds, stream);
  }
}

}  // namespace fasq
