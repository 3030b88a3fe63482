// Prefill GEMM kernels: variant selection and launch.
#include "fasq_gemm_mfma.h"
#include "fasq_gemv_launch.h"

namespace fasq {

namespace {

template <int BITS, int D, int MODE, int BM, int BN, int WGM, int WGN>
hipError_t launch_gemm_variant(const GemmArgs& a, int lds, hipStream_t stream) {
  auto kern = k_gemm_mfma<BITS, D, MODE, BM, BN, WGM, WGN>;
  if (plan_record("k_gemm_mfma", {BITS, D, MODE, BM, BN, WGM, WGN})) return hipSuccess;
  hipError_t e = prepare_kernel(kern);
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM));
  hipLaunchKernelGGL(kern, grid, dim3(WGM * WGN * kWave), lds, stream, a);
  return hipGetLastError();
}

// Tile shapes: 128 x 128 on 2 x 2 waves, or 128 x 256 on 2 x 4 waves (half the
// X re-reads per output, two waves per SIMD) when there are tiles enough.
enum GemmTile { kTile128x128 = 0, kTile128x256 = 1 };

template <int BITS, int D, int MODE>
hipError_t launch_gemm_tile(const GemmArgs& a, int tile, int lds, hipStream_t stream) {
  if (tile == kTile128x256) return launch_gemm_variant<BITS, D, MODE, 128, 256, 2, 4>(a, lds, stream);
  return launch_gemm_variant<BITS, D, MODE, 128, 128, 2, 2>(a, lds, stream);
}

template <int BITS, int D>
hipError_t launch_gemm_mode(const GemmArgs& a, int mode, int tile, int lds, hipStream_t stream) {
  switch (mode) {
    case CB_REPL: return launch_gemm_tile<BITS, D, CB_REPL>(a, tile, lds, stream);
    case CB_LDS: return launch_gemm_tile<BITS, D, CB_LDS>(a, tile, lds, stream);
    default: return launch_gemm_tile<BITS, D, CB_GLOBAL>(a, tile, lds, stream);
  }
}

template <int BITS>
hipError_t launch_gemm_bits(const GemmArgs& a, int d, int mode, int tile, int lds, hipStream_t stream) {
  switch (d) {
    case 1: return launch_gemm_mode<BITS, 1>(a, mode, tile, lds, stream);
    case 2: return launch_gemm_mode<BITS, 2>(a, mode, tile, lds, stream);
    case 4: return launch_gemm_mode<BITS, 4>(a, mode, tile, lds, stream);
    default:
      if constexpr (BITS == 12) return hipErrorNotSupported;  // 4 ids = 6 bytes: not dword aligned
      else return launch_gemm_mode<BITS, 8>(a, mode, tile, lds, stream);
  }
}

}  // namespace

hipError_t launch_gemm_mfma(const Problem& p, const DeviceInfo& dev, hipStream_t stream) {
  const int d = p.d;
  if (!(d == 1 || d == 2 || d == 4 || d == 8)) return hipErrorNotSupported;
  if (p.idx_bits == 12 && d == 8) return hipErrorNotSupported;
  if (p.K % kGemmKC) return hipErrorNotSupported;
  if (p.R * 8 != p.S * p.idx_bits) return hipErrorNotSupported;
  if ((reinterpret_cast<uintptr_t>(p.x) & 15) || (reinterpret_cast<uintptr_t>(p.codebook) & 15) ||
      (reinterpret_cast<uintptr_t>(p.idx) & 15) || (p.R & 3))
    return hipErrorNotSupported;
  // id runs are copied as 4-byte words
  const int hb = (32 / d) * p.idx_bits / 8;
  if (hb % 4) return hipErrorNotSupported;

  const int mode = choose_cb_mode(p.C, d);
  const int cb_bytes = (int)cb_lds_bytes(mode, p.C, d);
  auto lds_of = [&](int bn) { return cb_bytes + kGemmStages * (128 * 128 + bn * 2 * hb); };
  const int64_t mt = (p.M + 127) / 128;
  int tile = kTile128x128;
  if (4 * mt * ((p.N + 255) / 256) >= 3 * (int64_t)dev.num_cus && lds_of(256) <= dev.lds_per_block)
    tile = kTile128x256;
  const int lds = lds_of(tile == kTile128x256 ? 256 : 128);
  if (lds > dev.lds_per_block) return hipErrorNotSupported;

  GemmArgs a;
  a.x = static_cast<const half_t*>(p.x);
  a.M = p.M;
  a.K = p.K;
  a.N = p.N;
  a.idx = static_cast<const uint8_t*>(p.idx);
  a.R = p.R;
  a.cb = static_cast<const half_t*>(p.codebook);
  a.C = (int)p.C;
  a.cb_lds_bytes = cb_bytes;
  a.y = static_cast<half_t*>(p.y);
  switch (p.idx_bits) {
    case 8: return launch_gemm_bits<8>(a, d, mode, tile, lds, stream);
    case 12: return launch_gemm_bits<12>(a, d, mode, tile, lds, stream);
    default: return launch_gemm_bits<16>(a, d, mode, tile, lds, stream);
  }
}

}  // namespace fasq
