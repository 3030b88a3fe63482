// The paper's prefill kernel design (FASQ Sec. 4.2, Alg. 3) on gfx950, kept
// beside the MFMA GEMM to measure the gap the paper reports between a lookup
// table GEMM and a matrix-core GEMM (Sec. 4.4, sequence length scaling).
//
//   LUT[t][s][k] = dot(x[t, s*d : (s+1)*d], codebook[k])        (build)
//   y[t][n]      = sum_s LUT[t][s][u(n, s)]                      (lookup)
//
// Output-stationary as in Alg. 3: a workgroup owns 8 tokens and 256 output
// features (one per thread, all 8 tokens in registers) and walks the
// subspaces in batches of SB.  The lookup tables of the next batch are built
// by all threads while the current batch is looked up, in two LDS buffers, so
// there is one barrier per batch (the paper has one per subspace).  Tables
// and sums are fp32.
#include "fasq_codebook.h"
#include "fasq_device.h"
#include "fasq_internal.h"

namespace fasq {

namespace {

constexpr int kLutThreads = 256;
constexpr int kLutTokens = 8;            // tokens per workgroup
constexpr int kLutEntries = 16384;       // fp32 table entries per buffer (64 KB)

struct LutArgs {
  const half_t* x;
  int64_t M, K, N;
  const uint8_t* idx;
  int64_t R;
  const half_t* cb;
  int C;
  half_t* y;
};

// Ids of subspaces s0 .. s0 + SB - 1 of one row (R bytes, S ids); subspaces
// past S read nothing and give id 0.
template <int BITS, int SB>
__device__ __forceinline__ void load_ids(const uint8_t* row, int64_t s0, int64_t S, int64_t R, uint32_t* u) {
#pragma unroll
  for (int j = 0; j < SB; ++j) u[j] = s0 + j < S ? load_id_bytes<BITS>(row, s0 + j, R) : 0u;
}

template <int BITS, int D, int SB>
__global__ __launch_bounds__(kLutThreads) void k_gemm_lut(LutArgs a) {
  constexpr int LT = kLutTokens;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  float* lut = reinterpret_cast<float*>(smem);  // [2][SB][LT][C]
  const int C = a.C;
  const int per_buf = SB * LT * C;
  const int64_t S = a.K / D;
  const int64_t nb = (S + SB - 1) / SB;
  const int64_t t0 = (int64_t)blockIdx.y * LT;
  const int64_t n = (int64_t)blockIdx.x * kLutThreads + threadIdx.x;
  const uint8_t* row = a.idx + (n < a.N ? n : 0) * a.R;

  // x slice of a batch in LDS (two buffers): [LT][SB][D] fp32, the same for
  // every thread.  Subspaces past S repeat the last one (never looked up).
  constexpr int XS = LT * SB * D;
  float* xs = lut + 2 * per_buf;
  auto stage_x = [&](int64_t b, float* dst) __attribute__((always_inline)) {
    for (int e = threadIdx.x; e < XS; e += kLutThreads) {
      const int t = e / (SB * D);
      const int j = (e / D) % SB;
      const int i = e % D;
      const int64_t tt = t0 + t < a.M ? t0 + t : a.M - 1;
      const int64_t s = b * SB + j < S ? b * SB + j : S - 1;
      dst[e] = static_cast<float>(a.x[tt * a.K + s * D + i]);
    }
  };
  // Thread i builds the table entries of codewords k = i, i + 256, ... (held
  // in registers) for every (subspace, token) of a batch.
  constexpr int CPT = 8 / SB;  // codewords per thread: SB * 8 * C <= 16384 gives C <= 256 * CPT
  float cw[CPT][D];
#pragma unroll
  for (int r = 0; r < CPT; ++r) {
    const int k = threadIdx.x + r * kLutThreads;
#pragma unroll
    for (int i = 0; i < D; ++i) cw[r][i] = k < C ? static_cast<float>(a.cb[(int64_t)k * D + i]) : 0.f;
  }
  auto build = [&](const float* xb, float* dst) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < SB; ++j) {
#pragma unroll
      for (int t = 0; t < LT; ++t) {
        float xv[D];
#pragma unroll
        for (int i = 0; i < D; ++i) xv[i] = xb[(t * SB + j) * D + i];
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
          const int k = threadIdx.x + r * kLutThreads;
          if (k < C) {
            float v = 0.f;
#pragma unroll
            for (int i = 0; i < D; ++i) v = __builtin_fmaf(xv[i], cw[r][i], v);
            dst[(j * LT + t) * C + k] = v;
          }
        }
      }
    }
  };

  float acc[LT];
#pragma unroll
  for (int t = 0; t < LT; ++t) acc[t] = 0.f;

  // Iteration b looks up batch b, builds the tables of batch b + 1 and
  // stages the x slice of batch b + 2; one barrier per batch.
  stage_x(0, xs);
  if (nb > 1) stage_x(1, xs + XS);
  __syncthreads();
  build(xs, lut);
  __syncthreads();
  uint32_t un[SB];  // ids of the next batch, loaded one batch ahead
  load_ids<BITS, SB>(row, 0, S, a.R, un);
  for (int64_t b = 0; b < nb; ++b) {
    float* cur = lut + (b & 1) * per_buf;
    uint32_t u[SB];
#pragma unroll
    for (int j = 0; j < SB; ++j) u[j] = un[j];
    if (b + 1 < nb) load_ids<BITS, SB>(row, (b + 1) * SB, S, a.R, un);
    if (b + 1 < nb) build(xs + ((b + 1) & 1) * XS, lut + ((b + 1) & 1) * per_buf);
#pragma unroll
    for (int j = 0; j < SB; ++j) {
      if (b * SB + j < S) {
#pragma unroll
        for (int t = 0; t < LT; ++t) acc[t] += cur[(j * LT + t) * C + u[j]];
      }
    }
    __syncthreads();  // tables of b + 1 built, x slice of b + 1 read: buffers of b and b + 1 swap roles
    if (b + 2 < nb) {
      stage_x(b + 2, xs + (b & 1) * XS);
      __syncthreads();
    }
  }
  if (n < a.N) {
#pragma unroll
    for (int t = 0; t < LT; ++t)
      if (t0 + t < a.M) a.y[(t0 + t) * a.N + n] = static_cast<half_t>(acc[t]);
  }
}

template <int BITS, int D, int SB>
hipError_t launch_lut(const LutArgs& a, hipStream_t stream) {
  auto kern = k_gemm_lut<BITS, D, SB>;
  if (plan_record("k_gemm_lut", {BITS, D, SB})) return hipSuccess;
  hipError_t e = prepare_kernel(kern);
  if (e != hipSuccess) return e;
  const int lds = (2 * SB * kLutTokens * a.C + 2 * kLutTokens * SB * D) * 4;
  dim3 grid((unsigned)((a.N + kLutThreads - 1) / kLutThreads), (unsigned)((a.M + kLutTokens - 1) / kLutTokens));
  return launch_kernel(kern, grid, dim3(kLutThreads), lds, stream, a);
}

template <int BITS, int D>
hipError_t launch_lut_sb(const LutArgs& a, int sb, hipStream_t stream) {
  switch (sb) {
    case 8: return launch_lut<BITS, D, 8>(a, stream);
    case 4: return launch_lut<BITS, D, 4>(a, stream);
    case 2: return launch_lut<BITS, D, 2>(a, stream);
    default: return launch_lut<BITS, D, 1>(a, stream);
  }
}

template <int BITS>
hipError_t launch_lut_d(const LutArgs& a, int d, int sb, hipStream_t stream) {
  switch (d) {
    case 1: return launch_lut_sb<BITS, 1>(a, sb, stream);
    case 2: return launch_lut_sb<BITS, 2>(a, sb, stream);
    case 4: return launch_lut_sb<BITS, 4>(a, sb, stream);
    default: return launch_lut_sb<BITS, 8>(a, sb, stream);
  }
}

}  // namespace

hipError_t launch_gemm_lut(const Problem& p, hipStream_t stream) {
  const int d = p.d;
  if (p.cb_stride != 0 || !(d == 1 || d == 2 || d == 4 || d == 8)) return hipErrorNotSupported;
  // subspaces per batch: as many as the two table buffers hold, up to 8
  int sb = 8;
  while (sb > 1 && (int64_t)sb * kLutTokens * p.C > kLutEntries) sb /= 2;
  if ((int64_t)sb * kLutTokens * p.C > kLutEntries) return hipErrorNotSupported;
  if ((p.N + kLutThreads - 1) / kLutThreads > 0x7fffffff || (p.M + kLutTokens - 1) / kLutTokens > 65535)
    return hipErrorNotSupported;
  LutArgs a;
  a.x = static_cast<const half_t*>(p.x);
  a.M = p.M;
  a.K = p.K;
  a.N = p.N;
  a.idx = static_cast<const uint8_t*>(p.idx);
  a.R = p.R;
  a.cb = static_cast<const half_t*>(p.codebook);
  a.C = (int)p.C;
  a.y = static_cast<half_t*>(p.y);
  switch (p.idx_bits) {
    case 8: return launch_lut_d<8>(a, d, sb, stream);
    case 12: return launch_lut_d<12>(a, d, sb, stream);
    default: return launch_lut_d<16>(a, d, sb, stream);
  }
}

}  // namespace fasq
