// Reconstruction kernel and the general-purpose PQ matmul kernel.
//
// The general kernel handles every valid argument combination (any M, K, N,
// d, C, id width, pointer alignment); the tuned GEMV/GEMM kernels cover the
// common shapes and fall back to it for the rest.
#include "fasq_device.h"
#include "fasq_internal.h"

namespace fasq {

// W_hat[n, s*d + i] = codebook[u(n, s)*d + i], moved as raw 16-bit patterns.
// One thread per (n, s); grid-stride over all N*S sub-vectors.
template <int BITS>
__global__ __launch_bounds__(256) void k_reconstruct(const uint8_t* __restrict__ idx, int64_t N, int64_t S,
                                                     int64_t R, int d, const uint16_t* __restrict__ cb,
                                                     int64_t cbs, uint16_t* __restrict__ w) {
  const int64_t total = N * S;
  const int64_t K = S * d;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t n = t / S;
    const int64_t s = t - n * S;
    const uint32_t u = load_id_bytes<BITS>(idx + n * R, s, R);
    const uint16_t* src = cb + s * cbs + (int64_t)u * d;
    uint16_t* dst = w + n * K + s * d;
    for (int i = 0; i < d; ++i) dst[i] = src[i];
  }
}

// y[m, n] = sum_s dot(x[m, s*d:(s+1)*d], codebook[u(n, s)]), fp32 accumulation
// (codebook s of subspace s at cb + s * cbs when the books are per subspace).
// One wave per output row n; lanes stride over the S sub-vectors; MB rows of
// x are accumulated at a time.  Codewords are read from global memory.
constexpr int kGenericMB = 8;

template <int BITS>
__global__ __launch_bounds__(256) void k_pq_generic(const half_t* __restrict__ x, int64_t M, int64_t K,
                                                    int64_t N, const uint8_t* __restrict__ idx, int64_t R,
                                                    int d, const half_t* __restrict__ cb, int64_t cbs,
                                                    half_t* __restrict__ y) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
  const int64_t S = K / d;
  for (int64_t n = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave; n < N; n += waves) {
    const uint8_t* row = idx + n * R;
    for (int64_t m0 = 0; m0 < M; m0 += kGenericMB) {
      const int mb = (int)((M - m0) < kGenericMB ? (M - m0) : kGenericMB);
      float acc[kGenericMB];
#pragma unroll
      for (int j = 0; j < kGenericMB; ++j) acc[j] = 0.f;
      for (int64_t s = lane; s < S; s += kWave) {
        const uint32_t u = load_id_bytes<BITS>(row, s, R);
        const half_t* c = cb + s * cbs + (int64_t)u * d;
        for (int i = 0; i < d; ++i) {
          const float cv = static_cast<float>(c[i]);
          const half_t* xp = x + m0 * K + s * d + i;
#pragma unroll
          for (int j = 0; j < kGenericMB; ++j)
            if (j < mb) acc[j] = __builtin_fmaf(static_cast<float>(xp[j * K]), cv, acc[j]);
        }
      }
#pragma unroll
      for (int j = 0; j < kGenericMB; ++j) {
        if (j < mb) {
          const float v = wave_sum(acc[j]);
          if (lane == 0) y[(m0 + j) * N + n] = static_cast<half_t>(v);
        }
      }
    }
  }
}

static int grid_for(int64_t items, int per_block, int max_blocks) {
  int64_t b = (items + per_block - 1) / per_block;
  if (b > max_blocks) b = max_blocks;
  if (b < 1) b = 1;
  return (int)b;
}

hipError_t launch_reconstruct(const Problem& p, void* w, hipStream_t stream) {
  const int64_t S = p.K / p.d;
  const int blocks = grid_for(p.N * S, 256, 65536);
  const uint8_t* idx = static_cast<const uint8_t*>(p.idx);
  const uint16_t* cb = static_cast<const uint16_t*>(p.codebook);
  uint16_t* out = static_cast<uint16_t*>(w);
  switch (p.idx_bits) {
    case 8: return launch_kernel(k_reconstruct<8>, dim3(blocks), dim3(256), 0, stream, idx, p.N, S, p.R, p.d, cb, p.cb_stride, out);
    case 12: return launch_kernel(k_reconstruct<12>, dim3(blocks), dim3(256), 0, stream, idx, p.N, S, p.R, p.d, cb, p.cb_stride, out);
    default: return launch_kernel(k_reconstruct<16>, dim3(blocks), dim3(256), 0, stream, idx, p.N, S, p.R, p.d, cb, p.cb_stride, out);
  }
}

hipError_t launch_generic(const Problem& p, hipStream_t stream) {
  if (plan_record("k_pq_generic", {p.idx_bits})) return hipSuccess;
  const int blocks = grid_for(p.N, 4, 8192);
  const half_t* x = static_cast<const half_t*>(p.x);
  const uint8_t* idx = static_cast<const uint8_t*>(p.idx);
  const half_t* cb = static_cast<const half_t*>(p.codebook);
  half_t* y = static_cast<half_t*>(p.y);
  switch (p.idx_bits) {
    case 8: return launch_kernel(k_pq_generic<8>, dim3(blocks), dim3(256), 0, stream, x, p.M, p.K, p.N, idx, p.R, p.d, cb, p.cb_stride, y);
    case 12: return launch_kernel(k_pq_generic<12>, dim3(blocks), dim3(256), 0, stream, x, p.M, p.K, p.N, idx, p.R, p.d, cb, p.cb_stride, y);
    default: return launch_kernel(k_pq_generic<16>, dim3(blocks), dim3(256), 0, stream, x, p.M, p.K, p.N, idx, p.R, p.d, cb, p.cb_stride, y);
  }
}

}  // namespace fasq
