// Calibration-free PQ encoding (FASQ Sec. 3.1.1, Alg. 1): Lloyd's k-means over
// the sub-vectors of a weight matrix, with one codebook shared by every
// subspace (the format the matmul kernels consume).
//
// Definition (the paper leaves these details open):
//   * point p = n * (K / d) + s is w[n, s*d : (s+1)*d]; W is [N x K] row-major,
//     so the points are P = N * K / d consecutive runs of d fp16 values;
//   * assignment: squared Euclidean distance evaluated in fp32 as
//     acc = 0; acc = acc + (w_i - c_i) * (w_i - c_i), i = 0 .. d-1, every
//     operation rounded separately (no fused multiply-add); the lowest index
//     wins a tie;
//   * update: the cluster sum is exact (an fp16 value times 2^24 is an
//     integer; |w| < 128 keeps the sums inside 64 bits), then
//     mean = (fp64(sum) * 2^-24) / fp64(count), rounded to fp16 (nearest,
//     ties to even); an empty cluster keeps its codeword;
//   * iters updates, then a last assignment against the final codebook gives
//     the ids, packed in the library's id format.
// Exact integer sums make the result independent of the order in which the
// atomics land: the encoder is deterministic.
#include "fasq_device.h"
#include "fasq_internal.h"

namespace fasq {

namespace {

constexpr int kEncThreads = 256;
constexpr int kEncPointsPerThread = 4;
constexpr int kEncTileFloats = 16384;                // codeword tile in LDS: 64 KB of fp32
constexpr int kEncAggBytes = 64 * 1024;              // per-workgroup cluster sums in LDS, when they fit
constexpr float kQScale = 16777216.0f;               // 2^24
constexpr double kQInv = 1.0 / 16777216.0;

// fp64 -> fp16, round to nearest, ties to even, by integer operations on the
// fp64 encoding (one rounding step; inputs are finite).
__device__ __forceinline__ uint16_t f64_to_f16_rne(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  const int ex = (int)((b >> 52) & 0x7FF);
  if (ex == 0) return sign;  // zero or an fp64 subnormal: far below half the smallest fp16
  const uint64_t m = (b & ((uint64_t(1) << 52) - 1)) | (uint64_t(1) << 52);  // 53-bit significand
  const int e = ex - 1023;  // v = m * 2^(e - 52)
  if (e > 15) return sign | 0x7C00u;
  int shift;  // bits of m below the fp16 result's last place
  if (e >= -14) shift = 42;            // normal: 11 significant bits kept
  else if (e >= -25) shift = 28 - e;   // subnormal: result in units of 2^-24
  else return sign;                    // below 2^-25: rounds to zero
  const uint64_t q = m >> shift;
  const uint64_t rem = m & ((uint64_t(1) << shift) - 1);
  const uint64_t half = uint64_t(1) << (shift - 1);
  uint32_t r = (uint32_t)q + ((rem > half || (rem == half && (q & 1))) ? 1u : 0u);
  if (e >= -14) {
    // r in [2^10, 2^11]; a carry to 2^11 moves up one binade
    int ee = e + 15;
    if (r == 0x800u) { r = 0x400u; ++ee; }
    if (ee >= 31) return sign | 0x7C00u;
    return sign | (uint16_t)(ee << 10) | (uint16_t)(r & 0x3FFu);
  }
  // subnormal result r * 2^-24, r <= 2^10 (2^10 is the smallest normal, exponent field 1)
  return sign | (uint16_t)r;
}

__global__ void k_enc_copy(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

__global__ void k_enc_zero(int64_t* __restrict__ p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// Squared distance in fp32, operations in the defined order, no contraction.
template <int D>
__device__ __forceinline__ float sq_dist(const float* p, const float* c, int d) {
#pragma clang fp contract(off)
  float acc = 0.f;
  if constexpr (D > 0) {
#pragma unroll
    for (int i = 0; i < D; ++i) {
      const float diff = p[i] - c[i];
      acc = acc + diff * diff;
    }
  } else {
    for (int i = 0; i < d; ++i) {
      const float diff = p[i] - c[i];
      acc = acc + diff * diff;
    }
  }
  return acc;
}

// Assignment of every point to its nearest codeword; with ACCUM the points'
// exact fixed-point values and counts are added to the cluster sums (through
// a per-workgroup LDS table when AGG).  D = 0: runtime d <= 16.
template <int D, bool ACCUM, bool AGG>
__global__ __launch_bounds__(kEncThreads) void k_enc_assign(const half_t* __restrict__ w, int64_t P, int d,
                                                            const half_t* __restrict__ cb, int C,
                                                            uint32_t* __restrict__ assign,
                                                            int64_t* __restrict__ sums,
                                                            int64_t* __restrict__ counts) {
  constexpr int DM = D > 0 ? D : 16;
  constexpr int PPT = kEncPointsPerThread;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  float* tile = reinterpret_cast<float*>(smem);                       // [ct][d] fp32 codewords
  int64_t* agg = reinterpret_cast<int64_t*>(smem + kEncTileFloats * 4);  // [C][d + 1] sums, counts
  const int dd = D > 0 ? D : d;
  const int ct = kEncTileFloats / dd;  // codewords per tile
  const int ntiles = (C + ct - 1) / ct;

  if constexpr (AGG) {
    for (int i = threadIdx.x; i < C * (dd + 1); i += blockDim.x) agg[i] = 0;
  }

  const int64_t group = (int64_t)kEncThreads * PPT;
  bool staged = false;
  for (int64_t g0 = blockIdx.x * group; g0 < P; g0 += (int64_t)gridDim.x * group) {
    float pv[PPT][DM];
    float best[PPT];
    uint32_t bk[PPT];
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const int64_t p = g0 + (int64_t)j * kEncThreads + threadIdx.x;
      const int64_t pc = p < P ? p : P - 1;
#pragma unroll
      for (int i = 0; i < DM; ++i) pv[j][i] = (i < dd) ? static_cast<float>(w[pc * dd + i]) : 0.f;
      best[j] = __builtin_inff();
      bk[j] = 0;
    }
    for (int t = 0; t < ntiles; ++t) {
      const int k0 = t * ct;
      const int nk = C - k0 < ct ? C - k0 : ct;
      if (!(staged && ntiles == 1)) {
        __syncthreads();  // everyone is done with the previous tile
        for (int i = threadIdx.x; i < nk * dd; i += blockDim.x) tile[i] = static_cast<float>(cb[(int64_t)k0 * dd + i]);
        __syncthreads();
        staged = true;
      }
      for (int k = 0; k < nk; ++k) {
        const float* c = tile + k * dd;
#pragma unroll
        for (int j = 0; j < PPT; ++j) {
          const float dist = sq_dist<D>(pv[j], c, dd);
          if (dist < best[j]) {  // strict: the lowest index keeps a tie
            best[j] = dist;
            bk[j] = (uint32_t)(k0 + k);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const int64_t p = g0 + (int64_t)j * kEncThreads + threadIdx.x;
      if (p >= P) continue;
      assign[p] = bk[j];
      if constexpr (ACCUM) {
        const uint32_t k = bk[j];
        for (int i = 0; i < dd; ++i) {
          const int64_t q = (int64_t)(pv[j][i] * kQScale);  // exact: an integer below 2^31
          if constexpr (AGG) atomicAdd(reinterpret_cast<unsigned long long*>(&agg[k * (dd + 1) + i]),
                                       (unsigned long long)q);
          else atomicAdd(reinterpret_cast<unsigned long long*>(&sums[(int64_t)k * dd + i]), (unsigned long long)q);
        }
        if constexpr (AGG) atomicAdd(reinterpret_cast<unsigned long long*>(&agg[k * (dd + 1) + dd]), 1ull);
        else atomicAdd(reinterpret_cast<unsigned long long*>(&counts[k]), 1ull);
      }
    }
  }
  if constexpr (ACCUM && AGG) {
    __syncthreads();
    for (int k = threadIdx.x; k < C; k += blockDim.x) {
      const int64_t cnt = agg[k * (dd + 1) + dd];
      if (cnt == 0) continue;
      for (int i = 0; i < dd; ++i)
        atomicAdd(reinterpret_cast<unsigned long long*>(&sums[(int64_t)k * dd + i]),
                  (unsigned long long)agg[k * (dd + 1) + i]);
      atomicAdd(reinterpret_cast<unsigned long long*>(&counts[k]), (unsigned long long)cnt);
    }
  }
}

// New codewords: each non-empty cluster's rounded mean; empty ones are kept.
__global__ void k_enc_update(uint16_t* __restrict__ cb, const int64_t* __restrict__ sums,
                             const int64_t* __restrict__ counts, int C, int d) {
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < (int64_t)C * d;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = t / d;
    const int64_t cnt = counts[k];
    if (cnt == 0) continue;
    const double mean = (static_cast<double>(sums[t]) * kQInv) / static_cast<double>(cnt);
    cb[t] = f64_to_f16_rne(mean);
  }
}

// ids [N x S] (uint32) -> packed rows of R bytes.  One thread per id pair
// for 12-bit ids (three bytes), per id otherwise.
template <int BITS>
__global__ void k_enc_pack(const uint32_t* __restrict__ ids, int64_t N, int64_t S, int64_t R,
                           uint8_t* __restrict__ idx) {
  const int64_t per_row = BITS == 12 ? (S + 1) / 2 : S;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * per_row;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t n = t / per_row;
    const int64_t j = t - n * per_row;
    uint8_t* row = idx + n * R;
    const uint32_t* u = ids + n * S;
    if constexpr (BITS == 8) {
      row[j] = (uint8_t)u[j];
    } else if constexpr (BITS == 16) {
      row[2 * j] = (uint8_t)(u[j] & 0xFF);
      row[2 * j + 1] = (uint8_t)(u[j] >> 8);
    } else {
      const uint32_t a = u[2 * j];
      const uint32_t b = 2 * j + 1 < S ? u[2 * j + 1] : 0u;  // the pad nibble of an odd row is 0
      row[3 * j] = (uint8_t)(a & 0xFF);
      if (3 * j + 1 < R) row[3 * j + 1] = (uint8_t)((a >> 8) | ((b & 0xF) << 4));
      if (3 * j + 2 < R) row[3 * j + 2] = (uint8_t)(b >> 4);
    }
  }
}

inline unsigned grid_for(int64_t n, int threads) {
  const int64_t g = (n + threads - 1) / threads;
  return (unsigned)(g < 65536 ? (g > 0 ? g : 1) : 65536);
}

template <int D>
hipError_t launch_assign_d(const half_t* w, int64_t P, int d, const half_t* cb, int C, uint32_t* assign,
                           int64_t* sums, int64_t* counts, bool accum, const DeviceInfo& dev, hipStream_t stream) {
  const int dd = D > 0 ? D : d;
  const bool agg = accum && (int64_t)C * (dd + 1) * 8 <= kEncAggBytes;
  const int lds = kEncTileFloats * 4 + (agg ? C * (dd + 1) * 8 : 0);
  const int64_t groups = (P + (int64_t)kEncThreads * kEncPointsPerThread - 1) / ((int64_t)kEncThreads * kEncPointsPerThread);
  // enough workgroups to fill the chip; more would only repeat the codebook staging and the LDS flushes
  int64_t blocks = 4 * (int64_t)dev.num_cus;
  if (blocks > groups) blocks = groups;
  if (blocks < 1) blocks = 1;
  auto go = [&](auto kern) {
    hipError_t e = prepare_kernel(kern);
    if (e != hipSuccess) return e;
    return launch_kernel(kern, dim3((unsigned)blocks), dim3(kEncThreads), lds, stream, w, P, d, cb, C, assign, sums,
                         counts);
  };
  if (!accum) return go(k_enc_assign<D, false, false>);
  return agg ? go(k_enc_assign<D, true, true>) : go(k_enc_assign<D, true, false>);
}

hipError_t launch_assign(const half_t* w, int64_t P, int d, const half_t* cb, int C, uint32_t* assign, int64_t* sums,
                         int64_t* counts, bool accum, const DeviceInfo& dev, hipStream_t stream) {
  switch (d) {
    case 1: return launch_assign_d<1>(w, P, d, cb, C, assign, sums, counts, accum, dev, stream);
    case 2: return launch_assign_d<2>(w, P, d, cb, C, assign, sums, counts, accum, dev, stream);
    case 4: return launch_assign_d<4>(w, P, d, cb, C, assign, sums, counts, accum, dev, stream);
    case 8: return launch_assign_d<8>(w, P, d, cb, C, assign, sums, counts, accum, dev, stream);
    default: return launch_assign_d<0>(w, P, d, cb, C, assign, sums, counts, accum, dev, stream);
  }
}

}  // namespace

int64_t encode_workspace_bytes(int64_t N, int64_t K, int d, int64_t C) {
  const int64_t P = N * (K / d);
  const int64_t head = ((C * d + C) * 8 + 255) / 256 * 256;
  return head + P * 4;
}

hipError_t launch_encode(const EncodeProblem& e, const DeviceInfo& dev, hipStream_t stream) {
  const int64_t S = e.K / e.d;
  const int64_t P = e.N * S;
  const int d = e.d;
  const int C = (int)e.C;
  uint8_t* ws = static_cast<uint8_t*>(e.workspace);
  int64_t* sums = reinterpret_cast<int64_t*>(ws);
  int64_t* counts = sums + (int64_t)C * d;
  uint32_t* assign = reinterpret_cast<uint32_t*>(ws + ((e.C * d + e.C) * 8 + 255) / 256 * 256);
  const half_t* w = static_cast<const half_t*>(e.w);
  uint16_t* cb = static_cast<uint16_t*>(e.codebook);
  const int64_t cbn = (int64_t)C * d;
  hipError_t err;
  if (e.init != e.codebook) {
    err = launch_kernel(k_enc_copy, dim3(grid_for(cbn, 256)), dim3(256), 0, stream,
                        static_cast<const uint16_t*>(e.init), cb, cbn);
    if (err != hipSuccess) return err;
  }
  for (int it = 0; it < e.iters; ++it) {
    err = launch_kernel(k_enc_zero, dim3(grid_for(cbn + C, 256)), dim3(256), 0, stream, sums, cbn + C);
    if (err != hipSuccess) return err;
    err = launch_assign(w, P, d, reinterpret_cast<const half_t*>(cb), C, assign, sums, counts, true, dev, stream);
    if (err != hipSuccess) return err;
    err = launch_kernel(k_enc_update, dim3(grid_for(cbn, 256)), dim3(256), 0, stream, cb, sums, counts, C, d);
    if (err != hipSuccess) return err;
  }
  err = launch_assign(w, P, d, reinterpret_cast<const half_t*>(cb), C, assign, sums, counts, false, dev, stream);
  if (err != hipSuccess) return err;
  const int64_t per_row = e.idx_bits == 12 ? (S + 1) / 2 : S;
  const unsigned g = grid_for(e.N * per_row, 256);
  uint8_t* idx = static_cast<uint8_t*>(e.idx);
  switch (e.idx_bits) {
    case 8: return launch_kernel(k_enc_pack<8>, dim3(g), dim3(256), 0, stream, assign, e.N, S, e.R, idx);
    case 12: return launch_kernel(k_enc_pack<12>, dim3(g), dim3(256), 0, stream, assign, e.N, S, e.R, idx);
    default: return launch_kernel(k_enc_pack<16>, dim3(g), dim3(256), 0, stream, assign, e.N, S, e.R, idx);
  }
}

}  // namespace fasq
