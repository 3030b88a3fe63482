// Prefill GEMM: Y[M x N] = X[M x K] . W_hat^T with W_hat decoded tile by tile.
//
// Design (gfx950, wave64, v_mfma_f32_32x32x16_f16):
//   * A workgroup of WGM x WGN waves owns a BM x BN output tile, each wave
//     owning (BM/WGM) x (BN/WGN) = FM x FN MFMA tiles of 32 x 32 with fp32
//     accumulators in registers.
//   * K is walked in chunks of 64.  Each chunk's X tile (BM x 64 fp16) and
//     packed-id tile (BN columns) are copied from global memory straight
//     into LDS (global_load_lds), NS - 1 chunks ahead, into a ring of NS LDS
//     stages: the copies need no registers, so the loads of several chunks
//     are in flight while one is computed.  Small tiles take a deeper ring:
//     a workgroup that computes a chunk in a few hundred cycles waits on
//     memory latency unless many chunks are in flight.  X rows are 128 B
//     with their 16-byte granules XOR-swizzled by (row / 2) mod 8, so the
//     MFMA operand reads of one LDS cycle hit distinct banks.
//   * W_hat is never written to memory, not even to LDS: each lane decodes
//     the ids of its own B-operand column from the staged id tile and
//     gathers the codewords from the LDS codebook into the MFMA B registers.
//     The order of K inside a chunk is permuted identically for A and B
//     (allowed: the contraction is a sum over K), so that lane half h reads
//     one contiguous run of 32/d ids per chunk.
//   * Software pipeline: each wave reads the A and B operands of k-step
//     t + 1 from LDS while the matrix cores work on step t.
//   * Synchronisation: one workgroup barrier per chunk, in the middle of it
//     (after an explicit wait for this wave's copies of the next chunk):
//     every wave's copies of the next chunk are in, and every wave is done
//     with the stage about to be refilled.
//   * Epilogue: fp32 -> fp16 once, direct stores.
#pragma once

#include "fasq_device.h"
#include "fasq_codebook.h"
#include "fasq_internal.h"

namespace fasq {

constexpr int kGemmKC = 64;          // K per chunk

struct GemmArgs {
  const half_t* x;
  int64_t M, K, N;
  const uint8_t* idx;
  int64_t R;
  const half_t* cb;
  int C;
  int cb_lds_bytes;
  half_t* y;
  int ksplit;  // workgroups along K (grid z); above 1 the partials go to ws
  float* ws;   // [ksplit][M][N] fp32 partial sums when ksplit > 1
};

// Bytes of one packed-id run (one lane half, one chunk) and of one stage.
template <int BITS, int D>
__host__ __device__ constexpr int gemm_run_bytes() { return (32 / D) * BITS / 8; }
template <int BITS, int D, int BM, int BN>
__host__ __device__ constexpr int gemm_stage_bytes() { return BM * 128 + BN * 2 * gemm_run_bytes<BITS, D>(); }

// Ring depth of a tile: the wanted depth, reduced until the copies a wave
// keeps in flight, (depth - 2) chunks of them, fit the 6-bit vmcnt counter.
__host__ __device__ constexpr int gemm_ring_depth(int bits, int d, int bm, int bn, int waves, int want) {
  const int loads = bm / waves / 8 + bn * ((32 / d) * bits / 8 * 2 / 4) / (waves * 64);
  int ns = want;
  while (ns > 3 && loads * (ns - 2) >= 64) --ns;
  return ns;
}

// Copy 16 (or 4) bytes per lane from global memory into LDS: lane i's data
// lands at lds + 16 i (4 i).
__device__ __forceinline__ void copy16_to_lds(const void* src, uint8_t* lds) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}
__device__ __forceinline__ void copy4_to_lds(const void* src, uint8_t* lds) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds, 4, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt out of range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt with only the LDS/scalar counter constrained, to zero.
__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (0x7 << 4) | (0 << 8));
}

// KG > 1 splits K inside the workgroup: KG groups of WGM x WGN waves, each
// with its own ring, take the chunks c = KG * it + kg (group kg, iteration
// it) of the same output tile, and their accumulators are summed through LDS
// in group order at the end.  Small grids use it to keep several waves per
// SIMD busy.
template <int BITS, int D, int MODE, int BM, int BN, int WGM, int WGN, int NS, int KG>
__global__ __launch_bounds__(WGM * WGN * KG * 64) void k_gemm_mfma(GemmArgs a) {
  constexpr int WAVES = WGM * WGN;                 // waves per K group
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int HB = gemm_run_bytes<BITS, D>();    // bytes per lane half per chunk
  constexpr int IPS = 8 / D;                       // ids per k-step per lane
  constexpr int XR = BM / WAVES;                   // X tile rows copied by each wave
  constexpr int XI = XR / 8;                       // X copy instructions per wave per chunk (8 rows each)
  constexpr int IW = 2 * HB / 4;                   // id words per column per chunk
  constexpr int II = BN * IW / (WAVES * kWave);    // id copy instructions per wave per chunk
  constexpr int LPC = XI + II;                     // vector-memory instructions per wave per chunk
  constexpr int XBYTES = BM * 128;
  constexpr int SBYTES = gemm_stage_bytes<BITS, D, BM, BN>();
  static_assert(WM % 32 == 0 && WN % 32 == 0 && XR % 8 == 0, "tile does not split over the waves");
  static_assert(HB % 4 == 0, "index run must be whole dwords");
  static_assert((BN * IW) % (WAVES * kWave) == 0, "id tile must split evenly over the workgroup");
  static_assert(NS >= 3 && LPC * (NS - 2) < 64, "ring depth out of range for vmcnt");

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int tid = threadIdx.x;
  // K group and wave index as wave-uniform (scalar) values: a branch on them
  // is a real jump.  (MFMA ignores the execution mask, so a group's skipped
  // chunk must not become a masked branch.)
  const int kg = __builtin_amdgcn_readfirstlane(tid / (WAVES * kWave));
  const int wave = __builtin_amdgcn_readfirstlane((tid / kWave) % WAVES), lane = tid % kWave;
  const int wm = wave / WGN, wn = wave % WGN;
  const int h = lane >> 5, l32 = lane & 31;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const int64_t n0 = (int64_t)blockIdx.x * BN;
  // K range of this workgroup: chunks [c_begin, c_begin + nchunks) of K / 64
  const int all_chunks = (int)(a.K / kGemmKC);
  const int c_begin = (int)((int64_t)blockIdx.z * all_chunks / a.ksplit);
  const int nchunks = (int)((int64_t)(blockIdx.z + 1) * all_chunks / a.ksplit) - c_begin;
  const int niter = (nchunks + KG - 1) / KG;       // chunks per group (the last ones may lie past K)
  uint8_t* ring = smem + a.cb_lds_bytes + kg * (NS * SBYTES);  // NS stages of [X tile][id tile]
  // data chunk of iteration it, clamped into K for the copies
  auto chunk_of = [&](int it) { const int c = it * KG + kg; return c < nchunks ? c : nchunks - 1; };

  // ---- copy sources of this lane (rows >= M read row M - 1, columns >= N
  //      read column 0: they are computed but never stored)
  const half_t* xsrc[XI];
#pragma unroll
  for (int j = 0; j < XI; ++j) {
    const int r = wave * XR + j * 8 + lane / 8;        // tile row
    const int g = (lane % 8) ^ ((r >> 1) & 7);         // granule stored in slot lane % 8
    const int64_t m = m0 + r;
    xsrc[j] = a.x + (m < a.M ? m : a.M - 1) * a.K + g * 8;
  }
  const uint8_t* isrc[II];
#pragma unroll
  for (int j = 0; j < II; ++j) {
    const int gl = (wave * II + j) * kWave + lane;     // word slot in the id tile
    const int64_t n = n0 + gl / IW;
    isrc[j] = a.idx + (n < a.N ? n : 0) * a.R + (gl % IW) * 4;
  }
  auto issue = [&](int lc, int stage) {
    const int c = c_begin + lc;
    uint8_t* sb = ring + stage * SBYTES;
#pragma unroll
    for (int j = 0; j < XI; ++j)
      copy16_to_lds(xsrc[j] + (int64_t)c * kGemmKC, sb + (wave * XR + j * 8) * 128);
#pragma unroll
    for (int j = 0; j < II; ++j)
      copy4_to_lds(isrc[j] + (int64_t)c * (2 * HB), sb + XBYTES + (wave * II + j) * kWave * 4);
  };

  // The codebook (L2-resident) is staged first.
  CbStage cst;
  cb_fetch<D, MODE>(a.cb, a.C, cst);
  cb_store<D, MODE>(smem, a.cb, a.C, cst);
  __syncthreads();

#pragma unroll
  for (int s = 0; s < NS - 1; ++s) issue(chunk_of(s), s);

  float16_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[fm][fn][i] = 0.f;

  const uint32_t lane_off = cb_lane_off<D, MODE>(lane);

  // Operands of one k-step: FM A fragments from the X tile, FN B fragments
  // gathered from the codebook.
  struct Ops {
    half8_t a[FM];
    half8_t b[FN];
  };
  auto read_ids = [&](int stage, uint32_t (&ids)[FN][HB / 4]) {
    const uint8_t* ib = ring + stage * SBYTES + XBYTES;
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const uint8_t* p = ib + (wn * WN + fn * 32 + l32) * (2 * HB) + h * HB;
#pragma unroll
      for (int w = 0; w < HB / 4; ++w) ids[fn][w] = reinterpret_cast<const uint32_t*>(p)[w];
    }
  };
  auto read_ops = [&](Ops& o, int stage, const uint32_t (&ids)[FN][HB / 4], int t) {
    const uint8_t* xb = ring + stage * SBYTES;
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) o.b[fn] = gather8<BITS, D, MODE>(a.cb, lane_off, ids[fn], t * IPS);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int r = wm * WM + fm * 32 + l32;
      const int slot = (h * 4 + t) ^ ((r >> 1) & 7);
      o.a[fm] = *reinterpret_cast<const half8_t*>(xb + r * 128 + slot * 16);
    }
  };
  // Four-wave tiles (one wave per SIMD, or two K groups) pin the order: the
  // reads of the next step stay ahead of this step's MFMAs (scheduling
  // barriers on both sides), and each step starts with an explicit wait for
  // the reads of the step before.  Two steps of reads (16 with d = 4) are
  // more than the LDS counter can name, so the compiler's own wait, placed
  // after the next step's reads, would wait for those as well.  The
  // eight-wave tiles measured faster with the compiler's interleaving (the
  // other wave of the SIMD covers the waits).
  constexpr bool kPinSteps = WAVES == 4;
  auto step_reads = [&](Ops& o, int stage, const uint32_t (&ids)[FN][HB / 4], int t) {
    if constexpr (kPinSteps) {
      __builtin_amdgcn_sched_barrier(0);
      wait_lgkmcnt0();
    }
    read_ops(o, stage, ids, t);
  };
  auto mfma_step = [&](const Ops& o, bool valid) {
    if constexpr (kPinSteps) __builtin_amdgcn_sched_barrier(0);
    if (KG > 1 && !valid) return;  // a group's last chunk past K
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(o.a[fm], o.b[fn], acc[fm][fn], 0, 0, 0);
    if constexpr (kPinSteps) __builtin_amdgcn_sched_barrier(0);
  };

  // Software pipeline: the operands of k-step t + 1 are read while the
  // matrix cores work on step t, across chunk boundaries too.  One step
  // ahead keeps at most one step's LDS reads (plus the next ids) in flight,
  // few enough for the 4-bit LDS counter, so each wait names exactly the
  // reads it needs.  The control flow is the same in every chunk (the last
  // one reads and copies a clamped chunk it does not use), so no join point
  // makes the compiler wait for every read in flight.  The workgroup barrier
  // sits after the chunk's first step: every wave has finished chunk c - 1
  // (its stage can be refilled) and, after waiting for its own copies,
  // chunk c + 1 is in LDS (its ids and first operands can be read).
  wait_vmcnt<LPC * (NS - 2)>();  // this wave's copies of chunk 0
  __builtin_amdgcn_s_barrier();  // everyone's
  uint32_t idc[FN][HB / 4], idn[FN][HB / 4];
  read_ids(0, idc);
  Ops oa, ob;
  read_ops(oa, 0, idc, 0);
  for (int c = 0; c < niter; ++c) {
    const int stage = c % NS;
    const int nstage = (c + 1) % NS;
    const bool valid = c * KG + kg < nchunks;
    step_reads(ob, stage, idc, 1);
    mfma_step(oa, valid);
    wait_vmcnt<LPC * (NS - 3)>();  // this wave's copies of chunk c + 1
    __builtin_amdgcn_s_barrier();  // everyone's; nobody reads chunk c - 1 any more
    issue(chunk_of(c + NS - 1 < niter ? c + NS - 1 : niter - 1), (c + NS - 1) % NS);
    read_ids(nstage, idn);
    step_reads(oa, stage, idc, 2);
    mfma_step(ob, valid);
    step_reads(ob, stage, idc, 3);
    mfma_step(oa, valid);
    step_reads(oa, nstage, idn, 0);
    mfma_step(ob, valid);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int w = 0; w < HB / 4; ++w) idc[fn][w] = idn[fn][w];
  }
  wait_vmcnt<0>();  // drain the clamped copies issued past the last chunk

  if constexpr (KG > 1) {
    // Groups 1 .. KG-1 leave their accumulators in LDS (16-byte vectors,
    // lanes contiguous), group 0 adds them in group order.
    float4_t* dump = reinterpret_cast<float4_t*>(smem);
    auto slot = [&](int g, int fm, int fn, int i4) {
      return ((((g - 1) * WAVES + wave) * FM + fm) * FN + fn) * 4 * kWave + i4 * kWave + lane;
    };
    __syncthreads();  // every group is done with its ring and the codebook
    if (kg > 0) {
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
#pragma unroll
          for (int i4 = 0; i4 < 4; ++i4)
            dump[slot(kg, fm, fn, i4)] = float4_t{acc[fm][fn][4 * i4], acc[fm][fn][4 * i4 + 1],
                                                  acc[fm][fn][4 * i4 + 2], acc[fm][fn][4 * i4 + 3]};
    }
    __syncthreads();
    if (kg > 0) return;
    for (int g = 1; g < KG; ++g) {
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
#pragma unroll
          for (int i4 = 0; i4 < 4; ++i4) {
            const float4_t v = dump[slot(g, fm, fn, i4)];
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[fm][fn][4 * i4 + k] += v[k];
          }
    }
  }

  // ---- epilogue: lane l holds rows (i/4)*8 + h*4 + i%4, column l32 of each
  //      32x32 tile; fp16 outputs, or this K range's fp32 partial sums
  float* part = a.ws + (int64_t)blockIdx.z * a.M * a.N;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t n = n0 + wn * WN + fn * 32 + l32;
      if (n >= a.N) continue;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t m = m0 + wm * WM + fm * 32 + (i / 4) * 8 + h * 4 + (i % 4);
        if (m >= a.M) continue;
        if (a.ksplit > 1) part[m * a.N + n] = acc[fm][fn][i];
        else a.y[m * a.N + n] = static_cast<half_t>(acc[fm][fn][i]);
      }
    }
  }
}

// y = fp16(sum over the K ranges, in range order, of the fp32 partials).
// (At most eight ranges: loading them all before the first add, as the
// per-subspace reduction does, measured 1 % slower at a split of two.)
// VEC: four outputs per thread (16-byte partial loads, one 8-byte store),
// taken when MN is a multiple of 4 and the buffers are aligned for it.
template <bool VEC>
__global__ void k_gemm_split_reduce(const float* __restrict__ ws, int64_t MN, int ksplit, half_t* __restrict__ y) {
  if constexpr (VEC) {
    const int64_t n4 = MN / 4;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
      float4_t s = float4_t{0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < ksplit; ++k) s += reinterpret_cast<const float4_t*>(ws + (int64_t)k * MN)[i];
      half4_t h;
      h[0] = static_cast<half_t>(s[0]);
      h[1] = static_cast<half_t>(s[1]);
      h[2] = static_cast<half_t>(s[2]);
      h[3] = static_cast<half_t>(s[3]);
      reinterpret_cast<half4_t*>(y)[i] = h;
    }
  } else {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < MN; i += (int64_t)gridDim.x * blockDim.x) {
      float s = 0.f;
      for (int k = 0; k < ksplit; ++k) s += ws[(int64_t)k * MN + i];
      y[i] = static_cast<half_t>(s);
    }
  }
}

}  // namespace fasq
