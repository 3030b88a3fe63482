// Host-side variant selection and launch of the decode GEMV (M <= 16).
#pragma once

#include <algorithm>
#include <atomic>

#include "fasq_gemv.h"
#include "fasq_internal.h"

namespace fasq {

constexpr int kLdsCodebookBudget = 64 * 1024;  // bytes of LDS a codebook may take
constexpr int kSliceReserve = 4 * 1024;        // LDS kept for row partials beside a codebook slice
constexpr int kMinSliceBytes = 32 * 1024;      // smaller slices: gather from global memory instead
constexpr int kReplMinIdsPerEntry = 16;        // replicate the codebook only above this many ids per workgroup and entry
constexpr int64_t kMtWideXMinRows = 64;        // two tokens: rows per CU from which x takes twice the registers
constexpr int64_t kM1TwoWgReplMinRows = 64;    // one token, replicated table: rows per CU from which two workgroups share a CU
static_assert(kMaxBatchLaunch <= kM1MaxParts && kMaxBatchLaunch <= kGemvMaxParts,
              "a grouped launch needs a part per matrix at least");

// Codebook placement for a call: replicated in LDS when the replicated table
// fits the budget, one copy in LDS when that fits, else global memory.
inline int choose_cb_mode(int64_t C, int d) {
  if ((C * d * 2) % 16 != 0) return CB_GLOBAL;
  if (cb_lds_bytes(CB_REPL, C, d) <= kLdsCodebookBudget) return CB_REPL;
  if (cb_lds_bytes(CB_LDS, C, d) <= kLdsCodebookBudget) return CB_LDS;
  return CB_GLOBAL;
}

// Cuts `count` matrices of units[i] units each (rows, or 16-row tiles) into
// parts of near-equal size, at most max_parts in all, every part taking the
// same number of workgroups.  A matrix with the largest parts is cut once
// more at each step; the cut kept is the one whose largest part per
// workgroup is smallest, with about one workgroup per CU in all.  cuts[i]
// receives the parts of matrix i; returns the number of parts.
constexpr int kMaxLaunchParts = 8;
static_assert(kM1MaxParts <= kMaxLaunchParts && kGemvMaxParts <= kMaxLaunchParts, "part cuts per launch");
inline int choose_part_cuts(const int64_t* units, int count, int64_t ncu, int max_parts, int* cuts) {
  auto largest = [&](const int* c) {
    int64_t r = 0;
    for (int i = 0; i < count; ++i) {
      const int64_t ri = (units[i] + c[i] - 1) / c[i];
      if (ri > r) r = ri;
    }
    return r;
  };
  int cur[kMaxLaunchParts];
  for (int i = 0; i < count; ++i) cur[i] = cuts[i] = 1;
  int nparts = count, best_parts = count;
  double best_cost = (double)largest(cur) / (double)(ncu / count > 0 ? ncu / count : 1);
  while (nparts < max_parts) {
    int j = -1;
    int64_t jr = 1;
    for (int i = 0; i < count; ++i) {
      const int64_t ri = (units[i] + cur[i] - 1) / cur[i];
      if (cur[i] < units[i] && ri > jr) { j = i; jr = ri; }
    }
    if (j < 0) break;
    ++cur[j];
    ++nparts;
    const double cost = (double)largest(cur) / (double)(ncu / nparts > 0 ? ncu / nparts : 1);
    if (cost < best_cost) {
      best_cost = cost;
      best_parts = nparts;
      for (int i = 0; i < count; ++i) cuts[i] = cur[i];
    }
  }
  return best_parts;
}

template <int BITS, int D, int T, int MODE, int MR>
hipError_t launch_gemv_variant(const GemvArgs& a, bool mask, int threads, dim3 blocks, int lds, hipStream_t stream) {
  if (a.nslab > 1) {  // x in slabs (T up to 4): the plan name carries a trailing 1
    if constexpr (T <= 4) {
      if (plan_record("k_gemv", {BITS, D, T, MODE, MR, 1, 1})) return hipSuccess;
      auto kern = k_gemv<BITS, D, T, MODE, MR, true, true>;
      hipError_t e = prepare_kernel(kern);
      if (e != hipSuccess) return e;
      return launch_kernel(kern, blocks, dim3(threads), lds, stream, a);
    } else {
      return hipErrorNotSupported;
    }
  }
  auto kern = mask ? k_gemv<BITS, D, T, MODE, MR, true, false> : k_gemv<BITS, D, T, MODE, MR, false, false>;
  if (plan_record("k_gemv", {BITS, D, T, MODE, MR, mask ? 1 : 0})) return hipSuccess;
  hipError_t e = prepare_kernel(kern);
  if (e != hipSuccess) return e;
  return launch_kernel(kern, blocks, dim3(threads), lds, stream, a);
}

template <int BITS, int MR, int D, int MODE>
hipError_t launch_gemv_t(const GemvArgs& a, int T, bool mask, int threads, dim3 blocks, int lds,
                         hipStream_t stream) {
  switch (T) {
    case 1: return launch_gemv_variant<BITS, D, 1, MODE, MR>(a, mask, threads, blocks, lds, stream);
    case 2: return launch_gemv_variant<BITS, D, 2, MODE, MR>(a, mask, threads, blocks, lds, stream);
    case 4: return launch_gemv_variant<BITS, D, 4, MODE, MR>(a, mask, threads, blocks, lds, stream);
    default: return launch_gemv_variant<BITS, D, 8, MODE, MR>(a, mask, threads, blocks, lds, stream);
  }
}

template <int BITS, int MR, int D>
hipError_t launch_gemv_mode(const GemvArgs& a, int mode, int T, bool mask, int threads, dim3 blocks, int lds,
                            hipStream_t stream) {
  switch (mode) {
    case CB_REPL: return launch_gemv_t<BITS, MR, D, CB_REPL>(a, T, mask, threads, blocks, lds, stream);
    case CB_LDS: return launch_gemv_t<BITS, MR, D, CB_LDS>(a, T, mask, threads, blocks, lds, stream);
    case CB_SLICE:  // only 16-bit ids address codebooks larger than LDS
      if constexpr (BITS == 16) return launch_gemv_t<BITS, MR, D, CB_SLICE>(a, T, mask, threads, blocks, lds, stream);
      else return hipErrorNotSupported;
    case CB_SPLIT:
      if constexpr (BITS == 16) return launch_gemv_t<BITS, MR, D, CB_SPLIT>(a, T, mask, threads, blocks, lds, stream);
      else return hipErrorNotSupported;
    default: return launch_gemv_t<BITS, MR, D, CB_GLOBAL>(a, T, mask, threads, blocks, lds, stream);
  }
}

// x of the 16-row-tile kernel is staged whole when its rows take at most
// kXWholeBytes of LDS, else in slabs of at most kXSlabBytes.  Both limits
// depend on M and K alone, never on the codebooks, so a matrix computes in
// the same order in a grouped launch and alone.
constexpr int64_t kXWholeBytes = 136 * 1024;
constexpr int64_t kXSlabBytes = 80 * 1024;

// T chunk columns per lane and wave, P waves per row: the smallest T that
// covers `cols` chunk columns with at most 16 waves (0: none does).
inline int gemv_pick_t(int64_t cols) {
  const int64_t qc = (cols + 3) / 4;  // chunk columns of the four K groups
  for (int t : {1, 2, 4, 8})
    if ((qc + t - 1) / t <= 16) return t;
  return 0;
}

// Whether x goes to registers (whole rows, no masked columns), else to LDS,
// whole or in slabs.
inline bool gemv_x_in_regs(int64_t CH, int G, int d) {
  const int T = gemv_pick_t(CH);
  if (T == 0) return false;
  const int64_t P0 = ((CH + 3) / 4 + T - 1) / T;
  return P0 * T * 4 == CH && T * (G * d / 8) <= 8;
}

// K split of the 16-row-tile kernel over workgroups, for one matrix whose
// M rows of x take more than kXSegBytes and do not go to registers, when the
// caller gives a workspace: K is cut into 2, 4 or 8 segments (gridDim.z) of
// whole chunk columns, each workgroup stages only its segment of x (whole)
// for kXSegBytes or less of x per segment, and a second kernel adds the
// segments' fp32 partials in segment order.  Each workgroup then stages a
// fraction of x for the same ids, where without the split the x staging of a
// workgroup outweighed its share of the index stream (tall K, few rows per
// workgroup).  The partials take at most kGemvSplitMaxWs bytes.
constexpr int64_t kXSegBytes = 64 * 1024;
constexpr int kGemvMaxSegs = 8;
constexpr int64_t kGemvSplitMaxWs = int64_t(4) << 20;
// From this many tokens on, a split launch sums each round of tiles as soon
// as it is done (two barriers per round) and keeps one workgroup per CU;
// below it, the partials of all the workgroup's tiles wait in LDS and the
// LDS they take caps the tiles per workgroup.  Measured (same box,
// alternating builds): down_proj 4096 x 14336 at 4 / 8 / 11 tokens 15.1 /
// 15.8 / 24.5 us without the rounds against 16.2 / 18.4 / 23.1 us with
// them; Qwen3-8B down_proj (4096 x 12288, 65536-entry codebook) at 4 / 16
// tokens 51.0 / 64.7 against 52.1 / 58.2 us.
constexpr int kRoundSumFromTokens = 11;
// The same rounds for a codebook whose head is in LDS and the rest read from
// global memory (CB_SPLIT), from this many tokens on: the head takes most of
// LDS, so with the partials of all its tiles a workgroup could hold one or
// two tiles, and every CU restaged the head for each of several workgroups.
// Qwen3-8B layer (kernel sum) at 4 / 16 tokens: 193.9 / 211.5 against
// 190.4 / 205.9 us with the rounds (same box, alternating builds).
constexpr int kRoundHeadFromTokens = 4;

struct GemvSplit {
  int nseg = 1;      // K segments (1: no split)
  int64_t chs = 0;   // chunk columns per segment
};

inline GemvSplit gemv_split_plan(const Problem& p) {
  GemvSplit sp;
  const int G = p.idx_bits == 8 ? 16 : 8;
  if (p.cb_stride != 0 || p.M < 2 || p.M > 16 || p.S % G) return sp;
  const int64_t CH = p.S / G;
  if (gemv_x_in_regs(CH, G, p.d)) return sp;
  const int64_t XCB = (int64_t)G * p.d * 2;
  const int64_t x_total = p.M * CH * XCB;
  if (x_total <= kXSegBytes) return sp;
  int ks = 2;
  while (ks < kGemvMaxSegs && x_total / ks > kXSegBytes) ks *= 2;
  const int64_t chs = ((CH + ks - 1) / ks + 3) / 4 * 4;
  const int nseg = (int)((CH + chs - 1) / chs);
  const int T = gemv_pick_t(chs);
  if (nseg < 2 || T == 0 || T > 4 || p.M * (chs * XCB + 16) > kXWholeBytes) return sp;
  if ((int64_t)nseg * p.M * p.N * 4 > kGemvSplitMaxWs) return sp;
  sp.nseg = nseg;
  sp.chs = chs;
  return sp;
}

namespace {
// y[o] = fp16(sum over the K segments, in segment order, of ws[seg][o]);
// every partial is loaded before the first add.
__global__ void k_gemv_seg_sum(const float* __restrict__ ws, int64_t MN, int nseg, half_t* __restrict__ y) {
  for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < MN; o += (int64_t)gridDim.x * blockDim.x) {
    float v[kGemvMaxSegs];
#pragma unroll
    for (int k = 0; k < kGemvMaxSegs; ++k)
      if (k < nseg) v[k] = ws[(int64_t)k * MN + o];
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kGemvMaxSegs; ++k)
      if (k < nseg) s += v[k];
    y[o] = static_cast<half_t>(s);
  }
}
}  // namespace

inline bool gemv_x_slabbed(const Problem& p) {
  const int G = p.idx_bits == 8 ? 16 : 8;
  if (p.S % G) return false;
  const int64_t CH = p.S / G;
  return !gemv_x_in_regs(CH, G, p.d) && p.M * (CH * G * p.d * 2 + 16) > kXWholeBytes;
}

// 2 to 16 tokens, one launch over
// `count` <= kGemvMaxParts matrices that share x, M, K, d and the id width:
// select the x slabs, T, P, Q, the codebook placement, the parts and the
// 16-row tiles per workgroup, and launch; hipErrorNotSupported when another
// kernel has to take the call.
template <int BITS, int MR>
hipError_t launch_gemv_bits(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream) {
  constexpr int G = Chunk<BITS>::G;
  constexpr int CBY = Chunk<BITS>::DW * 4;
  if (count < 1 || count > kGemvMaxParts) return hipErrorNotSupported;
  const Problem& p = ps[0];
  const int d = p.d;
  static_assert(MR == 16, "16 token slots");
  if (p.M < 2 || p.M > 16) return hipErrorNotSupported;
  if (!(d == 1 || d == 2 || d == 4 || d == 8)) return hipErrorNotSupported;
  if (p.S % G || p.K % 8) return hipErrorNotSupported;
  const int64_t CH = p.S / G;
  if (CH * CBY != p.R) return hipErrorNotSupported;
  if (16 * p.R >= (int64_t(1) << 24) || (reinterpret_cast<uintptr_t>(p.x) & 15)) return hipErrorNotSupported;
  int64_t maxC = 0, total_rows = 0;
  int64_t tiles_of[kGemvMaxParts];
  for (int i = 0; i < count; ++i) {
    const Problem& pi = ps[i];
    if (pi.M != p.M || pi.K != p.K || pi.d != d || pi.idx_bits != p.idx_bits || pi.x != p.x) return hipErrorNotSupported;
    if (pi.cb_stride != 0 || pi.N * pi.R >= (int64_t(1) << 32)) return hipErrorNotSupported;
    if ((reinterpret_cast<uintptr_t>(pi.idx) & (CBY == 16 ? 15 : 3)) || (reinterpret_cast<uintptr_t>(pi.codebook) & 15))
      return hipErrorNotSupported;
    maxC = std::max(maxC, pi.C);
    total_rows += pi.N;
    tiles_of[i] = (pi.N + 15) / 16;
  }

  const int XCB = G * d * 2;  // bytes of x per chunk column and token
  // x in registers (whole rows, no masked columns) needs no LDS
  const bool x_in_regs = gemv_x_in_regs(CH, G, d);
  int64_t CHS = CH;  // chunk columns per x slab
  // K split over workgroups with a caller workspace (one matrix): each
  // segment is one slab
  int nseg = 1;
  if (count == 1 && p.ws != nullptr && !(reinterpret_cast<uintptr_t>(p.ws) & 3)) {
    const GemvSplit sp = gemv_split_plan(p);
    if (sp.nseg > 1 && p.ws_bytes >= (int64_t)sp.nseg * p.M * p.N * 4) {
      nseg = sp.nseg;
      CHS = sp.chs;
    }
  }
  if (nseg == 1 && !x_in_regs && p.M * (CH * XCB + 16) > kXWholeBytes) {
    // at most 64 chunk columns of each K group per slab (T <= 4)
    const int64_t cmax = std::min<int64_t>(((kXSlabBytes / p.M - 16) / XCB) / 4 * 4, 256);
    if (cmax < 4) return hipErrorNotSupported;
    const int64_t ns = (CH + cmax - 1) / cmax;
    CHS = ((CH + ns - 1) / ns + 3) / 4 * 4;  // near-equal slabs, whole K groups
  }
  const int nslab = (int)((CH + CHS - 1) / CHS);
  const int T = gemv_pick_t(CHS);
  if (T == 0) return hipErrorNotSupported;
  const int P = (int)(((CHS + 3) / 4 + T - 1) / T);
  const int Q = 16 / P;
  const int PS = gemv_red_stride(P);  // floats per (row, token) pair of partials
  // lanes past the slab's (or the row's) last chunk column; slabbed x is
  // always read with the column checks (and never from registers)
  const bool mask = (int64_t)P * T * 4 != CHS || nslab > 1;
  const int threads = P * Q * kWave;

  // One codebook placement for the launch: the largest codebook decides it.
  int mode = choose_cb_mode(maxC, d);
  if (mode == CB_REPL && (total_rows + dev.num_cus - 1) / dev.num_cus * p.S < kReplMinIdsPerEntry * maxC) mode = CB_LDS;
  const int xs = (int)(CHS * XCB + 16);
  const int64_t x_bytes = x_in_regs ? 0 : p.M * (int64_t)xs;
  // The replicated table (up to 64 KB) gives way to one copy when it leaves
  // too little room beside x for one row group's partials.
  if (mode == CB_REPL &&
      cb_lds_bytes(CB_REPL, maxC, d) + x_bytes + (int64_t)Q * 16 * p.M * PS * 4 > dev.lds_per_block)
    mode = CB_LDS;
  // A codebook too large for the LDS budget still goes to LDS when all of it
  // fits beside x and the partials of two row groups (one slice, one pass).
  // More passes do not pay here: each pass costs as much as the whole
  // gather-from-L2 kernel at M >= 4.
  int sl_shift = 0;
  if (mode == CB_GLOBAL && (maxC * d * 2) % 16 == 0) {
    const int64_t red_min = 2 * (int64_t)Q * 16 * p.M * PS * 4;
    const int64_t room = dev.lds_per_block - x_bytes - (red_min > kSliceReserve ? red_min : kSliceReserve);
    while (sl_shift < 16 && (int64_t(2) << sl_shift) * d * 2 <= room) ++sl_shift;
    if ((int64_t(1) << sl_shift) * d * 2 >= kMinSliceBytes && (int64_t(1) << sl_shift) >= maxC) mode = CB_SLICE;
  }
  // Otherwise the first entries of the codebooks go to LDS, as many as fit
  // beside x and the partials of two row groups (whole 16-byte words, and no
  // more than the smallest codebook holds); ids past them gather from
  // global memory.
  int64_t head = 0;
  if (BITS == 16 && mode == CB_GLOBAL) {
    int64_t minC = maxC;
    for (int i = 0; i < count; ++i) minC = std::min(minC, ps[i].C);
    // the partials of one round of tiles beside the head when the launch
    // sums by rounds (below), else of two
    const int64_t red_min = (p.M >= kRoundHeadFromTokens ? 1 : 2) * (int64_t)Q * 16 * p.M * PS * 4;
    const int64_t room = dev.lds_per_block - x_bytes - std::max<int64_t>(red_min, kSliceReserve);
    const int64_t per_word = 16 / (2 * d);  // entries per 16-byte word
    head = std::min(room / (2 * d), minC) / per_word * per_word;
    if (head * d * 2 >= kMinSliceBytes) mode = CB_SPLIT;
  }
  if (mode != CB_GLOBAL && mode != CB_SPLIT)  // every codebook must be whole 16-byte words to be staged
    for (int i = 0; i < count; ++i)
      if ((ps[i].C * d * 2) % 16 != 0) return hipErrorNotSupported;
  const int cb_bytes = mode == CB_SLICE   ? (int)((int64_t(1) << sl_shift) * d * 2)
                       : mode == CB_SPLIT ? (int)(head * d * 2)
                                          : (int)cb_lds_bytes(mode, maxC, d);
  const int64_t avail = dev.lds_per_block - cb_bytes - x_bytes;

  // Parts: matrix i is cut into cuts[i] ranges of whole 16-row tiles; every
  // part gets the grid's x size in workgroups (its y size counts the parts).
  // Within a part, row tiles are dealt round-robin to the workgroups; each
  // workgroup gets a whole number of tiles per row group.
  int cuts[kGemvMaxParts];
  const int nparts = choose_part_cuts(tiles_of, count, dev.num_cus, kGemvMaxParts, cuts);
  int64_t ntiles = 0;  // tiles of the largest part
  for (int i = 0; i < count; ++i) ntiles = std::max(ntiles, (tiles_of[i] + cuts[i] - 1) / cuts[i]);
  int64_t nwg = std::max<int64_t>(dev.num_cus / (nparts * nseg), 1);
  if (nwg > (ntiles + Q - 1) / Q) nwg = (ntiles + Q - 1) / Q;
  int64_t tw = (ntiles + nwg - 1) / nwg;
  tw = (tw + Q - 1) / Q * Q;
  // summing by rounds, LDS holds one round of Q tiles' partials at a time
  const bool rounds = (nseg > 1 && p.M >= kRoundSumFromTokens) || (mode == CB_SPLIT && p.M >= kRoundHeadFromTokens);
  const int64_t tw_max = rounds ? (avail >= Q * 16 * p.M * PS * 4 ? tw : 0)
                                : avail / (16 * p.M * PS * 4) / Q * Q;
  if (tw_max < Q) return hipErrorNotSupported;
  if (tw > tw_max) {
    tw = tw_max;
    nwg = (ntiles + tw - 1) / tw;
  }
  if (nwg > 0x7fffffff || tw * 16 > 0x7fffffff) return hipErrorNotSupported;
  const int lds = (int)(cb_bytes + x_bytes + (rounds ? Q : tw) * 16 * p.M * PS * 4);

  GemvArgs a = {};
  a.x = static_cast<const half_t*>(p.x);
  a.M = p.M;
  a.K = p.K;
  a.R = p.R;
  a.CH = CH;
  a.CHS = (int)CHS;
  a.nslab = nslab;
  a.P = P;
  a.TW = (int)tw;
  a.cb_bytes = cb_bytes;
  a.xs = xs;
  a.x_bytes = (int)x_bytes;
  a.sl_shift = sl_shift;
  a.head = (int)head;
  a.seg_slabs = nseg > 1 ? 1 : nslab;
  a.ws = nseg > 1 ? static_cast<float*>(p.ws) : nullptr;
  a.ld_ws = p.N;
  a.round_sum = rounds ? 1 : 0;
  int k = 0;
  for (int i = 0; i < count; ++i) {
    const int64_t base = tiles_of[i] / cuts[i], extra = tiles_of[i] % cuts[i];
    int64_t row = 0;
    for (int c = 0; c < cuts[i]; ++c, ++k) {
      const int64_t rows = std::min((base + (c < extra ? 1 : 0)) * 16, ps[i].N - row);
      GemvPart& pt = a.part[k];
      pt.idx = static_cast<const uint8_t*>(ps[i].idx) + row * ps[i].R;
      pt.cb = static_cast<const half_t*>(ps[i].codebook);
      pt.y = static_cast<half_t*>(ps[i].y) + row;
      pt.N = rows;
      pt.ldy = ps[i].N;
      pt.C = (int)ps[i].C;
      pt.nsl = 1;
      pt.ws_row = row;
      row += rows;
    }
  }
  const dim3 grid((unsigned)nwg, (unsigned)nparts, (unsigned)nseg);
  hipError_t e;
  switch (d) {
    case 1: e = launch_gemv_mode<BITS, MR, 1>(a, mode, T, mask, threads, grid, lds, stream); break;
    case 2: e = launch_gemv_mode<BITS, MR, 2>(a, mode, T, mask, threads, grid, lds, stream); break;
    case 4: e = launch_gemv_mode<BITS, MR, 4>(a, mode, T, mask, threads, grid, lds, stream); break;
    default: e = launch_gemv_mode<BITS, MR, 8>(a, mode, T, mask, threads, grid, lds, stream); break;
  }
  if (e != hipSuccess || nseg == 1 || plan().active) return e;
  const int64_t mn = p.M * p.N;
  const int64_t rblocks = (mn + 255) / 256;
  return launch_kernel(k_gemv_seg_sum, dim3((unsigned)(rblocks < 65536 ? rblocks : 65536)), dim3(256), 0, stream,
                       static_cast<const float*>(p.ws), mn, nseg, static_cast<half_t*>(p.y));
}

}  // namespace fasq

namespace fasq {

template <typename K>
hipError_t launch_rows_kernel(K kern, const GemvM1Args& a, int threads, dim3 grid, int lds, hipStream_t stream) {
  hipError_t e = prepare_kernel(kern);
  if (e != hipSuccess) return e;
  return launch_kernel(kern, grid, dim3(threads), lds, stream, a);
}

// mt: token slots (1 or 2); two tokens only with the codebook in LDS.
template <int BITS, int D, int T, int MODE>
hipError_t launch_gemv_m1_variant(const GemvM1Args& a, int mt, bool mask, int threads, dim3 grid, int lds,
                                  hipStream_t stream) {
  if (mt == 1) {
    auto kern = mask ? k_gemv_m1<BITS, D, T, MODE, true> : k_gemv_m1<BITS, D, T, MODE, false>;
    if (plan_record("k_gemv_m1", {BITS, D, T, MODE, mask ? 1 : 0})) return hipSuccess;
    return launch_rows_kernel(kern, a, threads, grid, lds, stream);
  }
  if constexpr (MODE == CB_REPL || MODE == CB_LDS) {
    if (plan_record("k_gemv_mt", {BITS, D, T, MODE, mask ? 1 : 0, mt})) return hipSuccess;
    return launch_rows_kernel(mask ? k_gemv_mt<BITS, D, T, MODE, true, 2> : k_gemv_mt<BITS, D, T, MODE, false, 2>, a,
                              threads, grid, lds, stream);
  } else {
    return hipErrorNotSupported;
  }
}

template <int BITS, int D, int MODE>
hipError_t launch_gemv_m1_t(const GemvM1Args& a, int mt, int T, bool mask, int threads, dim3 grid, int lds,
                            hipStream_t stream) {
  switch (T) {
    case 1: return launch_gemv_m1_variant<BITS, D, 1, MODE>(a, mt, mask, threads, grid, lds, stream);
    case 2: return launch_gemv_m1_variant<BITS, D, 2, MODE>(a, mt, mask, threads, grid, lds, stream);
    case 4: return launch_gemv_m1_variant<BITS, D, 4, MODE>(a, mt, mask, threads, grid, lds, stream);
    default: return launch_gemv_m1_variant<BITS, D, 8, MODE>(a, mt, mask, threads, grid, lds, stream);
  }
}

template <int BITS, int D>
hipError_t launch_gemv_m1_mode(const GemvM1Args& a, int mt, int mode, int T, bool mask, int threads, dim3 grid,
                               int lds, hipStream_t stream) {
  switch (mode) {
    case CB_REPL: return launch_gemv_m1_t<BITS, D, CB_REPL>(a, mt, T, mask, threads, grid, lds, stream);
    case CB_LDS: return launch_gemv_m1_t<BITS, D, CB_LDS>(a, mt, T, mask, threads, grid, lds, stream);
    case CB_SLICE:  // only 16-bit ids address codebooks larger than LDS
      if constexpr (BITS == 16) return launch_gemv_m1_t<BITS, D, CB_SLICE>(a, mt, T, mask, threads, grid, lds, stream);
      else return hipErrorNotSupported;
    default: return launch_gemv_m1_t<BITS, D, CB_GLOBAL>(a, mt, T, mask, threads, grid, lds, stream);
  }
}

// One to kM1MaxTokens tokens, one launch over `count` <= kM1MaxParts
// matrices that share x, M, K, d and the id width: choose T (wave-wide loads
// per row part), P (waves per row), Q (row groups per workgroup), the parts
// and their workgroups and the rows per row group; hipErrorNotSupported when
// another kernel has to take the call.
template <int BITS>
hipError_t launch_gemv_m1_bits(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream) {
  constexpr int G = Chunk<BITS>::G;
  constexpr int CBY = Chunk<BITS>::DW * 4;
  if (count < 1 || count > kM1MaxParts) return hipErrorNotSupported;
  const Problem& p = ps[0];
  const int d = p.d;
  if (p.M < 1 || p.M > kM1MaxTokens) return hipErrorNotSupported;
  const int MT = (int)p.M;  // token slots of the kernel
  if (!(d == 1 || d == 2 || d == 4 || d == 8)) return hipErrorNotSupported;
  if (p.S % G || p.K % 8) return hipErrorNotSupported;
  const int64_t CH = p.S / G;
  if (CH * CBY != p.R) return hipErrorNotSupported;
  if (reinterpret_cast<uintptr_t>(p.x) & 15) return hipErrorNotSupported;
  int64_t maxC = 0, total_rows = 0;
  for (int i = 0; i < count; ++i) {
    const Problem& pi = ps[i];
    if (pi.M != p.M || pi.K != p.K || pi.d != d || pi.idx_bits != p.idx_bits || pi.x != p.x) return hipErrorNotSupported;
    if (pi.cb_stride != 0) return hipErrorNotSupported;
    if (pi.N * pi.R >= (int64_t(1) << 32)) return hipErrorNotSupported;
    if ((reinterpret_cast<uintptr_t>(pi.idx) & (CBY == 16 ? 15 : 3)) || (reinterpret_cast<uintptr_t>(pi.codebook) & 15))
      return hipErrorNotSupported;
    if (pi.C > maxC) maxC = pi.C;
    total_rows += pi.N;
  }

  const int SPC = G * d / 8;
  const int64_t CHW = (CH + 63) / 64;  // wave-wide loads per row
  // Two tokens and many rows per CU: twice the x registers, so that a wave
  // covers two wave-wide loads of a row (T = 2) with x in registers instead
  // of one load per row part (T = 1, two waves per row, a reduction per load).
  // Measured on the Llama-3-8B gate+up launch at two tokens: 14.65 against
  // 16.11 us; with few rows per CU (o_proj: 16) one load per part is faster.
  const int64_t rows_per_cu = (total_rows + dev.num_cus - 1) / dev.num_cus;
  const bool wide_x = MT > 1 && rows_per_cu >= kMtWideXMinRows && CH % (2 * 64) == 0;
  const int xregs = kRowsXRegs * (wide_x ? 2 : 1);
  const int tx = SPC * MT <= xregs ? xregs / (SPC * MT) : 0;  // largest T whose x slices fit the register budget
  int T = 0;
  for (int t : {8, 4, 2, 1}) {  // exact split, x in registers
    if (t <= tx && CHW % t == 0 && CHW / t <= 16) { T = t; break; }
  }
  if (T == 0) {
    for (int t : {1, 2, 4, 8}) {  // exact split, x from LDS
      if (CHW % t == 0 && CHW / t <= 16) { T = t; break; }
    }
  }
  if (T == 0) {
    for (int t : {1, 2, 4, 8}) {
      if ((CHW + t - 1) / t <= 16) { T = t; break; }
    }
  }
  if (T == 0) return hipErrorNotSupported;
  const int P = (int)((CHW + T - 1) / T);
  const bool mask = (int64_t)P * T * 64 != CH;

  // One codebook placement for the launch: the largest codebook decides it.
  // A codebook too large for LDS is staged slice by slice (one pass over the
  // rows per slice) when its slices fit beside x and the row partials.
  int mode = choose_cb_mode(maxC, d);
  // The replicated table costs each workgroup C * 256 bytes of LDS writes; a
  // workgroup with few ids to gather is faster with one copy.
  if (mode == CB_REPL && (total_rows + dev.num_cus - 1) / dev.num_cus * p.S < kReplMinIdsPerEntry * maxC)
    mode = CB_LDS;
  const int64_t xw = p.K / 8;                                  // 16-byte words of x per token
  const int64_t x_bytes = MT * (xw + (xw + 15) / 16) * 16;     // one unused word after every 16
  int sl_shift = 0;
  if (mode == CB_GLOBAL && (maxC * d * 2) % 16 == 0) {
    const int64_t room = dev.lds_per_block - x_bytes - kSliceReserve;
    while (sl_shift < 16 && (int64_t(2) << sl_shift) * d * 2 <= room) ++sl_shift;
    if ((int64_t(1) << sl_shift) * d * 2 >= kMinSliceBytes) mode = CB_SLICE;
  }
  if (MT > 1 && mode != CB_REPL && mode != CB_LDS) return hipErrorNotSupported;  // several tokens: codebook in LDS
  if (mode != CB_GLOBAL)  // every codebook must be whole 16-byte words to be staged
    for (int i = 0; i < count; ++i)
      if ((ps[i].C * d * 2) % 16 != 0) return hipErrorNotSupported;
  const int cb_bytes = mode == CB_SLICE ? (int)((int64_t(1) << sl_shift) * d * 2) : (int)cb_lds_bytes(mode, maxC, d);
  // Workgroup slots per CU: two workgroups of at most 8 waves when a wave
  // owns whole rows (P = 1) and two workgroups' LDS fits side by side, unless
  // few rows per CU meet the replicated table (two stagings of it per CU would
  // then cost more than the second workgroup hides); else one of up to 16.
  // Measured on the Llama-3-8B layers against one workgroup per CU: gate+up
  // 12.07 against 12.37 us at 4 bits, q+k+v 6.43 against 6.67 and gate+up
  // 11.95 against 12.17 at 3 bits; slower on the 4-bit q+k+v and o_proj
  // (6.10 against 5.55 and 5.05 against 4.68, 24 and 16 rows per CU) and on
  // the 3-bit down_proj (P = 7: 9.50 against 8.75).
  const int wgcu = P == 1 && 2 * (cb_bytes + x_bytes) < dev.lds_per_block &&
                           (mode != CB_REPL || rows_per_cu >= kM1TwoWgReplMinRows)
                       ? 2
                       : 1;
  const int64_t avail = dev.lds_per_block / wgcu - cb_bytes - x_bytes;

  // Q row groups per workgroup: enough workgroups to cover every slot for
  // small N, up to 16 waves per CU.
  const int64_t ncu = (int64_t)dev.num_cus * wgcu;
  int64_t Q = (total_rows + ncu - 1) / ncu;
  if (Q > 16 / wgcu / P) Q = 16 / wgcu / P;
  if (Q < 1) Q = 1;

  // Parts: matrix i is cut into best[i] ranges of near-equal row counts, and
  // every part gets the same number of workgroups (the grid's x size; its y
  // size counts the parts).
  int64_t rows_of[kM1MaxParts];
  int best[kM1MaxParts];
  for (int i = 0; i < count; ++i) rows_of[i] = ps[i].N;
  const int nparts = choose_part_cuts(rows_of, count, ncu, kM1MaxParts, best);
  int64_t max_rows = 0;
  for (int i = 0; i < count; ++i) max_rows = std::max(max_rows, (ps[i].N + best[i] - 1) / best[i]);
  int64_t wpp = ncu / nparts;  // workgroups per part
  if (wpp > (max_rows + Q - 1) / Q) wpp = (max_rows + Q - 1) / Q;  // no workgroup without a row group
  if (wpp < 1) wpp = 1;
  int64_t nrw = (max_rows + wpp * Q - 1) / (wpp * Q);
  const int64_t nrw_max = avail / (4 * Q * P * MT);
  if (nrw_max < 1) return hipErrorNotSupported;
  if (nrw > nrw_max) {  // LDS bound: more workgroups than CUs
    nrw = nrw_max;
    wpp = (max_rows + nrw * Q - 1) / (nrw * Q);
  }
  // 32-bit buffer offsets must cover every row the pipeline reads, including
  // the rows it reads ahead past the last one (those load zeros).
  for (int i = 0; i < count; ++i)
    if ((wpp * Q * (nrw + kGemvPipe / T + 1)) * ps[i].R >= (int64_t(1) << 32)) return hipErrorNotSupported;
  if (wpp > 0x7fffffff || nrw * T > 0x7fffffff) return hipErrorNotSupported;
  const int lds = (int)(cb_bytes + x_bytes + Q * nrw * P * MT * 4);
  const int threads = (int)(P * Q * kWave);

  GemvM1Args a = {};
  a.x = static_cast<const half_t*>(p.x);
  a.K = p.K;
  a.R = p.R;
  a.CH = CH;
  a.P = P;
  a.NRW = (int)nrw;
  a.cb_bytes = cb_bytes;
  a.x_bytes = (int)x_bytes;
  a.sl_shift = sl_shift;
  a.wpp = (int)wpp;
  a.M = (int)p.M;
  int k = 0;
  for (int i = 0; i < count; ++i) {
    const int64_t base = ps[i].N / best[i], extra = ps[i].N % best[i];
    int64_t row = 0;
    for (int c = 0; c < best[i]; ++c, ++k) {
      const int64_t rows = base + (c < extra ? 1 : 0);
      GemvM1Part& pt = a.part[k];
      pt.idx = static_cast<const uint8_t*>(ps[i].idx) + row * ps[i].R;
      pt.cb = static_cast<const half_t*>(ps[i].codebook);
      pt.y = static_cast<half_t*>(ps[i].y) + row;
      pt.N = rows;
      pt.ldy = ps[i].N;
      pt.C = (int)ps[i].C;
      pt.nsl = mode == CB_SLICE ? (int)((ps[i].C + (int64_t(1) << sl_shift) - 1) >> sl_shift) : 1;
      row += rows;
    }
  }
  const dim3 grid((unsigned)wpp, (unsigned)nparts);
  switch (d) {
    case 1: return launch_gemv_m1_mode<BITS, 1>(a, MT, mode, T, mask, threads, grid, lds, stream);
    case 2: return launch_gemv_m1_mode<BITS, 2>(a, MT, mode, T, mask, threads, grid, lds, stream);
    case 4: return launch_gemv_m1_mode<BITS, 4>(a, MT, mode, T, mask, threads, grid, lds, stream);
    default: return launch_gemv_m1_mode<BITS, 8>(a, MT, mode, T, mask, threads, grid, lds, stream);
  }
}

}  // namespace fasq
