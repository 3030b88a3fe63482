// Prefill GEMM kernels: variant selection and launch.
#include "fasq_gemm_mfma.h"
#include "fasq_gemv_launch.h"

namespace fasq {

namespace {

template <int BITS, int D, int MODE, int BM, int BN, int WGM, int WGN, int WANT, int KG>
hipError_t launch_gemm_variant(const GemmArgs& a, int lds, hipStream_t stream) {
  constexpr int NS = gemm_ring_depth(BITS, D, BM, BN, WGM * WGN, WANT);
  auto kern = k_gemm_mfma<BITS, D, MODE, BM, BN, WGM, WGN, NS, KG>;
  if (plan_record("k_gemm_mfma", {BITS, D, MODE, BM, BN, WGM, WGN, NS, KG})) return hipSuccess;
  hipError_t e = prepare_kernel(kern);
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM), (unsigned)a.ksplit);
  return launch_kernel(kern, grid, dim3(WGM * WGN * KG * kWave), lds, stream, a);
}

// Tile shapes, largest first: 256 x 256 and 128 x 256 on 2 x 4 waves (two
// waves per SIMD; 128 x 64 and 64 x 64 per wave), 128 x 128, 64 x 128 and
// 64 x 64 on 2 x 2 waves, with the LDS ring depth of each.  The launcher
// takes the largest tile whose grid covers at least 3/4 of the CUs, else the
// smallest.  A 128 x 64 wave tile reads 0.75 KB of LDS operands per MFMA
// against 1 KB for 64 x 64, which lifts the LDS-bound MFMA loop; its ring
// leaves no room for the replicated codebook, so it gathers from the
// half-row table (CB_HALF) where that fits, else from one copy.
// The 64-row tiles (small grids) also split K over KG groups of waves inside
// the workgroup, with a shallower ring per group.
struct GemmTileShape {
  int bm, bn, ns;
};
// Build-time switches for measuring variants against each other (the
// defaults are the measured choices): the ring depth of the 256 x 256 tile
// (4 fits only with one codebook copy), and whether that tile may use the
// half-row table (0: one copy).
#ifndef FASQ_GEMM_BIG_NS
#define FASQ_GEMM_BIG_NS 3
#endif
#ifndef FASQ_GEMM_HALF
#define FASQ_GEMM_HALF 1
#endif
constexpr GemmTileShape kGemmTiles[] = {
    {256, 256, FASQ_GEMM_BIG_NS}, {128, 256, 4}, {128, 128, 4}, {64, 128, 8}, {64, 64, 8}};
constexpr int kGemmNumTiles = 5;
// K groups tried for the 64-row tiles, in order.  Two groups (two waves per
// SIMD) with the replicated codebook measured best; four groups only fit
// with one codebook copy, whose bank conflicts cost more than they gain.
constexpr int kGemmSplitGroups[] = {2, 1};
inline int gemm_group_ring(int kg, int ns) { return kg == 1 ? ns : kg == 2 ? 4 : 3; }

inline int gemm_tile_waves(int t) { return kGemmTiles[t].bn == 256 ? 8 : 4; }
// The 256 x 256 tile keeps its operands in registers only when few ids make
// a K step: d >= 4 with 8- or 12-bit ids (the others spill).
constexpr bool gemm_big_tile_fits(int bits, int d) { return d >= 4 && bits <= 12; }

// Whether tile t splits the id copies evenly over its waves (and, for the
// 256 x 256 tile, fits the registers).
inline bool gemm_tile_ok(int t, int hb, int bits, int d) {
  if (t == 0 && !gemm_big_tile_fits(bits, d)) return false;
  return (kGemmTiles[t].bn * (2 * hb / 4)) % (gemm_tile_waves(t) * kWave) == 0;
}

template <int BITS, int D, int MODE, int BM, int BN, int NS1>
hipError_t launch_gemm_groups(const GemmArgs& a, int kg, int lds, hipStream_t stream) {
  switch (kg) {
    case 2: return launch_gemm_variant<BITS, D, MODE, BM, BN, 2, 2, 4, 2>(a, lds, stream);
    default: return launch_gemm_variant<BITS, D, MODE, BM, BN, 2, 2, NS1, 1>(a, lds, stream);
  }
}

template <int BITS, int D, int MODE>
hipError_t launch_gemm_tile(const GemmArgs& a, int tile, int kg, int lds, hipStream_t stream) {
  constexpr int IW = 2 * gemm_run_bytes<BITS, D>() / 4;
  switch (tile) {
    case 0:
      if constexpr (gemm_big_tile_fits(BITS, D))
        return launch_gemm_variant<BITS, D, MODE, 256, 256, 2, 4, kGemmTiles[0].ns, 1>(a, lds, stream);
      else return hipErrorNotSupported;
    case 1: return launch_gemm_variant<BITS, D, MODE, 128, 256, 2, 4, kGemmTiles[1].ns, 1>(a, lds, stream);
    case 3:
      if constexpr ((128 * IW) % 256 == 0)
        return launch_gemm_groups<BITS, D, MODE, 64, 128, kGemmTiles[3].ns>(a, kg, lds, stream);
      else return hipErrorNotSupported;
    case 4:
      if constexpr ((64 * IW) % 256 == 0)
        return launch_gemm_groups<BITS, D, MODE, 64, 64, kGemmTiles[4].ns>(a, kg, lds, stream);
      else return hipErrorNotSupported;
    default: return launch_gemm_variant<BITS, D, MODE, 128, 128, 2, 2, kGemmTiles[2].ns, 1>(a, lds, stream);
  }
}

template <int BITS, int D>
hipError_t launch_gemm_mode(const GemmArgs& a, int mode, int tile, int kg, int lds, hipStream_t stream) {
  switch (mode) {
    case CB_REPL: return launch_gemm_tile<BITS, D, CB_REPL>(a, tile, kg, lds, stream);
    case CB_LDS: return launch_gemm_tile<BITS, D, CB_LDS>(a, tile, kg, lds, stream);
    case CB_HALF:  // the 256 x 256 tile only
      if constexpr (gemm_big_tile_fits(BITS, D))
        return launch_gemm_variant<BITS, D, CB_HALF, 256, 256, 2, 4, kGemmTiles[0].ns, 1>(a, lds, stream);
      else return hipErrorNotSupported;
    default: return launch_gemm_tile<BITS, D, CB_GLOBAL>(a, tile, kg, lds, stream);
  }
}

template <int BITS>
hipError_t launch_gemm_bits(const GemmArgs& a, int d, int mode, int tile, int kg, int lds, hipStream_t stream) {
  switch (d) {
    case 1: return launch_gemm_mode<BITS, 1>(a, mode, tile, kg, lds, stream);
    case 2: return launch_gemm_mode<BITS, 2>(a, mode, tile, kg, lds, stream);
    case 4: return launch_gemm_mode<BITS, 4>(a, mode, tile, kg, lds, stream);
    default:
      if constexpr (BITS == 12) return hipErrorNotSupported;  // 4 ids = 6 bytes: not dword aligned
      else return launch_gemm_mode<BITS, 8>(a, mode, tile, kg, lds, stream);
  }
}

}  // namespace

// The launch plan of a call: tile, K groups, codebook placement, LDS bytes
// and the workgroups along K (ksplit > 1 needs ksplit * M * N * 4 bytes of
// workspace); false when the tuned kernel does not apply.
struct GemmPlan {
  int tile = 0, kg = 1, mode = 0, lds = 0, ksplit = 1;
};

// K ranges per output tile when the grid leaves CUs idle: enough to reach
// about one workgroup per CU, at most kGemmMaxSplit, each range at least
// kGemmMinSplitChunks chunks of 64 per K group.
constexpr int kGemmMaxSplit = 8;
constexpr int kGemmMinSplitChunks = 4;

bool gemm_plan(const Problem& p, const DeviceInfo& dev, GemmPlan* out) {
  const int d = p.d;
  if (p.cb_stride != 0) return false;
  if (!(d == 1 || d == 2 || d == 4 || d == 8)) return false;
  if (p.idx_bits == 12 && d == 8) return false;
  if (p.K % kGemmKC) return false;
  if (p.R * 8 != p.S * p.idx_bits) return false;
  if ((reinterpret_cast<uintptr_t>(p.x) & 15) || (reinterpret_cast<uintptr_t>(p.codebook) & 15) ||
      (reinterpret_cast<uintptr_t>(p.idx) & 15) || (p.R & 3))
    return false;
  // id runs are copied as 4-byte words
  const int hb = (32 / d) * p.idx_bits / 8;
  if (hb % 4) return false;

  int mode = choose_cb_mode(p.C, d);
  auto lds_of = [&](int t, int kg, int m) {
    const GemmTileShape& ts = kGemmTiles[t];
    const int ns = gemm_ring_depth(p.idx_bits, d, ts.bm, ts.bn, gemm_tile_waves(t), gemm_group_ring(kg, ts.ns));
    const int64_t lds = cb_lds_bytes(m, p.C, d) + (int64_t)kg * ns * (ts.bm * 128 + ts.bn * 2 * hb);
    const int64_t dump = (int64_t)(kg - 1) * ts.bm * ts.bn * 4;  // accumulators of groups 1 .. kg-1
    return lds > dump ? lds : dump;
  };
  auto tiles_of = [&](int t) {
    return ((p.M + kGemmTiles[t].bm - 1) / kGemmTiles[t].bm) * ((p.N + kGemmTiles[t].bn - 1) / kGemmTiles[t].bn);
  };
  // The codebook placement of tile t: the call's; else, for the replicated
  // table, the half-row table (256 x 256 tile) or one LDS copy, whichever
  // fits beside the tile's ring first (-1: none fits).
  auto mode_of = [&](int t) {
    if (lds_of(t, 1, mode) <= dev.lds_per_block) return mode;
    if (FASQ_GEMM_HALF && mode == CB_REPL && t == 0 && lds_of(t, 1, CB_HALF) <= dev.lds_per_block)
      return (int)CB_HALF;
    if (mode == CB_REPL && lds_of(t, 1, CB_LDS) <= dev.lds_per_block) return (int)CB_LDS;
    return -1;
  };
  int tile = -1;
  for (int t = 0; t < kGemmNumTiles && tile < 0; ++t)
    if (gemm_tile_ok(t, hb, p.idx_bits, d) && mode_of(t) >= 0 && 4 * tiles_of(t) >= 3 * (int64_t)dev.num_cus) tile = t;
  for (int t = kGemmNumTiles - 1; t >= 0 && tile < 0; --t)
    if (gemm_tile_ok(t, hb, p.idx_bits, d) && mode_of(t) >= 0) tile = t;
  if (tile < 0) return false;
  mode = mode_of(tile);
  // K groups for the 64-row tiles: the first count in kGemmSplitGroups that
  // fits, with the replicated codebook or, failing that, one copy.
  int kg = 1;
  if (kGemmTiles[tile].bm == 64) {
    bool done = false;
    for (int g : kGemmSplitGroups) {
      for (int m : {mode, (int)CB_LDS}) {
        if (m == CB_LDS && mode != CB_REPL && mode != CB_LDS) continue;
        if (lds_of(tile, g, m) <= dev.lds_per_block) { kg = g; mode = m; done = true; break; }
      }
      if (done) break;
    }
  }
  const int lds = (int)lds_of(tile, kg, mode);
  int ksplit = 1;
  const int64_t tiles = tiles_of(tile);
  const int64_t chunks = p.K / kGemmKC;
  while (ksplit < kGemmMaxSplit && tiles * (ksplit + 1) <= dev.num_cus &&
         chunks / (ksplit + 1) >= (int64_t)kGemmMinSplitChunks * kg)
    ++ksplit;
  out->tile = tile;
  out->kg = kg;
  out->mode = mode;
  out->lds = lds;
  out->ksplit = ksplit;
  return true;
}

// Whether a decode call with a workspace runs faster on this GEMM: from 12
// tokens on, when the decode kernel would have to stage x in slabs (rows of
// x too long for LDS) and the GEMM splits K with its codebook in LDS.
// Measured on the Llama-3-8B down_proj shape (4096 x 14336, d = 2, C = 256):
// 12 tokens 29.3 us on the decode kernel against 25.6 us on the GEMM, 16
// tokens 35.7 against 26.5 us (8 tokens: 22.0 against 26.6); with x whole in
// LDS or registers (gate_proj 16 tokens: 15.9 against 25.3 us), or a
// codebook the GEMM has to gather from global memory (65536 entries), the
// decode kernel is the faster one.
bool decode_prefers_gemm(const Problem& p, const DeviceInfo& dev) {
  if (p.M < kGemmFromTokens || p.M > kGemvMaxTokens || !gemv_x_slabbed(p)) return false;
  GemmPlan pl;
  if (!gemm_plan(p, dev, &pl)) return false;
  return pl.ksplit > 1 && (pl.mode == CB_REPL || pl.mode == CB_HALF || pl.mode == CB_LDS);
}

int64_t gemv_split_workspace_bytes(const Problem& p) {
  const GemvSplit sp = gemv_split_plan(p);
  return sp.nseg > 1 ? (int64_t)sp.nseg * p.M * p.N * 4 : 0;
}

int64_t gemm_workspace_bytes(const Problem& p, const DeviceInfo& dev) {
  GemmPlan pl;
  if (!gemm_plan(p, dev, &pl) || pl.ksplit == 1) return 0;
  return (int64_t)pl.ksplit * p.M * p.N * 4;
}

hipError_t launch_gemm_mfma(const Problem& p, const DeviceInfo& dev, hipStream_t stream, void* workspace,
                            int64_t workspace_bytes) {
  GemmPlan pl;
  if (!gemm_plan(p, dev, &pl)) return hipErrorNotSupported;
  const int d = p.d;
  // the K split only with a workspace that holds its partials
  if (pl.ksplit > 1 && (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 3) ||
                        workspace_bytes < (int64_t)pl.ksplit * p.M * p.N * 4))
    pl.ksplit = 1;
  const int tile = pl.tile, kg = pl.kg, mode = pl.mode, lds = pl.lds;
  const int cb_bytes = (int)cb_lds_bytes(mode, p.C, d);

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
  a.ksplit = pl.ksplit;
  a.ws = static_cast<float*>(workspace);
  hipError_t e;
  switch (p.idx_bits) {
    case 8: e = launch_gemm_bits<8>(a, d, mode, tile, kg, lds, stream); break;
    case 12: e = launch_gemm_bits<12>(a, d, mode, tile, kg, lds, stream); break;
    default: e = launch_gemm_bits<16>(a, d, mode, tile, kg, lds, stream); break;
  }
  if (e != hipSuccess || a.ksplit == 1 || plan().active) return e;
  const int64_t mn = p.M * p.N;
  const bool vec = mn % 4 == 0 && (reinterpret_cast<uintptr_t>(workspace) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(p.y) & 7) == 0;
  const int64_t blocks = ((vec ? mn / 4 : mn) + 255) / 256;
  const dim3 grid((unsigned)(blocks < 65536 ? blocks : 65536));
  if (vec)
    return launch_kernel(k_gemm_split_reduce<true>, grid, dim3(256), 0, stream, static_cast<const float*>(workspace),
                         mn, a.ksplit, a.y);
  return launch_kernel(k_gemm_split_reduce<false>, grid, dim3(256), 0, stream, static_cast<const float*>(workspace),
                       mn, a.ksplit, a.y);
}

}  // namespace fasq
