// Decode GEMV with one codebook per subspace (FASQ Sec. 3.1.1, Eq.
// lut-accumulate with its per-subspace tables; Sec. 4.1 splits the subspaces
// over blocks the same way), for M <= 16 tokens.
//
//   y[m, n] = sum_s dot(x[m, s*d : (s+1)*d], codebook_s[u(n, s)])
//
// The books of all subspaces (S x C x d fp16, 2 MB for a 4096-wide layer at
// d = 2, C = 256) do not fit in LDS, so K is split over workgroups: workgroup
// (row block rb, segment ks) stages the books of the NCH * G subspaces of its
// segment (up to 144 KB) into LDS once, then streams the id segments of its
// rows.  Lane l of a wave-wide load holds chunk l % NCH (G ids, 16 or 12
// bytes) of row l / NCH of the segment, so one load reads 64 / NCH rows of
// NCH * 16 contiguous bytes.  The lane gathers each codeword from the book of
// its subspace and accumulates the dot products with x in fp32; the NCH lanes
// of a row sum their partials (DPP), and the row's fp32 partial for this
// segment goes to the workspace.  A second kernel adds the segments of every
// row in segment order and rounds to fp16 once: deterministic, no atomics.
// One token keeps the lane's x slice in registers.  Several tokens (d <= 4)
// stage the segment's slice of every row of x in LDS after the books; the
// lane gathers its G codewords once per chunk and takes the dot products
// with each token's slice in turn, so the ids and the gathers are shared by
// all tokens.
#include "fasq_codebook.h"
#include "fasq_device.h"
#include "fasq_internal.h"

namespace fasq {

namespace {

constexpr int kSubThreads = 1024;               // 16 waves
constexpr int kSubBookBytes = 144 * 1024;       // LDS for the books of one segment
constexpr int kSubMaxNch = 16;                  // chunks per row segment (lanes per row)
constexpr int kSubMaxTokens = 16;               // tokens of the multi-token kernel

struct SubArgs {
  const half_t* x;
  int64_t M, K;       // tokens, row length of x
  int x_off;          // several tokens: LDS byte offset of the staged x slices
  int64_t N;
  const uint8_t* idx;
  int64_t R;          // bytes per id row
  int64_t CH;         // chunks per row
  const half_t* cb;   // [S x C x d]
  int C;
  int KS;             // segments
  int64_t rows_per_block;
  float* ws;          // [KS x M x N] fp32 partials
};

// Codeword of book b (LDS byte address base + (b * C + u) * 2D) dotted with
// the D x values at xv, added to acc.
template <int D>
__device__ __forceinline__ float dot_codeword(uint32_t addr, const uint32_t* xv, float acc) {
  if constexpr (D == 1) {
    const half_t c = __builtin_bit_cast(half_t, *lds_at<uint16_t>(addr));
    const half_t xh = __builtin_bit_cast(half_t, (uint16_t)(xv[0] & 0xFFFF));
    return __builtin_fmaf(static_cast<float>(xh), static_cast<float>(c), acc);
  } else {
    uint32_t c[D / 2];
    read_codeword_lds<D>(addr, c);
#pragma unroll
    for (int k = 0; k < D / 2; ++k) acc = dot2(xv[k], c[k], acc);
    return acc;
  }
}

// XL: several tokens, x slices staged in LDS (see the file comment).
template <int BITS, int D, int NCH, bool XL>
__global__ __launch_bounds__(kSubThreads) void k_gemv_sub(SubArgs a) {
  constexpr int G = Chunk<BITS>::G;
  constexpr int DW = Chunk<BITS>::DW;
  constexpr int CBY = DW * 4;
  constexpr int RPL = kWave / NCH;             // rows per wave-wide load
  constexpr int XW = D == 1 ? 1 : D / 2;       // dwords of x per id (D == 1: the low half)
  constexpr int XSB = G * D * 2;               // bytes of one chunk's x slice (one token)
  // several tokens: x words per token, and LDS words per token with one
  // unused word after every 16, so that the 16 lanes of one LDS read cycle,
  // one chunk apart, hit distinct banks
  constexpr int WPS = NCH * XSB / 16;
  constexpr int WPSP = WPS + (WPS + 15) / 16;
  static_assert(kWave % NCH == 0 && NCH <= kSubMaxNch, "NCH must divide the wave");
  static_assert(!XL || (D <= 4 && XSB % 16 == 0), "the multi-token kernel takes d <= 4");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int ks = (int)(blockIdx.x % a.KS);
  const int64_t rb = blockIdx.x / a.KS;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int waves = blockDim.x / kWave;
  const int c = lane % NCH;                     // chunk of the lane within the segment
  const int rl = lane / NCH;                    // row of the lane within a load
  const int64_t ch = (int64_t)ks * NCH + c;     // chunk within the row
  const bool cval = ch < a.CH;
  const int nbooks = (int)((a.CH - (int64_t)ks * NCH < NCH ? a.CH - (int64_t)ks * NCH : NCH) * G);

  // rows of this workgroup: [r0, r1); wave-wide loads j = wave, wave + waves, ...
  const int64_t r0 = rb * a.rows_per_block;
  const int64_t r1 = r0 + a.rows_per_block < a.N ? r0 + a.rows_per_block : a.N;
  const int nloads = (int)((r1 - r0 + RPL - 1) / RPL);
  const int mine = nloads > wave ? (nloads - wave + waves - 1) / waves : 0;

  const __amdgpu_buffer_rsrc_t rsrc = idx_rsrc(a.idx, (uint32_t)(a.N * a.R));
  auto offset_of = [&](int k) {  // k-th load of this wave; rows past N read zeros
    const int64_t row = r0 + (int64_t)(wave + k * waves) * RPL + rl;
    return (uint32_t)(row * a.R + (cval ? ch : 0) * CBY);
  };
  uint32_t buf0[DW], buf1[DW];
  if (mine > 0) buffer_chunk<BITS>(rsrc, offset_of(0), buf0);
  if (mine > 1) buffer_chunk<BITS>(rsrc, offset_of(1), buf1);

  // books of the segment -> LDS (16-byte words, consecutive threads)
  {
    const int words = nbooks * a.C * D * 2 / 16;
    const u32x4* src = reinterpret_cast<const u32x4*>(a.cb + ((int64_t)ks * NCH * G) * a.C * D);
    for (int base = threadIdx.x; base < words; base += 8 * blockDim.x) {
      u32x4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int w = base + k * blockDim.x;
        v[k] = src[w < words ? w : words - 1];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int w = base + k * blockDim.x;
        if (w < words) *reinterpret_cast<u32x4*>(smem + (uint32_t)w * 16) = v[k];
      }
    }
  }
  // several tokens: the segment's slice of every row of x (NCH chunks of G
  // ids, zeros past the row) after the books, 16-byte words
  if constexpr (XL) {
    const int words = (int)a.M * WPS;
    const int64_t seg0 = (int64_t)ks * NCH * G * D;  // first x element of the segment
    for (int w = threadIdx.x; w < words; w += blockDim.x) {
      const int m = w / WPS, k = w - m * WPS;
      const int64_t ch_w = (int64_t)ks * NCH + (k * 16) / XSB;  // chunk of the word
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (ch_w < a.CH) v = *reinterpret_cast<const u32x4*>(a.x + (int64_t)m * a.K + seg0 + (int64_t)k * 8);
      *reinterpret_cast<u32x4*>(smem + a.x_off + (uint32_t)(m * WPSP + k + (k >> 4)) * 16) = v;
    }
  }
  // one token: x of the lane's chunk, G * D halves, in registers
  uint32_t xv[XL ? 1 : G][XW];
  if constexpr (!XL) {
    const uint16_t* xs = reinterpret_cast<const uint16_t*>(a.x) + (cval ? ch : 0) * G * D;
#pragma unroll
    for (int i = 0; i < G; ++i) {
#pragma unroll
      for (int k = 0; k < XW; ++k) {
        const uint32_t lo = xs[i * D + 2 * k];
        const uint32_t hi = D == 1 ? 0u : (uint32_t)xs[i * D + 2 * k + 1];
        xv[i][k] = cval ? (lo | (hi << 16)) : 0u;  // a chunk past the row contributes 0
      }
    }
  }
  __syncthreads();

  const uint32_t book0 = (uint32_t)c * G;  // first book of the lane's chunk
  auto compute = [&](const uint32_t* w, int k) {
    const int64_t row = r0 + (int64_t)(wave + k * waves) * RPL + rl;
    if constexpr (XL) {
      // the chunk's G codewords (zeros past the row end: no staged books)
      uint32_t cw[G][XW];
#pragma unroll
      for (int i = 0; i < G; ++i) {
#pragma unroll
        for (int q = 0; q < XW; ++q) cw[i][q] = 0u;
        if (cval) read_codeword_lds<D>(((book0 + i) * (uint32_t)a.C + stream_id<BITS>(w, i)) * (2 * D), cw[i]);
      }
      const uint32_t cw0 = (uint32_t)c * (XSB / 16);  // first word of the lane's chunk
      const uint32_t xs0 = (uint32_t)a.x_off + (cw0 + (cw0 >> 4)) * 16;
      for (int m = 0; m < (int)a.M; ++m) {
        uint32_t xs[G * D / 2 > 0 ? G * D / 2 : 1];
#pragma unroll
        for (int q = 0; q < XSB / 16; ++q) {
          const u32x4 v = *lds_at<u32x4>(xs0 + (uint32_t)m * (WPSP * 16) + (uint32_t)q * 16);
          xs[4 * q] = v[0]; xs[4 * q + 1] = v[1]; xs[4 * q + 2] = v[2]; xs[4 * q + 3] = v[3];
        }
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < G; ++i) {
          if constexpr (D == 1) {
            const uint16_t xh = (uint16_t)(xs[i / 2] >> (16 * (i % 2)));
            const half_t xf = __builtin_bit_cast(half_t, xh);
            const half_t cf = __builtin_bit_cast(half_t, (uint16_t)(cw[i][0] & 0xFFFFu));
            acc = __builtin_fmaf(static_cast<float>(xf), static_cast<float>(cf), acc);
          } else {
#pragma unroll
            for (int q = 0; q < XW; ++q) acc = dot2(xs[i * XW + q], cw[i][q], acc);
          }
        }
        acc = group_sum<NCH>(acc);
        if (c == 0 && row < r1) a.ws[((int64_t)ks * a.M + m) * a.N + row] = acc;
      }
    } else {
      float acc = 0.f;
      if (cval) {  // a chunk past the row end (last segment) has no staged books
#pragma unroll
        for (int i = 0; i < G; ++i)
          acc = dot_codeword<D>(((book0 + i) * (uint32_t)a.C + stream_id<BITS>(w, i)) * (2 * D), xv[i], acc);
      }
      acc = group_sum<NCH>(acc);
      if (c == 0 && row < r1) a.ws[(int64_t)ks * a.N + row] = acc;
    }
  };
  for (int k = 0; k < mine; k += 2) {
    compute(buf0, k);
    if (k + 2 < mine) buffer_chunk<BITS>(rsrc, offset_of(k + 2), buf0);
    if (k + 1 < mine) {
      compute(buf1, k + 1);
      if (k + 3 < mine) buffer_chunk<BITS>(rsrc, offset_of(k + 3), buf1);
    }
  }
}

// y[m, n] = fp16(sum over segments, in segment order, of ws[ks][m][n]).
// The partials are read kSumBatch at a time, every load issued before the
// first add (a load inside the add loop would wait for each one in turn),
// and added in segment order, so the sum keeps its order and its bits.
constexpr int kSumBatch = 8;
__global__ void k_sub_reduce(const float* __restrict__ ws, int64_t MN, int KS, half_t* __restrict__ y) {
  for (int64_t o = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; o < MN; o += (int64_t)gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int k0 = 0; k0 < KS; k0 += kSumBatch) {
      float v[kSumBatch];
#pragma unroll
      for (int j = 0; j < kSumBatch; ++j)
        if (k0 + j < KS) v[j] = ws[(int64_t)(k0 + j) * MN + o];
#pragma unroll
      for (int j = 0; j < kSumBatch; ++j)
        if (k0 + j < KS) s += v[j];
    }
    y[o] = static_cast<half_t>(s);
  }
}

// The split of a call: chunks per segment (NCH), segments (KS) and row
// blocks; false when the tuned kernel does not apply.
struct SubPlan {
  int nch = 0, ks = 0;
  int64_t rb = 0, rows = 0;
};

// LDS bytes of the staged x slices of M tokens over nch chunks: one unused
// 16-byte word after every 16 (see the kernel).
inline int64_t sub_x_bytes(int64_t M, int nch, int G, int d) {
  const int64_t wps = (int64_t)nch * G * d * 2 / 16;  // words per token
  return M * (wps + (wps + 15) / 16) * 16;
}

bool sub_plan(const Problem& p, const DeviceInfo& dev, SubPlan* out) {
  if (p.M < 1 || p.M > kSubMaxTokens || p.cb_stride != p.C * p.d) return false;
  const int d = p.d;
  if (!(d == 1 || d == 2 || d == 4 || d == 8)) return false;
  if (p.M > 1 && (d > 4 || (reinterpret_cast<uintptr_t>(p.x) & 15) || (p.K * 2) % 16)) return false;
  const int G = p.idx_bits == 8 ? 16 : 8;
  const int CBY = p.idx_bits == 12 ? 12 : 16;
  if (p.S % G || p.R != p.S / G * CBY) return false;
  if ((p.C * d * 2) % 16) return false;
  if ((reinterpret_cast<uintptr_t>(p.idx) & 3) || (reinterpret_cast<uintptr_t>(p.codebook) & 15) ||
      (reinterpret_cast<uintptr_t>(p.x) & 3))
    return false;
  if ((p.N + kWave) * p.R >= (int64_t(1) << 32)) return false;  // loads read up to one load past N
  const int64_t per_chunk = (int64_t)G * p.C * d * 2;  // book bytes per chunk of ids
  auto x_bytes = [&](int n) { return p.M > 1 ? sub_x_bytes(p.M, n, G, d) : 0; };  // staged x (several tokens)
  int nch = kSubMaxNch;
  while (nch > 1 && (nch * per_chunk > kSubBookBytes || nch * per_chunk + x_bytes(nch) > dev.lds_per_block)) nch /= 2;
  if (per_chunk > kSubBookBytes || per_chunk + x_bytes(1) > dev.lds_per_block) return false;
  const int64_t CH = p.S / G;
  const int64_t ks = (CH + nch - 1) / nch;
  // row blocks: about one workgroup per CU in all, each with whole loads
  int64_t rb = (dev.num_cus + ks - 1) / ks;
  const int64_t rpl = kWave / nch;
  if (rb > (p.N + rpl - 1) / rpl) rb = (p.N + rpl - 1) / rpl;
  if (rb < 1) rb = 1;
  int64_t rows = (p.N + rb - 1) / rb;
  rows = (rows + rpl - 1) / rpl * rpl;
  rb = (p.N + rows - 1) / rows;
  if (rb * ks > 0x7fffffff) return false;
  out->nch = nch;
  out->ks = (int)ks;
  out->rb = rb;
  out->rows = rows;
  return true;
}

template <int BITS, int D, int NCH>
hipError_t launch_sub(const SubArgs& a, int blocks, int lds, hipStream_t stream) {
  const bool xl = a.M > 1;
  if constexpr (D > 4) {
    if (xl) return hipErrorNotSupported;
  }
  auto kern = xl ? k_gemv_sub<BITS, D, NCH, D <= 4> : k_gemv_sub<BITS, D, NCH, false>;
  if (plan_record("k_gemv_sub", {BITS, D, NCH, xl ? 1 : 0})) return hipSuccess;
  hipError_t e = prepare_kernel(kern);
  if (e != hipSuccess) return e;
  return launch_kernel(kern, dim3(blocks), dim3(kSubThreads), lds, stream, a);
}

template <int BITS, int D>
hipError_t launch_sub_nch(const SubArgs& a, int nch, int blocks, int lds, hipStream_t stream) {
  switch (nch) {
    case 16: return launch_sub<BITS, D, 16>(a, blocks, lds, stream);
    case 8: return launch_sub<BITS, D, 8>(a, blocks, lds, stream);
    case 4: return launch_sub<BITS, D, 4>(a, blocks, lds, stream);
    case 2: return launch_sub<BITS, D, 2>(a, blocks, lds, stream);
    default: return launch_sub<BITS, D, 1>(a, blocks, lds, stream);
  }
}

template <int BITS>
hipError_t launch_sub_d(const SubArgs& a, int d, int nch, int blocks, int lds, hipStream_t stream) {
  switch (d) {
    case 1: return launch_sub_nch<BITS, 1>(a, nch, blocks, lds, stream);
    case 2: return launch_sub_nch<BITS, 2>(a, nch, blocks, lds, stream);
    case 4: return launch_sub_nch<BITS, 4>(a, nch, blocks, lds, stream);
    default: return launch_sub_nch<BITS, 8>(a, nch, blocks, lds, stream);
  }
}

}  // namespace

int64_t gemv_sub_workspace_bytes(const Problem& p, const DeviceInfo& dev) {
  SubPlan sp;
  if (!sub_plan(p, dev, &sp)) return 0;
  return (int64_t)sp.ks * p.M * p.N * 4;
}

hipError_t launch_gemv_sub(const Problem& p, void* workspace, int64_t workspace_bytes, const DeviceInfo& dev,
                           hipStream_t stream) {
  SubPlan sp;
  if (!sub_plan(p, dev, &sp)) return hipErrorNotSupported;
  if (workspace == nullptr || workspace_bytes < (int64_t)sp.ks * p.M * p.N * 4 ||
      (reinterpret_cast<uintptr_t>(workspace) & 3))
    return hipErrorNotSupported;
  const int G = p.idx_bits == 8 ? 16 : 8;
  const int books = (int)((int64_t)sp.nch * G * p.C * p.d * 2);
  SubArgs a;
  a.x = static_cast<const half_t*>(p.x);
  a.M = p.M;
  a.K = p.K;
  a.x_off = books;
  a.N = p.N;
  a.idx = static_cast<const uint8_t*>(p.idx);
  a.R = p.R;
  a.CH = p.S / G;
  a.cb = static_cast<const half_t*>(p.codebook);
  a.C = (int)p.C;
  a.KS = sp.ks;
  a.rows_per_block = sp.rows;
  a.ws = static_cast<float*>(workspace);
  const int lds = books + (p.M > 1 ? (int)sub_x_bytes(p.M, sp.nch, G, p.d) : 0);
  const int blocks = (int)(sp.rb * sp.ks);
  hipError_t e;
  switch (p.idx_bits) {
    case 8: e = launch_sub_d<8>(a, p.d, sp.nch, blocks, lds, stream); break;
    case 12: e = launch_sub_d<12>(a, p.d, sp.nch, blocks, lds, stream); break;
    default: e = launch_sub_d<16>(a, p.d, sp.nch, blocks, lds, stream); break;
  }
  if (e != hipSuccess || plan().active) return e;
  const int64_t rblocks = (p.M * p.N + 255) / 256;
  return launch_kernel(k_sub_reduce, dim3((unsigned)(rblocks < 65536 ? rblocks : 65536)), dim3(256), 0, stream,
                       static_cast<const float*>(workspace), p.M * p.N, sp.ks, static_cast<half_t*>(p.y));
}

}  // namespace fasq
