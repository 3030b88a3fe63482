/*
 * fasq.h - product-quantized (PQ) weight matmul for AMD Instinct MI355X (gfx950).
 *
 * The operation (FASQ, Sec. 3.1.2, Eq. lut-accumulate; Sec. 2.2):
 *
 *   A weight matrix W_hat with N output features and K input features is never
 *   stored densely.  Each output row n is cut along K into S = K / d
 *   sub-vectors of length d, and sub-vector s is replaced by the id u(n, s) of
 *   one of C fp16 codewords:
 *
 *       W_hat[n, s*d + i] = codebook[u(n, s) * d + i]        (0 <= i < d)
 *       y[m, n]           = sum_s dot(x[m, s*d : s*d + d], codebook[u(n, s)])
 *                         = (x . W_hat^T)[m, n]
 *
 *   One codebook is shared by every sub-vector of the matrix (the paper's
 *   per-subspace tables with all tables equal).
 *
 * Layouts (all buffers are DEVICE memory, owned and allocated by the caller):
 *   x        fp16 [M x K], row-major, contiguous.
 *   y        fp16 [M x N], row-major, contiguous; every element is written
 *            (no zeroing needed).  Accumulation is fp32; each output is rounded
 *            to fp16 (round to nearest even) exactly once.
 *   codebook fp16 [C x d], row-major.
 *   idx      N rows of R = fasq_idx_row_bytes(K, d, idx_bits) bytes, back to
 *            back (row n starts at byte n*R).  Within a row the ids form one
 *            least-significant-bit-first bit stream: id s occupies stream bits
 *            [idx_bits*s, idx_bits*s + idx_bits), and stream bit t is bit
 *            (t mod 8) of byte (t div 8).  So idx_bits = 8 is one byte per id,
 *            16 a little-endian byte pair, and 12 packs two ids in three bytes
 *            (b0 = u0 & 0xFF, b1 = (u0 >> 8) | (u1 & 0xF) << 4, b2 = u1 >> 4).
 *            The pad bits of an odd 12-bit row are ignored.
 *
 * Conventions:
 *   - Every call is asynchronous on `stream` (0 = the null stream).  The
 *     library allocates no device memory and, outside launch lists (below),
 *     keeps no pointer after returning, so the calls may be captured in a
 *     hipGraph.  The plain entry
 *     points use no scratch memory; the _ex calls and the encoder take a
 *     caller-owned workspace argument for theirs.
 *   - Argument checks run before any HIP call.  A bad argument returns
 *     FASQ_ERR_INVALID_ARG and launches nothing.  A failed launch returns
 *     FASQ_ERR_HIP.  fasq_last_error() then describes the failure (per calling
 *     thread).  A fault inside a kernel surfaces at the caller's next
 *     synchronisation.
 *   - Preconditions that are NOT checked: every id is < C (an id >= C reads
 *     outside the codebook); x, y, idx and codebook do not overlap.
 *   - Calls that share no output buffer may run concurrently from any thread.
 *   - Results are deterministic: the same inputs give the same bits.
 */
#ifndef FASQ_H
#define FASQ_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FASQ_ABI_VERSION 6

typedef enum {
  FASQ_OK = 0,
  FASQ_ERR_INVALID_ARG = 1, /* a size, pointer or format argument is invalid */
  FASQ_ERR_UNSUPPORTED = 2, /* valid, but no kernel handles this combination */
  FASQ_ERR_HIP = 3,         /* the HIP runtime reported an error */
  FASQ_ERR_HOST_MEMORY = 4  /* host memory for a launch list could not be allocated */
} fasq_status;

/*
 * Decode regime (FASQ Sec. 4.1, the batch-1 GEMV of the decode phase):
 * y[M x N] = x[M x K] . W_hat^T.  Tuned for M <= 16 (M = 1 is token-by-token
 * decode); any M >= 1 is accepted and computed correctly.  This is also the
 * batch-adaptive entry point the paper leaves to future work (Sec. 4.4,
 * batch size): rows of x beyond 16, or operands the decode kernels cannot
 * hold on chip, go to the prefill kernel of fasq_pq_gemm.
 *
 *   x, M, K     activations, fp16 [M x K]
 *   N           output features (rows of the index table)
 *   idx         packed ids, N rows of fasq_idx_row_bytes(K, d, idx_bits) bytes
 *   idx_bits    8, 12 or 16
 *   d           sub-vector length, d >= 1, K % d == 0
 *   codebook, C fp16 [C x d], 1 <= C <= 2^idx_bits
 *   y           output, fp16 [M x N]
 *   stream      HIP stream the kernels are queued on
 *
 * Returns FASQ_OK, FASQ_ERR_INVALID_ARG (M, K, N < 1; d < 1; K % d != 0;
 * idx_bits not in {8, 12, 16}; C outside [1, 2^idx_bits]; a NULL pointer) or
 * FASQ_ERR_HIP.
 */
fasq_status fasq_pq_gemv(const void* x, int64_t M, int64_t K, int64_t N,
                         const void* idx, int idx_bits, int d,
                         const void* codebook, int64_t C,
                         void* y, hipStream_t stream);

/*
 * Decode regime over several weight matrices that read the same activations
 * (FASQ Sec. 4.1; in a decoder layer the q, k and v projections share their
 * input, and so do the gate and up projections): for i < count,
 *
 *   y[i][M x N[i]] = x[M x K] . W_hat_i^T
 *
 * with W_hat_i given by idx[i] (N[i] rows of fasq_idx_row_bytes(K, d,
 * idx_bits) bytes) and codebook[i] (fp16 [C[i] x d]).  x, M, K, idx_bits and d
 * are shared; every array holds `count` entries and lives in HOST memory,
 * while the buffers it points to are device memory.  For M <= 16 up to eight
 * matrices run in one launch; when no grouped kernel applies (d = 3, for
 * instance) the matrices are computed one call after another.  Every y[i] is
 * bit-for-bit what fasq_pq_gemv would write for matrix i alone.
 *
 * Returns FASQ_ERR_INVALID_ARG when count < 1, an array is NULL, or any
 * matrix fails the checks of fasq_pq_gemv (fasq_last_error() names the
 * matrix); FASQ_ERR_HIP on a launch error.  The y buffers must not overlap
 * one another or any input.
 */
fasq_status fasq_pq_gemv_batched(const void* x, int64_t M, int64_t K, int count,
                                 const void* const* idx, const int64_t* N,
                                 const void* const* codebook, const int64_t* C,
                                 void* const* y, int idx_bits, int d, hipStream_t stream);

/*
 * Prefill regime (FASQ Sec. 4.2: many tokens share one weight matrix).  Same
 * operation, arguments, layouts and errors as fasq_pq_gemv; built for M in the
 * tens to thousands.  Weight tiles are decoded from the ids into on-chip
 * memory and contracted with matrix-core (MFMA) instructions, fp16 inputs,
 * fp32 accumulation.
 */
fasq_status fasq_pq_gemm(const void* x, int64_t M, int64_t K, int64_t N,
                         const void* idx, int idx_bits, int d,
                         const void* codebook, int64_t C,
                         void* y, hipStream_t stream);

/*
 * fasq_pq_gemm with a workspace (FASQ Sec. 4.2 splits the subspaces, i.e. K,
 * over blocks; Sec. 4.4 tunes the split for the prefill length).  When the
 * output tiles alone leave compute units idle (small M or N), the tuned
 * kernel also splits K over up to 8 workgroups per tile, which write fp32
 * partial sums to the workspace; a second kernel adds them in a fixed order
 * and rounds once to fp16 (deterministic for a given shape and device).
 *
 *   workspace  device scratch of at least fasq_pq_gemm_ex_workspace_bytes()
 *              bytes (4-byte aligned; may be NULL when that is 0); contents
 *              are overwritten.  A NULL or smaller workspace runs exactly
 *              fasq_pq_gemm (no split).
 *
 * Other arguments, layouts and errors as fasq_pq_gemm, plus
 * FASQ_ERR_INVALID_ARG for workspace_bytes < 0.
 */
fasq_status fasq_pq_gemm_ex(const void* x, int64_t M, int64_t K, int64_t N,
                            const void* idx, int idx_bits, int d,
                            const void* codebook, int64_t C,
                            void* y, void* workspace, int64_t workspace_bytes,
                            hipStream_t stream);

/* Workspace bytes fasq_pq_gemm_ex splits K with on the current device (0
 * when it would not split), -1 for invalid sizes. */
int64_t fasq_pq_gemm_ex_workspace_bytes(int64_t M, int64_t K, int64_t N, int idx_bits, int d, int64_t C);

/*
 * The paper's own prefill kernel design (FASQ Sec. 4.2, Alg. 3), kept for
 * comparison with fasq_pq_gemm: per token and subspace a lookup table of the
 * C dot products x_s . codebook[k] is built in LDS (fp32), and every output
 * feature adds up its table entries.  No matrix cores.  Same arguments,
 * layouts and errors as fasq_pq_gemm, plus FASQ_ERR_UNSUPPORTED when d is not
 * in {1, 2, 4, 8} or C > 2048 (the tables would not fit in LDS).
 */
fasq_status fasq_pq_gemm_lut(const void* x, int64_t M, int64_t K, int64_t N,
                             const void* idx, int idx_bits, int d,
                             const void* codebook, int64_t C,
                             void* y, hipStream_t stream);

/*
 * Decode regime with the paper's general codebook layout (FASQ Sec. 3.1.1:
 * T_cluster is [N_ss x K_s x SZ_ss], one codebook per subspace; Eq.
 * lut-accumulate):
 *
 *   y[m, n] = sum_s dot(x[m, s*d : (s+1)*d], codebook[s * cb_stride + u(n, s) * d .. + d])
 *
 *   cb_stride  0: one codebook [C x d] shared by every subspace (exactly
 *              fasq_pq_gemv); C * d: one codebook per subspace, the S = K / d
 *              books back to back, fp16 [S x C x d].  Other values are invalid.
 *   workspace  device scratch of at least fasq_pq_gemv_ex_workspace_bytes()
 *              bytes (4-byte aligned; NULL when that is 0), for the fp32
 *              partial sums of the K split; contents are overwritten
 *
 * Other arguments, layouts and errors as fasq_pq_gemv.  With per-subspace
 * books and M <= 16 the tuned kernel splits K over workgroups whose books fit
 * in LDS and adds the partials in a fixed order (deterministic; each token's
 * output has the bits a call with that token alone gives); for M > 1 it needs
 * d <= 4 and x 16-byte aligned with K * 2 a multiple of 16.  Other shapes, or
 * a workspace that is too small, take the general kernel.  With one shared
 * codebook the call is fasq_pq_gemv, except that the workspace lets the
 * prefill GEMM split K as fasq_pq_gemm_ex does where the GEMM takes the call:
 * beyond 16 tokens, where no decode kernel applies, and, from 12 tokens on,
 * where the decode kernel would stage x in slabs and the GEMM keeps its
 * codebook in LDS (the measured crossover of Sec. 4.4's batch-size trade-off);
 * and it lets the decode kernel for 3 to 16 tokens split K over workgroups
 * where the rows of x outweigh a workgroup's share of the ids (tall K, few
 * rows: 2 to 8 segments, at most 4 MiB of fp32 partials, added in segment
 * order by a second kernel; deterministic, though not the bits of the
 * unsplit call).
 */
fasq_status fasq_pq_gemv_ex(const void* x, int64_t M, int64_t K, int64_t N,
                            const void* idx, int idx_bits, int d,
                            const void* codebook, int64_t C, int64_t cb_stride,
                            void* y, void* workspace, int64_t workspace_bytes,
                            hipStream_t stream);

/* Workspace bytes fasq_pq_gemv_ex uses on the current device for these sizes
 * (per-subspace books: the tuned kernel's partials; one shared codebook: the
 * K split of the GEMM fallback), 0 when none is used, -1 for invalid sizes. */
int64_t fasq_pq_gemv_ex_workspace_bytes(int64_t M, int64_t K, int64_t N, int idx_bits, int d,
                                        int64_t C, int64_t cb_stride);

/*
 * fasq_pq_gemv_ex for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * Same operation, arguments (minus the workspace), layouts and results as
 * fasq_pq_gemv_ex: the scratch that call would take from a caller workspace
 * (the per-subspace K split, the decode kernel's K split, or the K split of
 * the GEMM fallback) comes from
 * a static device array the library holds on every GPU it runs on, of
 * fasq_noalloc_scratch_bytes() = FASQ_NOALLOC_SCRATCH_BYTES bytes, kept until
 * the process ends.  The call allocates nothing: no hipMalloc, no allocating
 * library routine.  Its device address is looked up once per device, on the
 * first call made with that device current.
 *
 * Every call on one GPU shares that GPU's array, and the array keeps the last
 * call's contents: calls that overlap on one GPU (concurrent streams or
 * threads) race on it and must be serialised by the caller.  Calls on
 * different GPUs do not interact.
 *
 * Returns FASQ_ERR_INVALID_ARG for the checks of fasq_pq_gemv_ex and when
 * fasq_pq_gemv_ex_workspace_bytes() of these sizes exceeds the array
 * (fasq_last_error() gives both figures; such calls need fasq_pq_gemv_ex
 * with a workspace), FASQ_ERR_HIP when the array cannot be located or a
 * launch fails.
 */
#define FASQ_NOALLOC_SCRATCH_BYTES (16 * 1024 * 1024)
fasq_status fasq_pq_gemv_ex_noalloc(const void* x, int64_t M, int64_t K, int64_t N,
                                    const void* idx, int idx_bits, int d,
                                    const void* codebook, int64_t C, int64_t cb_stride,
                                    void* y, hipStream_t stream);

/* Bytes of the per-device scratch array of fasq_pq_gemv_ex_noalloc. */
int64_t fasq_noalloc_scratch_bytes(void);

/*
 * Calibration-free PQ encoding of one weight matrix (FASQ Sec. 3.1.1, Alg. 1):
 * Lloyd's k-means over the N * K / d sub-vectors of w, with one codebook of C
 * codewords shared by every subspace (the format the matmul entry points
 * consume).  No calibration data: only the weights.
 *
 *   w              fp16 [N x K], row-major; sub-vector p = n * (K / d) + s is
 *                  w[n, s*d : (s+1)*d]; finite, |w| < 128 (unchecked)
 *   d, C, idx_bits sub-vector length (1 <= d <= 16), codewords, id width
 *   init_codebook  fp16 [C x d], the starting codewords (for example C
 *                  distinct sub-vectors of w chosen at random); may be the
 *                  same buffer as `codebook`
 *   iters          Lloyd iterations (assignment, then update), >= 0
 *   codebook       out: fp16 [C x d], the codewords after `iters` updates
 *   idx            out: N rows of fasq_idx_row_bytes(K, d, idx_bits) bytes,
 *                  the nearest codeword of every sub-vector under the final
 *                  codebook, in the packed format of fasq_pq_gemv
 *   workspace      device scratch of at least
 *                  fasq_pq_encode_workspace_bytes(N, K, d, C) bytes, 8-byte
 *                  aligned; its contents are overwritten
 *
 * Arithmetic (the paper leaves it open): squared distances in fp32, summed
 * over the d components in order without fused multiply-add, the lowest index
 * winning a tie; cluster sums formed exactly (every fp16 value is a multiple
 * of 2^-24), the mean divided out in fp64 and rounded to fp16 (nearest, ties
 * to even); an empty cluster keeps its codeword.  The result does not depend
 * on scheduling: repeated calls give identical bits.
 *
 * Asynchronous on `stream`; the caller owns every buffer.  Returns
 * FASQ_ERR_INVALID_ARG (sizes; d does not divide K; idx_bits not in
 * {8, 12, 16}; C outside [1, 2^idx_bits]; iters < 0; a NULL or misaligned
 * pointer; a workspace that is too small), FASQ_ERR_UNSUPPORTED (d > 16) or
 * FASQ_ERR_HIP.
 */
fasq_status fasq_pq_encode(const void* w, int64_t N, int64_t K, int d, int64_t C, int idx_bits,
                           const void* init_codebook, int iters, void* codebook, void* idx,
                           void* workspace, int64_t workspace_bytes, hipStream_t stream);

/* Workspace bytes fasq_pq_encode needs for these sizes; -1 if they are invalid
 * (N, K < 1; d does not divide K; C outside [1, 65536]). */
int64_t fasq_pq_encode_workspace_bytes(int64_t N, int64_t K, int d, int64_t C);

/*
 * Launch lists: the kernel launches of a sequence of library calls, recorded
 * once and queued again as often as needed, for callers that issue the same
 * calls with the same buffers at every step (a serving loop's decode step, a
 * benchmark) and want to pay only for the launches: no argument checks, no
 * kernel selection, no HIP graph.  Between fasq_launch_list_begin and
 * fasq_launch_list_end, every fasq_* compute call made on the calling thread
 * (fasq_pq_gemv, _batched, _ex, _ex_noalloc, fasq_pq_gemm, _ex, _lut,
 * fasq_pq_reconstruct, fasq_pq_encode) validates its arguments and chooses its
 * kernels as usual, then appends its launches (kernel, grid, block, LDS bytes
 * and a copy of the argument values) to the list instead of queueing them; its
 * `stream` argument is ignored.  fasq_launch_list_run queues every recorded
 * launch, in recording order, on `stream`.  A run computes what the recorded
 * calls would have computed at that point of the stream, bit for bit.
 *
 * The list holds the device addresses the calls were given (inputs, outputs,
 * workspaces, the static array of fasq_pq_gemv_ex_noalloc): they must stay
 * valid while the list may run, and a run reads and writes their contents as
 * they are when it executes.  A list records for the device current at
 * fasq_launch_list_begin and runs only with that device current (its
 * recorded launches from later begin/end pairs are appended and must be on
 * the same device).  A call that fails while recording returns its error and
 * may leave part of its launches in the list: destroy such a list.
 *
 *   fasq_launch_list_create   *list = a new, empty list.  FASQ_ERR_INVALID_ARG
 *                             (list is NULL), FASQ_ERR_HOST_MEMORY.
 *   fasq_launch_list_begin    the calling thread records into `list`.
 *                             FASQ_ERR_INVALID_ARG when list is NULL, the
 *                             thread already records a list, the list records
 *                             on another thread, or it holds launches for
 *                             another device; FASQ_ERR_HIP when no device is
 *                             current.
 *   fasq_launch_list_end      stop recording.  FASQ_ERR_INVALID_ARG when
 *                             `list` does not record on the calling thread.
 *   fasq_launch_list_run      queue the launches on `stream` (asynchronous).
 *                             FASQ_ERR_INVALID_ARG when list is NULL, it
 *                             records, the calling thread records a list, or
 *                             another device is current; FASQ_ERR_HIP when a
 *                             launch fails (fasq_last_error() names which;
 *                             the launches before it are queued).  An empty
 *                             list queues nothing.  Runs from several threads
 *                             may share a list.
 *   fasq_launch_list_size     launches recorded, -1 for a NULL list.
 *   fasq_launch_list_destroy  free the list (and stop recording into it on the
 *                             calling thread); NULL is ignored.  Launches
 *                             already queued are not affected.  No other
 *                             thread may record into the list, or run it,
 *                             while it is destroyed, and no thread may
 *                             record into a list that another thread runs.
 */
typedef struct fasq_launch_list fasq_launch_list;
fasq_status fasq_launch_list_create(fasq_launch_list** list);
fasq_status fasq_launch_list_begin(fasq_launch_list* list);
fasq_status fasq_launch_list_end(fasq_launch_list* list);
fasq_status fasq_launch_list_run(const fasq_launch_list* list, hipStream_t stream);
int64_t fasq_launch_list_size(const fasq_launch_list* list);
void fasq_launch_list_destroy(fasq_launch_list* list);

/*
 * Decode W_hat explicitly (the reconstruction the paper's reconstruction-free
 * kernels avoid, Sec. 3.1.2).  Writes fp16 [N x K] to `w`; every element is a
 * bit-for-bit copy of a codebook entry (signed zeros, subnormals, NaN
 * payloads preserved).  Diagnostic only: it is how the decoder is tested.
 * Errors as for fasq_pq_gemv.
 */
fasq_status fasq_pq_reconstruct(const void* idx, int64_t N, int64_t K, int idx_bits, int d,
                                const void* codebook, int64_t C, void* w,
                                hipStream_t stream);

/*
 * Bytes of one packed index row: ceil((K / d) * idx_bits / 8).  Each of the
 * K / d sub-vectors of a row stores one codeword id of ceil(log2 K_s) bits
 * (FASQ Sec. 3.2, the index term of the storage footprint); ids are packed
 * as the bit stream described at the top of this file.  Returns -1 when
 * K < 1, d < 1, K % d != 0 or idx_bits is not 8, 12 or 16.  Host only.
 */
int64_t fasq_idx_row_bytes(int64_t K, int d, int idx_bits);

/* Static, human-readable name of a status code. */
const char* fasq_status_string(fasq_status s);

/*
 * Detail of the calling thread's most recent failed call ("" if none).  The
 * string stays valid until the thread's next fasq_* call.
 */
const char* fasq_last_error(void);

/* FASQ_ABI_VERSION of the built library. */
int fasq_abi_version(void);

/*
 * Diagnostic: the name of the kernel instantiation that fasq_pq_gemv
 * (regime 0), fasq_pq_gemm (regime 1) or fasq_pq_gemv_batched over two or
 * more matrices of these sizes (regime 2) would launch with 16-byte-aligned
 * buffers, e.g. "k_gemv_m1<8, 2, 2, 0, 0>" (template arguments in
 * declaration order).  Launches nothing; needs a current HIP
 * device.  Returns "" for invalid arguments or when no device is available.
 * The string is thread-local and valid until the thread's next fasq_* call.
 */
const char* fasq_pq_plan(int regime, int64_t M, int64_t K, int64_t N, int idx_bits, int d, int64_t C);

#ifdef __cplusplus
}
#endif

#endif /* FASQ_H */
