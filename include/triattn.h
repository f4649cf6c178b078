/*
 * triattn: triangle self-attention (starting and ending node) for MI355X.
 *
 * The operation is MegaFold's memory-efficient 3D attention (arXiv
 * 2506.20686, Section IV-A; forward and backward definitions in the appendix
 * table "EvoAttention's forward and backward passes"), extended with the
 * AF3 sigmoid gate.  For every pair (a, b) of an N x N pair map and head h:
 *
 *   starting node, row r = a, query q = b, keys k:
 *     s_k = scale * <Q[r][q][h], K[r][k][h]> + bias[q][k][h],  valid iff mask[r][k]
 *     out[r][q][h] = sigmoid(G[r][q][h]) * sum_k softmax(s)_k V[r][k][h]
 *   ending node, row j = b, query i = a, keys k:
 *     s_k = scale * <Q[i][j][h], K[k][j][h]> + bias[k][i][h],  valid iff mask[k][j]
 *     out[i][j][h] = sigmoid(G[i][j][h]) * sum_k softmax(s)_k V[k][j][h]
 *
 * The softmax over keys is streamed (online max and sum) and the N^3 H logit
 * tensor never exists in memory (Section IV-A); the forward saves one fp32
 * log-sum-exp per (pair, head) for the backward pass, which recomputes the
 * probabilities from it.  The bias gradient is a sum over the pair-row axis
 * (appendix table); it is reduced in a fixed order, so results are bitwise
 * reproducible (the paper's atomics are not).
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are DEVICE memory owned by the caller, C-contiguous
 *     with the last index fastest:
 *       q, k, v, g, out, dout, dq, dk, dv, dg : [n][n][h][d]   (dtype)
 *       bias, dbias                             : [n][n][h]      (dtype)
 *       lse                                     : [n][n][h]      (fp32)
 *       mask                                    : [n][n]         (uint8, 0 = masked)
 *     Tensor pointers must be 16-byte aligned.  mask may be NULL (all valid).
 *   - A masked key gets weight exactly 0.  A query with no valid key gets
 *     out = 0, lse = -inf and contributes nothing to any gradient.
 *   - Inputs must be finite, except that bias entries may be -inf: an
 *     additive -inf excludes that key for that query like the mask does (a
 *     query whose valid keys all carry -inf is treated as one with no valid
 *     key).  Device code is compiled on the assumption that no NaN reaches it
 *     (-fno-honor-nans), so a NaN input gives unspecified results.
 *   - dtype TRIATTN_BF16: bfloat16 tensors, fp32 accumulation, outputs
 *     rounded to nearest even.  TRIATTN_F32: fp32 throughout.
 *   - d must be 32; the whole-map and batched calls also take d = 16 and
 *     d = 64.  bf16 d = 16 runs the 32-channel kernels' 16-channel variants
 *     on the tensors as they are; fp32 d = 16 runs the d = 32 kernels on
 *     zero-padded copies held in the workspace (zero channels add exact
 *     zeros: the results are those of d = 16).  bf16 d = 64 runs the DMA
 *     kernels' 64-channel variants, fp32 d = 64 register-staged kernels built
 *     for 64 channels.  1 <= n <= 8192, 1 <= h <= 64.  scale must be finite and
 *     positive (1/sqrt(d) is the usual choice).
 *   - The library never allocates or frees memory and never synchronises:
 *     work is enqueued on `stream` (a hipStream_t; NULL is the default stream)
 *     and the caller supplies a device workspace of at least the size the
 *     matching *_workspace_bytes call reports.  Outputs are fully
 *     overwritten.  Calls that share a workspace must not overlap.
 *   - Errors: every function returns a triattn_status.  Arguments are checked
 *     before any HIP call is made, so an invalid call has no effect.  A HIP
 *     launch failure returns TRIATTN_ERR_HIP.  Nothing aborts.
 *   - Determinism: the same arguments on the same device give bitwise
 *     identical results.
 */
#ifndef TRIATTN_H
#define TRIATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TRIATTN_OK = 0,
  TRIATTN_ERR_INVALID_ARG = 1, /* null pointer, bad enum, size or scale out of range */
  TRIATTN_ERR_UNSUPPORTED = 2, /* a value the library does not implement (e.g. d = 128) */
  TRIATTN_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  TRIATTN_ERR_HIP = 4,         /* a HIP launch reported an error */
  TRIATTN_ERR_TOO_LARGE = 5    /* more scratch than tri_attn_fwd_noalloc holds */
} triattn_status;

typedef enum { TRIATTN_STARTING = 0, TRIATTN_ENDING = 1 } triattn_node;
typedef enum { TRIATTN_F32 = 0, TRIATTN_BF16 = 1 } triattn_dtype;

/* Bytes of device workspace tri_attn_fwd needs for these sizes, written to
 * *bytes.  Pure host arithmetic. */
int tri_attn_fwd_workspace_bytes(int node, int dtype, int64_t n, int64_t h, int64_t d,
                                 size_t* bytes);

/* Forward pass (Section IV-A: online-softmax streaming over key tiles,
 * log-sum-exp saved).  Writes out [n][n][h][d] (dtype, gated) and lse
 * [n][n][h] (fp32, natural log; -inf for a query with no valid key). */
int tri_attn_fwd(int node, int dtype, int64_t n, int64_t h, int64_t d, float scale,
                 const void* q, const void* k, const void* v, const void* g, const void* bias,
                 const uint8_t* mask, void* out, float* lse, void* workspace,
                 size_t workspace_bytes, void* stream);

/* The forward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results (bitwise) and rules as tri_attn_fwd, without the
 * workspace: the library keeps it in a device array of
 * TRIATTN_FWD_NOALLOC_SCRATCH_BYTES that each GPU it runs on holds from the
 * library's first use until the process ends; the call itself allocates and
 * frees nothing.  Sizes whose forward workspace (tri_attn_fwd_workspace_bytes)
 * exceeds the array return TRIATTN_ERR_TOO_LARGE (N = 768 at h = 4, d = 32
 * needs about 9.5 MiB; fp32 d = 16 needs its padded copies too).  `stream` must
 * belong to the current device (TRIATTN_ERR_INVALID_ARG otherwise).  Every
 * call on one GPU shares that GPU's array: calls that may overlap on one GPU
 * (different streams, no ordering between them) race and must not be made;
 * calls on one stream are ordered and safe. */
#define TRIATTN_FWD_NOALLOC_SCRATCH_BYTES (32u << 20)
int tri_attn_fwd_noalloc(int node, int dtype, int64_t n, int64_t h, int64_t d, float scale,
                         const void* q, const void* k, const void* v, const void* g,
                         const void* bias, const uint8_t* mask, void* out, float* lse,
                         void* stream);

/* Bytes of device workspace tri_attn_bwd needs for these sizes. */
int tri_attn_bwd_workspace_bytes(int node, int dtype, int64_t n, int64_t h, int64_t d,
                                 size_t* bytes);

/* Backward pass of L = sum(dout * out) (appendix backward listing and
 * table: D = rowsum(dO * O), dS = P (dP - D), dK/dV stage, dQ stage, bias
 * gradient summed over rows in fixed order).  Takes the forward's inputs,
 * its out and lse, and dout; writes dq, dk, dv, dg [n][n][h][d] and dbias
 * [n][n][h], all in dtype.  The mask and scale get no gradient. */
int tri_attn_bwd(int node, int dtype, int64_t n, int64_t h, int64_t d, float scale,
                 const void* q, const void* k, const void* v, const void* g, const void* bias,
                 const uint8_t* mask, const void* out, const float* lse, const void* dout,
                 void* dq, void* dk, void* dv, void* dg, void* dbias, void* workspace,
                 size_t workspace_bytes, void* stream);

/* A batch of `batch` independent pair maps (each sample with its own bias
 * and mask): tensors gain a leading batch axis,
 *   q, k, v, g, out, dout, dq, dk, dv, dg : [batch][n][n][h][d]
 *   bias, dbias, lse                        : [batch][n][n][h]
 *   mask                                    : [batch][n][n]  (NULL = all valid)
 * and sample b gives exactly what tri_attn_fwd / tri_attn_bwd give for its
 * slices, bitwise.  With a workspace of the size the *_batched_workspace_bytes
 * calls report (one copy of the unbatched workspace per sample), every kernel
 * is launched once for the whole batch (the sample is the grid's third
 * index), which keeps the GPU full when one sample's grid is small.  With the
 * unbatched workspace size (tri_attn_fwd_workspace_bytes /
 * tri_attn_bwd_workspace_bytes for n, h, d) the samples run one after another
 * on `stream` and share it.  fp32 d = 16 always runs sample by sample, and so
 * do batches above 65535.  The base pointers follow the unbatched rules;
 * 1 <= batch <= 2^20.  The per-sample slices of bias, dbias, lse and mask need
 * only element alignment. */
int tri_attn_fwd_batched_workspace_bytes(int node, int dtype, int64_t batch, int64_t n,
                                         int64_t h, int64_t d, size_t* bytes);
int tri_attn_bwd_batched_workspace_bytes(int node, int dtype, int64_t batch, int64_t n,
                                         int64_t h, int64_t d, size_t* bytes);
int tri_attn_fwd_batched(int node, int dtype, int64_t batch, int64_t n, int64_t h, int64_t d,
                         float scale, const void* q, const void* k, const void* v, const void* g,
                         const void* bias, const uint8_t* mask, void* out, float* lse,
                         void* workspace, size_t workspace_bytes, void* stream);
int tri_attn_bwd_batched(int node, int dtype, int64_t batch, int64_t n, int64_t h, int64_t d,
                         float scale, const void* q, const void* k, const void* v, const void* g,
                         const void* bias, const uint8_t* mask, const void* out,
                         const float* lse, const void* dout, void* dq, void* dk, void* dv,
                         void* dg, void* dbias, void* workspace, size_t workspace_bytes,
                         void* stream);

/* Starting node over a contiguous range of rows: one GPU's share of the
 * pair representation when it is split into contiguous shards along one
 * sequence axis (Section IV-B, sequence parallelism).  Rows of the starting
 * node are independent attention problems, so a range of `rows` rows
 * (1 <= rows <= n) gives exactly those rows of the whole call's results.
 * Tensors are local to the range, row 0 being the range's first row:
 *   q, k, v, g, out, dout, dq, dk, dv, dg : [rows][n][h][d]  (dtype)
 *   lse                                     : [rows][n][h]     (fp32)
 *   mask                                    : [rows][n]        (uint8; NULL = all valid)
 *   bias                                    : [n][n][h]        (dtype, the whole map)
 *   dbias_partial                           : [n][n][h]        (fp32)
 * dbias_partial is this range's term of the bias gradient, the sum over its
 * rows, kept in fp32: the whole gradient is the sum of every range's term
 * (in a fixed order for reproducible results), rounded once.  The ending
 * node's shards are starting-node shards of the transposed map (ending =
 * starting applied to T(q), T(k), T(v), T(g) with bias^T and mask^T, T
 * swapping the two pair axes), which is where the re-shard between the two
 * nodes puts them.  Size, pointer, workspace, stream and error rules as
 * above; rows outside [1, n] is TRIATTN_ERR_INVALID_ARG. */
int tri_attn_rows_fwd_workspace_bytes(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d,
                                      size_t* bytes);

/* Forward pass of rows [0, rows) of a range (same outputs as tri_attn_fwd
 * for those rows). */
int tri_attn_rows_fwd(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d, float scale,
                      const void* q, const void* k, const void* v, const void* g,
                      const void* bias, const uint8_t* mask, void* out, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of device workspace tri_attn_rows_bwd needs for these sizes. */
int tri_attn_rows_bwd_workspace_bytes(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d,
                                      size_t* bytes);

/* Backward pass of a range: dq, dk, dv, dg of its rows (as tri_attn_bwd
 * gives them) and its fp32 bias-gradient term dbias_partial. */
int tri_attn_rows_bwd(int dtype, int64_t n, int64_t rows, int64_t h, int64_t d, float scale,
                      const void* q, const void* k, const void* v, const void* g,
                      const void* bias, const uint8_t* mask, const void* out, const float* lse,
                      const void* dout, void* dq, void* dk, void* dv, void* dg,
                      float* dbias_partial, void* workspace, size_t workspace_bytes,
                      void* stream);

/* Fused layer-norm + linear projection (Section IV, fused layer-norm &
 * linear projection; forward formulas in the appendix table of fused
 * operators): the step that produces the attention inputs from the pair
 * representation.  For every row of x [m][k]:
 *   o1 = (x - mean) * rstd * gamma + beta,  rstd = 1 / sqrt(var + eps),
 *        mean and var (biased) over the row's k features;
 *   o2 = o1 W,  W [k][ncols],  ncols = cols[0] + ... + cols[n_out - 1].
 * o2's columns are written into n_out row-major tensors: outs[i] receives
 * columns cols[0] + ... + cols[i - 1] onwards as [m][cols[i]] (for triangle
 * attention: Q, K, V, G [n*n][h*d] and the bias logits [n*n][h]).  mean and
 * rstd [m] (fp32) are saved for the backward pass.
 *   dtype: TRIATTN_BF16 only (x, gamma [k], beta [k], w and the outputs;
 *          fp32 statistics and accumulation); TRIATTN_ERR_UNSUPPORTED else.
 *   k must be 128; 1 <= n_out <= 8; every cols[i] a positive multiple of 4
 *   and ncols <= 1024; m >= 1; eps finite and >= 0.
 *   cols and outs are host arrays; tensor pointers are device memory,
 *   16-byte aligned.  No workspace.  Same stream and error rules as above. */
int tri_ln_linear_fwd(int dtype, int64_t m, int64_t k, int n_out, const int64_t* cols, float eps,
                      const void* x, const void* gamma, const void* beta, const void* w,
                      void* const* outs, float* mean, float* rstd, void* stream);

/* Bytes of device workspace tri_ln_linear_bwd needs for these sizes. */
int tri_ln_linear_bwd_workspace_bytes(int dtype, int64_t m, int64_t k, int n_out,
                                      const int64_t* cols, size_t* bytes);

/* Backward pass of the fused layer-norm + linear projection for
 * L = sum(do2 * o2) (appendix table of fused operators: do1 = do2 W^T,
 * dW = o1^T do2, dgamma = sum over rows of do1 * xhat, dbeta = sum over
 * rows of do1, dx = rstd (do1 gamma - c1 xhat - c2) with c1, c2 the row
 * means over the k features of xhat do1 gamma and of do1 gamma).  Takes the
 * forward's x, gamma, beta, w and its saved mean and rstd, and douts: n_out
 * tensors [m][cols[i]] holding do2 split like the forward's outputs.
 * Writes dx [m][k] (dtype), dw [k][ncols], dgamma [k] and dbeta [k] (fp32,
 * sums over rows taken in a fixed order: bitwise reproducible).
 *   Same size rules as tri_ln_linear_fwd, and ncols <= 544 and
 *   (m + 32) * max(k, cols[i]) * 2 < 2^31 (TRIATTN_ERR_UNSUPPORTED else).
 *   Same pointer, workspace, stream and error rules as above. */
int tri_ln_linear_bwd(int dtype, int64_t m, int64_t k, int n_out, const int64_t* cols,
                      const void* x, const void* gamma, const void* beta, const void* w,
                      const float* mean, const float* rstd, const void* const* douts, void* dx,
                      float* dw, float* dgamma, float* dbeta, void* workspace,
                      size_t workspace_bytes, void* stream);

/* Fused transition layer (Section IV: fused layer-norm & linear projection,
 * fused SwiGLU, fused transition layer; forward and backward in the
 * appendix listing of the transition layer).  For every row x of x [m][c]:
 *   o1 = (x - mean) * rstd * gamma + beta,  rstd = 1 / sqrt(var + eps),
 *        mean and var (biased) over the row's c features;
 *   [a | b] = o1 W1,  W1 [c][2f]: a = columns 0..f-1, b = columns f..2f-1;
 *   u = a * sigmoid(a) * b                    (SwiGLU)
 *   out = u W2,  W2 [f][c].
 * out [m][c] (dtype) and mean, rstd [m] (fp32, saved for the backward).
 * Neither [a | b] nor u is written to memory.
 *   dtype: TRIATTN_BF16 only (x, gamma [c], beta [c], W1, W2, out; fp32
 *          statistics and accumulation), TRIATTN_ERR_UNSUPPORTED else.
 *   c must be 128; f a multiple of 128, at most 2048; 1 <= m <= 2^31;
 *   eps finite and >= 0.  Pointers are device memory, 16-byte aligned.
 *   The workspace (size from the matching call) holds the weights in the
 *   order the kernels read them.  Same stream and error rules as above. */
int tri_transition_fwd_workspace_bytes(int dtype, int64_t m, int64_t c, int64_t f,
                                       size_t* bytes);
int tri_transition_fwd(int dtype, int64_t m, int64_t c, int64_t f, float eps, const void* x,
                       const void* gamma, const void* beta, const void* w1, const void* w2,
                       void* out, float* mean, float* rstd, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Backward of the transition layer for L = sum(dout * out): takes the
 * forward's x, gamma, beta, W1, W2, its saved mean and rstd, and dout
 * [m][c]; recomputes [a | b] and writes dx [m][c] (dtype) and dW1 [c][2f],
 * dW2 [f][c], dgamma [c], dbeta [c] (fp32 sums over rows taken in a fixed
 * order: bitwise reproducible).  With du = dout W2^T:
 *   da = du * b * sigmoid(a) * (1 + a (1 - sigmoid(a))),  db = du * a * sigmoid(a),
 *   dW2 = u^T dout,  dW1 = o1^T [da | db],  do1 = [da | db] W1^T,
 *   dgamma = sum over rows of do1 * xhat,  dbeta = sum over rows of do1,
 *   dx = rstd (do1 gamma - c1 xhat - c2), c1 and c2 the row means of
 *   xhat do1 gamma and of do1 gamma.
 * Same size, pointer, workspace, stream and error rules as the forward. */
int tri_transition_bwd_workspace_bytes(int dtype, int64_t m, int64_t c, int64_t f,
                                       size_t* bytes);
int tri_transition_bwd(int dtype, int64_t m, int64_t c, int64_t f, const void* x,
                       const void* gamma, const void* beta, const void* w1, const void* w2,
                       const float* mean, const float* rstd, const void* dout, void* dx,
                       float* dw1, float* dw2, float* dgamma, float* dbeta, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Static, human-readable name of a status code ("unknown status" otherwise). */
const char* tri_attn_status_string(int status);

/* Per-kernel timing, for benchmarks and profiling (not part of the paper's
 * method).  While enabled, every entry point records a pair of HIP events
 * on its stream around each kernel it launches.  The switch and the
 * accumulated times are process-wide; enable it only while no other thread
 * is calling the library.  Off by default. */
int tri_attn_timing_enable(int on);

/* Restricts the per-kernel timing to the kernels whose bit is set in `mask`
 * (bit i: kernel i in tri_attn_timing_read's numbering); 0, the default,
 * times every kernel.  Each timed launch records two events, which costs
 * the stream a little time, so a benchmark can time only the kernel it
 * needs.  Process-wide, like tri_attn_timing_enable.  Returns TRIATTN_OK. */
int tri_attn_timing_select(uint64_t mask);

/* Waits for the recorded events of kernel `index` (0, 1, ... in launch-site
 * order; TRIATTN_ERR_INVALID_ARG past the last one) and returns its name
 * (static string), the summed elapsed milliseconds and the launch count
 * since the last reset.  TRIATTN_ERR_HIP if an event call failed. */
int tri_attn_timing_read(int index, const char** name, double* total_ms, int64_t* launches);

/* Clears the accumulated times and counts (after waiting for pending
 * events); returns TRIATTN_ERR_HIP if an event call had failed. */
int tri_attn_timing_reset(void);

/* Calibration kernel for the MFMA-activity counters (not part of the paper's
 * method): `blocks` workgroups of 4 waves, each wave running `iters` rounds of
 * eight bf16 v_mfma_f32_32x32x16 (32768 flop each) and nothing else, then
 * writing one float per thread to out [blocks * 256] (device memory).
 * 1 <= blocks <= 2^20, 1 <= iters <= 2^24; asynchronous on `stream`. */
int tri_attn_mfma_probe(int64_t blocks, int64_t iters, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TRIATTN_H */
