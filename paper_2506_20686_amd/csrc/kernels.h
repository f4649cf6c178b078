// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace triattn {

// Geometry of one call.  A pair tensor X[a][b][h][c] is addressed through
// (row, position): the starting node has row = a and position = b, the
// ending node row = b and position = a, so the ending node is the same
// kernel with the two strides swapped; no transpose copy is made.
struct Geom {
  int n;     // tokens per pair axis (queries and keys of a row)
  int nr;    // rows this call computes (n, or a row range's length)
  int H;     // heads
  int np;    // n rounded up to a multiple of 32
  int nkt;   // np / 32 key tiles
  int d;     // channels per head: 32, or 64 (register-staged kernels only)
  int64_t sRow, sPos;  // element strides of [nr][n][H][d] tensors
  int64_t lRow, lPos;  // element strides of [n][n][H] tensors (lse)
  float scale;         // softmax scale on Q K^T
  // Batched launches (bf16, 32 channels): sample s = blockIdx.z of a grid
  // with `batch` layers finds its tensors `s` strides past the first sample's
  // and its own workspace `s * bWs` bytes past the first.  batch = 1 and zero
  // strides otherwise.
  int batch;
  int64_t bPair;  // elements of one sample's [n][n][H][d] tensor
  int64_t bBias;  // elements of one sample's [n][n][H] tensor (bias, dbias, lse)
  int64_t bMask;  // bytes of one sample's [n][n] mask
  int64_t bWs;    // bytes of one sample's workspace
};

// This block's sample of a batched launch (0 otherwise).
__device__ inline int64_t sample_id() { return (int64_t)blockIdx.z; }
template <typename P>
__device__ inline P* at_sample(P* p, int64_t stride) {
  return p ? p + sample_id() * stride : p;
}
template <typename P>
__device__ inline P* ws_at_sample(P* p, int64_t bytes) {
  return p ? (P*)((char*)p + sample_id() * bytes) : p;
}
template <typename P>
__device__ inline const P* ws_at_sample(const P* p, int64_t bytes) {
  return p ? (const P*)((const char*)p + sample_id() * bytes) : p;
}

// Workspace pieces (device pointers), see api.hip for sizes.
struct Prep {
  float* bt;       // [H][np/32][np/32][1024] bias(q, k) / scale in accumulator order,
                   //   lanes <-> queries (zero padded)
  float* btT;      // the same with lanes <-> keys (backward only; may be null)
  uint32_t* kbits; // [nr][nkt]    bit e of word t: key 32 t + e is valid for that row
  uint32_t* rowfull;  // [nr]    1 iff every key < n is valid for that row, else 0
};

struct BwdWs {
  float* lse2;   // [H][nr][np]  lse * log2(e); +inf where the query has no valid key
  float* dsum;   // [H][nr][np]  -D, D = rowsum(dO * O) (stored negated: it enters as -D)
  void* da;      // [nr][n][H][32] dtype: dA = dO * sigmoid(G), laid out like dO
  void* dalo;    // bf16 only: dA - bf16(dA) rounded to bf16 (null for fp32)
  float* slabs;  // [nrc][H][np][np] per-row-chunk partial bias gradients
  int nrc;       // row chunks of the bias-gradient reduction
};

template <typename T>
hipError_t launch_prep(const Geom& g, int node, const T* bias, const uint8_t* mask, const Prep& p,
                       hipStream_t s);
template <typename T>
hipError_t launch_fwd(const Geom& g, const Prep& p, const T* q, const T* k, const T* v,
                      const T* gate, T* out, float* lse, hipStream_t s);
// dbias_f32, when not null, receives the bias gradient in fp32 (a row range's
// partial sum, to be added to other ranges' before rounding) and dbias is unused.
template <typename T>
hipError_t launch_bwd(const Geom& g, int node, const Prep& p, const BwdWs& w, const T* q,
                      const T* k, const T* v, const T* gate, const T* out, const float* lse,
                      const T* dout, T* dq, T* dk, T* dv, T* dg, T* dbias, float* dbias_f32,
                      hipStream_t s);

// d = 16 through the d = 32 kernels (pad.hip): rows of 16 channels copied
// into rows of 32 with zeros, and back.
hipError_t launch_pad16(const void* src, void* dst, int64_t rows, int elem_bytes, hipStream_t s);
hipError_t launch_unpad16(const void* src, void* dst, int64_t rows, int elem_bytes,
                          hipStream_t s);

// ---- fused layer-norm + linear projection (lnl.hip) ---------------------------------
constexpr int LNL_K = 128;       // features per row (the pair channel width)
constexpr int LNL_MAX_OUT = 8;   // output tensors o2's columns are split into
constexpr int LNL_MAX_TILES = 32;  // 32-column output tiles (N <= 1024)

// Output columns one workgroup keeps resident in LDS as W^T (a launch covers
// N in ceil(N / LNL_GROUP) column groups).
constexpr int LNL_GROUP = 544;

// Where 32-column output tile T goes.  fast: all 32 columns lie in one
// output i, 16-byte aligned (w and off multiples of 8), and (m + 32) w 2
// bytes fit a buffer resource; the tile is then stored with buffer stores
// at base + ((row w + off + 8 c) 2) bytes, rows past m dropped by the
// resource's range check.  Other tiles use the per-quad table.
struct LnlTile {
  bf16* base;  // out[i]
  int off;     // first column of the tile inside output i
  int w;       // width of output i
  int fast;
  int pad;
};

struct LnlArgs {
  int64_t m;                     // rows
  int ncols;                     // output columns N (sum of the outputs' widths)
  int gw;                        // columns per workgroup group (multiple of 32)
  int n_out;                     // output tensors
  int start[LNL_MAX_OUT + 1];    // first column of each output; start[n_out] = N
  float eps;
  const bf16 *x, *gamma, *beta;  // x [m][K], gamma and beta [K]
  const bf16* w;                 // W [K][N]
  bf16* out[LNL_MAX_OUT];        // output i: [m][start[i + 1] - start[i]]
  float *mean, *rstd;            // [m], saved for the backward
  LnlTile tile[LNL_MAX_TILES];
};

hipError_t launch_lnl_fwd(const LnlArgs& a, hipStream_t s);

// Backward (N <= LNL_GROUP).  Row sums go through per-workgroup partial
// slabs: gpart [nwg][K + 1][np] holds, per workgroup of the row-sum kernel,
// G = xhat^T dO2 (rows 0..K-1) and s = column sums of dO2 (row K); gsum
// [K + 1][np] their fixed-order totals.
struct LnlBwdArgs {
  int64_t m;
  int ncols, np, n_out;
  int start[LNL_MAX_OUT + 1];
  const bf16 *x, *gamma, *beta, *w;  // forward inputs
  const float *mean, *rstd;          // forward statistics
  const bf16* dout[LNL_MAX_OUT];     // dO2 split like the forward's outputs
  bf16* dx;                          // [m][K]
  float *dw, *dgamma, *dbeta;        // [K][N], [K], [K]
  float *gpart, *gsum;               // workspace
  int nwg;                           // workgroups of the row-sum kernel
  LnlTile tile[LNL_MAX_TILES];       // dO2 source of each 32-column tile
};

// Workgroups of the row-sum kernel and workspace bytes for m rows, np columns.
int lnl_bwd_partials(int64_t m);
size_t lnl_bwd_workspace(int64_t m, int np);
hipError_t launch_lnl_bwd(const LnlBwdArgs& a, hipStream_t s);

// ---- fused transition layer (trn.hip) -----------------------------------------------
constexpr int TRN_C = 128;         // features per row (the pair channel width)
constexpr int TRN_FC = 32;         // hidden columns per weight chunk
constexpr int TRN_FWD_IMG = 24576; // bytes of one chunk's forward weight image
constexpr int TRN_BWD_IMG = 40960; // bytes of one chunk's backward weight image
constexpr int TRN_GROUP = 128;     // hidden columns per workgroup of the weight-gradient kernel

struct TrnFwdArgs {
  int64_t m;                     // rows
  int f;                         // hidden width F (a multiple of TRN_GROUP)
  float eps;
  const bf16 *x, *gamma, *beta;  // x [m][C], gamma and beta [C]
  const bf16 *w1, *w2;           // W1 [C][2F], W2 [F][C]
  char* img;                     // workspace: F / 32 forward chunk images
  bf16* out;                     // [m][C]
  float *mean, *rstd;            // [m], saved for the backward
};

struct TrnBwdArgs {
  int64_t m;
  int f;
  const bf16 *x, *gamma, *beta, *w1, *w2;
  const float *mean, *rstd;      // forward statistics
  const bf16* dout;              // [m][C]
  bf16* dx;                      // [m][C]
  float *dw1, *dw2, *dgamma, *dbeta;  // [C][2F], [F][C], [C], [C]
  char* img;                     // workspace: F / 32 backward chunk images
  float* part;                   // workspace: nparts partial sums (see trn_part_floats)
  float* gsum;                   // workspace: G [C][2F] and s [2F] totals
  int nparts;                    // row partitions of the weight-gradient kernel
};

// Floats of one partial-sum block: G [C][2F], s [2F], dW2 [F][C].
__host__ __device__ inline int64_t trn_part_floats(int f) { return (int64_t)TRN_C * 2 * f + 2 * f + (int64_t)f * TRN_C; }
int trn_bwd_parts(int64_t m, int f);
hipError_t launch_trn_fwd(const TrnFwdArgs& a, hipStream_t s);
hipError_t launch_trn_bwd(const TrnBwdArgs& a, hipStream_t s);

}  // namespace triattn
