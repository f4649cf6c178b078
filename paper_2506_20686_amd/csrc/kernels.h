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
  int n;     // tokens per pair axis
  int H;     // heads
  int np;    // n rounded up to a multiple of 32
  int nkt;   // np / 32 key tiles
  int64_t sRow, sPos;  // element strides of [n][n][H][32] tensors
  int64_t lRow, lPos;  // element strides of [n][n][H] tensors (lse)
  float scale;         // softmax scale on Q K^T
};

// Workspace pieces (device pointers), see api.hip for sizes.
struct Prep {
  float* bt;       // [H][np/32][np/32][1024] bias(q, k) / scale in accumulator order,
                   //   lanes <-> queries (zero padded)
  float* btT;      // the same with lanes <-> keys (backward only; may be null)
  uint32_t* kbits; // [n][nkt]     bit e of word t: key 32 t + e is valid for that row
  uint32_t* rowfull;  // [n]     1 iff every key < n is valid for that row, else 0
};

struct BwdWs {
  float* lse2;   // [H][n][np]  lse * log2(e); +inf where the query has no valid key
  float* dsum;   // [H][n][np]  -D, D = rowsum(dO * O) (stored negated: it enters as -D)
  void* da;      // [n][n][H][32] dtype: dA = dO * sigmoid(G), laid out like dO
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
template <typename T>
hipError_t launch_bwd(const Geom& g, int node, const Prep& p, const BwdWs& w, const T* q,
                      const T* k, const T* v, const T* gate, const T* out, const float* lse,
                      const T* dout, T* dq, T* dk, T* dv, T* dg, T* dbias, hipStream_t s);

// ---- fused layer-norm + linear projection (lnl.hip) ---------------------------------
constexpr int LNL_K = 128;       // features per row (the pair channel width)
constexpr int LNL_MAX_OUT = 8;   // output tensors o2's columns are split into

struct LnlArgs {
  int64_t m;                     // rows
  int ncols;                     // output columns N (sum of the outputs' widths)
  int np;                        // N rounded up to a multiple of 32
  int n_out;                     // output tensors
  int start[LNL_MAX_OUT + 1];    // first column of each output; start[n_out] = N
  float eps;
  const bf16 *x, *gamma, *beta;  // x [m][K], gamma and beta [K]
  const bf16* wt;                // W^T [np][K] (prepared in the workspace)
  bf16* out[LNL_MAX_OUT];        // output i: [m][start[i + 1] - start[i]]
  float *mean, *rstd;            // [m], saved for the backward
};

hipError_t launch_lnl_fwd(const LnlArgs& a, bf16* wt, const bf16* w, hipStream_t s);

}  // namespace triattn
