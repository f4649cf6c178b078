// Fused transition layer (MegaFold Section IV: fused layer-norm & linear
// projection, fused SwiGLU and the fused transition layer built from them;
// forward and backward in the appendix listing of the transition layer).
// Per row x of the pair representation (C = 128 features):
//   o1 = (x - mean) rstd * gamma + beta
//   [a | b] = o1 W1              W1 [C][2F]
//   u = a sigmoid(a) b           (SwiGLU)
//   out = u W2                   W2 [F][C]
//
// Differences from the paper's design (separate layer-norm-linear, SwiGLU
// and matmul kernels with o1 and o2 written to memory, atomics for the
// weight gradients), for gfx950:
//  - the forward is ONE kernel: a wave keeps its 32 rows' normalised
//    features and its output accumulators in registers and walks the hidden
//    width in chunks of 32 columns; [a | b] and u of a chunk never leave the
//    registers (u goes straight from the accumulators into the B operand of
//    the W2 product);
//  - the backward recomputes [a | b] instead of reading it back (the matrix
//    cores have room, HBM does not): one kernel computes dx (du, the
//    recomputed a and b, dh = [da | db], do1 = dh W1^T, the layer-norm
//    backward), a second one the sums over rows per column group of the
//    hidden width (G = xhat^T dh, s = column sums of dh, dW2 = u^T dout),
//    each into its own partial-sum block, reduced in a fixed order:
//    dW1 = gamma G + beta s^T, dgamma = sum_n W1 o G, dbeta = W1 s
//    (o1 = xhat gamma + beta regrouped), bitwise reproducible;
//  - products are formed transposed where that keeps a lane on one row
//    (out^T = W2^T u^T, do1^T = W1 dh^T), so the elementwise steps stay in
//    the lane that holds the row.
//
// Weights reach the kernels through per-chunk images that a small packing
// kernel writes into the workspace in LDS order (bank-permuted rows, the
// contraction slots of the accumulator-fed operands already in accumulator
// order); a workgroup streams them into a two-slot LDS ring.
#include <algorithm>

#include "dma.h"
#include "kernels.h"
#include "timing.h"

namespace triattn {

namespace {

constexpr int TRN_WAVES = 8;
constexpr int TRN_THREADS = 64 * TRN_WAVES;
constexpr int TRN_NT = TRN_C / 16;  // MFMA steps over the features
constexpr int TRN_ROWS = 32 * TRN_WAVES;  // rows per workgroup block

// image layout of one chunk j (hidden columns fb = 32 j .. fb + 31):
//   forward : A1a [0, 8K)  A1b [8K, 16K)  A2 [16K, 24K)
//   backward: A1a [0, 8K)  A1b [8K, 16K)  A3 [16K, 24K)  A4 [24K, 40K)
// A1a / A1b: W1^T rows fb + r (a) / F + fb + r (b), 16 chunks of 8 features.
// A2: W2^T for output tile t, row r = output column 32 t + r, 4 chunks
//     (k-step s, half g) of hidden columns in accumulator order.
// A3: W2 rows fb + r, 16 chunks of 8 output columns.
// A4: W1 for feature tile t, row r = feature 32 t + r, 8 chunks (k-step
//     s = 0..3, half g): s < 2 the a columns, s >= 2 the b columns of the
//     chunk, in accumulator order.
constexpr int OFF_A1B = 8192, OFF_A2 = 16384, OFF_A3 = 16384, OFF_A4 = 24576;

// 256-byte rows: chunk c of row r at slot c ^ (r % 16).
__device__ inline uint32_t w256_off(int r, int c) { return r * 256 + 16 * (c ^ (r & 15)); }
// A2 tile rows of 64 bytes.
__device__ inline uint32_t a2_off(int t, int r, int c) {
  return t * 2048 + r * 64 + 16 * (c ^ ((r >> 2) & 3));
}
// A4 tile rows of 128 bytes.
__device__ inline uint32_t a4_off(int t, int r, int c) {
  return t * 4096 + r * 128 + 16 * (c ^ ((r >> 1) & 7));
}
// Accumulator order of a 16-wide contraction step s: slot e of half g holds
// index 16 s + 8 (e / 4) + 4 g + e % 4 (the rows a 32x32 accumulator gives
// a lane in its registers 8 s .. 8 s + 7).
__device__ inline int acc_k(int s, int g, int e) { return 16 * s + 8 * (e >> 2) + 4 * g + (e & 3); }

__device__ inline float sigm(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

__device__ inline f32x4 mma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---- weight images -------------------------------------------------------------------

// One thread per 16-byte slot of the images of all chunks.
__global__ __launch_bounds__(256) void trn_pack_kernel(const bf16* w1, const bf16* w2, int f,
                                                       int bwd, char* img) {
  const int img_bytes = bwd ? TRN_BWD_IMG : TRN_FWD_IMG;
  const int per = img_bytes / 16;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)(f / TRN_FC) * per) return;
  const int j = (int)(idx / per), q = (int)(idx % per), fb = TRN_FC * j;
  const int n1 = 2 * f;  // W1 row length
  bf16x8 v;
  if (q < 1024) {  // A1a, A1b
    const int r = (q & 511) >> 4, c = (q & 15) ^ (r & 15);
    const int col = (q < 512 ? 0 : f) + fb + r;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = w1[(int64_t)(8 * c + e) * n1 + col];
  } else if (!bwd) {  // A2
    const int q2 = q - 1024, t = q2 >> 7, r = (q2 & 127) >> 2, c = (q2 & 3) ^ ((r >> 2) & 3);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = w2[(int64_t)(fb + acc_k(c >> 1, c & 1, e)) * TRN_C + 32 * t + r];
  } else if (q < 1536) {  // A3
    const int q3 = q - 1024, r = q3 >> 4, c = (q3 & 15) ^ (r & 15);
    v = *(const bf16x8*)(w2 + (int64_t)(fb + r) * TRN_C + 8 * c);
  } else {  // A4
    const int q4 = q - 1536, t = q4 >> 8, r = (q4 & 255) >> 3, c = (q4 & 7) ^ ((r >> 1) & 7);
    const int s = c >> 1, g = c & 1;
    const int base = (s < 2 ? 0 : f) + fb;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = w1[(int64_t)(32 * t + r) * n1 + base + acc_k(s & 1, g, e)];
  }
  // write the slot where the reader expects it (the index already is the slot)
  *(bf16x8*)(img + (int64_t)j * img_bytes + 16 * q) = v;
}

// Stream chunk images through a two-slot LDS ring: each thread copies
// N 16-byte pieces.
template <int N>
struct Stage {
  f32x4 v[N];
  __device__ inline void load(const char* src, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = *(const f32x4*)(src + 16 * (tid + i * TRN_THREADS));
  }
  __device__ inline void store(char* dst, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) *(f32x4*)(dst + 16 * (tid + i * TRN_THREADS)) = v[i];
  }
};

// Row statistics and o1 (bf16, the B operand over the features) of a lane's
// row: half g holds features 16 t + 8 g .. + 7.
__device__ inline void ln_row(const bf16x8 (&xr)[TRN_NT], const float (&gb)[2][TRN_C], int g,
                              float eps, float& mean, float& rstd, bf16x8 (&of)[TRN_NT]) {
  float xv[TRN_NT][8];
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xv[t][e] = (float)xr[t][e];
      s += xv[t][e];
    }
  mean = wave_xor32_sum(s) * (1.f / TRN_C);
  float v = 0.f;
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xv[t][e] -= mean;
      v = fmaf(xv[t][e], xv[t][e], v);
    }
  rstd = 1.f / sqrtf(wave_xor32_sum(v) * (1.f / TRN_C) + eps);
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 16 * t + 8 * g + e;
      of[t][e] = (bf16)fmaf(xv[t][e] * rstd, gb[0][k], gb[1][k]);
    }
}

// o1 from saved statistics.
__device__ inline void ln_row_saved(const bf16x8 (&xr)[TRN_NT], const float (&gb)[2][TRN_C], int g,
                                    float mean, float rstd, bf16x8 (&of)[TRN_NT]) {
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 16 * t + 8 * g + e;
      of[t][e] = (bf16)fmaf(((float)xr[t][e] - mean) * rstd, gb[0][k], gb[1][k]);
    }
}

__device__ inline void load_row(const bf16* base, int64_t row, int64_t m, int g,
                                bf16x8 (&xr)[TRN_NT]) {
  const bf16* p = base + (row < m ? row : m - 1) * TRN_C + 8 * g;
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t) xr[t] = *(const bf16x8*)(p + 16 * t);
}

// h^T tile of the chunk in `img` (a or b half): rows = hidden columns,
// lanes = rows of x.
__device__ inline f32x16 h_tile(const char* img, const uint32_t (&a1)[TRN_NT],
                                const bf16x8 (&of)[TRN_NT]) {
  f32x16 acc = {};
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t) acc = Mma<bf16>::mma(*(const bf16x8*)(img + a1[t]), of[t], acc);
  return acc;
}

// Store a lane's 4 x 16 accumulated values (feature 32 t + 8 j + 4 g + i)
// of its row as bf16, 8 bytes per run.
__device__ inline void store_row(bf16* base, int64_t row, int g, const f32x16 (&acc)[4]) {
  bf16* p = base + row * TRN_C + 4 * g;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *(bf16x4*)(p + 32 * t + 8 * j) =
          bf16x4{(bf16)acc[t][4 * j], (bf16)acc[t][4 * j + 1], (bf16)acc[t][4 * j + 2],
                 (bf16)acc[t][4 * j + 3]};
}

// ---- forward -------------------------------------------------------------------------
//
// Persistent workgroups of 8 waves (one per CU); a workgroup takes blocks of
// 256 rows (32 per wave) and, per block, streams the F / 32 chunk images,
// two chunks per ring slot (one barrier per 64 hidden columns).

constexpr int FWD_CPS = 2;  // chunk images per ring slot

__global__ __launch_bounds__(TRN_THREADS, 1) void trn_fwd_kernel(TrnFwdArgs a) {
  __shared__ __align__(16) char ring[2][FWD_CPS * TRN_FWD_IMG];
  __shared__ __align__(16) float gb[2][TRN_C];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6;
  const int64_t nblk = (a.m + TRN_ROWS - 1) / TRN_ROWS;
  if ((int64_t)blockIdx.x >= nblk) return;  // whole workgroup, before any barrier
  const int nst = a.f / TRN_FC / FWD_CPS;  // ring stages per block (F is a multiple of 128)
  const int64_t nsteps = (nblk - blockIdx.x + gridDim.x - 1) / gridDim.x * nst;
  constexpr int PER = FWD_CPS * TRN_FWD_IMG / 16 / TRN_THREADS;
  Stage<PER> st;
  st.load(a.img, tid);
  if (tid < TRN_C) {
    gb[0][tid] = (float)a.gamma[tid];
    gb[1][tid] = (float)a.beta[tid];
  }
  st.store(ring[0], tid);
  __syncthreads();

  uint32_t a1[TRN_NT], a2[4][2];
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t) a1[t] = w256_off(l32, 2 * t + g);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int s = 0; s < 2; ++s) a2[t][s] = OFF_A2 + a2_off(t, l32, 2 * s + g);

  int64_t step = 0;
  for (int64_t blk = blockIdx.x; blk < nblk; blk += gridDim.x) {
    const int64_t row = blk * TRN_ROWS + wave * 32 + l32;
    bf16x8 xr[TRN_NT], of[TRN_NT];
    load_row(a.x, row, a.m, g, xr);
    float mean, rstd;
    ln_row(xr, gb, g, a.eps, mean, rstd, of);
    if (row < a.m && g == 0) {
      a.mean[row] = mean;
      a.rstd[row] = rstd;
    }
    f32x16 acc[4] = {};
    for (int j = 0; j < nst; ++j, ++step) {
      const char* slot = ring[step & 1];
      const bool more = step + 1 < nsteps;
      if (more)
        st.load(a.img + (int64_t)(j + 1 == nst ? 0 : j + 1) * FWD_CPS * TRN_FWD_IMG, tid);
#pragma unroll
      for (int c = 0; c < FWD_CPS; ++c) {
        const char* cur = slot + c * TRN_FWD_IMG;
        const f32x16 ha = h_tile(cur, a1, of);
        const f32x16 hb = h_tile(cur + OFF_A1B, a1, of);
        bf16x8 uf[2];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float x = ha[v];
          uf[v >> 3][v & 7] = (bf16)(x * sigm(x) * hb[v]);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int s = 0; s < 2; ++s)
            acc[t] = Mma<bf16>::mma(*(const bf16x8*)(cur + a2[t][s]), uf[s], acc[t]);
      }
      if (more) st.store(ring[(step + 1) & 1], tid);
      __syncthreads();
    }
    if (row < a.m) store_row(a.out, row, g, acc);
  }
}

// ---- backward: dx ----------------------------------------------------------------------

__global__ __launch_bounds__(TRN_THREADS, 1) void trn_bwd_dx_kernel(TrnBwdArgs a) {
  __shared__ __align__(16) char ring[2][TRN_BWD_IMG];
  __shared__ __align__(16) float gb[2][TRN_C];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6;
  const int64_t nblk = (a.m + TRN_ROWS - 1) / TRN_ROWS;
  if ((int64_t)blockIdx.x >= nblk) return;
  const int nch = a.f / TRN_FC;
  const int64_t nsteps = (nblk - blockIdx.x + gridDim.x - 1) / gridDim.x * nch;
  constexpr int PER = TRN_BWD_IMG / 16 / TRN_THREADS;
  Stage<PER> st;
  st.load(a.img, tid);
  if (tid < TRN_C) {
    gb[0][tid] = (float)a.gamma[tid];
    gb[1][tid] = (float)a.beta[tid];
  }
  st.store(ring[0], tid);
  __syncthreads();

  uint32_t a1[TRN_NT], a4[4][4];
#pragma unroll
  for (int t = 0; t < TRN_NT; ++t) a1[t] = w256_off(l32, 2 * t + g);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int s = 0; s < 4; ++s) a4[t][s] = OFF_A4 + a4_off(t, l32, 2 * s + g);

  int64_t step = 0;
  for (int64_t blk = blockIdx.x; blk < nblk; blk += gridDim.x) {
    const int64_t row = blk * TRN_ROWS + wave * 32 + l32;
    const int64_t rc = row < a.m ? row : a.m - 1;
    bf16x8 xr[TRN_NT], of[TRN_NT], df[TRN_NT];
    load_row(a.x, row, a.m, g, xr);
    load_row(a.dout, row, a.m, g, df);
    const float mean = a.mean[rc], rstd = a.rstd[rc];
    ln_row_saved(xr, gb, g, mean, rstd, of);
    f32x16 d1[4] = {};  // do1^T: feature 32 t + acc row, lane <-> row
    for (int j = 0; j < nch; ++j, ++step) {
      const char* cur = ring[step & 1];
      const bool more = step + 1 < nsteps;
      if (more) st.load(a.img + (int64_t)(j + 1 == nch ? 0 : j + 1) * TRN_BWD_IMG, tid);
      const f32x16 ha = h_tile(cur, a1, of);
      const f32x16 hb = h_tile(cur + OFF_A1B, a1, of);
      const f32x16 du = h_tile(cur + OFF_A3, a1, df);  // du^T = W2 rows . dout^T
      bf16x8 dh[4];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float x = ha[v], sg = sigm(x), silu = x * sg;
        dh[v >> 3][v & 7] = (bf16)(du[v] * hb[v] * sg * (1.f + x * (1.f - sg)));
        dh[2 + (v >> 3)][v & 7] = (bf16)(du[v] * silu);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          d1[t] = Mma<bf16>::mma(*(const bf16x8*)(cur + a4[t][s]), dh[s], d1[t]);
      if (more) st.store(ring[(step + 1) & 1], tid);
      __syncthreads();
    }
    // layer-norm backward: wdy = do1 gamma, dx = rstd (wdy - c1 xhat - c2)
    float xh[4][16], wdy[4][16];
    float c1 = 0.f, c2 = 0.f;
    const bf16* xp = a.x + rc * TRN_C + 4 * g;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x4 xv = *(const bf16x4*)(xp + 32 * t + 8 * j);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = 32 * t + 8 * j + 4 * g + i, v = 4 * j + i;
          xh[t][v] = ((float)xv[i] - mean) * rstd;
          wdy[t][v] = d1[t][v] * gb[0][k];
          c1 = fmaf(xh[t][v], wdy[t][v], c1);
          c2 += wdy[t][v];
        }
      }
    c1 = wave_xor32_sum(c1) * (1.f / TRN_C);
    c2 = wave_xor32_sum(c2) * (1.f / TRN_C);
    f32x16 dx[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) dx[t][v] = (wdy[t][v] - c1 * xh[t][v] - c2) * rstd;
    if (row < a.m) store_row(a.dx, row, g, dx);
  }
}

// ---- backward: sums over rows ----------------------------------------------------------
//
// Workgroup (part p, column group cg): rows of part p, hidden columns
// cg * 128 .. + 127.  Wave w owns hidden columns f0 = cg * 128 + 16 w .. + 15
// and keeps W1's a and b columns and W2's rows for them in LDS (fragment
// order).  Per block of 32 rows (o1, xhat and dout staged in LDS by all
// threads, shared by the waves):
//   hC  [32 rows x 32 cols]  = o1 . W1[:, a cols | b cols]      (lane <-> column)
//   duC [32 rows x 32 cols]  = dout . W2^T[:, f cols, twice]     (both halves)
//   the a lane and the b lane of a column swap values, so each has a, b, du:
//   dh = da (a lanes) or db (b lanes), u = a sigmoid(a) b
//   G  [128 features x 32 cols] += xhat^T dh,  s += column sums of dh
//   dW2 [16 f x 128 out] += u^T dout       (16x16x32 MFMAs)
// The x and dout tiles are stored as four 32-column blocks of 64-byte rows
// (blk_off), so their transposed reads are the attention kernels' ones.

// One ring slot: o1 (bf16), xhat (bf16), dout and the low part of o1
// (o1 - bf16(o1), rounded to bf16) tiles of 32 rows, each as four 32-column
// blocks of 64-byte rows (blk_off).  The staging threads normalise once per
// block for all waves.  a and b are recomputed from o1 as the pair hi + lo:
// rounding o1 to one bf16 moves a and b by up to 2^-9 of the l2 norm of
// their terms, which is large against a or b where the terms cancel, and a
// sum over a few rows does not average that out.
// Blocks sit W_BLK bytes apart (2 KB + 64): the staging stores of one wave
// touch the four blocks of a row at once, and the extra 64 bytes put them on
// different banks.  Every read stays inside one block.
constexpr int W_BLK = 2048 + 64;
constexpr int W_TILE = 4 * W_BLK;
constexpr int W_SLOT = 4 * W_TILE;
constexpr int W_XH = W_TILE, W_DO = 2 * W_TILE, W_OL = 3 * W_TILE;

__global__ __launch_bounds__(TRN_THREADS, 1) void trn_bwd_w_kernel(TrnBwdArgs a, int64_t rpp) {
  __shared__ __align__(16) char ring[2][W_SLOT];
  __shared__ __align__(16) float gb[2][TRN_C];
  // each wave's B operands W2[fl][k], fragment-major (the W2 fragments of
  // lanes 16..31 of each half repeat lanes 0..15); those of W1 stay in
  // registers
  __shared__ __align__(16) bf16x8 wf2[TRN_WAVES][TRN_NT][32];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6, q = lane >> 4;
  const int f = a.f, p = blockIdx.x, cg = blockIdx.y;
  const int f0 = cg * TRN_GROUP + 16 * wave;
  const bool is_a = l32 < 16;
  const int hcol = (is_a ? 0 : f) + f0 + (l32 & 15);  // this lane's column of W1 / dW1
  const int fl = f0 + (l32 & 15);                     // its hidden column
  const int64_t r0 = (int64_t)p * rpp, r1 = r0 + rpp < a.m ? r0 + rpp : a.m;
  const int nb = r1 > r0 ? (int)((r1 - r0 + 31) / 32) : 0;

  if (tid < TRN_C) {
    gb[0][tid] = (float)a.gamma[tid];
    gb[1][tid] = (float)a.beta[tid];
  }
  // the wave's B operands W1[k][hcol] (registers) and W2[fl][k] (LDS),
  // k = 16 s + 8 g + e, kept for the whole launch
  bf16x8 w1r[TRN_NT];
#pragma unroll
  for (int s = 0; s < TRN_NT; ++s) {
#pragma unroll
    for (int e = 0; e < 8; ++e) w1r[s][e] = a.w1[(int64_t)(16 * s + 8 * g + e) * 2 * f + hcol];
    if (is_a) wf2[wave][s][16 * g + l32] = *(const bf16x8*)(a.w2 + (int64_t)fl * TRN_C + 16 * s + 8 * g);
  }
  __syncthreads();  // gamma, beta

  // staging: thread tid takes 8 features (chunk tid % 16) of row tid / 16:
  // x, dout and the row's statistics; it writes o1 and xhat in bf16 and dout
  const int sr = tid >> 4, sc = tid & 15;
  const uint32_t soff = (sc >> 2) * W_BLK + blk_off(sr, sc & 3);
  struct Staged {
    bf16x8 x, d;
    float mean, rstd;
  };
  auto stage_load = [&](int ib, Staged& v) {
    const int64_t row = r0 + 32 * (int64_t)ib + sr;
    const bool ok = row < r1;
    const int64_t rc = ok ? row : r0;
    v.x = *(const bf16x8*)(a.x + rc * TRN_C + 8 * sc);
    v.d = ok ? *(const bf16x8*)(a.dout + rc * TRN_C + 8 * sc) : bf16x8{};  // no contribution
    v.mean = a.mean[rc];
    v.rstd = a.rstd[rc];
  };
  auto stage_store = [&](char* slot, const Staged& v) {
    bf16x8 o1, ol, xh;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float h = ((float)v.x[e] - v.mean) * v.rstd;
      xh[e] = (bf16)h;
      const float o = fmaf(h, gb[0][8 * sc + e], gb[1][8 * sc + e]);
      o1[e] = (bf16)o;
      ol[e] = (bf16)(o - (float)o1[e]);
    }
    *(bf16x8*)(slot + soff) = o1;
    *(bf16x8*)(slot + W_XH + soff) = xh;
    *(bf16x8*)(slot + W_DO + soff) = v.d;
    *(bf16x8*)(slot + W_OL + soff) = ol;
  };
  Staged sv;
  if (nb > 0) {
    stage_load(0, sv);
    stage_store(ring[0], sv);
  }
  __syncthreads();

  f32x16 G[4] = {};
  f32x4 W2a[8] = {};
  float ssum = 0.f;
  const TrAddr tr(lane);
  // dout transposed reads for the 16x16x32 B operand: lane group q takes rows
  // 16 (q % 2) + 4 (q / 2) + {0..3} and + 8 + {0..3}; supplying lane 4 e + j
  // of the group addresses row +e, columns 4 j .. + 3 of the 16-column tile
  const int qi = lane & 15, qe = qi >> 2, qj = qi & 3;
  // the odd groups read their second quad of rows first: rows r and r + 16
  // share banks, rows r + 24 and r do not (blk_off's permutation), so the two
  // groups of each half-wave never read the same banks together
  const int qrow = 16 * (q & 1) + 4 * (q >> 1) + qe;
  const int qfirst = qrow + 8 * (q & 1), qsecond = qrow + 8 * (1 - (q & 1));
  for (int ib = 0; ib < nb; ++ib) {
    const char* cur = ring[ib & 1];
    const bool more = ib + 1 < nb;
    if (more) stage_load(ib + 1, sv);
    // o1 and dout as A operands (lane <-> row l32, features 16 s + 8 g ..)
    f32x16 hC = {}, duC = {};
#pragma unroll
    for (int s = 0; s < TRN_NT; ++s) {
      const uint32_t o = (s >> 1) * W_BLK + blk_off(l32, 2 * (s & 1) + g);
      hC = Mma<bf16>::mma(*(const bf16x8*)(cur + o), w1r[s], hC);
      hC = Mma<bf16>::mma(*(const bf16x8*)(cur + W_OL + o), w1r[s], hC);
      duC = Mma<bf16>::mma(*(const bf16x8*)(cur + W_DO + o), wf2[wave][s][16 * g + (l32 & 15)],
                           duC);
    }
    // a and b of the same hidden column sit in lanes l and l ^ 16 (rows of
    // 16 lanes: a in the even rows, b in the odd ones).  v_permlane16_swap
    // of h with itself leaves the even-row value (a) in its first result and
    // the odd-row value (b) in its second, in every lane.  Both lanes then
    // compute u; the a lane keeps da, the b lane db (selects, no branches).
    f32x16 dh, u;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(hC[v]),
                                                      __float_as_uint(hC[v]), false, false);
      const float av = __uint_as_float(r[0]), bv = __uint_as_float(r[1]);
      const float sg = sigm(av), silu = av * sg;
      const float fa = bv * fmaf(silu, 1.f - sg, sg);  // b sigmoid(a) (1 + a (1 - sigmoid(a)))
      dh[v] = duC[v] * (is_a ? fa : silu);
      u[v] = silu * bv;
      ssum += dh[v];
    }
    // G += xhat^T dh: A = xhat^T (lane <-> feature 32 t + l32, rows in
    // accumulator order), B = dh from the registers as the pair hi + lo of
    // bf16 numbers (with both xhat and dh rounded once, a sum over a few rows
    // whose dh columns differ in size sits near the bf16 bound)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bf16x8 bf, bl;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf[e] = (bf16)dh[8 * s + e];
        bl[e] = (bf16)(dh[8 * s + e] - (float)bf[e]);
      }
#pragma unroll
      for (int t = 0; t < 4; t += 2) {
        const uint32_t b0 = lds_addr(cur + W_XH + t * W_BLK), b1 = b0 + W_BLK;
        s16x4 rr[4];
        tr_read4_wait(b0 + tr.off(16 * s), b0 + tr.off(16 * s + 8), b1 + tr.off(16 * s),
                      b1 + tr.off(16 * s + 8), rr);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          G[t + h] = Mma<bf16>::mma(tr_frag(rr, h), bf, G[t + h]);
          G[t + h] = Mma<bf16>::mma(tr_frag(rr, h), bl, G[t + h]);
        }
      }
    }
    // dW2 += u^T dout: A = u (lane <-> hidden column; group q takes the rows
    // of registers 8 (q % 2) .. + 7, the odd groups their upper quad first),
    // B = dout^T reads of the same rows in the same order
    bf16x8 ua;
#pragma unroll
    for (int e = 0; e < 8; ++e) ua[e] = (bf16)((q & 1) ? u[e < 4 ? 12 + e : 4 + e] : u[e]);
#pragma unroll
    for (int ot = 0; ot < 8; ot += 2) {
      // tiles ot and ot + 1 are the two 16-column halves of one 32-column block
      const uint32_t tb = lds_addr(cur + W_DO + (ot >> 1) * W_BLK);
      const int half = 8 * (qj & 1);
      const uint32_t c0 = 2 * 0 + (qj >> 1), c1 = 2 * 1 + (qj >> 1);
      s16x4 rr[4];
      tr_read4_wait(tb + blk_off(qfirst, c0) + half, tb + blk_off(qsecond, c0) + half,
                    tb + blk_off(qfirst, c1) + half, tb + blk_off(qsecond, c1) + half, rr);
      W2a[ot] = mma16(ua, tr_frag(rr, 0), W2a[ot]);
      W2a[ot + 1] = mma16(ua, tr_frag(rr, 1), W2a[ot + 1]);
    }
    if (more) stage_store(ring[(ib + 1) & 1], sv);
    __syncthreads();
  }

  // partial sums of part p: G [C][2F], s [2F], dW2 [F][C]
  float* out = a.part + (int64_t)p * trn_part_floats(f);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v)
      out[(int64_t)(32 * t + acc_row(v, g)) * 2 * f + hcol] = G[t][v];
  ssum += __shfl_xor(ssum, 32);
  if (g == 0) out[(int64_t)TRN_C * 2 * f + hcol] = ssum;
  float* w2o = out + (int64_t)TRN_C * 2 * f + 2 * f;
  // 16x16 accumulator: lane l holds column l % 16 of output tile ot and
  // hidden rows 4 (l / 16) + i of the wave's 16
#pragma unroll
  for (int ot = 0; ot < 8; ++ot)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w2o[(int64_t)(f0 + 4 * q + i) * TRN_C + 16 * ot + qi] = W2a[ot][i];
}

// Fixed-order sum of the partial blocks: G and s into gsum, dW2 into its output.
__global__ __launch_bounds__(256) void trn_reduce_kernel(TrnBwdArgs a) {
  const int64_t per = trn_part_floats(a.f);
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= per) return;
  float s = 0.f;
  for (int p = 0; p < a.nparts; ++p) s += a.part[(int64_t)p * per + i];
  const int64_t ng = (int64_t)TRN_C * 2 * a.f + 2 * a.f;
  if (i < ng)
    a.gsum[i] = s;
  else
    a.dw2[i - ng] = s;
}

// dW1 = gamma G + beta s^T, dgamma = sum_n W1 o G, dbeta = W1 s; one
// workgroup per feature, fixed-order tree over the columns.
__global__ __launch_bounds__(256) void trn_finish_kernel(TrnBwdArgs a) {
  __shared__ float red[2][256];
  const int k = blockIdx.x, tid = threadIdx.x, n = 2 * a.f;
  const float gm = (float)a.gamma[k], bt = (float)a.beta[k];
  const float* G = a.gsum + (int64_t)k * n;
  const float* s = a.gsum + (int64_t)TRN_C * n;
  float dg = 0.f, db = 0.f;
  for (int c = tid; c < n; c += 256) {
    const float w = (float)a.w1[(int64_t)k * n + c];
    a.dw1[(int64_t)k * n + c] = gm * G[c] + bt * s[c];
    dg = fmaf(w, G[c], dg);
    db = fmaf(w, s[c], db);
  }
  red[0][tid] = dg;
  red[1][tid] = db;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) {
      red[0][tid] += red[0][tid + w];
      red[1][tid] += red[1][tid + w];
    }
    __syncthreads();
  }
  if (tid == 0) {
    a.dgamma[k] = red[0][0];
    a.dbeta[k] = red[1][0];
  }
}

constexpr int TRN_GRID = 256;  // persistent workgroups (one per CU)

}  // namespace

int trn_bwd_parts(int64_t m, int f) {
  const int groups = f / TRN_GROUP;
  int p = TRN_GRID / groups;
  if (p < 1) p = 1;
  const int64_t blocks = (m + 31) / 32;
  if (p > blocks) p = (int)blocks;
  return p;
}

hipError_t launch_trn_fwd(const TrnFwdArgs& a, hipStream_t s) {
  const int64_t slots = (int64_t)(a.f / TRN_FC) * (TRN_FWD_IMG / 16);
  {
    KernelTimer t(K_TRN_PACK, s);
    hipLaunchKernelGGL(trn_pack_kernel, dim3((unsigned)((slots + 255) / 256)), dim3(256), 0, s,
                       a.w1, a.w2, a.f, 0, a.img);
  }
  const int64_t nblk = (a.m + TRN_ROWS - 1) / TRN_ROWS;
  {
    KernelTimer t(K_TRN_FWD, s);
    hipLaunchKernelGGL(trn_fwd_kernel, dim3((unsigned)std::min<int64_t>(nblk, TRN_GRID)),
                       dim3(TRN_THREADS), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_trn_bwd(const TrnBwdArgs& a, hipStream_t s) {
  const int64_t slots = (int64_t)(a.f / TRN_FC) * (TRN_BWD_IMG / 16);
  {
    KernelTimer t(K_TRN_PACK, s);
    hipLaunchKernelGGL(trn_pack_kernel, dim3((unsigned)((slots + 255) / 256)), dim3(256), 0, s,
                       a.w1, a.w2, a.f, 1, a.img);
  }
  const int64_t nblk = (a.m + TRN_ROWS - 1) / TRN_ROWS;
  {
    KernelTimer t(K_TRN_BWD_DX, s);
    hipLaunchKernelGGL(trn_bwd_dx_kernel, dim3((unsigned)std::min<int64_t>(nblk, TRN_GRID)),
                       dim3(TRN_THREADS), 0, s, a);
  }
  {
    // rows per part: a multiple of 32
    const int64_t blocks = (a.m + 31) / 32;
    const int64_t rpp = (blocks + a.nparts - 1) / a.nparts * 32;
    KernelTimer t(K_TRN_BWD_W, s);
    hipLaunchKernelGGL(trn_bwd_w_kernel, dim3((unsigned)a.nparts, (unsigned)(a.f / TRN_GROUP)),
                       dim3(TRN_THREADS), 0, s, a, rpp);
  }
  {
    const int64_t per = trn_part_floats(a.f);
    KernelTimer t(K_TRN_REDUCE, s);
    hipLaunchKernelGGL(trn_reduce_kernel, dim3((unsigned)((per + 255) / 256)), dim3(256), 0, s,
                       a);
  }
  {
    KernelTimer t(K_TRN_FINISH, s);
    hipLaunchKernelGGL(trn_finish_kernel, dim3(TRN_C), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace triattn
