// Fused layer-norm + linear projection (MegaFold Section IV, "fused
// layer-norm & linear projection"; forward and backward formulas in the
// appendix table of fused operators), the step that turns the pair
// representation into the triangle-attention inputs:
//   o1 = (x - mean) rstd * gamma + beta   per row of x [M][K],
//   o2 = o1 W                             (W [K][N], no bias),
// with o2's columns written into n_out separate row-major tensors (for the
// attention: Q, K, V, G and the bias logits), so no split copy follows.
//
// Differences from the paper's two-kernel Triton design, for gfx950:
//  - K = 128 (the pair channel width) fits one wave's registers, so the row
//    statistics are computed inside the projection kernel (no separate
//    mean/var pass): a lane holds half a row, two passes over registers give
//    mean and the biased variance, and the normalised row goes straight into
//    the MFMA operand registers in bf16;
//  - the product is formed transposed, o2^T = W^T o1^T (lane <-> row), so
//    each lane stores runs of four consecutive output columns of its row;
//  - the backward's sums over rows (dW, dgamma, dbeta) go to per-block
//    partial sums reduced in a fixed order instead of atomics.
#include <algorithm>

#include "dma.h"
#include "kernels.h"
#include "timing.h"

namespace triattn {

// ---- forward --------------------------------------------------------------------------
//
// Persistent workgroups of LNF_WAVES waves, one per CU.  W^T of the
// workgroup's column group stays in LDS for the whole launch (read once per
// workgroup); each wave walks 32-row units u = its global wave index + i *
// (waves in the grid), prefetching the next unit's rows while the current
// one is computed.
//
// LDS W^T: row n (an output column) is 256 bytes = 16 chunks of 8 features;
// chunk c of row n sits at chunk slot c ^ (n % 16), so the A-fragment read
// (32 consecutive rows, one chunk each) hits 8 distinct 16-byte bank groups
// in every aligned run of 8 lanes.
//
// Output tiles (32 rows x 32 columns) pass through a 2 KB LDS tile per wave
// so that each store instruction writes 16 rows x 64 contiguous bytes.
// Tiles that lie inside one output (all but a narrow output such as the
// bias logits) are stored with buffer stores whose range check drops the
// rows past m, so their epilogue has no branches and the compiler can
// interleave it with the next tile's MFMAs.

constexpr int LNF_WAVES = 8;
constexpr int LNF_NT = LNL_K / 16;  // MFMA contraction steps over the features
constexpr int LNF_TILES = LNL_GROUP / 32;

// Output address of a run of 4 columns: p + row * w.  v8: the run and the
// next 4 columns are one 16-byte aligned run of the same output.
typedef __attribute__((address_space(1))) bf16 gbf16;  // global memory (not flat)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 gu32x4;
typedef __attribute__((address_space(1))) u32x2 gu32x2;
struct LnlQuad {
  gbf16* p;
  int w;
  int v8;
};

__device__ inline uint32_t lnf_wt_off(int n, int c) { return n * 256 + 16 * (c ^ (n & 15)); }

// Byte offset of 16-byte chunk c (columns 8 c .. 8 c + 7) of row r of a
// staged 32 x 32 bf16 tile (64-byte rows, chunks permuted by row pairs).
__device__ inline uint32_t lnf_stage_off(int r, int c) { return r * 64 + 16 * (c ^ ((r >> 1) & 3)); }

// One wave's 32 rows (lane <-> row m, half g holds features 16 t + 8 g .. + 7).
// Rows past the end read the last row (their results are never stored), so
// the loads are unconditional and the compiler can count them in its waits.
__device__ inline void lnf_load_rows(const LnlArgs& a, int64_t m, int g, bf16x8 (&xr)[LNF_NT]) {
  const bf16* p = a.x + (m < a.m ? m : a.m - 1) * LNL_K + 8 * g;
#pragma unroll
  for (int t = 0; t < LNF_NT; ++t) xr[t] = *(const bf16x8*)(p + 16 * t);
}

__device__ inline void lnf_load_a(bf16x8 (&af)[LNF_NT], const uint32_t (&aoff)[LNF_NT], int nt) {
#pragma unroll
  for (int t = 0; t < LNF_NT; ++t) af[t] = lds_load16<bf16x8>(aoff[t] + nt * 8192);
}

// One 32 x 32 output tile: o2^T[n][m] = sum_k W^T[n][k] o1[m][k].
__device__ inline f32x16 lnf_tile(const bf16x8 (&af)[LNF_NT], const bf16x8 (&of)[LNF_NT]) {
  f32x16 acc = {};
#pragma unroll
  for (int t = 0; t < LNF_NT; ++t) acc = Mma<bf16>::mma(af[t], of[t], acc);
  return acc;
}

// Lane (row l32, half g) holds columns 8 j + 4 g + 0..3 of the tile in
// acc[4 j ..]: write them to the wave's LDS tile, then read back chunk
// lane % 4 of rows lane / 4 and lane / 4 + 16.
__device__ inline void lnf_stage(const f32x16& acc, char* stage, int lane, u32x4 (&v)[2]) {
  const int l32 = lane & 31, g = lane >> 5;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bf16x4 x{(bf16)acc[4 * j], (bf16)acc[4 * j + 1], (bf16)acc[4 * j + 2],
                   (bf16)acc[4 * j + 3]};
    *(bf16x4*)(stage + lnf_stage_off(l32, j) + 8 * g) = x;
  }
#pragma unroll
  for (int rr = 0; rr < 2; ++rr)
    v[rr] = *(const u32x4*)(stage + lnf_stage_off((lane >> 2) + 16 * rr, lane & 3));
}

// Store a tile that lies inside one output (LnlTile::fast).
__device__ inline void lnf_store_fast(const f32x16& acc, char* stage, const LnlTile& tl,
                                      int lane, int64_t m0, int64_t m) {
  u32x4 v[2];
  lnf_stage(acc, stage, lane, v);
  const rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(tl.base, (short)0,
                                                     (int)(uint32_t)(m * tl.w * 2), 0x00020000);
  const uint32_t voff =
      ((uint32_t)(m0 + (lane >> 2)) * (uint32_t)tl.w + (uint32_t)(tl.off + 8 * (lane & 3))) * 2u;
  __builtin_amdgcn_raw_buffer_store_b128(v[0], r, voff, 0, 0);
  __builtin_amdgcn_raw_buffer_store_b128(v[1], r, voff + 32u * (uint32_t)tl.w, 0, 0);
}

// Store any tile: each 16-byte chunk goes out as one 16-byte run or two
// 8-byte runs per the quad table tq (the tile's 8 entries).
__device__ inline void lnf_store_any(const f32x16& acc, char* stage, const LnlQuad* tq, int lane,
                                     int64_t m0, int64_t mrows) {
  u32x4 v[2];
  lnf_stage(acc, stage, lane, v);
  const int c = lane & 3;
  const LnlQuad e0 = tq[2 * c], e1 = tq[2 * c + 1];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    const int64_t row = m0 + (lane >> 2) + 16 * rr;
    if (row >= mrows || e0.p == nullptr) continue;
    if (e0.v8) {
      *(gu32x4*)(e0.p + row * e0.w) = v[rr];
    } else {
      *(gu32x2*)(e0.p + row * e0.w) = u32x2{v[rr][0], v[rr][1]};
      if (e1.p != nullptr) *(gu32x2*)(e1.p + row * e1.w) = u32x2{v[rr][2], v[rr][3]};
    }
  }
}

__global__ __launch_bounds__(64 * LNF_WAVES) void lnl_fwd_kernel(LnlArgs a) {
  __shared__ __align__(16) bf16 wt[LNL_GROUP * LNL_K];  // W^T of the group
  __shared__ __align__(16) LnlQuad quad[LNL_GROUP / 4];
  __shared__ __align__(16) bf16 gb[2][LNL_K];           // gamma, beta
  __shared__ __align__(16) char stage[LNF_WAVES][32 * 64];
  __shared__ int order[LNF_TILES];                        // fast tiles first
  __shared__ int nfast_s;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = tid >> 6;
  const int c0 = blockIdx.y * a.gw;
  const int gn = min(a.gw, a.ncols - c0);  // columns of this group
  const int gnp = (gn + 31) & ~31;
  const int nq = gnp / 4;
  const int ntiles = gnp / 32;

  // W^T of the group (columns past the group are zero): all loads first
  {
    constexpr int NT = 64 * LNF_WAVES;
    constexpr int FILL = (LNL_K * (LNL_GROUP / 4) + NT - 1) / NT;
    bf16x4 wv[FILL];
#pragma unroll
    for (int i = 0; i < FILL; ++i) {
      const int idx = tid + i * NT, k = idx / nq, n = 4 * (idx - k * nq);
      wv[i] = (idx < LNL_K * nq && n < gn) ? *(const bf16x4*)(a.w + (int64_t)k * a.ncols + c0 + n)
                                           : bf16x4{};
    }
#pragma unroll
    for (int i = 0; i < FILL; ++i) {
      const int idx = tid + i * NT, k = idx / nq, n = 4 * (idx - k * nq);
      if (idx < LNL_K * nq) {
        char* base = (char*)wt + 2 * (k & 7);
#pragma unroll
        for (int e = 0; e < 4; ++e) *(bf16*)(base + lnf_wt_off(n + e, k >> 3)) = wv[i][e];
      }
    }
  }
  // output address of every run of 4 columns of the group
  for (int q = tid; q < nq; q += 64 * LNF_WAVES) {
    LnlQuad e{nullptr, 0, 0};
    if (4 * q < gn) {
      const int col = c0 + 4 * q;
      int i = 0;
      while (i + 1 < a.n_out && col >= a.start[i + 1]) ++i;
      const int w = a.start[i + 1] - a.start[i], off = col - a.start[i];
      e.p = (gbf16*)(a.out[i] + off);
      e.w = w;
      e.v8 = (w % 8 == 0 && off % 8 == 0) ? 1 : 0;
    }
    quad[q] = e;
  }
  if (tid < LNL_K) {
    gb[0][tid] = a.gamma[tid];
    gb[1][tid] = a.beta[tid];
  }
  if (tid == 0) {
    int nf = 0;
    for (int nt = 0; nt < ntiles; ++nt)
      if (a.tile[c0 / 32 + nt].fast) order[nf++] = nt;
    int k = nf;
    for (int nt = 0; nt < ntiles; ++nt)
      if (!a.tile[c0 / 32 + nt].fast) order[k++] = nt;
    nfast_s = nf;
  }
  __syncthreads();

  uint32_t aoff[LNF_NT];
#pragma unroll
  for (int t = 0; t < LNF_NT; ++t) aoff[t] = lds_addr(wt) + lnf_wt_off(l32, 2 * t + g);
  char* st = stage[wave];
  const int nfast = nfast_s;
  const bool stats_out = blockIdx.y == 0;
  const int64_t units = (a.m + 31) / 32;
  const int64_t stride = (int64_t)gridDim.x * LNF_WAVES;
  int64_t u = (int64_t)blockIdx.x * LNF_WAVES + wave;
  bf16x8 xr[LNF_NT];
  lnf_load_rows(a, u * 32 + l32, g, xr);
  // tile id (uniform) of position i of the order
  auto tile_at = [&](int i) { return __builtin_amdgcn_readfirstlane(order[i]); };

  for (; u < units; u += stride) {
    // gamma and beta are re-read from LDS per unit rather than held in registers
    asm volatile("" ::: "memory");
    const int64_t m0 = u * 32, m = m0 + l32;
    // row statistics: this lane's 64 features, then the other half (lane ^ 32);
    // two passes over the registers (mean, then the centred sum of squares)
    float xv[LNF_NT][8];
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < LNF_NT; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xv[t][e] = (float)xr[t][e];
        s += xv[t][e];
      }
    const float mean = wave_xor32_sum(s) * (1.f / LNL_K);
    float v = 0.f;
#pragma unroll
    for (int t = 0; t < LNF_NT; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xv[t][e] -= mean;
        v = fmaf(xv[t][e], xv[t][e], v);
      }
    const float var = wave_xor32_sum(v) * (1.f / LNL_K);
    const float rstd = 1.f / sqrtf(var + a.eps);
    if (stats_out && m < a.m && g == 0) {
      a.mean[m] = mean;
      a.rstd[m] = rstd;
    }
    // o1 = xhat gamma + beta as the B operand (contraction over the features)
    bf16x8 of[LNF_NT];
#pragma unroll
    for (int t = 0; t < LNF_NT; ++t) {
      const bf16x8 gm = *(const bf16x8*)(&gb[0][16 * t + 8 * g]);
      const bf16x8 bt = *(const bf16x8*)(&gb[1][16 * t + 8 * g]);
#pragma unroll
      for (int e = 0; e < 8; ++e) of[t][e] = (bf16)fmaf(xv[t][e] * rstd, (float)gm[e], (float)bt[e]);
    }
    lnf_load_rows(a, (u + stride) * 32 + l32, g, xr);  // next unit

    // Tiles inside one output: the MFMAs of the next tile are issued before
    // this one is stored (positions past the last are clamped; their results
    // are unused), and two accumulators alternate so no tile is copied.
    bf16x8 af[LNF_NT];
    if (nfast > 0) {
      const int last = nfast - 1;
      int t0 = tile_at(0);
      lnf_load_a(af, aoff, t0);
      f32x16 acc0 = lnf_tile(af, of), acc1;
      int t1 = tile_at(min(1, last));
      lnf_load_a(af, aoff, t1);
      for (int i = 0; i < nfast; i += 2) {
        acc1 = lnf_tile(af, of);
        const int t2 = tile_at(min(i + 2, last));
        lnf_load_a(af, aoff, t2);
        lnf_store_fast(acc0, st, a.tile[c0 / 32 + t0], lane, m0, a.m);
        if (i + 1 >= nfast) break;
        acc0 = lnf_tile(af, of);
        const int t3 = tile_at(min(i + 3, last));
        lnf_load_a(af, aoff, t3);
        lnf_store_fast(acc1, st, a.tile[c0 / 32 + t1], lane, m0, a.m);
        t0 = t2;
        t1 = t3;
      }
    }
    // the other tiles
    for (int i = nfast; i < ntiles; ++i) {
      const int t = tile_at(i);
      lnf_load_a(af, aoff, t);
      const f32x16 acc = lnf_tile(af, of);
      lnf_store_any(acc, st, quad + t * 8, lane, m0, a.m);
    }
  }
}

hipError_t launch_lnl_fwd(const LnlArgs& a, hipStream_t s) {
  const int groups = (a.ncols + a.gw - 1) / a.gw;
  const int64_t units = (a.m + 31) / 32;
  const int64_t per_group = std::max<int64_t>(1, 256 / groups);
  const int nwg = (int)std::min<int64_t>(per_group, (units + LNF_WAVES - 1) / LNF_WAVES);
  KernelTimer t(K_LNL_FWD, s);
  hipLaunchKernelGGL(lnl_fwd_kernel, dim3((unsigned)nwg, (unsigned)groups), dim3(64 * LNF_WAVES),
                     0, s, a);
  return hipGetLastError();
}

// ---- backward -------------------------------------------------------------------------
//
// Per row (appendix table of fused operators):  do1 = dO2 W^T,
//   wdy = do1 gamma,  c1 = sum_k xhat wdy / K,  c2 = sum_k wdy / K,
//   dx = rstd (wdy - c1 xhat - c2).
// The sums over rows are regrouped so that they all come from one pass over
// dO2 and x:  G = xhat^T dO2 [K][N] and s = sum_m dO2 [N] give
//   dW = o1^T dO2 = gamma G + beta s^T,  dgamma = sum_n W G,  dbeta = W s.
// Kernels: lnl_bwd_dx (dx), lnl_bwd_g (G and s per workgroup, partial
// slabs), lnl_reduce (the slabs summed in a fixed order), lnl_finish (dW,
// dgamma, dbeta).

// lnl_bwd_dx: persistent workgroups of LBX_WAVES waves, W resident in LDS as
// rows k of 16-byte chunks of 8 columns (chunk c of row k at slot c ^ (k % 8),
// 72 chunk slots per row), each wave walking 32-row units.  do1^T tiles
// [32 k][32 m] = W rows x dO2 rows^T: the dO2 B fragments (lane <-> row m,
// 8 consecutive columns) come straight from HBM.  The 16-column steps of
// the leading fast tiles (whole 32-column pieces of one output) form one
// stream across the wave's units, LBX_AHEAD fragments in flight, so the next
// unit's first fragments are in flight during this unit's epilogue; the
// remaining steps read two 4-column pieces each.  No load sits in a branch:
// a load whose result joins another value makes the wave wait for it there.
constexpr int LBX_WAVES = 8;
constexpr int LBX_PITCH = 72 * 16;
constexpr int LBX_AHEAD = 8;  // fast-step fragments in flight per lane (a multiple of 4)
constexpr int LBX_SLOW_AHEAD = 2;  // other steps whose fragments are loaded at the unit's start

__device__ inline uint32_t lbx_w_off(int k, int c) { return k * LBX_PITCH + 16 * (c ^ (k & 7)); }

// dO2 fragment of fast step s (columns 16 s + 8 g .. + 7, inside one output)
// for row mrow; zeros past the last row, or everywhere if !real.
__device__ inline bf16x8 lbx_load_fast(const LnlBwdArgs& a, int s, int g, uint32_t mrow, bool real) {
  const LnlTile& tl = a.tile[s >> 1];
  const rsrc_t r = buf_rsrc_n(tl.base, real ? (uint32_t)(a.m * tl.w * 2) : 0u);
  const uint32_t voff = (mrow * (uint32_t)tl.w + (uint32_t)(tl.off + 16 * (s & 1) + 8 * g)) * 2u;
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

// dO2 fragment of any step s for row m from two 4-column pieces of the quad
// table.  Both loads are always issued (a missing piece reads x's first
// bytes instead) and the pieces are zeroed after they arrive (lbx_slow_value).
struct LbxSlow {
  u32x2 lo, hi;
  bool lok, hok;
};
__device__ inline LbxSlow lbx_load_slow(const LnlBwdArgs& a, const LnlQuad* quad, int s, int g,
                                        int64_t m) {
  const int q = 2 * (2 * s + g);
  const LnlQuad e0 = quad[q], e1 = quad[q + 1];
  const bool ok = m < a.m;
  LbxSlow r;
  r.lok = ok && e0.p;
  r.hok = ok && e1.p;
  const gu32x2* dummy = (const gu32x2*)(gbf16*)a.x;
  const gu32x2* p0 = r.lok ? (const gu32x2*)(e0.p + m * e0.w) : dummy;
  const gu32x2* p1 = r.hok ? (const gu32x2*)(e1.p + m * e1.w) : dummy;
  r.lo = *p0;
  r.hi = *p1;
  return r;
}
__device__ inline bf16x8 lbx_slow_value(const LbxSlow& r) {
  const u32x2 lo = r.lok ? r.lo : u32x2{0u, 0u}, hi = r.hok ? r.hi : u32x2{0u, 0u};
  return __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
}

// Output address table of the dO2 slices (as the forward's, for reading).
__device__ inline void lnl_quad_table(const int* start, int n_out, bf16* const* ptrs, int ncols,
                                      int nq, LnlQuad* quad, int tid, int nthreads) {
  for (int q = tid; q < nq; q += nthreads) {
    LnlQuad e{nullptr, 0, 0};
    const int col = 4 * q;
    if (col < ncols) {
      int i = 0;
      while (i + 1 < n_out && col >= start[i + 1]) ++i;
      const int w = start[i + 1] - start[i], off = col - start[i];
      e.p = (gbf16*)(ptrs[i] + off);
      e.w = w;
      e.v8 = (w % 8 == 0 && off % 8 == 0) ? 1 : 0;
    }
    quad[q] = e;
  }
}

// The dx kernel's 16-column steps: those holding a column below N (host side).
static int lbx_steps(const LnlBwdArgs& a) { return (a.ncols + 15) / 16; }

// Steps [0, nf) of the fast-step stream: the 16-column steps of the leading
// fast tiles, rounded down to a multiple of LBX_AHEAD (host side).
static int lbx_fast_steps(const LnlBwdArgs& a) {
  const int nsteps = lbx_steps(a);
  int nt = 0;
  while (2 * nt < nsteps && a.tile[nt].fast) ++nt;
  return std::min(2 * nt, nsteps) / LBX_AHEAD * LBX_AHEAD;
}

// STREAM: at least one block of fast steps and at most LBX_SLOW_AHEAD other
// steps, all loaded at the unit's start, so that no load of the unit loop is
// conditional and the waits count the loads exactly (a wait that cannot count
// them waits for all, the next unit's fragments included).
template <bool STREAM>
__global__ __launch_bounds__(64 * LBX_WAVES) void lnl_bwd_dx_kernel(LnlBwdArgs a, int nf) {
  __shared__ __align__(16) char wk[LNL_K * LBX_PITCH];
  __shared__ __align__(16) LnlQuad quad[LNL_GROUP / 4];
  __shared__ __align__(16) float gam[LNL_K];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nq = a.np / 4;
  {  // W [K][N] into LDS (columns past N zero): all loads first, none in a
     // branch (an element outside W reads W's first one and is zeroed)
    constexpr int NT = 64 * LBX_WAVES;
    constexpr int FILL = (LNL_K * (LNL_GROUP / 4) + NT - 1) / NT;
    u32x2 wv[FILL];
#pragma unroll
    for (int i = 0; i < FILL; ++i) {
      const int idx = tid + i * NT, k = idx / nq, q = idx - k * nq;
      const bool ok = idx < LNL_K * nq && 4 * q < a.ncols;
      const u32x2 v = *(const u32x2*)(a.w + (ok ? (int64_t)k * a.ncols + 4 * q : 0));
      wv[i] = ok ? v : u32x2{0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < FILL; ++i) {
      const int idx = tid + i * NT, k = idx / nq, q = idx - k * nq;
      if (idx < LNL_K * nq) *(u32x2*)(wk + lbx_w_off(k, q >> 1) + 8 * (q & 1)) = wv[i];
    }
  }
  lnl_quad_table(a.start, a.n_out, (bf16* const*)a.dout, a.ncols, nq, quad, tid, 64 * LBX_WAVES);
  if (tid < LNL_K) gam[tid] = (float)a.gamma[tid];
  __syncthreads();

  // The rows of a k tile enter the A operand permuted: operand row
  // r = 8 j + 4 h + i (the accumulator rows that lane half h holds) reads W
  // row 16 (j / 2) + 8 h + 4 (j % 2) + i, so that a lane ends up with two runs
  // of 8 consecutive features per k tile (k = 32 kt + 16 a + 8 g + e in
  // acc[kt][8 a + e]) and reads x and writes dx 16 bytes at a time.
  const int wrow = 16 * (l32 >> 4) + 8 * ((l32 >> 2) & 1) + 4 * ((l32 >> 3) & 1) + (l32 & 3);
  // A fragment of (k tile kt, step s): W row 32 kt + wrow, chunk
  // 2 s + g = 8 (s / 4) + (2 (s % 4) + g)  ->  ao[s % 4] + kt * 32 rows + 128 (s / 4)
  uint32_t ao[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) ao[s4] = lds_addr(wk) + lbx_w_off(wrow, 2 * s4 + g);
  const int nsteps = (a.ncols + 15) / 16;  // as lbx_steps: later steps would multiply zeros
  const int ns = nsteps - nf;              // the steps after the fast-step stream (nf: lbx_fast_steps)
  const int64_t units = (a.m + 31) / 32;
  const int64_t stride = (int64_t)gridDim.x * LBX_WAVES;
  const int64_t u0 = (int64_t)blockIdx.x * LBX_WAVES + wave;
  // the fast-step stream: position s of unit u, then step 0 of unit u + stride
  bf16x8 bq[LBX_AHEAD];
#pragma unroll
  for (int d = 0; d < LBX_AHEAD; ++d)
    bq[d] = lbx_load_fast(a, d, g, (uint32_t)(u0 * 32 + l32), nf > 0 && u0 < units);
  if constexpr (STREAM) {
    // eight empty stores (a zero-length range drops them): the unit loop
    // is then entered with the same operations in flight as at its back edge
    // (fragments, then a unit's stores), so the waits of a unit's first
    // block count the stores and need not wait for them
    const rsrc_t none = buf_rsrc_n(a.dx, 0u);
#pragma unroll
    for (int f = 0; f < 8; ++f) __builtin_amdgcn_raw_buffer_store_b128(u32x4{0u, 0u, 0u, 0u}, none, 16u * f, 0, 0);
  }
  f32x16 acc[4] = {};  // zero at the start of every unit
  for (int64_t u = u0; u < units; u += stride) {
    const int64_t m = u * 32 + l32;
    const bool mok = m < a.m;
    // this row's x at k = 32 kt + 16 a + 8 g + 0..7 (xq[2 kt + a]) and its
    // statistics (for the epilogue).  Every load of the loop is issued
    // unconditionally (a row past m reads the last row and is zeroed), so the
    // waits can count them.
    const int64_t mc = mok ? m : a.m - 1;
    u32x4 xq[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const u32x4 v = *(const u32x4*)(a.x + mc * LNL_K + 16 * f + 8 * g);
      xq[f] = mok ? v : u32x4{0u, 0u, 0u, 0u};
    }
    const float mean0 = a.mean[mc], rstd0 = a.rstd[mc];
    const float mean = mok ? mean0 : 0.f, rstd = mok ? rstd0 : 0.f;
    LbxSlow sl[LBX_SLOW_AHEAD];  // the first other steps (a step past the last reads the last)
#pragma unroll
    for (int i = 0; i < LBX_SLOW_AHEAD; ++i) sl[i] = lbx_load_slow(a, quad, min(nf + i, nsteps - 1), g, m);

    auto mma_step = [&](int s, const bf16x8& b) {
      const uint32_t ad = lds_addr(wk) + lbx_w_off(wrow, 2 * s + g);
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
        acc[kt] = Mma<bf16>::mma(lds_load16<bf16x8>(ad + kt * 32 * LBX_PITCH), b, acc[kt]);
    };
    const int64_t un = u + stride;
    auto fast_block = [&](int s0) {  // steps s0 .. s0 + LBX_AHEAD - 1
      const bool wrap = s0 + LBX_AHEAD >= nf;  // the refills belong to the next unit
      const uint32_t mrow = (uint32_t)((wrap ? un : u) * 32 + l32);
      const bool real = !wrap || un < units;
#pragma unroll
      for (int d = 0; d < LBX_AHEAD; ++d) {
        const int s = s0 + d;
        const uint32_t ad = ao[d % 4] + 128 * (s >> 2);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
          acc[kt] = Mma<bf16>::mma(lds_load16<bf16x8>(ad + kt * 32 * LBX_PITCH), bq[d], acc[kt]);
        // the refill after the use: it can reuse the fragment's registers
        bq[d] = lbx_load_fast(a, wrap ? d : s + LBX_AHEAD, g, mrow, real);
      }
    };
    if constexpr (STREAM) {
      // at least one block (nf >= LBX_AHEAD), the first outside the loop: its
      // waits can count this unit's x loads and the last unit's stores as
      // issued after its fragments, and the waits after the loop know that
      // the last block's loads were issued after everything else
      fast_block(0);
      for (int s0 = LBX_AHEAD; s0 < nf; s0 += LBX_AHEAD) fast_block(s0);
    } else {
      for (int s0 = 0; s0 < nf; s0 += LBX_AHEAD) fast_block(s0);
    }
#pragma unroll
    for (int i = 0; i < LBX_SLOW_AHEAD; ++i)
      if (i < ns) mma_step(nf + i, lbx_slow_value(sl[i]));
    if constexpr (!STREAM)
      for (int i = LBX_SLOW_AHEAD; i < ns; ++i) mma_step(nf + i, lbx_slow_value(lbx_load_slow(a, quad, nf + i, g, m)));
    // lane (row m, half g) holds do1[m][32 kt + 16 a + 8 g + e] in acc[kt][8 a + e].
    // gamma is read from LDS per unit: an offset the compiler cannot see
    // through keeps it from holding all 64 values in registers across the loop.
    int gz = 8 * g;
    asm volatile("" : "+v"(gz));
    const float* const gl = gam + gz;
    float c1 = 0.f, c2 = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int a2 = 0; a2 < 2; ++a2) {
        const bf16x8 xv = __builtin_bit_cast(bf16x8, xq[2 * kt + a2]);
        const f32x4 g0 = *(const f32x4*)(gl + 32 * kt + 16 * a2), g1 = *(const f32x4*)(gl + 32 * kt + 16 * a2 + 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = ((float)xv[e] - mean) * rstd;
          const float wdy = acc[kt][8 * a2 + e] * (e < 4 ? g0[e] : g1[e - 4]);
          c1 = fmaf(xh, wdy, c1);
          c2 += wdy;
        }
      }
    c1 = wave_xor32_sum(c1) * (1.f / LNL_K);
    c2 = wave_xor32_sum(c2) * (1.f / LNL_K);
    u32x4 pk[8];  // dx of the lane's 64 features, bf16
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int a2 = 0; a2 < 2; ++a2) {
        const bf16x8 xv = __builtin_bit_cast(bf16x8, xq[2 * kt + a2]);
        const f32x4 g0 = *(const f32x4*)(gl + 32 * kt + 16 * a2), g1 = *(const f32x4*)(gl + 32 * kt + 16 * a2 + 4);
        bf16x8 d;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = ((float)xv[e] - mean) * rstd;
          d[e] = (bf16)(rstd * (acc[kt][8 * a2 + e] * (e < 4 ? g0[e] : g1[e - 4]) - c1 * xh - c2));
        }
        pk[2 * kt + a2] = __builtin_bit_cast(u32x4, d);
      }
    // The next unit's accumulators are zeroed (and tied) before the stores are
    // issued, so the stores' data and the accumulators never share registers:
    // no write to the accumulators has to wait for a store to read its data.
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) acc[kt] = f32x16{};
    asm volatile("" : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]) : : "memory");
    // every lane stores (the buffer range drops rows past m): no branch, so
    // the waits of the next unit can count the stores
    const rsrc_t rdx = buf_rsrc_n(a.dx, (uint32_t)(a.m * LNL_K * 2));
    const uint32_t vdx = (uint32_t)m * (uint32_t)(LNL_K * 2) + 16u * (uint32_t)g;
#pragma unroll
    for (int f = 0; f < 8; ++f) __builtin_amdgcn_raw_buffer_store_b128(pk[f], rdx, vdx + 32u * f, 0, 0);
  }
}

// lnl_bwd_g: persistent workgroups of LBG_WAVES waves; each workgroup walks
// 32-row units u = blockIdx + i * gridDim, staging the unit's x, mean, rstd
// and dO2 rows in LDS with buffer-resource DMA (rows past m read as zeros)
// into a ring of up to three slots, two units ahead.  A wave issues the same
// pieces for every unit and nothing else, so it knows exactly how many of its
// loads may still be in flight when a unit must have landed.  Wave w accumulates the G tiles
// (k tile w % 4, column tiles w / 4 + 2 i) over all its units in registers:
// A = xhat^T (transposed x reads, normalised in registers), B = dO2
// (transposed reads), contraction over the unit's 32 rows.  One wave of each
// column tile also sums its B fragments into s.  At the end each workgroup writes
// its slab of gpart.
constexpr int LBG_WAVES = 8;
constexpr int LBG_STAGE = 148 * 1024;  // ring bytes
constexpr int LBG_MAXOPS = 64;
constexpr int LBG_TPW = (LNL_GROUP / 32 + 1) / 2;  // column tiles per wave (at most)

struct LbgOp {
  const char* src;    // tensor base
  uint32_t rowbytes;  // bytes per row of the tensor
  uint32_t voff;      // byte offset of this 1 KB piece inside the unit's rows
  uint32_t lds;       // destination offset inside a slot
  uint32_t nbytes;    // bytes of the tensor (range of the buffer resource)
};

// Rows of 256 bytes (x, and dO2 outputs 128 columns wide) are staged with
// their 16-byte chunks permuted: chunk c of row p sits at slot c ^ 4 (p % 4),
// so the transposed reads of 4 consecutive rows hit four different 64-byte
// bank windows.  The DMA writes a piece's lanes to consecutive LDS bytes, so
// the lane that fills slot c' of row p loads chunk c' ^ 4 (p % 4).
__device__ inline uint32_t lbg_swz_lane(int lane) {
  const int r = lane >> 4;
  return 256u * r + 16u * ((lane & 15) ^ (4 * (r & 3)));
}
__device__ inline uint32_t lbg_swz_off(int p, int col) {  // byte offset of (row p, column col)
  return p * 256 + 16 * ((col >> 3) ^ (4 * (p & 3))) + 2 * (col & 7);
}

// The A operand's staged reads of a unit, one wait for all: x^T at
// xa (+ 2048 j, four transposed reads) and the mean and rstd of its
// positions at sp (runs at + 0, 32, 64, 96 and, for rstd, + 1024).
__device__ inline void lbg_a_reads(uint32_t xa, uint32_t sp, s16x4 (&xr)[4], f32x4 (&st)[8]) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %12\n\tds_read_b64_tr_b16 %1, %12 offset:2048\n\t"
      "ds_read_b64_tr_b16 %2, %12 offset:4096\n\tds_read_b64_tr_b16 %3, %12 offset:6144\n\t"
      "ds_read_b128 %4, %13\n\tds_read_b128 %5, %13 offset:32\n\t"
      "ds_read_b128 %6, %13 offset:1024\n\tds_read_b128 %7, %13 offset:1056\n\t"
      "ds_read_b128 %8, %13 offset:64\n\tds_read_b128 %9, %13 offset:96\n\t"
      "ds_read_b128 %10, %13 offset:1088\n\tds_read_b128 %11, %13 offset:1120\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(xr[0]), "=&v"(xr[1]), "=&v"(xr[2]), "=&v"(xr[3]), "=&v"(st[0]), "=&v"(st[1]),
        "=&v"(st[2]), "=&v"(st[3]), "=&v"(st[4]), "=&v"(st[5]), "=&v"(st[6]), "=&v"(st[7])
      : "v"(xa), "v"(sp));
}

// Transposed reads of three B tiles (four each, at b[t] + j s[t]), one wait.
__device__ inline void lbg_b_reads3(const uint32_t (&b)[3], const uint32_t (&st)[3], s16x4 (&r)[12]) {
  uint32_t ad[12];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) ad[4 * t + j] = b[t] + j * st[t];
  asm volatile(
      "ds_read_b64_tr_b16 %0, %12\n\tds_read_b64_tr_b16 %1, %13\n\t"
      "ds_read_b64_tr_b16 %2, %14\n\tds_read_b64_tr_b16 %3, %15\n\t"
      "ds_read_b64_tr_b16 %4, %16\n\tds_read_b64_tr_b16 %5, %17\n\t"
      "ds_read_b64_tr_b16 %6, %18\n\tds_read_b64_tr_b16 %7, %19\n\t"
      "ds_read_b64_tr_b16 %8, %20\n\tds_read_b64_tr_b16 %9, %21\n\t"
      "ds_read_b64_tr_b16 %10, %22\n\tds_read_b64_tr_b16 %11, %23\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]),
        "=&v"(r[6]), "=&v"(r[7]), "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11])
      : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(ad[4]), "v"(ad[5]), "v"(ad[6]),
        "v"(ad[7]), "v"(ad[8]), "v"(ad[9]), "v"(ad[10]), "v"(ad[11]));
}

// s_waitcnt vmcnt(n) for a wave-uniform n in [0, 15].
__device__ inline void wait_vm_n(int n) {
  switch (n) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<1>(); break;
    case 2: wait_vm<2>(); break;
    case 3: wait_vm<3>(); break;
    case 4: wait_vm<4>(); break;
    case 5: wait_vm<5>(); break;
    case 6: wait_vm<6>(); break;
    case 7: wait_vm<7>(); break;
    case 8: wait_vm<8>(); break;
    case 9: wait_vm<9>(); break;
    case 10: wait_vm<10>(); break;
    case 11: wait_vm<11>(); break;
    case 12: wait_vm<12>(); break;
    case 13: wait_vm<13>(); break;
    case 14: wait_vm<14>(); break;
    default: wait_vm<15>(); break;
  }
}

__global__ __launch_bounds__(64 * LBG_WAVES) void lnl_bwd_g_kernel(LnlBwdArgs a) {
  __shared__ __align__(16) char stage[LBG_STAGE];
  __shared__ LbgOp ops[LBG_MAXOPS];
  __shared__ uint32_t qreg[LNL_GROUP / 4];  // per 4 columns: staged region (offset in a slot)
  __shared__ uint32_t qcol[LNL_GROUP / 4];  // first column inside the output
  __shared__ uint32_t qpitch[LNL_GROUP / 4];  // row pitch in bytes (0: past N, read zeros)
  __shared__ int nops_s, slot_s;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5;
  const int wave = tid >> 6;
  const int nq = a.np / 4, ntiles = a.np / 32;
  const uint32_t mb = (uint32_t)a.m;  // rows fit 32 bits (checked by the caller)
  if (tid == 0) {
    int no = 0;
    uint32_t lds = 0;
    for (int j = 0; j < 8; ++j)
      ops[no++] = LbgOp{(const char*)a.x, 2 * LNL_K, 1024u * j, lds + 1024u * j, mb * 2 * LNL_K};
    lds += 8192;
    ops[no++] = LbgOp{(const char*)a.mean, 4, 0, lds, mb * 4};
    ops[no++] = LbgOp{(const char*)a.rstd, 4, 0, lds + 1024, mb * 4};
    lds += 2048;
    int region[LNL_MAX_OUT];
    for (int i = 0; i < a.n_out; ++i) {
      const uint32_t w = a.start[i + 1] - a.start[i], bytes = 64 * w, nop = (bytes + 1023) / 1024;
      region[i] = lds;
      for (uint32_t j = 0; j < nop; ++j)
        ops[no++] = LbgOp{(const char*)a.dout[i], 2 * w, 1024u * j, lds + 1024u * j, mb * 2 * w};
      lds += 1024 * nop;
    }
    // then 64 zero bytes; a slot is a multiple of 256 bytes
    const uint32_t zero = lds;
    for (int q = 0; q < nq; ++q) {
      const int col = 4 * q;
      if (col < a.ncols) {
        int i = 0;
        while (i + 1 < a.n_out && col >= a.start[i + 1]) ++i;
        qreg[q] = region[i];
        qcol[q] = col - a.start[i];
        qpitch[q] = 2 * (a.start[i + 1] - a.start[i]);
      } else {
        qreg[q] = zero;
        qcol[q] = 0;
        qpitch[q] = 0;
      }
    }
    nops_s = no;
    slot_s = (int)((zero + 64 + 255) & ~255u);
  }
  __syncthreads();
  const int nops = nops_s, sb = slot_s;
  const int nslots = LBG_STAGE / sb >= 3 ? 3 : 2;
  const int ahead = nslots - 1;                          // units in flight beyond the current
  const int nw = nops > wave ? (nops - wave + LBG_WAVES - 1) / LBG_WAVES : 0;  // pieces per unit
  const uint32_t zoff = (uint32_t)sb - 64;
  if (tid < 16 * nslots) *(uint32_t*)(stage + (tid >> 4) * sb + zoff + 4 * (tid & 15)) = 0u;
  __syncthreads();

  // this wave's tiles
  const int kt = wave & 3, t0 = wave >> 2;
  const int nt_w = t0 < ntiles ? (ntiles - t0 + 1) / 2 : 0;
  // transposed-read addresses: lane supplies position pe (+ p0) and columns
  // 16 (G % 2) + 4 j of its tile (TrAddr's pattern over row-major rows)
  const int G = lane >> 4, jj = lane & 3, pe = ((lane & 15) >> 2) + 4 * (G >> 1);
  const int cq = 4 * (G & 1) + jj;  // quad of the tile this lane supplies
  const uint32_t sbase = lds_addr(stage);
  const uint32_t xa = sbase + lbg_swz_off(pe, 32 * kt + 4 * cq);
  uint32_t ba[LBG_TPW], bp[LBG_TPW];
#pragma unroll
  for (int i = 0; i < LBG_TPW; ++i) {
    const int T = t0 + 2 * i, q = T < ntiles ? 8 * T + cq : 0;
    const uint32_t pitch = qpitch[q];
    bp[i] = pitch;
    ba[i] = sbase + qreg[q] +
            (pitch == 256 ? lbg_swz_off(pe, qcol[q]) : pe * pitch + 2 * qcol[q]);
  }
  // this wave's DMA pieces (the same for every unit)
  const uint32_t lplain = 16u * lane, lswz = lbg_swz_lane(lane);
  const uint32_t sa = sbase + 8192;  // mean (+ 1024: rstd)

  f32x16 acc[LBG_TPW] = {};
  float ssum[LBG_TPW] = {};
  const bf16x2 one2 = {(bf16)1.f, (bf16)1.f};
  const int64_t units = (a.m + 31) / 32;
  // this wave's pieces of a unit (the same nw for every unit); the two
  // statistics pieces need only the unit's 32 x 4 bytes.  The table is read
  // once, before the loop, and its fields made wave-uniform, so the buffer
  // resources live in scalar registers and each piece is one instruction.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  constexpr int MAXW = LBG_MAXOPS / LBG_WAVES;  // pieces per wave, at most
  rsrc_t prs[MAXW];
  uint32_t prow[MAXW], pvo[MAXW], plds[MAXW];
#pragma unroll
  for (int i = 0; i < MAXW; ++i) {
    const LbgOp op = ops[min(wave_u + LBG_WAVES * i, nops - 1)];
    // (readfirstlane returns int: widen through uint32_t, never sign-extend)
    const uint64_t src =
        (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)op.src) |
        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)((uintptr_t)op.src >> 32))
         << 32);
    const uint32_t nbytes = __builtin_amdgcn_readfirstlane(op.nbytes);
    prs[i] = __builtin_amdgcn_make_buffer_rsrc((void*)(uintptr_t)src, (short)0, (int)nbytes, 0x00020000);
    prow[i] = __builtin_amdgcn_readfirstlane(op.rowbytes);
    pvo[i] = __builtin_amdgcn_readfirstlane(op.voff);
    plds[i] = __builtin_amdgcn_readfirstlane(op.lds);
  }
  auto issue = [&](int64_t u, int slot) {
    if (u >= units) return;
#pragma unroll
    for (int i = 0; i < MAXW; ++i) {
      if (i >= nw) break;
      const uint32_t voff = (uint32_t)u * 32u * prow[i] + pvo[i] + (prow[i] == 256 ? lswz : lplain);
      if (prow[i] != 4 || lane < 8) dma16b(prs[i], voff, stage + slot * sb + plds[i]);
    }
  };
  int64_t u = blockIdx.x;
  for (int i = 0; i < ahead; ++i) issue(u + (int64_t)i * gridDim.x, i);
  for (int it = 0; u < units; ++it, u += gridDim.x) {
    const int slot = it % nslots;
    // this unit's pieces have landed once at most those of the units issued
    // after it are in flight
    int later = 0;
    for (int i = 1; i < ahead; ++i) later += u + (int64_t)i * gridDim.x < units ? 1 : 0;
    wait_vm_n(later * nw);
    lds_barrier();  // for every wave; and the slot refilled next is free
    issue(u + (int64_t)ahead * gridDim.x, (it + ahead) % nslots);
    const uint32_t so = slot * sb;
    // A = xhat^T: x of positions {4 g + 0..3, 8 + 4 g + 0..3} (+ 16 u) at
    // channels 32 kt + l32, normalised with those positions' statistics
    s16x4 xr[4];
    f32x4 st[8];  // per half h: mean of the two runs of 4, then their rstd
    lbg_a_reads(xa + so, sa + so + 16 * g, xr, st);
    bf16x8 af[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bf16x8 xv = tr_frag(xr, h);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        af[h][e] = (bf16)(((float)xv[e] - st[4 * h][e]) * st[4 * h + 2][e]);
        af[h][4 + e] = (bf16)(((float)xv[4 + e] - st[4 * h + 1][e]) * st[4 * h + 3][e]);
      }
    }
    // the B tiles three at a time (one wait per three)
#pragma unroll
    for (int i0 = 0; i0 < LBG_TPW; i0 += 3) {
      if (i0 >= nt_w) break;
      uint32_t b[3], bst[3];
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int i = min(i0 + t, LBG_TPW - 1);
        const bool ok = i0 + t < nt_w;  // else a harmless read of the first tile
        b[t] = (ok ? ba[i] : ba[i0]) + so;
        bst[t] = 8 * (ok ? bp[i] : bp[i0]);
      }
      s16x4 br[12];
      lbg_b_reads3(b, bst, br);
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int i = i0 + t;
        if (i < LBG_TPW && i < nt_w) {
          const s16x4 bt[4] = {br[4 * t], br[4 * t + 1], br[4 * t + 2], br[4 * t + 3]};
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const bf16x8 bf = tr_frag(bt, h);
            acc[i] = Mma<bf16>::mma(af[h], bf, acc[i]);
            if (i % 4 == kt)  // column sums: each tile by one of its four waves
            {
              ssum[i] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(bf, bf, 0, 1), one2,
                                                        ssum[i], false);
              ssum[i] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(bf, bf, 2, 3), one2,
                                                        ssum[i], false);
              ssum[i] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(bf, bf, 4, 5), one2,
                                                        ssum[i], false);
              ssum[i] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(bf, bf, 6, 7), one2,
                                                        ssum[i], false);
            }
          }
        }
      }
    }
  }
  wait_vm<0>();  // the pieces issued past the last unit land before the wave ends
  // this workgroup's slab: G rows k = 32 kt + 8 j + 4 g + i, column 32 T + l32
  float* slab = a.gpart + (int64_t)blockIdx.x * (LNL_K + 1) * a.np;
  const int l32 = lane & 31;
#pragma unroll
  for (int i = 0; i < LBG_TPW; ++i) {
    if (i < nt_w) {
      const int n = 32 * (t0 + 2 * i) + l32;
#pragma unroll
      for (int v = 0; v < 16; ++v) slab[(int64_t)(32 * kt + acc_row(v, g)) * a.np + n] = acc[i][v];
      if (i % 4 == kt) {
        const float st = wave_xor32_sum(ssum[i]);
        if (g == 0) slab[(int64_t)LNL_K * a.np + n] = st;
      }
    }
  }
}

// gsum[r][n] = sum over workgroups p (in order p = c, c + 8, ..., then the 8
// chains c = 0..7 in order) of gpart[p][r][n]; one workgroup per (row r,
// 128 columns).
__global__ __launch_bounds__(256) void lnl_reduce_kernel(LnlBwdArgs a) {
  __shared__ f32x4 red[8][32];
  const int r = blockIdx.y, t = threadIdx.x, n4 = t & 31, c = t >> 5;
  const int n = blockIdx.x * 128 + 4 * n4;
  f32x4 s = {};
  if (n < a.np)
    for (int p = c; p < a.nwg; p += 8)
      s += *(const f32x4*)(a.gpart + ((int64_t)p * (LNL_K + 1) + r) * a.np + n);
  red[c][n4] = s;
  __syncthreads();
  if (t < 32 && n < a.np) {
    f32x4 tot = red[0][t];
#pragma unroll
    for (int i = 1; i < 8; ++i) tot += red[i][t];
    *(f32x4*)(a.gsum + (int64_t)r * a.np + n) = tot;
  }
}

// dW[k][n] = gamma_k G[k][n] + beta_k s[n];  dgamma[k] = sum_n W[k][n] G[k][n];
// dbeta[k] = sum_n W[k][n] s[n]  (per-thread partials, then a fixed tree).
__global__ __launch_bounds__(256) void lnl_finish_kernel(LnlBwdArgs a) {
  __shared__ float rg[256], rb[256];
  const int k = blockIdx.x, t = threadIdx.x;
  const float gk = (float)a.gamma[k], bk = (float)a.beta[k];
  const float* G = a.gsum + (int64_t)k * a.np;
  const float* S = a.gsum + (int64_t)LNL_K * a.np;
  float pg = 0.f, pb = 0.f;
  for (int n = t; n < a.ncols; n += 256) {
    const float gv = G[n], sv = S[n], wv = (float)a.w[(int64_t)k * a.ncols + n];
    a.dw[(int64_t)k * a.ncols + n] = fmaf(gk, gv, bk * sv);
    pg = fmaf(wv, gv, pg);
    pb = fmaf(wv, sv, pb);
  }
  rg[t] = pg;
  rb[t] = pb;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (t < h) {
      rg[t] += rg[t + h];
      rb[t] += rb[t + h];
    }
    __syncthreads();
  }
  if (t == 0) {
    a.dgamma[k] = rg[0];
    a.dbeta[k] = rb[0];
  }
}

int lnl_bwd_partials(int64_t m) { return (int)std::min<int64_t>(256, (m + 31) / 32); }

size_t lnl_bwd_workspace(int64_t m, int np) {
  const size_t slab = (size_t)(LNL_K + 1) * np * sizeof(float);
  return (size_t)lnl_bwd_partials(m) * slab + slab;
}

hipError_t launch_lnl_bwd(const LnlBwdArgs& a, hipStream_t s) {
  const int64_t units = (a.m + 31) / 32;
  {
    KernelTimer t(K_LNL_BWD_DX, s);
    const int nwg = (int)std::min<int64_t>(256, (units + LBX_WAVES - 1) / LBX_WAVES);
    const int nf = lbx_fast_steps(a);
    if (nf >= LBX_AHEAD && lbx_steps(a) - nf <= LBX_SLOW_AHEAD)
      hipLaunchKernelGGL(lnl_bwd_dx_kernel<true>, dim3(nwg), dim3(64 * LBX_WAVES), 0, s, a, nf);
    else
      hipLaunchKernelGGL(lnl_bwd_dx_kernel<false>, dim3(nwg), dim3(64 * LBX_WAVES), 0, s, a, nf);
  }
  {
    KernelTimer t(K_LNL_BWD_G, s);
    hipLaunchKernelGGL(lnl_bwd_g_kernel, dim3(a.nwg), dim3(64 * LBG_WAVES), 0, s, a);
  }
  {
    KernelTimer t(K_LNL_REDUCE, s);
    hipLaunchKernelGGL(lnl_reduce_kernel, dim3((a.np + 127) / 128, LNL_K + 1), dim3(256), 0, s, a);
  }
  {
    KernelTimer t(K_LNL_FINISH, s);
    hipLaunchKernelGGL(lnl_finish_kernel, dim3(LNL_K), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace triattn
