// Triangle-attention backward (MegaFold appendix: backward listing and the
// EvoAttention table).  Every kernel recomputes P = exp(S - LSE) from the
// saved log-sum-exp; nothing of size N^3 is stored.
//
//   bwd_prep : dG = dO * O * (1 - sigmoid(G)), dA = dO * sigmoid(G) (the
//              gradient of the ungated output), lse in base 2 --
//              elementwise over the pair map.  For bf16,
//              dA is kept as a pair hi + lo of bf16 numbers and dP = dA V^T
//              takes both (one extra MFMA): rounding dA to a single bf16
//              makes sum_k P dP drift from D, and that drift accumulates
//              in the row sum of the bias gradient.
//   dkdv     : the paper's first stage -- per (row, head, key block), loop
//              over query tiles: dV += P^T dA, dK += scale dS^T Q.
//   dq       : the paper's second stage without the bias -- per (row, head,
//              query block), loop over key tiles: dQ += scale dS K.  It runs
//              first and also produces D = rowsum(dO * O) in the form
//              sum_k P dP (equal in exact arithmetic, table of the appendix):
//              taken from the same P and dP the other kernels recompute, it
//              keeps sum_k dS = 0, which D from the bf16-rounded output O
//              does not (visible when one key takes all the weight).
//   db       : the bias gradient dB[q][k] = sum over rows of dS[row][q][k].
//              The paper adds dS into dBias with atomics; here each
//              workgroup owns a (query block, key block, head, row chunk)
//              tile, keeps its partial sum in registers over the rows of the
//              chunk and stores it to a slab; db_reduce adds the slabs in
//              chunk order.  No atomics, so the result is reproducible.
#include <type_traits>

#include "dma.h"
#include "kernels.h"
#include "stage.h"
#include "timing.h"

namespace triattn {

template <typename T>
constexpr bool kSplitDA = std::is_same<T, bf16>::value;

// ---- elementwise preparation -------------------------------------------------------

// Four threads per (pair, head): thread t handles channels 8 (t % 4) .. +7,
// so every load and store is 16 contiguous bytes and a wave covers 16 whole
// (pair, head) rows.
template <typename T>
__global__ __launch_bounds__(256) void bwd_prep_kernel(Geom G, int node, const T* out,
                                                       const float* lse, const T* gate,
                                                       const T* dout, T* dg, T* da,
                                                       T* dalo, float* lse2) {
  const int64_t tix = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t idx = tix >> 2;  // (a, b, h)
  const int64_t total = (int64_t)G.n * G.n * G.H;
  if (idx >= total) return;
  const int64_t base = idx * HEAD_DIM + 8 * (tix & 3);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const f32x4 go = load4(dout + base + 4 * j), oo = load4(out + base + 4 * j);
    const f32x4 gg = load4(gate + base + 4 * j);
    f32x4 dgv, dav;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float sg = 1.f / (1.f + __expf(-gg[e]));
      dgv[e] = go[e] * oo[e] * (1.f - sg);
      dav[e] = go[e] * sg;
    }
    store4(dg + base + 4 * j, dgv);
    store4(da + base + 4 * j, dav);
    if constexpr (kSplitDA<T>) {
      f32x4 lo;
#pragma unroll
      for (int e = 0; e < 4; ++e) lo[e] = dav[e] - (float)(bf16)dav[e];
      store4(dalo + base + 4 * j, lo);
    }
  }
  if ((tix & 3) == 0) {
    const int h = (int)(idx % G.H);
    const int64_t pair = idx / G.H;
    const int a = (int)(pair / G.n), b = (int)(pair % G.n);
    const int row = node == 0 ? a : b, qi = node == 0 ? b : a;
    const float l = lse[idx];
    lse2[((int64_t)h * G.n + row) * G.np + qi] = l == neg_inf() ? pos_inf() : l * LOG2E;
  }
}

// Queries n .. np-1 of every row: no valid key (+inf) and D = 0.
__global__ __launch_bounds__(256) void bwd_pad_kernel(Geom G, float* lse2, float* dsum) {
  const int pad = G.np - G.n;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)G.H * G.n * pad) return;
  const int64_t hr = idx / pad;
  const int64_t at = hr * G.np + G.n + (int)(idx % pad);
  lse2[at] = pos_inf();
  dsum[at] = 0.f;
}

constexpr int BWD_WAVES = 4;
constexpr int BWD_BLK = BWD_WAVES * TILE;

template <typename T>
struct BwdArgs {
  Geom g;
  const float *bt, *btT;
  const uint32_t* kbits;
  const T *q, *k, *v, *da;
  const T* dalo;  // bf16 only: dA - bf16(dA), also rounded to bf16
  const float* lse2;
  float* dsum;  // -D per (head, row, query): written by dq_kernel, read after
  T *dq, *dk, *dv;
  float* slabs;
  int nblk;  // 128-wide blocks per axis
  int nrc;   // row chunks (db)
  int rpc;   // rows per chunk (db)
};

// ---- dQ (and D) ----------------------------------------------------------------------

// Per (row, head, 128 queries): stream the row's keys in blocks of 64 (K, K^T
// and V staged in LDS, double-buffered).  dQ = scale (X - D Y) with
// X = sum_k P dP K, Y = sum_k P K and D = sum_k P dP, all from one pass.
template <typename T>
__global__ __launch_bounds__(256, 2) void dq_kernel(BwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int qb = w % a.nblk, rh = w / a.nblk;
  const int r = rh % G.n, h = rh / G.n;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * BWD_BLK + wave * TILE;
  const bool active = q0 < G.n;
  const int q = q0 + l32;  // lane <-> query
  const bool qok = q < G.n;

  __shared__ __align__(16) T ks[2 * ROW_TILE];    // K   [key][channel]
  __shared__ __align__(16) T kT[2 * TRANS_TILE];  // K^T [channel][key]
  __shared__ __align__(16) T vs[2 * ROW_TILE];    // V   [key][channel]

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
  const T* kr = a.k + rowbase;
  const T* vr = a.v + rowbase;
  const int last = G.n - 1;
  typename M::frag qf[M::KCH], daf[M::KCH], dalf[M::KCH];
  float l2 = pos_inf();
  zero_frags<T>(dalf);
  if (qok) {
    row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
    row_frags(a.da + rowbase + (int64_t)q * G.sPos, g, daf);
    if constexpr (kSplitDA<T>) row_frags(a.dalo + rowbase + (int64_t)q * G.sPos, g, dalf);
    l2 = a.lse2[((int64_t)h * G.n + r) * G.np + q];
  } else {
    zero_frags<T>(qf);
    zero_frags<T>(daf);
  }
  const float c1 = G.scale * LOG2E;
  f32x16 xt = {}, yt = {};
  float dpart = 0.f;
  const uint32_t* kb = a.kbits + (int64_t)r * G.nkt;
  const int nblk = (G.nkt + 1) >> 1;
  const int qt = active ? q0 / TILE : 0;
  auto bias_tile = [&](int kt) {
    return load_frag_tile(frag_tile(a.bt, h, qt, min(kt, G.nkt - 1), G.nkt), lane);
  };

  auto sub_tile = [&](const T* ksb, const T* kTb, const T* vsb, const f32x16& bias, uint32_t bits,
                      int u) {
    // S^T = bias + K Q^T (lane <-> query, registers <-> keys)
    typename M::frag af[M::KCH];
    row_frags(ksb + (32 * u + l32) * LDS_ROW, g, af);
    f32x16 s = M::mma(af[0], qf[0], bias);
#pragma unroll
    for (int t = 1; t < M::KCH; ++t) s = M::mma(af[t], qf[t], s);
    if (bits != 0xffffffffu) mask_rows(s, bits, g);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2));
    // dP^T = V dA^T, then P dP and its running sum D
    row_frags(vsb + (32 * u + l32) * LDS_ROW, g, af);
    f32x16 dp = M::mma(af[0], daf[0], f32x16{});
#pragma unroll
    for (int t = 1; t < M::KCH; ++t) dp = M::mma(af[t], daf[t], dp);
    if constexpr (kSplitDA<T>) {
#pragma unroll
      for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], dalf[t], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      dp[v] *= s[v];
      dpart += dp[v];
    }
    // X^T += K^T (P dP)^T,  Y^T += K^T P^T (contraction over the keys)
    typename M::frag pf[M::PCH], xf[M::PCH];
    quad_frags(kTb + l32 * LDS_TROW + 32 * u, g, xf);
    acc_frags(dp, pf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) xt = M::mma(xf[t], pf[t], xt);
    acc_frags(s, pf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) yt = M::mma(xf[t], pf[t], yt);
  };

  PairPiece<T> kp;
  RowPiece<T> vp;
  uint64_t bb = block_bits(kb, G.nkt, 0);
  kp.load(kr, G.sPos, 0, last, tid);
  vp.load(vr, G.sPos, 0, last, tid);
  f32x16 bA0 = bias_tile(0), bA1 = bias_tile(1), bB0, bB1;
  kp.validate(tid, bb);
  kp.store_rows(ks, tid);
  kp.store_trans(kT, tid);
  vp.store(vs, tid, bb);
  __syncthreads();
  auto step = [&](int b, const f32x16& c0, const f32x16& c1, f32x16& n0, f32x16& n1) {
    const int bn = min(b + 1, nblk - 1);
    const uint64_t bbn = block_bits(kb, G.nkt, bn);
    kp.load(kr, G.sPos, bn * SPAN, last, tid);
    vp.load(vr, G.sPos, bn * SPAN, last, tid);
    n0 = bias_tile(2 * bn);
    n1 = bias_tile(2 * bn + 1);
    const int buf = b & 1;
    if (active) {
      const T* ksb = ks + buf * ROW_TILE;
      const T* kTb = kT + buf * TRANS_TILE;
      const T* vsb = vs + buf * ROW_TILE;
      if ((uint32_t)bb) sub_tile(ksb, kTb, vsb, c0, (uint32_t)bb, 0);
      if ((uint32_t)(bb >> 32)) sub_tile(ksb, kTb, vsb, c1, (uint32_t)(bb >> 32), 1);
    }
    if (b + 1 < nblk) {
      kp.validate(tid, bbn);
      kp.store_rows(ks + (buf ^ 1) * ROW_TILE, tid);
      kp.store_trans(kT + (buf ^ 1) * TRANS_TILE, tid);
      vp.store(vs + (buf ^ 1) * ROW_TILE, tid, bbn);
    }
    __syncthreads();
    bb = bbn;
  };
  for (int b = 0; b < nblk; b += 2) {
    step(b, bA0, bA1, bB0, bB1);
    if (b + 1 >= nblk) break;
    step(b + 1, bB0, bB1, bA0, bA1);
  }
  if (!active) return;
  const float dsum = wave_xor32_sum(dpart);
  if (!qok) return;
  if (g == 0) a.dsum[((int64_t)h * G.n + r) * G.np + q] = -dsum;  // stored negated
  const int64_t base = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f32x4 x;
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = (xt[4 * j + e] - dsum * yt[4 * j + e]) * G.scale;
    store4(a.dq + base + 8 * j + 4 * g, x);
  }
}

// bf16 dQ (and D) with asynchronous LDS staging (see dma.h).  One workgroup
// = 4 waves = 64 queries x 2 rows of one head: wave w owns query tile w % 2
// (lane <-> query) of row r0 + w / 2.  Keys stream in blocks of 32; per
// block, K and V of both rows and the query-major bias tiles of the 64
// queries (shared by the two rows) are copied HBM -> LDS by DMA into a ring
// of QD_SLOTS slots.  K^T fragments for the dQ products come from the
// transposing LDS read of the row-major K block.
constexpr int QD_BLK = 32 * 64;                     // 2 KB: 32 keys x 32 channels
constexpr int QD_K = 0, QD_V = 2 * QD_BLK;          // [row] blocks
constexpr int QD_BIAS = 4 * QD_BLK;                 // 2 query tiles x 4 KB
constexpr int QD_SLOT = QD_BIAS + 2 * 4096;
// Two slots (32 KB) let four workgroups share a CU, four waves per SIMD
// (measured 0.73 ms against 0.81-0.85 ms with three slots and three waves
// per SIMD at N = 768).
constexpr int QD_SLOTS = 2;
constexpr int QD_OPS = 4;                           // DMA ops per thread per block

__global__ __launch_bounds__(256, 4) void dq_dma_kernel(BwdArgs<bf16> a, int nqb) {
  using M = Mma<bf16>;
  using F = bf16x8;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nrg = (G.n + 1) / 2;
  const int qb = w % nqb, rg = (w / nqb) % nrg, h = w / (nqb * nrg);
  const int r0 = rg * 2;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qtl = wave & 1, ri = wave >> 1;
  const int r = min(r0 + ri, G.n - 1);
  const bool rok = r0 + ri < G.n;
  const int q0 = qb * 64 + qtl * TILE;
  const int q = q0 + l32;
  const bool active = rok && q0 < G.n;
  const bool qok = q < G.n;
  const int nkt = G.nkt, last = G.n - 1;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[QD_SLOTS * QD_SLOT];

  // ---- this lane's query: Q, dA (hi, lo) fragments and lse2
  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
  F qf[M::KCH], daf[M::KCH], dalf[M::KCH];
  float l2 = pos_inf();
  if (qok) {
    row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
    row_frags(a.da + rowbase + (int64_t)q * G.sPos, g, daf);
    row_frags(a.dalo + rowbase + (int64_t)q * G.sPos, g, dalf);
    l2 = a.lse2[((int64_t)h * G.n + r) * G.np + q];
  } else {
    zero_frags<bf16>(qf);
    zero_frags<bf16>(daf);
    zero_frags<bf16>(dalf);
  }
  // plain register loads: let them complete before any DMA is issued (with
  // both kinds outstanding the compiler would wait for every DMA at each use)
  wait_vm<0>();

  // ---- DMA lanes.  Ops 0, 1: K, V of both rows (wave w: row w / 2,
  // positions 16 (w % 2) + lane / 4).  Ops 2, 3: bias tile j of the 64
  // queries, quarter w.
  const int dri = wave >> 1;
  const int dp = 16 * (wave & 1) + (lane >> 2), dc = (lane & 3) ^ swz(dp);
  const int64_t drb = (int64_t)min(r0 + dri, last) * G.sRow + (int64_t)h * HEAD_DIM + 8 * dc;
  auto issue = [&](int t, int slot) {
    char* sl = smem + slot * QD_SLOT;
    const int64_t o = drb + (int64_t)min(t * TILE + dp, last) * G.sPos;
    dma16(a.k + o, sl + QD_K + dri * QD_BLK + 1024 * (wave & 1));
    dma16(a.v + o, sl + QD_V + dri * QD_BLK + 1024 * (wave & 1));
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const float* bsrc = frag_tile(a.bt, h, min(qb * 2 + j, nkt - 1), t, nkt);
      dma16((const char*)bsrc + 1024 * wave + 16 * lane, sl + QD_BIAS + j * 4096 + 1024 * wave);
    }
  };

  // ---- LDS read addresses (slot 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t rk0 = base + ri * QD_BLK + l32 * 64 + 16 * (g ^ sw);
  const uint32_t rk1 = base + ri * QD_BLK + l32 * 64 + 16 * ((2 + g) ^ sw);
  const TrAddr ta(lane);
  const uint32_t rtr = base + QD_K + ri * QD_BLK + ta.off(0);
  const uint32_t rtr8 = base + QD_K + ri * QD_BLK + ta.off(8) - 8 * 64;
  const uint32_t rb = base + QD_BIAS + qtl * 4096 + lane * 16;

  f32x16 xt = {}, yt = {};
  float dpart = 0.f;

#pragma unroll
  for (int j = 0; j < QD_SLOTS - 1; ++j) issue(min(j, nkt - 1), j);
  for (int t = 0; t < nkt; ++t) {
    const uint32_t so = (t % QD_SLOTS) * QD_SLOT;
    wait_vm<(QD_SLOTS - 2) * QD_OPS>();  // block t has landed
    lds_barrier();
    // key bits of both rows: the same in every wave, so the branch below (it
    // holds a barrier) is uniform across the workgroup
    const uint32_t w0 = const_load(a.kbits + (int64_t)r0 * nkt + t);
    const uint32_t w1 = r0 + 1 < G.n ? const_load(a.kbits + (int64_t)(r0 + 1) * nkt + t) : 0u;
    if ((w0 & (r0 + 1 < G.n ? w1 : 0xffffffffu)) != 0xffffffffu) {
      // zero V rows of keys invalid for a row (P = 0 there, and 0 times a
      // non-finite dP would not be); thread t < 128: row t / 64, key t / 2 % 32
      if (tid < 128) {
        const uint32_t wb = (tid >> 6) ? w1 : w0;
        if (!((wb >> ((tid >> 1) & 31)) & 1u))
          *(f32x4*)(smem + so + QD_V + 32 * tid) = f32x4{},
                   *(f32x4*)(smem + so + QD_V + 32 * tid + 16) = f32x4{};
      }
      __syncthreads();
    }
    // block t + QD_SLOTS - 1 into the slot of block t - 1
    issue(min(t + QD_SLOTS - 1, nkt - 1), (t + QD_SLOTS - 1) % QD_SLOTS);
    const uint32_t bits = ri ? w1 : w0;
    if (!active || bits == 0u) continue;
    // S^T = bias + K Q^T (lane <-> query, registers <-> keys)
    f32x16 sv;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 y = lds_load16<f32x4>(rb + so + 1024 * j);
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[4 * j + e] = y[e];
    }
    {
      const F k0 = lds_load16<F>(rk0 + so + QD_K), k1 = lds_load16<F>(rk1 + so + QD_K);
      sv = M::mma(k1, qf[1], M::mma(k0, qf[0], sv));
    }
    if (bits != 0xffffffffu) mask_rows(sv, bits, g);
#pragma unroll
    for (int v = 0; v < 16; ++v) sv[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2));
    // dP^T = V dA^T (hi and lo parts), then P dP and its running sum D
    f32x16 dp;
    {
      const F v0 = lds_load16<F>(rk0 + so + QD_V), v1 = lds_load16<F>(rk1 + so + QD_V);
      dp = M::mma(v0, daf[0], f32x16{});
      dp = M::mma(v1, daf[1], dp);
      dp = M::mma(v0, dalf[0], dp);
      dp = M::mma(v1, dalf[1], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      dp[v] *= sv[v];
      dpart += dp[v];
    }
    // X^T += K^T (P dP)^T,  Y^T += K^T P^T (contraction over the block's keys)
    const uint32_t tk = rtr + so, tk8 = rtr8 + so;
    s16x4 xk[4];
    xk[0] = ds_read_tr<0>(tk);
    xk[1] = ds_read_tr<8 * 64>(tk8);
    xk[2] = ds_read_tr<16 * 64>(tk);
    xk[3] = ds_read_tr<24 * 64>(tk8);
    F pf[M::PCH], xf[M::PCH];
    acc_frags(dp, xf);
    acc_frags(sv, pf);
    tr_wait(xk);
#pragma unroll
    for (int u = 0; u < M::PCH; ++u) {
      xt = M::mma(tr_frag(xk, u), xf[u], xt);
      yt = M::mma(tr_frag(xk, u), pf[u], yt);
    }
  }
  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active) return;
  const float dsum = wave_xor32_sum(dpart);
  if (!qok) return;
  if (g == 0) a.dsum[((int64_t)h * G.n + r) * G.np + q] = -dsum;  // stored negated
  const int64_t gb = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f32x4 x;
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = (xt[4 * j + e] - dsum * yt[4 * j + e]) * G.scale;
    store4(a.dq + gb + 8 * j + 4 * g, x);
  }
}

// ---- dK, dV --------------------------------------------------------------------------

// Per (row, head, 128 keys; wave <-> 32 keys, lane <-> key): stream the row's
// queries in blocks of 64 (Q, Q^T, dA, dA^T, the low part of dA, lse2 and -D
// staged in LDS, double-buffered).  The paper's first backward stage.
template <typename T>
__global__ __launch_bounds__(256, 2) void dkdv_kernel(BwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int kbk = w % a.nblk, rh = w / a.nblk;
  const int r = rh % G.n, h = rh / G.n;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int kt = kbk * BWD_WAVES + wave;  // this wave's key tile
  const bool active = kt < G.nkt;
  const uint32_t bits = active ? a.kbits[(int64_t)r * G.nkt + kt] : 0u;
  const int key = kt * TILE + l32;
  const bool kvalid = (bits >> l32) & 1u;
  const bool work = bits != 0u;  // some key of this wave is valid for the row

  __shared__ __align__(16) T qs[2 * ROW_TILE];      // Q    [query][channel]
  __shared__ __align__(16) T qT[2 * TRANS_TILE];    // Q^T  [channel][query]
  __shared__ __align__(16) T das[2 * ROW_TILE];     // dA
  __shared__ __align__(16) T daT[2 * TRANS_TILE];   // dA^T
  __shared__ __align__(16) T dals[kSplitDA<T> ? 2 * ROW_TILE : 1];  // low part of dA
  __shared__ __align__(16) float l2s[2 * SPAN];     // lse2 of the block's queries
  __shared__ __align__(16) float nds[2 * SPAN];     // -D of the block's queries

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
  const T* qr = a.q + rowbase;
  const T* dar = a.da + rowbase;
  const T* dalr = kSplitDA<T> ? a.dalo + rowbase : nullptr;
  const int last = G.n - 1;
  typename M::frag kf[M::KCH], vf[M::KCH];
  if (kvalid) {
    row_frags(a.k + rowbase + (int64_t)key * G.sPos, g, kf);
    row_frags(a.v + rowbase + (int64_t)key * G.sPos, g, vf);
  } else {
    zero_frags<T>(kf);
    zero_frags<T>(vf);
  }
  const float c1 = G.scale * LOG2E;
  f32x16 dkt = {}, dvt = {};
  const int ktc = active ? kt : 0;  // key tile of the key-major bias (0 for idle waves)
  const float* l2row = a.lse2 + ((int64_t)h * G.n + r) * G.np;
  const float* drow = a.dsum + ((int64_t)h * G.n + r) * G.np;
  const int nblk = (G.nkt + 1) >> 1;  // query blocks of 64
  const float kmask = kvalid ? 0.f : neg_inf();
  auto bias_tile = [&](int t) {
    f32x16 x = load_frag_tile(frag_tile(a.btT, h, ktc, min(t, G.nkt - 1), G.nkt), lane);
#pragma unroll
    for (int v = 0; v < 16; ++v) x[v] += kmask;  // -inf for a masked key
    return x;
  };

  PairPiece<T> qp, dap;
  RowPiece<T> dlp;
  float sv = 0.f;  // thread < 64: lse2 of query tid; 64 <= thread < 128: -D of query tid-64
  const int sq = tid & 63;
  auto load_block = [&](int b) {
    qp.load(qr, G.sPos, b * SPAN, last, tid);
    dap.load(dar, G.sPos, b * SPAN, last, tid);
    if constexpr (kSplitDA<T>) dlp.load(dalr, G.sPos, b * SPAN, last, tid);
    const int qi = min(b * SPAN + sq, G.np - 1);
    sv = tid < SPAN ? l2row[qi] : drow[qi];
  };
  auto store_block = [&](int b, int bf) {
    const uint64_t vb = range_bits64(b * SPAN, G.n);
    qp.validate(tid, vb);
    dap.validate(tid, vb);
    qp.store_rows(qs + bf * ROW_TILE, tid);
    qp.store_trans(qT + bf * TRANS_TILE, tid);
    dap.store_rows(das + bf * ROW_TILE, tid);
    dap.store_trans(daT + bf * TRANS_TILE, tid);
    if constexpr (kSplitDA<T>) dlp.store(dals + bf * ROW_TILE, tid, vb);
    const bool in = b * SPAN + sq < G.np;  // queries n..np-1 carry +inf / 0 already
    if (tid < SPAN)
      l2s[bf * SPAN + sq] = in ? sv : pos_inf();
    else if (tid < 2 * SPAN)
      nds[bf * SPAN + sq] = in ? sv : 0.f;
  };
  auto sub_tile = [&](int bf, const f32x16& bias, int u) {
    const T* qsb = qs + bf * ROW_TILE;
    // S = bias + Q K^T (lane <-> key, registers <-> queries)
    typename M::frag af[M::KCH];
    row_frags(qsb + (32 * u + l32) * LDS_ROW, g, af);
    f32x16 s = M::mma(af[0], kf[0], bias);
#pragma unroll
    for (int t = 1; t < M::KCH; ++t) s = M::mma(af[t], kf[t], s);
    // P = exp2(S scale log2 e - lse2[query])
    const f32x16 l2 = load_quads(l2s + bf * SPAN + 32 * u + 4 * g);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2[v]));
    // dP - D = dA V^T - D, then dS = P (dP - D)
    row_frags(das + bf * ROW_TILE + (32 * u + l32) * LDS_ROW, g, af);
    f32x16 dp = M::mma(af[0], vf[0], load_quads(nds + bf * SPAN + 32 * u + 4 * g));
#pragma unroll
    for (int t = 1; t < M::KCH; ++t) dp = M::mma(af[t], vf[t], dp);
    if constexpr (kSplitDA<T>) {
      row_frags(dals + bf * ROW_TILE + (32 * u + l32) * LDS_ROW, g, af);
#pragma unroll
      for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], vf[t], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) dp[v] *= s[v];
    // dV^T += dA^T P,  dK^T += Q^T dS (contraction over the block's queries)
    typename M::frag pf[M::PCH], xf[M::PCH];
    acc_frags(s, pf);
    quad_frags(daT + bf * TRANS_TILE + l32 * LDS_TROW + 32 * u, g, xf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) dvt = M::mma(xf[t], pf[t], dvt);
    acc_frags(dp, pf);
    quad_frags(qT + bf * TRANS_TILE + l32 * LDS_TROW + 32 * u, g, xf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) dkt = M::mma(xf[t], pf[t], dkt);
  };

  load_block(0);
  f32x16 bA0 = bias_tile(0), bA1 = bias_tile(1), bB0, bB1;
  store_block(0, 0);
  __syncthreads();
  auto step = [&](int b, const f32x16& c0, const f32x16& c1, f32x16& n0, f32x16& n1) {
    const int bn = min(b + 1, nblk - 1);
    load_block(bn);
    n0 = bias_tile(2 * bn);
    n1 = bias_tile(2 * bn + 1);
    const int buf = b & 1;
    if (work) {
      sub_tile(buf, c0, 0);
      if (2 * b + 1 < G.nkt) sub_tile(buf, c1, 1);
    }
    if (b + 1 < nblk) store_block(bn, buf ^ 1);
    __syncthreads();
  };
  for (int b = 0; b < nblk; b += 2) {
    step(b, bA0, bA1, bB0, bB1);
    if (b + 1 >= nblk) break;
    step(b + 1, bB0, bB1, bA0, bA1);
  }
  if (!active || key >= G.n) return;
  const int64_t base = rowbase + (int64_t)key * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c0 = 8 * j + 4 * g;
    f32x4 x, y;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = dvt[4 * j + e];
      y[e] = dkt[4 * j + e] * G.scale;
    }
    store4(a.dv + base + c0, x);
    store4(a.dk + base + c0, y);
  }
}

// bf16 dK, dV with asynchronous LDS staging (see dma.h).  One workgroup =
// 8 waves = 128 keys x 2 rows of one head: wave w owns key tile w % 4 of
// the block (lane <-> key) in row r0 + w / 4.  Queries stream in blocks of
// 32; per block, Q, dA and its low part of both rows, their lse2 and D, and
// the key-major bias tiles of the 128 keys (shared by the two rows) are
// copied HBM -> LDS by DMA into a ring of KD_SLOTS slots.  Q^T and dA^T
// fragments come from the transposing LDS read of the same row-major
// blocks.
constexpr int KD_ROWS = 2;
constexpr int KD_BLK = 32 * 64;                        // 2 KB: 32 positions x 32 channels
constexpr int KD_Q = 0, KD_DA = 2 * KD_BLK, KD_LO = 4 * KD_BLK;  // [row] blocks
constexpr int KD_BIAS = 6 * KD_BLK;                    // 4 key tiles x 4 KB
constexpr int KD_L2 = KD_BIAS + 4 * 4096;              // lse2 [row][32], then -D [row][32]
constexpr int KD_SLOT = KD_L2 + 4 * 128;
// Ring depth (blocks in flight + 1).  Two slots (58 KB) let two workgroups
// share a CU: four waves per SIMD hide more latency than a deeper ring with
// two (measured: 0.82 ms against 0.98-1.07 ms with four slots at N = 768).
constexpr int KD_SLOTS = 2;
constexpr int KD_OPS = 4;    // DMA ops per thread per block

__global__ __launch_bounds__(512, KD_SLOTS <= 2 ? 2 : 1) void dkdv_dma_kernel(BwdArgs<bf16> a) {
  using M = Mma<bf16>;
  using F = bf16x8;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nrg = (G.n + KD_ROWS - 1) / KD_ROWS;
  const int kbk = w % a.nblk, rg = (w / a.nblk) % nrg, h = w / (a.nblk * nrg);
  const int r0 = rg * KD_ROWS;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ri = wave >> 2;                 // row of this wave (0, 1)
  const int r = min(r0 + ri, G.n - 1);
  const bool rok = r0 + ri < G.n;
  const int kt = kbk * 4 + (wave & 3);      // this wave's key tile
  const int nkt = G.nkt, last = G.n - 1;
  const bool active = rok && kt < nkt;
  const uint32_t bits = active ? const_load(a.kbits + (int64_t)r * nkt + kt) : 0u;
  const int key = kt * TILE + l32;
  const bool kvalid = (bits >> l32) & 1u;
  const bool work = bits != 0u;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[KD_SLOTS * KD_SLOT];

  // ---- the wave's keys: K and V fragments (zero for invalid keys, so that
  // non-finite values there cannot reach the products)
  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
  F kf[M::KCH], vf[M::KCH];
  if (kvalid) {
    row_frags(a.k + rowbase + (int64_t)key * G.sPos, g, kf);
    row_frags(a.v + rowbase + (int64_t)key * G.sPos, g, vf);
  } else {
    zero_frags<bf16>(kf);
    zero_frags<bf16>(vf);
  }
  // the fragments are plain register loads: let them complete before any
  // DMA is issued (with both kinds outstanding the compiler would wait for
  // every DMA at each use)
  wait_vm<0>();

  // ---- DMA lanes.  Op 0: Q and dA of both rows (wave w: block w / 2 of
  // [Q0, Q1, dA0, dA1], positions 16 (w % 2) + lane / 4).  Op 1: waves 0-3
  // the low part of dA, waves 4-7 lse2 / -D (lanes 0..7, 128 bytes each).
  // Ops 2, 3: bias tiles 4 KB each, wave w: tile 2 (op - 2) + w / 4,
  // quarter w % 4.
  const int dpl = 16 * (wave & 1) + (lane >> 2);
  int64_t drow[KD_ROWS];
#pragma unroll
  for (int i = 0; i < KD_ROWS; ++i)
    drow[i] = (int64_t)min(r0 + i, last) * G.sRow + (int64_t)h * HEAD_DIM;
  const int b0 = wave >> 1;  // op 0 block: 0 Q0, 1 Q1, 2 dA0, 3 dA1
  const bf16* src0 = b0 < 2 ? a.q : a.da;
  const int64_t row0 = (b0 & 1) ? drow[1] : drow[0];
  const int64_t row1 = (wave >> 1 & 1) ? drow[1] : drow[0];  // op 1 (waves 0-3): dalo row
  const int lrow = min(r0 + (wave & 1), last);                // op 1 (waves 4-7): lse2 / -D row
  const float* lsrc = (wave & 2) ? a.dsum : a.lse2;
  auto issue = [&](int t, int slot) {
    char* sl = smem + slot * KD_SLOT;
    const int p = min(t * TILE + dpl, last);
    const int c = (lane & 3) ^ swz(dpl);
    dma16(src0 + row0 + (int64_t)p * G.sPos + 8 * c, sl + b0 * KD_BLK + 1024 * (wave & 1));
    if (wave < 4) {
      dma16(a.dalo + row1 + (int64_t)p * G.sPos + 8 * c,
            sl + KD_LO + (wave >> 1) * KD_BLK + 1024 * (wave & 1));
    } else if (lane < 8) {
      dma16(lsrc + ((int64_t)h * G.n + lrow) * G.np + t * TILE + 4 * lane,
            sl + KD_L2 + 128 * (wave - 4));
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int tl = 2 * j + (wave >> 2);
      const float* bsrc = frag_tile(a.btT, h, min(kbk * 4 + tl, nkt - 1), t, nkt);
      dma16((const char*)bsrc + 1024 * (wave & 3) + 16 * lane,
            sl + KD_BIAS + tl * 4096 + 1024 * (wave & 3));
    }
  };

  // ---- LDS read addresses (slot 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t rq0 = base + ri * KD_BLK + l32 * 64 + 16 * (g ^ sw);
  const uint32_t rq1 = base + ri * KD_BLK + l32 * 64 + 16 * ((2 + g) ^ sw);
  const TrAddr ta(lane);
  const uint32_t rtr = base + ri * KD_BLK + ta.off(0);
  const uint32_t rtr8 = base + ri * KD_BLK + ta.off(8) - 8 * 64;
  const uint32_t rb = base + KD_BIAS + (wave & 3) * 4096 + lane * 16;
  const uint32_t rl = base + KD_L2 + ri * 128 + 16 * g;  // + 32 j: lse2 quad j; + 256: D

  f32x16 dkt = {}, dvt = {};
  const float kmask = kvalid ? 0.f : neg_inf();
  auto quads = [&](uint32_t at) {
    f32x16 x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 y = lds_load16<f32x4>(at + 32 * j);
#pragma unroll
      for (int e = 0; e < 4; ++e) x[4 * j + e] = y[e];
    }
    return x;
  };

#pragma unroll
  for (int j = 0; j < KD_SLOTS - 1; ++j) issue(min(j, nkt - 1), j);
  for (int t = 0; t < nkt; ++t) {
    const uint32_t so = (t % KD_SLOTS) * KD_SLOT;
    // block t has landed (the KD_SLOTS - 2 blocks after it may be in flight)
    wait_vm<(KD_SLOTS - 2) * KD_OPS>();
    lds_barrier();
    // block t + KD_SLOTS - 1 into the slot of block t - 1 (a copy of the last
    // block past the end keeps the wait counts uniform)
    issue(min(t + KD_SLOTS - 1, nkt - 1), (t + KD_SLOTS - 1) % KD_SLOTS);
    if (!work) continue;
    // S = bias + Q K^T (registers <-> queries, lane <-> key)
    f32x16 sv;
    {
      f32x16 bias;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 y = lds_load16<f32x4>(rb + so + 1024 * j);
#pragma unroll
        for (int e = 0; e < 4; ++e) bias[4 * j + e] = y[e];
      }
      if (bits != 0xffffffffu) {
#pragma unroll
        for (int v = 0; v < 16; ++v) bias[v] += kmask;  // -inf for an invalid key
      }
      const F q0 = lds_load16<F>(rq0 + so + KD_Q), q1 = lds_load16<F>(rq1 + so + KD_Q);
      sv = M::mma(q1, kf[1], M::mma(q0, kf[0], bias));
    }
    // P = exp2(S c1 - lse2[query])
    const f32x16 l2 = quads(rl + so);
#pragma unroll
    for (int v = 0; v < 16; ++v) sv[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2[v]));
    // dP - D = dA V^T - D (hi and lo parts of dA), then dS = P (dP - D)
    const F d0 = lds_load16<F>(rq0 + so + KD_DA), d1 = lds_load16<F>(rq1 + so + KD_DA);
    const F e0 = lds_load16<F>(rq0 + so + KD_LO), e1 = lds_load16<F>(rq1 + so + KD_LO);
    f32x16 dp = quads(rl + so + 256);  // -D
    dp = M::mma(d0, vf[0], dp);
    dp = M::mma(d1, vf[1], dp);
    dp = M::mma(e0, vf[0], dp);
    dp = M::mma(e1, vf[1], dp);
#pragma unroll
    for (int v = 0; v < 16; ++v) dp[v] *= sv[v];
    // dV^T += dA^T P,  dK^T += Q^T dS (contraction over the block's queries)
    const uint32_t tq = rtr + so + KD_Q, td = rtr + so + KD_DA;
    const uint32_t tq8 = rtr8 + so + KD_Q, td8 = rtr8 + so + KD_DA;
    s16x4 xa[4], xq[4];
    xa[0] = ds_read_tr<0>(td);
    xa[1] = ds_read_tr<8 * 64>(td8);
    xa[2] = ds_read_tr<16 * 64>(td);
    xa[3] = ds_read_tr<24 * 64>(td8);
    xq[0] = ds_read_tr<0>(tq);
    xq[1] = ds_read_tr<8 * 64>(tq8);
    xq[2] = ds_read_tr<16 * 64>(tq);
    xq[3] = ds_read_tr<24 * 64>(tq8);
    F pf[M::PCH], sf[M::PCH];
    acc_frags(sv, pf);
    acc_frags(dp, sf);
    tr_wait(xa);
    tr_wait(xq);
#pragma unroll
    for (int u = 0; u < M::PCH; ++u) {
      dvt = M::mma(tr_frag(xa, u), pf[u], dvt);
      dkt = M::mma(tr_frag(xq, u), sf[u], dkt);
    }
  }
  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active || key >= G.n) return;
  const int64_t gb = rowbase + (int64_t)key * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c0 = 8 * j + 4 * g;
    f32x4 x, y;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = dvt[4 * j + e];
      y[e] = dkt[4 * j + e] * G.scale;
    }
    store4(a.dv + gb + c0, x);
    store4(a.dk + gb + c0, y);
  }
}

// ---- dBias ---------------------------------------------------------------------------

constexpr int DB_WAVES = 8;  // 4 query tiles x 2 key halves
constexpr int DB_ROWS = 2 * SPAN;  // keys (and queries) per workgroup block

// One workgroup: 128 queries x 128 keys of one head, summed over the rows of
// one row chunk.  Wave w owns query tile w % 4 (lane <-> query) and key tiles
// 2 (w / 4), 2 (w / 4) + 1.  Per row, K and V of the 128 keys and Q, dA (and
// its low part), lse2 and -D of the 128 queries are loaded with coalesced
// 16-byte pieces (issued before the previous row's compute) and staged in
// LDS.  The bias tiles stay in registers for all rows.
template <typename T>
__global__ __launch_bounds__(512, 1) void db_kernel(BwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int kbk = w % a.nblk;
  const int qb = (w / a.nblk) % a.nblk;
  const int rc = (w / (a.nblk * a.nblk)) % a.nrc;
  const int h = w / (a.nblk * a.nblk * a.nrc);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int qw = (wave & 3) * TILE;  // this wave's queries within the block
  const int q0 = qb * DB_ROWS + qw;
  const int kh = wave >> 2;  // key half of the block
  const bool active = q0 < G.n;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) T ks[2 * ROW_TILE];   // K  [key][channel] of the 128 keys
  __shared__ __align__(16) T vs[2 * ROW_TILE];   // V
  __shared__ __align__(16) T qs[2 * ROW_TILE];   // Q  [query][channel] of the 128 queries
  __shared__ __align__(16) T das[2 * ROW_TILE];  // dA
  __shared__ __align__(16) T dals[kSplitDA<T> ? 2 * ROW_TILE : 1];
  __shared__ __align__(16) float l2s[DB_ROWS];   // lse2 of the queries (+inf: none valid)
  __shared__ __align__(16) float nds[DB_ROWS];   // -D

  const int kt0 = kbk * BWD_WAVES;  // first key tile of the block
  const int kstart = kt0 * TILE, qstart = qb * DB_ROWS;
  const int last = G.n - 1;
  f32x16 binit[2], acc[2];
  const int qt = active ? q0 / TILE : 0;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    acc[u] = f32x16{};
    binit[u] =
        load_frag_tile(frag_tile(a.bt, h, qt, min(kt0 + 2 * kh + u, G.nkt - 1), G.nkt), lane);
  }
  auto row_bits = [&](int r, int half) -> uint64_t {
    return block_bits(a.kbits + (int64_t)r * G.nkt, G.nkt, (kt0 >> 1) + half);
  };
  const int r0 = rc * a.rpc, r1 = min(G.n, r0 + a.rpc);

  // thread -> (half of the 128 positions, piece index within the half)
  const int half = tid >> 8, pt = tid & 255;
  const uint64_t qvalid = range_bits64(qstart + SPAN * half, G.n);
  RowPiece<T> kp, vp, qp, dap, dlp;
  float sv = 0.f;  // thread < 128: lse2 of query tid; 128 <= thread < 256: -D of query tid-128
  const int sq = min(qstart + (tid & 127), G.np - 1);
  auto load_row = [&](int r) {
    const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
    kp.load(a.k + rowbase, G.sPos, kstart + SPAN * half, last, pt);
    vp.load(a.v + rowbase, G.sPos, kstart + SPAN * half, last, pt);
    qp.load(a.q + rowbase, G.sPos, qstart + SPAN * half, last, pt);
    dap.load(a.da + rowbase, G.sPos, qstart + SPAN * half, last, pt);
    if constexpr (kSplitDA<T>) dlp.load(a.dalo + rowbase, G.sPos, qstart + SPAN * half, last, pt);
    const int64_t at = ((int64_t)h * G.n + r) * G.np + sq;
    sv = tid < DB_ROWS ? a.lse2[at] : a.dsum[at];
  };
  auto store_row = [&](int r) {
    const uint64_t kv = row_bits(r, half);
    kp.store(ks + half * ROW_TILE, pt, kv);
    vp.store(vs + half * ROW_TILE, pt, kv);
    qp.store(qs + half * ROW_TILE, pt, qvalid);
    dap.store(das + half * ROW_TILE, pt, qvalid);
    if constexpr (kSplitDA<T>) dlp.store(dals + half * ROW_TILE, pt, qvalid);
    const bool in = qstart + (tid & 127) < G.n;
    if (tid < DB_ROWS)
      l2s[tid] = in ? sv : pos_inf();
    else if (tid < 2 * DB_ROWS)
      nds[tid - DB_ROWS] = in ? sv : 0.f;
  };

  if (r0 < r1) {
    load_row(r0);
    store_row(r0);
  }
  __syncthreads();
  for (int r = r0; r < r1; ++r) {
    const uint64_t bb = row_bits(r, kh);  // this wave's two key tiles
    load_row(min(r + 1, r1 - 1));         // the last row reloads itself, unused
    const float l2 = l2s[qw + l32];
    if (active && bb != 0ull && !__all(l2 == pos_inf())) {
      typename M::frag qf[M::KCH], daf[M::KCH], dalf[M::KCH];
      row_frags(qs + (qw + l32) * LDS_ROW, g, qf);
      row_frags(das + (qw + l32) * LDS_ROW, g, daf);
      if constexpr (kSplitDA<T>) row_frags(dals + (qw + l32) * LDS_ROW, g, dalf);
      const f32x16 ndv = splat16(nds[qw + l32]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint32_t bits = (uint32_t)(bb >> (32 * u));
        if (bits == 0u) continue;
        const int off = (SPAN * kh + 32 * u + l32) * LDS_ROW;
        typename M::frag af[M::KCH];
        row_frags(ks + off, g, af);
        f32x16 s = M::mma(af[0], qf[0], binit[u]);
#pragma unroll
        for (int t = 1; t < M::KCH; ++t) s = M::mma(af[t], qf[t], s);
        if (bits != 0xffffffffu) mask_rows(s, bits, g);
        row_frags(vs + off, g, af);
        f32x16 dp = M::mma(af[0], daf[0], ndv);
#pragma unroll
        for (int t = 1; t < M::KCH; ++t) dp = M::mma(af[t], daf[t], dp);
        if constexpr (kSplitDA<T>) {
#pragma unroll
          for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], dalf[t], dp);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v)
          acc[u][v] += __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2)) * dp[v];
      }
    }
    __syncthreads();  // everyone is done with row r's tiles
    if (r + 1 < r1) store_row(r + 1);
    __syncthreads();
  }
  if (!active) return;
  float* slab = a.slabs + (((int64_t)rc * G.H + h) * G.np + q0 + l32) * G.np + 4 * g;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int kt = kt0 + 2 * kh + u;
    if (kt >= G.nkt) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = acc[u][4 * j + e];
      *(f32x4*)(slab + kt * TILE + 8 * j) = x;
    }
  }
}

// bf16 bias gradient with asynchronous LDS staging (see dma.h).  One
// workgroup: 128 queries x 64 keys of one head, summed over the rows of one
// row chunk; wave w owns query tile w % 4 (lane <-> query) and key tile
// w / 4 of the block.  Per row, K and V of the 64 keys and Q, dA, its low
// part, lse2 and -D of the 128 queries land in LDS by DMA through a ring of
// two slots (33 KB each), one row ahead; two workgroups share a CU (four
// waves per SIMD) to hide the latency of each wave's dependent MFMA and
// vector steps.
constexpr int DBD_Q = 128, DBD_K = 64;        // queries and keys per workgroup block
constexpr int DBD_KV = DBD_K * 64;            // 4 KB: K (or V) of the block's keys
constexpr int DBD_QB = DBD_Q * 64;            // 8 KB: Q (or dA, dA low) of the queries
constexpr int DBD_OK = 0, DBD_OV = DBD_KV, DBD_OQ = 2 * DBD_KV;
constexpr int DBD_ODA = DBD_OQ + DBD_QB, DBD_OLO = DBD_ODA + DBD_QB;
constexpr int DBD_LD = DBD_OLO + DBD_QB;      // lse2 [128], then -D [128]
constexpr int DBD_SLOT = DBD_LD + 1024;
constexpr int DBD_SLOTS = 2;
constexpr int DBD_OPS = 5;                    // DMA ops per thread per row

__global__ __launch_bounds__(512, 2) void db_dma_kernel(BwdArgs<bf16> a, int nkb) {
  using M = Mma<bf16>;
  using F = bf16x8;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int kbk = w % nkb;
  const int qb = (w / nkb) % a.nblk;
  const int rc = (w / (nkb * a.nblk)) % a.nrc;
  const int h = w / (nkb * a.nblk * a.nrc);
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qtl = wave & 3, ktl = wave >> 2;
  const int qstart = qb * DBD_Q, kstart = kbk * DBD_K;
  const int q = qstart + qtl * TILE + l32;  // this lane's query
  const int kt = kbk * 2 + ktl;             // this wave's key tile
  const bool active = qstart + qtl * TILE < G.n && kt < G.nkt;
  const bool qok = q < G.n;
  const int last = G.n - 1;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[DBD_SLOTS * DBD_SLOT];

  f32x16 binit, acc = {};
  {
    const int qt = active ? qstart / TILE + qtl : 0;
    binit = load_frag_tile(frag_tile(a.bt, h, qt, min(kt, G.nkt - 1), G.nkt), lane);
  }
  // the bias tile is a plain register load: let it complete before any DMA
  // is issued (with both kinds outstanding the compiler would wait for every
  // DMA at each use of binit)
  wait_vm<0>();

  // ---- DMA lanes.  Op 0: K (waves 0-3) and V (waves 4-7) of the 64 keys,
  // wave w % 4 moving positions 16 (w % 4) + lane / 4.  Ops 1-3: Q, dA, dA
  // low of the 128 queries, position tid / 4.  Op 4: lse2 (waves 0-3) and
  // -D (waves 4-7), 128 bytes per wave (lanes 0..7).
  const int hb = h * HEAD_DIM;
  const int kp = 16 * (wave & 3) + (lane >> 2), kc = (lane & 3) ^ swz(kp);
  const int64_t kofs = (int64_t)min(kstart + kp, last) * G.sPos + 8 * kc + hb;
  const bf16* kvsrc = wave < 4 ? a.k : a.v;
  const int qp = tid >> 2, qc = (tid & 3) ^ swz(qp);
  const int64_t qofs = (int64_t)min(qstart + qp, last) * G.sPos + 8 * qc + hb;
  const int lq = min(qstart + 32 * (wave & 3) + 4 * lane, G.np - 4);
  const float* ldsrc = wave < 4 ? a.lse2 : a.dsum;
  auto issue = [&](int r, int slot) {
    char* sl = smem + slot * DBD_SLOT;
    const int64_t rb = (int64_t)r * G.sRow;
    dma16(kvsrc + rb + kofs, sl + (wave < 4 ? DBD_OK : DBD_OV) + 1024 * (wave & 3));
    dma16(a.q + rb + qofs, sl + DBD_OQ + 1024 * wave);
    dma16(a.da + rb + qofs, sl + DBD_ODA + 1024 * wave);
    dma16(a.dalo + rb + qofs, sl + DBD_OLO + 1024 * wave);
    if (lane < 8)
      dma16(ldsrc + ((int64_t)h * G.n + r) * G.np + lq, sl + DBD_LD + 128 * wave);
  };

  // ---- LDS read addresses (slot 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t qpos = base + (uint32_t)(qtl * TILE + l32) * 64;
  const uint32_t rq0 = qpos + 16 * (g ^ sw), rq1 = qpos + 16 * ((2 + g) ^ sw);
  const uint32_t kpos = base + (uint32_t)(ktl * TILE + l32) * 64;
  const uint32_t rk0 = kpos + 16 * (g ^ sw), rk1 = kpos + 16 * ((2 + g) ^ sw);
  const uint32_t rl = base + DBD_LD + (qtl * TILE + l32) * 4;

  const int r0 = rc * a.rpc, r1 = min(G.n, r0 + a.rpc);
  const int nr = r1 - r0;
  const int nkt = G.nkt;
  auto kword = [&](int r, int t) -> uint32_t {
    return t < nkt ? const_load(a.kbits + (int64_t)r * nkt + t) : 0u;
  };

  if (nr > 0) issue(r0, 0);
  for (int i = 0; i < nr; ++i) {
    const int r = r0 + i;
    const uint32_t so = (i % DBD_SLOTS) * DBD_SLOT;
    wait_vm<(DBD_SLOTS - 2) * DBD_OPS>();  // row r has landed
    lds_barrier();
    const uint32_t w0 = kword(r, kbk * 2), w1 = kword(r, kbk * 2 + 1);
    if ((w0 & w1) != 0xffffffffu) {
      // zero V rows of keys invalid for the row (P = 0 there, and 0 times a
      // non-finite dP would not be); thread t < 256: key t / 4, 16 bytes
      if (tid < 256) {
        const uint32_t wb = (tid >> 7) ? w1 : w0;
        if (!((wb >> ((tid >> 2) & 31)) & 1u)) *(f32x4*)(smem + so + DBD_OV + 16 * tid) = f32x4{};
      }
      __syncthreads();
    }
    // row r + 1 into the other slot (a copy of the last row past the end
    // keeps the wait counts uniform)
    issue(r0 + min(i + DBD_SLOTS - 1, nr - 1), (i + DBD_SLOTS - 1) % DBD_SLOTS);
    const uint32_t bits = ktl ? w1 : w0;
    if (!active || bits == 0u) continue;
    float l2 = *(const TRIATTN_LDS float*)(uintptr_t)(rl + so);
    const float nd = *(const TRIATTN_LDS float*)(uintptr_t)(rl + so + 512);
    if (!qok) l2 = pos_inf();
    const F q0 = lds_load16<F>(rq0 + so + DBD_OQ), q1 = lds_load16<F>(rq1 + so + DBD_OQ);
    const F k0 = lds_load16<F>(rk0 + so + DBD_OK), k1 = lds_load16<F>(rk1 + so + DBD_OK);
    f32x16 sv = M::mma(k1, q1, M::mma(k0, q0, binit));  // S^T = bias + K Q^T
    if (bits != 0xffffffffu) mask_rows(sv, bits, g);
    const F d0 = lds_load16<F>(rq0 + so + DBD_ODA), d1 = lds_load16<F>(rq1 + so + DBD_ODA);
    const F e0 = lds_load16<F>(rq0 + so + DBD_OLO), e1 = lds_load16<F>(rq1 + so + DBD_OLO);
    const F v0 = lds_load16<F>(rk0 + so + DBD_OV), v1 = lds_load16<F>(rk1 + so + DBD_OV);
    f32x16 dpv = M::mma(v0, d0, splat16(nd));  // dP^T - D = V dA^T - D (hi and lo parts)
    dpv = M::mma(v1, d1, dpv);
    dpv = M::mma(v0, e0, dpv);
    dpv = M::mma(v1, e1, dpv);
#pragma unroll
    for (int v = 0; v < 16; ++v)
      acc[v] += __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2)) * dpv[v];
  }
  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active) return;
  float* slab = a.slabs + (((int64_t)rc * G.H + h) * G.np + qstart + qtl * TILE + l32) * G.np +
                kt * TILE + 4 * g;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f32x4 x;
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = acc[4 * j + e];
    *(f32x4*)(slab + 8 * j) = x;
  }
}

// dbias at (query q, key k, head h) = sum of the slabs in chunk order; the
// starting node stores it at [q][k][h], the ending node at [k][q][h].
template <typename T>
__global__ __launch_bounds__(256) void db_reduce_kernel(Geom G, int node, int nrc,
                                                        const float* slabs, T* dbias) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (h, q, k), k fastest
  const int64_t n = G.n;
  if (idx >= (int64_t)G.H * n * n) return;
  const int k = (int)(idx % n), q = (int)((idx / n) % n), h = (int)(idx / (n * n));
  const int64_t plane = (int64_t)G.np * G.np;
  const float* p = slabs + (int64_t)h * plane + (int64_t)q * G.np + k;
  float s = 0.f;
  for (int c = 0; c < nrc; ++c) s += p[(int64_t)c * G.H * plane];
  const int64_t at = node == 0 ? ((int64_t)q * n + k) * G.H + h : ((int64_t)k * n + q) * G.H + h;
  dbias[at] = (T)s;
}

template <typename T>
hipError_t launch_bwd(const Geom& g, int node, const Prep& p, const BwdWs& ws, const T* q,
                      const T* k, const T* v, const T* gate, const T* out, const float* lse,
                      const T* dout, T* dq, T* dk, T* dv, T* dg, T* dbias, hipStream_t s) {
  T* da = (T*)ws.da;
  T* dalo = (T*)ws.dalo;
  const int64_t npair = (int64_t)g.n * g.n * g.H;
  {
    KernelTimer t(K_BWD_PREP, s);
    hipLaunchKernelGGL(bwd_prep_kernel<T>, dim3((unsigned)((4 * npair + 255) / 256)), dim3(256),
                       0, s, g, node, out, lse, gate, dout, dg, da, dalo, ws.lse2);
  }
  if (g.np > g.n) {
    const int64_t npad = (int64_t)g.H * g.n * (g.np - g.n);
    KernelTimer t(K_BWD_PAD, s);
    hipLaunchKernelGGL(bwd_pad_kernel, dim3((unsigned)((npad + 255) / 256)), dim3(256), 0, s, g,
                       ws.lse2, ws.dsum);
  }
  BwdArgs<T> a{g, p.bt, p.btT, p.kbits, q, k, v, da, dalo, ws.lse2, ws.dsum, dq, dk, dv, ws.slabs,
               (g.n + BWD_BLK - 1) / BWD_BLK, ws.nrc, (g.n + ws.nrc - 1) / ws.nrc};
  const int64_t nrow = (int64_t)a.nblk * g.n * g.H;
  {
    // the dQ kernel first: it produces D for the other two
    KernelTimer t(K_DQ, s);
    if constexpr (std::is_same<T, bf16>::value) {
      const int nqb = (g.n + 63) / 64;
      const int64_t nwg = (int64_t)nqb * ((g.n + 1) / 2) * g.H;
      hipLaunchKernelGGL(dq_dma_kernel, dim3((unsigned)nwg), dim3(256), 0, s, a, nqb);
    } else {
      hipLaunchKernelGGL(dq_kernel<T>, dim3((unsigned)nrow), dim3(256), 0, s, a);
    }
  }
  {
    KernelTimer t(K_DKDV, s);
    if constexpr (std::is_same<T, bf16>::value) {
      const int64_t nwg = (int64_t)a.nblk * ((g.n + KD_ROWS - 1) / KD_ROWS) * g.H;
      hipLaunchKernelGGL(dkdv_dma_kernel, dim3((unsigned)nwg), dim3(512), 0, s, a);
    } else {
      hipLaunchKernelGGL(dkdv_kernel<T>, dim3((unsigned)nrow), dim3(256), 0, s, a);
    }
  }
  {
    const int64_t ndb = (int64_t)a.nblk * a.nblk * ws.nrc * g.H;
    KernelTimer t(K_DB, s);
    if constexpr (std::is_same<T, bf16>::value) {
      const int nkb = (g.n + DBD_K - 1) / DBD_K;
      const int64_t nwg = (int64_t)a.nblk * nkb * ws.nrc * g.H;
      hipLaunchKernelGGL(db_dma_kernel, dim3((unsigned)nwg), dim3(512), 0, s, a, nkb);
    } else
      hipLaunchKernelGGL(db_kernel<T>, dim3((unsigned)ndb), dim3(64 * DB_WAVES), 0, s, a);
  }
  {
    const int64_t nred = (int64_t)g.H * g.n * g.n;
    KernelTimer t(K_DB_REDUCE, s);
    hipLaunchKernelGGL(db_reduce_kernel<T>, dim3((unsigned)((nred + 255) / 256)), dim3(256), 0, s,
                       g, node, ws.nrc, ws.slabs, dbias);
  }
  return hipGetLastError();
}

template hipError_t launch_bwd<bf16>(const Geom&, int, const Prep&, const BwdWs&, const bf16*,
                                     const bf16*, const bf16*, const bf16*, const bf16*,
                                     const float*, const bf16*, bf16*, bf16*, bf16*, bf16*,
                                     bf16*, hipStream_t);
template hipError_t launch_bwd<float>(const Geom&, int, const Prep&, const BwdWs&, const float*,
                                      const float*, const float*, const float*, const float*,
                                      const float*, const float*, float*, float*, float*, float*,
                                      float*, hipStream_t);

}  // namespace triattn
