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
//              over query tiles: dV += P^T dA, dK += scale dS^T Q (in
//              dkdv.hip, launched from here).
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

#include "bwd.h"
#include "dma.h"
#include "kernels.h"
#include "stage.h"
#include "timing.h"

namespace triattn {

// ---- elementwise preparation -------------------------------------------------------

// Four threads per (pair, head) (two for D = 16): thread t handles channels
// 8 TPH c + 8 (t % TPH) .. +7 for c < NC, so every load and store is 16
// contiguous bytes (bf16) and a wave covers 16 (32) whole (pair, head) rows.  All of a thread's loads are
// issued before its first store (the compiler may not move loads past stores
// to memory that could alias them).  Grid: x over the (b, h) entries of one
// pair row a = blockIdx.y (all index arithmetic in 32 bits but the row
// offset).
template <typename T>
struct Vec8 {
  float x[8];
};
__device__ inline Vec8<bf16> load8(const bf16* p) {
  const bf16x8 v = *(const bf16x8*)p;
  Vec8<bf16> r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r.x[e] = (float)v[e];
  return r;
}
__device__ inline Vec8<float> load8(const float* p) {
  const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
  Vec8<float> r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    r.x[e] = a[e];
    r.x[4 + e] = b[e];
  }
  return r;
}
__device__ inline void store8(bf16* p, const float (&x)[8]) {
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (bf16)x[e];
  *(bf16x8*)p = v;
}
__device__ inline void store8(float* p, const float (&x)[8]) {
  *(f32x4*)p = f32x4{x[0], x[1], x[2], x[3]};
  *(f32x4*)(p + 4) = f32x4{x[4], x[5], x[6], x[7]};
}

template <typename T, int D = HEAD_DIM>
__global__ __launch_bounds__(256) void bwd_prep_kernel(Geom G, int node, const T* out,
                                                       const float* lse, const T* gate,
                                                       const T* dout, T* dg, T* da,
                                                       T* dalo, float* lse2) {
  out = at_sample(out, G.bPair);
  gate = at_sample(gate, G.bPair);
  dout = at_sample(dout, G.bPair);
  dg = at_sample(dg, G.bPair);
  lse = at_sample(lse, G.bBias);
  da = ws_at_sample(da, G.bWs);
  dalo = ws_at_sample(dalo, G.bWs);
  lse2 = ws_at_sample(lse2, G.bWs);
  constexpr int TPH = D == 16 ? 2 : 4;  // threads per (pair, head)
  constexpr int NC = D / (8 * TPH);     // 8-channel chunks per thread
  constexpr int CS = 8 * TPH;           // channel stride between a thread's chunks
  const uint32_t tix = blockIdx.x * 256u + threadIdx.x;
  const uint32_t in_row = tix / TPH;  // b * H + h
  if (in_row >= (uint32_t)(G.n * G.H)) return;
  const int pa = blockIdx.y;
  const int64_t idx = (int64_t)pa * (G.n * G.H) + in_row;  // (a, b, h)
  const int64_t base = idx * D + 8 * (tix % TPH);
  Vec8<T> go[NC], oo[NC], gg[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    go[c] = load8(dout + base + CS * c);
    oo[c] = load8(out + base + CS * c);
    gg[c] = load8(gate + base + CS * c);
  }
  const float l = tix % TPH == 0 ? lse[idx] : 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    float dgv[8], dav[8], lo[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float sg = fast_rcp(1.f + __expf(-gg[c].x[e]));  // as the forward's gate
      dgv[e] = go[c].x[e] * oo[c].x[e] * (1.f - sg);
      dav[e] = go[c].x[e] * sg;
      lo[e] = dav[e] - (float)(bf16)dav[e];
    }
    store8(dg + base + CS * c, dgv);
    store8(da + base + CS * c, dav);
    if constexpr (kSplitDA<T>) store8(dalo + base + CS * c, lo);
  }
  if (tix % TPH == 0) {
    const int b = (int)(in_row / (uint32_t)G.H), h = (int)(in_row - (uint32_t)b * G.H);
    const int row = node == 0 ? pa : b, qi = node == 0 ? b : pa;
    lse2[((int64_t)h * G.nr + row) * G.np + qi] = l == neg_inf() ? pos_inf() : l * LOG2E;
  }
}

// Queries n .. np-1 of every row: no valid key (+inf) and D = 0.
__global__ __launch_bounds__(256) void bwd_pad_kernel(Geom G, float* lse2, float* dsum) {
  lse2 = ws_at_sample(lse2, G.bWs);
  dsum = ws_at_sample(dsum, G.bWs);
  const int pad = G.np - G.n;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)G.H * G.nr * pad) return;
  const int64_t hr = idx / pad;
  const int64_t at = hr * G.np + G.n + (int)(idx % pad);
  lse2[at] = pos_inf();
  dsum[at] = 0.f;
}

// ---- dQ (and D) ----------------------------------------------------------------------

// Per (row, head, 128 queries): stream the row's keys in blocks of 64 (K, K^T
// and V staged in LDS, double-buffered).  dQ = scale (X - D Y) with
// X = sum_k P dP K, Y = sum_k P K and D = sum_k P dP, all from one pass.
template <typename T, int D>
__global__ __launch_bounds__(256, 2) void dq_kernel(BwdArgs<T> a) {
  to_sample(a);
  using M = Mma<T>;
  using TL = Tiles<D>;
  constexpr int KCH = kch<T, D>();
  constexpr int NO = D / 32;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int qb = w % a.nblk, rh = w / a.nblk;
  const int r = rh % G.nr, h = rh / G.nr;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * BWD_BLK + wave * TILE;
  const bool active = q0 < G.n;
  const int q = q0 + l32;  // lane <-> query
  const bool qok = q < G.n;

  __shared__ __align__(16) T ks[2 * TL::ROWT];    // K   [key][channel]
  __shared__ __align__(16) T kT[2 * TL::TRANS];  // K^T [channel][key]
  __shared__ __align__(16) T vs[2 * TL::ROWT];    // V   [key][channel]

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * D;
  const T* kr = a.k + rowbase;
  const T* vr = a.v + rowbase;
  const int last = G.n - 1;
  typename M::frag qf[KCH], daf[KCH], dalf[KCH];
  float l2 = pos_inf();
  zero_frags(dalf);
  if (qok) {
    row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
    row_frags(a.da + rowbase + (int64_t)q * G.sPos, g, daf);
    if constexpr (kSplitDA<T>) row_frags(a.dalo + rowbase + (int64_t)q * G.sPos, g, dalf);
    l2 = a.lse2[((int64_t)h * G.nr + r) * G.np + q];
  } else {
    zero_frags(qf);
    zero_frags(daf);
  }
  const float c1 = G.scale * LOG2E;
  f32x16 xt[NO] = {}, yt[NO] = {};
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
    typename M::frag af[KCH];
    row_frags(ksb + (32 * u + l32) * TL::ROW, g, af);
    f32x16 s = M::mma(af[0], qf[0], bias);
#pragma unroll
    for (int t = 1; t < KCH; ++t) s = M::mma(af[t], qf[t], s);
    if (bits != 0xffffffffu) mask_rows(s, bits, g);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2));
    // dP^T = V dA^T, then P dP and its running sum D
    row_frags(vsb + (32 * u + l32) * TL::ROW, g, af);
    f32x16 dp = M::mma(af[0], daf[0], f32x16{});
#pragma unroll
    for (int t = 1; t < KCH; ++t) dp = M::mma(af[t], daf[t], dp);
    if constexpr (kSplitDA<T>) {
#pragma unroll
      for (int t = 0; t < KCH; ++t) dp = M::mma(af[t], dalf[t], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      dp[v] *= s[v];
      dpart += dp[v];
    }
    // X^T += K^T (P dP)^T,  Y^T += K^T P^T (contraction over the keys)
    typename M::frag pf[M::PCH], sf[M::PCH], xf[M::PCH];
    acc_frags(dp, pf);
    acc_frags(s, sf);
#pragma unroll
    for (int c = 0; c < NO; ++c) {
      quad_frags(kTb + (32 * c + l32) * LDS_TROW + 32 * u, g, xf);
#pragma unroll
      for (int t = 0; t < M::PCH; ++t) xt[c] = M::mma(xf[t], pf[t], xt[c]);
#pragma unroll
      for (int t = 0; t < M::PCH; ++t) yt[c] = M::mma(xf[t], sf[t], yt[c]);
    }
  };

  PairPiece<T, D> kp;
  RowPiece<T, D> vp;
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
      const T* ksb = ks + buf * TL::ROWT;
      const T* kTb = kT + buf * TL::TRANS;
      const T* vsb = vs + buf * TL::ROWT;
      if ((uint32_t)bb) sub_tile(ksb, kTb, vsb, c0, (uint32_t)bb, 0);
      if ((uint32_t)(bb >> 32)) sub_tile(ksb, kTb, vsb, c1, (uint32_t)(bb >> 32), 1);
    }
    if (b + 1 < nblk) {
      kp.validate(tid, bbn);
      kp.store_rows(ks + (buf ^ 1) * TL::ROWT, tid);
      kp.store_trans(kT + (buf ^ 1) * TL::TRANS, tid);
      vp.store(vs + (buf ^ 1) * TL::ROWT, tid, bbn);
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
  if (g == 0) a.dsum[((int64_t)h * G.nr + r) * G.np + q] = -dsum;  // stored negated
  const int64_t base = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int c = 0; c < NO; ++c)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        x[e] = (xt[c][4 * j + e] - dsum * yt[c][4 * j + e]) * G.scale;
      store4(a.dq + base + 32 * c + 8 * j + 4 * g, x);
    }
}

// bf16 dQ (and D) with asynchronous LDS staging (see dma.h).  One workgroup
// = QD_ROWS x QD_QT waves = 32 QD_QT queries x QD_ROWS rows of one head:
// wave w owns query tile w % QD_QT (lane <-> query) of row r0 + w / QD_QT.
// Keys stream in tiles of 32; per tile, K and V of the rows and the
// query-major bias tiles of the queries (shared by the rows) are copied
// HBM -> LDS by DMA into a ring of QD_SLOTS slots.  K^T fragments for the
// dQ products come from the transposing LDS read of the row-major K tile.
// The DMAs go through buffer resources advanced in scalar registers, and
// the loop is unrolled by the ring length, so no vector instruction is
// spent on addresses.
#ifndef QD_ROWS_CFG
#define QD_ROWS_CFG 2
#endif
#ifndef QD_QT_CFG
#define QD_QT_CFG 2
#endif
#ifndef QD_SLOTS_CFG
#define QD_SLOTS_CFG 2
#endif
constexpr int QD_ROWS = QD_ROWS_CFG, QD_QT = QD_QT_CFG, QD_SLOTS = QD_SLOTS_CFG;
constexpr int QD_WAVES = QD_ROWS * QD_QT;
constexpr int QD_BLK = 32 * 64;                         // 2 KB: 32 keys x 32 channels
// Slot layout: K tiles [channel half][row], V tiles [channel half][row], then
// QD_QT bias tiles (fp32, 4 KB each).  A 64-channel head keeps each position
// as two 32-channel halves (24 KB slots, two waves per SIMD); 16- and
// 32-channel heads have one (16 KB slots, four waves per SIMD).
template <int D>
struct QdL {
  static constexpr int NH = D == 64 ? 2 : 1;         // 32-channel halves per position
  static constexpr int HQ = QD_ROWS * QD_BLK;        // one half's tiles of the rows
  static constexpr int K = 0, V = NH * HQ;
  static constexpr int BIAS = 2 * NH * HQ;
  static constexpr int SLOT = BIAS + QD_QT * 4096;
  static constexpr int KVU = 4 * QD_ROWS * NH;       // 1 KB K/V DMA units per tile
  static constexpr int UNITS = KVU + 4 * QD_QT;      // and the bias quarters
  static constexpr int OPS = UNITS / QD_WAVES;       // DMA ops per thread per tile
  static constexpr int WPE = D == 64 ? 2 : 4;        // waves per SIMD
  static_assert(UNITS % QD_WAVES == 0, "DMA units must split evenly over the waves");
  // source of unit u: K or V rows of channel half c, or bias tile t
  static constexpr int source(int u) {
    return u < KVU ? 2 * ((u >> 1) / (2 * QD_ROWS)) + ((u >> 1) % (2 * QD_ROWS) < QD_ROWS ? 0 : 1)
                   : 2 * NH + (u - KVU) / 4;
  }
  // whether the OPS units of every wave share one source
  static constexpr bool one_source() {
    for (int w = 0; w < QD_WAVES; ++w)
      for (int j = 1; j < OPS; ++j)
        if (source(OPS * w + j) != source(OPS * w)) return false;
    return true;
  }
  static_assert(QD_SLOTS * SLOT <= 65536, "slot offsets must fit the LDS immediate");
};

// D = 16, 32 or 64 channels per head (see dma.h for 16).
template <int D>
__global__ __launch_bounds__(64 * QD_WAVES) __attribute__((amdgpu_waves_per_eu(QdL<D>::WPE, QdL<D>::WPE))) void dq_dma_kernel(BwdArgs<bf16> a, int nqb) {
  to_sample(a);
  using M = Mma<bf16>;
  using F = bf16x8;
  using L = QdL<D>;
  constexpr int NH = L::NH;
  constexpr int QD_OPS = L::OPS;
  constexpr int KC = D == 16 ? 1 : D / 16;  // 16-channel MFMA steps of a contraction over channels
  constexpr int KA = D == 64 ? 4 : 2;       // fragment slots per operand row
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nrg = (G.nr + QD_ROWS - 1) / QD_ROWS;
  const int qb = w % nqb, rg = (w / nqb) % nrg, h = w / (nqb * nrg);
  const int r0 = rg * QD_ROWS;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qtl = wave % QD_QT, ri = wave / QD_QT;
  const int last = G.nr - 1;  // last row
  const int r = min(r0 + ri, last);
  const bool rok = r0 + ri < G.nr;
  const int q0 = qb * 32 * QD_QT + qtl * TILE;
  const int q = q0 + l32;
  const bool active = rok && q0 < G.n;
  const bool qok = q < G.n;
  const int nkt = G.nkt;
  const int nrows = min(QD_ROWS, G.nr - r0);  // rows of this group that exist
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[QD_SLOTS * L::SLOT];

  // ---- this lane's query: Q, dA (hi, lo) fragments and lse2
  const int64_t hb = (int64_t)h * D;
  const int64_t rowbase = (int64_t)r * G.sRow + hb;
  F qf[KA], daf[KA], dalf[KA];
  float l2 = pos_inf();
  if (active && qok) {
    if constexpr (D == 64) {
      row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
      row_frags(a.da + rowbase + (int64_t)q * G.sPos, g, daf);
      row_frags(a.dalo + rowbase + (int64_t)q * G.sPos, g, dalf);
    } else {
      row_frags_d<D>(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
      row_frags_d<D>(a.da + rowbase + (int64_t)q * G.sPos, g, daf);
      row_frags_d<D>(a.dalo + rowbase + (int64_t)q * G.sPos, g, dalf);
    }
    l2 = a.lse2[((int64_t)h * G.nr + r) * G.np + q];
  } else {
    zero_frags(qf);
    zero_frags(daf);
    zero_frags(dalf);
  }
  bool rows_full = true;
  for (int i = 0; i < nrows; ++i) rows_full = rows_full && const_load(a.rowfull + r0 + i) != 0u;
  // the plain register loads above stay in flight with the first DMAs: the
  // first step's full wait (vmcnt 0) precedes every use of their registers

  // ---- DMA lanes.  Unit u = QD_OPS w + j of wave w: u < KVU: keys
  // 16 (u % 2) + lane / 4 of tile b = (u / 2) % (2 QD_ROWS) of [K rows, V
  // rows], channel half (u / 2) / (2 QD_ROWS); otherwise quarter v % 4 of
  // bias tile v / 4, v = u - KVU.  Lane offsets are fixed; the source bases
  // advance by one key tile per issue.
  const int64_t tensor = (int64_t)G.nr * G.n * G.H * D;
  const int64_t tstep = (int64_t)TILE * G.sPos;
  const void* src[QD_OPS];
  const void* srcend[QD_OPS];
  int64_t adv[QD_OPS];  // bytes per tile
  uint32_t voff[QD_OPS];
  char* dst[QD_OPS];
  bool dok[QD_OPS];  // this lane has a chunk to copy (not: channels 16..31 of a 16-channel head)
#pragma unroll
  for (int j = 0; j < QD_OPS; ++j) {
    const int u = QD_OPS * wave + j;
    if (u < L::KVU) {
      const int blk = (u >> 1) % (2 * QD_ROWS), c = (u >> 1) / (2 * QD_ROWS), half = u & 1;
      const bf16* t = blk < QD_ROWS ? a.k : a.v;
      const int p = 16 * half + (lane >> 2);
      src[j] = t + (int64_t)min(r0 + blk % QD_ROWS, last) * G.sRow + hb;
      srcend[j] = t + tensor;
      adv[j] = tstep * 2;
      voff[j] = (uint32_t)(((int64_t)p * G.sPos + 32 * c + 8 * ((lane & 3) ^ swz(p))) * 2);
      dst[j] = smem + (blk < QD_ROWS ? L::K : L::V) + c * L::HQ + (blk % QD_ROWS) * QD_BLK +
               1024 * half;
      dok[j] = chunk_exists<D == 16 ? 16 : 32>(p, lane & 3);
    } else {
      const int v = u - L::KVU, tl = v >> 2, qu = v & 3;
      src[j] = a.bt + ((int64_t)h * nkt + qb * QD_QT + tl) * nkt * 1024;
      srcend[j] = a.bt + (int64_t)G.H * nkt * nkt * 1024;
      adv[j] = 4096;
      voff[j] = (uint32_t)(1024 * qu + 16 * lane);
      dst[j] = smem + L::BIAS + tl * 4096 + 1024 * qu;
      dok[j] = true;
    }
  }
  // When the units of every wave come from one source (the K rows, the V rows
  // or one bias tile, of one channel half), one walking resource serves a
  // wave's units, the rows told apart by their lane offsets.  Otherwise (64
  // channels: six units from two sources per wave) each unit's pointer moves
  // and its resource is rebuilt per tile: six walking resources held in
  // scalar registers outgrow them (their spills cost dQ about 10% at 64 channels).
  constexpr bool ONE = L::one_source();
  Walk wk[1];
  if constexpr (ONE) wk[0] = Walk(src[0], srcend[0], adv[0]);
  if constexpr (ONE) {
#pragma unroll
    for (int j = 1; j < QD_OPS; ++j)
      voff[j] += (uint32_t)((const char*)src[j] - (const char*)src[0]);
  }
  int issued = 0;
  auto issue = [&](int slot) {
    // tiles past the last copy nothing (empty resources) but keep the wait
    // counts uniform
    const bool real = issued < nkt;
    if constexpr (ONE) {
      const rsrc_t rs = wk[0].rsrc(real);
#pragma unroll
      for (int j = 0; j < QD_OPS; ++j)
        if (dok[j]) dma16b(rs, voff[j], dst[j] + slot * L::SLOT);
      wk[0].advance();
    } else {
#pragma unroll
      for (int j = 0; j < QD_OPS; ++j) {
        // records from the unit's pointer to its tensor's end (capped at 2^32 - 1)
        const uint64_t len = real ? (uint64_t)((const char*)srcend[j] - (const char*)src[j]) : 0u;
        const rsrc_t rs = buf_rsrc_n(src[j], (len >> 32) != 0 ? 0xffffffffu : (uint32_t)len);
        if (dok[j]) dma16b(rs, voff[j], dst[j] + slot * L::SLOT);
        if (real) src[j] = (const char*)src[j] + adv[j];
      }
    }
    ++issued;
  };

  // ---- LDS read addresses (slot 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t rk0 = base + ri * QD_BLK + l32 * 64 + 16 * (g ^ sw);
  const uint32_t rk1 = base + ri * QD_BLK + l32 * 64 + 16 * ((2 + g) ^ sw);
  const TrAddr ta(lane);
  const uint32_t rtr = base + L::K + ri * QD_BLK + ta.off(0);
  const uint32_t rtr8 = base + L::K + ri * QD_BLK + ta.off(8) - 8 * 64;
  const uint32_t rb = base + L::BIAS + qtl * 4096 + lane * 16;
  // K (region L::K) or V (L::V) fragment t (channels 16 t + 8 g .. +7) of this wave's row
  auto rfrag = [&](uint32_t region, int t) {
    return lds_load16<F>((t & 1 ? rk1 : rk0) + (t >> 1) * L::HQ + region);
  };

  f32x16 xt[NH] = {}, yt[NH] = {};
  float dpart = 0.f;

  // the loop; FULL: every key of every row of the group is valid
  auto run = [&](auto full_c) {
    constexpr bool FULL = decltype(full_c)::value;
    auto step = [&](int t, auto slot) {
      constexpr int S = decltype(slot)::value;
      constexpr uint32_t so = S * L::SLOT;
      // key bits of tile t for this wave's row (0 for a row past the end)
      uint32_t bits = 0;
      if constexpr (FULL) {
        bits = rok ? in_range_bits(t, G.n) : 0u;
        wait_vm<(QD_SLOTS - 2) * QD_OPS>();  // tile t has landed
        lds_barrier();
        issue((S + QD_SLOTS - 1) % QD_SLOTS);  // tile t + QD_SLOTS - 1 into the slot of tile t - 1
      } else {
        uint32_t wr[QD_ROWS];  // per row of the group
#pragma unroll
        for (int i = 0; i < QD_ROWS; ++i)
          wr[i] = i < nrows ? const_load(a.kbits + (int64_t)(r0 + i) * nkt + t) : 0u;
        wait_vm<(QD_SLOTS - 2) * QD_OPS>();
        lds_barrier();
        bool full = true;
#pragma unroll
        for (int i = 0; i < QD_ROWS; ++i) full = full && (i >= nrows || wr[i] == 0xffffffffu);
        if (!full) {
          // zero V rows of keys invalid for a row (P = 0 there, and 0 times a
          // non-finite dP would not be); thread t < 32 QD_ROWS: row t / 32, key t % 32
          if (tid < 32 * QD_ROWS) {
            uint32_t wb = 0;
#pragma unroll
            for (int i = 0; i < QD_ROWS; ++i)
              if ((tid >> 5) == i) wb = wr[i];
            if (!((wb >> (tid & 31)) & 1u)) {
              char* z = smem + so + L::V + (tid >> 5) * QD_BLK + 64 * (tid & 31);
#pragma unroll
              for (int c = 0; c < NH; ++c)
#pragma unroll
                for (int e = 0; e < 4; ++e) *(f32x4*)(z + c * L::HQ + 16 * e) = f32x4{};
            }
          }
          __syncthreads();
        }
        issue((S + QD_SLOTS - 1) % QD_SLOTS);
#pragma unroll
        for (int i = 0; i < QD_ROWS; ++i)
          if (ri == i) bits = wr[i];
      }
      if (!active || bits == 0u) return;
      // S^T = bias + K Q^T (lane <-> query, registers <-> keys)
      f32x16 sv;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 y = lds_load16<f32x4>(rb + so + 1024 * j);
#pragma unroll
        for (int e = 0; e < 4; ++e) sv[4 * j + e] = y[e];
      }
#pragma unroll
      for (int t = 0; t < KC; ++t) sv = M::mma(rfrag(so + L::K, t), qf[t], sv);
      if (bits != 0xffffffffu) mask_rows(sv, bits, g);
#pragma unroll
      for (int v = 0; v < 16; ++v) sv[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2));
      // dP^T = V dA^T (hi and lo parts), then P dP and its running sum D
      f32x16 dp;
      {
        F vf[KA];
#pragma unroll
        for (int t = 0; t < KC; ++t) vf[t] = rfrag(so + L::V, t);
        dp = M::mma(vf[0], daf[0], f32x16{});
#pragma unroll
        for (int t = 1; t < KC; ++t) dp = M::mma(vf[t], daf[t], dp);
#pragma unroll
        for (int t = 0; t < KC; ++t) dp = M::mma(vf[t], dalf[t], dp);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        dp[v] *= sv[v];
        dpart += dp[v];
      }
      // X^T += K^T (P dP)^T,  Y^T += K^T P^T (contraction over the tile's keys)
      F pf[M::PCH], xf[M::PCH];
      acc_frags(dp, xf);
      acc_frags(sv, pf);
      auto half = [&](auto cc) {  // K^T fragments of channel half c
        constexpr int c = decltype(cc)::value;
        constexpr uint32_t ho = so + c * L::HQ;
        s16x4 xk[4];
        xk[0] = ds_read_tr<ho>(rtr);
        xk[1] = ds_read_tr<ho + 8 * 64>(rtr8);
        xk[2] = ds_read_tr<ho + 16 * 64>(rtr);
        xk[3] = ds_read_tr<ho + 24 * 64>(rtr8);
        tr_wait(xk);
#pragma unroll
        for (int u = 0; u < M::PCH; ++u) {
          xt[c] = M::mma(tr_frag(xk, u), xf[u], xt[c]);
          yt[c] = M::mma(tr_frag(xk, u), pf[u], yt[c]);
        }
      };
      half(std::integral_constant<int, 0>{});
      if constexpr (NH == 2) half(std::integral_constant<int, 1>{});
    };
#pragma unroll
    for (int j = 0; j < QD_SLOTS - 1; ++j) issue(j);
    for (int t = 0; t < nkt; t += QD_SLOTS) {
      step(t, slot_c<0>{});
      if (t + 1 >= nkt) break;
      step(t + 1, slot_c<1 % QD_SLOTS>{});
      if (QD_SLOTS < 3 || t + 2 >= nkt) continue;
      step(t + 2, slot_c<2 % QD_SLOTS>{});
    }
  };
  if (rows_full)
    run(std::true_type{});
  else
    run(std::false_type{});
  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active) return;
  const float dsum = wave_xor32_sum(dpart);
  if (!qok) return;
  if (g == 0) a.dsum[((int64_t)h * G.nr + r) * G.np + q] = -dsum;  // stored negated
  const int64_t gb = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int c = 0; c < NH; ++c)
#pragma unroll
    for (int j = 0; j < (D == 16 ? 2 : 4); ++j) {  // the quads of channels 32 c + 8 j + 4 g .. +3 < D
      f32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = (xt[c][4 * j + e] - dsum * yt[c][4 * j + e]) * G.scale;
      store4(a.dq + gb + 32 * c + 8 * j + 4 * g, x);
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
template <typename T, int D>
__global__ __launch_bounds__(512, 1) void db_kernel(BwdArgs<T> a) {
  to_sample(a);
  using M = Mma<T>;
  using TL = Tiles<D>;
  constexpr int KCH = kch<T, D>();
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

  __shared__ __align__(16) T ks[2 * TL::ROWT];   // K  [key][channel] of the 128 keys
  __shared__ __align__(16) T vs[2 * TL::ROWT];   // V
  __shared__ __align__(16) T qs[2 * TL::ROWT];   // Q  [query][channel] of the 128 queries
  __shared__ __align__(16) T das[2 * TL::ROWT];  // dA
  __shared__ __align__(16) T dals[kSplitDA<T> ? 2 * TL::ROWT : 1];
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
  const int r0 = rc * a.rpc, r1 = min(G.nr, r0 + a.rpc);

  // thread -> (half of the 128 positions, piece index within the half)
  const int half = tid >> 8, pt = tid & 255;
  const uint64_t qvalid = range_bits64(qstart + SPAN * half, G.n);
  RowPiece<T, D> kp, vp, qp, dap, dlp;
  float sv = 0.f;  // thread < 128: lse2 of query tid; 128 <= thread < 256: -D of query tid-128
  const int sq = min(qstart + (tid & 127), G.np - 1);
  auto load_row = [&](int r) {
    const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * D;
    kp.load(a.k + rowbase, G.sPos, kstart + SPAN * half, last, pt);
    vp.load(a.v + rowbase, G.sPos, kstart + SPAN * half, last, pt);
    qp.load(a.q + rowbase, G.sPos, qstart + SPAN * half, last, pt);
    dap.load(a.da + rowbase, G.sPos, qstart + SPAN * half, last, pt);
    if constexpr (kSplitDA<T>) dlp.load(a.dalo + rowbase, G.sPos, qstart + SPAN * half, last, pt);
    const int64_t at = ((int64_t)h * G.nr + r) * G.np + sq;
    sv = tid < DB_ROWS ? a.lse2[at] : a.dsum[at];
  };
  auto store_row = [&](int r) {
    const uint64_t kv = row_bits(r, half);
    kp.store(ks + half * TL::ROWT, pt, kv);
    vp.store(vs + half * TL::ROWT, pt, kv);
    qp.store(qs + half * TL::ROWT, pt, qvalid);
    dap.store(das + half * TL::ROWT, pt, qvalid);
    if constexpr (kSplitDA<T>) dlp.store(dals + half * TL::ROWT, pt, qvalid);
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
      typename M::frag qf[KCH], daf[KCH], dalf[KCH];
      row_frags(qs + (qw + l32) * TL::ROW, g, qf);
      row_frags(das + (qw + l32) * TL::ROW, g, daf);
      if constexpr (kSplitDA<T>) row_frags(dals + (qw + l32) * TL::ROW, g, dalf);
      const f32x16 ndv = splat16(nds[qw + l32]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint32_t bits = (uint32_t)(bb >> (32 * u));
        if (bits == 0u) continue;
        const int off = (SPAN * kh + 32 * u + l32) * TL::ROW;
        typename M::frag af[KCH];
        row_frags(ks + off, g, af);
        f32x16 s = M::mma(af[0], qf[0], binit[u]);
#pragma unroll
        for (int t = 1; t < KCH; ++t) s = M::mma(af[t], qf[t], s);
        if (bits != 0xffffffffu) mask_rows(s, bits, g);
        row_frags(vs + off, g, af);
        f32x16 dp = M::mma(af[0], daf[0], ndv);
#pragma unroll
        for (int t = 1; t < KCH; ++t) dp = M::mma(af[t], daf[t], dp);
        if constexpr (kSplitDA<T>) {
#pragma unroll
          for (int t = 0; t < KCH; ++t) dp = M::mma(af[t], dalf[t], dp);
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
// workgroup = 16 waves = 128 queries x 128 keys of one head, summed over
// the rows of one row chunk; wave w owns query tile w % 4 (lane <-> query)
// and key tile w / 4 of the block.  Per row, K and V of the 128 keys and Q,
// dA, its low part, lse2 and -D of the 128 queries (41 KB) land in LDS by
// DMA through a three-slot ring, two rows ahead, and are shared by the 16
// waves; one workgroup per CU runs four waves per SIMD.  The DMAs go
// through buffer resources whose bases advance by one row in scalar
// registers, so no vector instruction is spent on addresses, and the bias
// tile of each wave stays in registers for all rows.
constexpr int DBD_Q = 128, DBD_K = 128;       // queries and keys per workgroup block
constexpr int DBD_WAVES = 16;
constexpr int DBD_KV = DBD_K * 64;            // 8 KB: K (or V) of the block's keys
constexpr int DBD_QB = DBD_Q * 64;            // 8 KB: Q (or dA, dA low) of the queries
constexpr int DBD_OK = 0, DBD_OV = DBD_KV, DBD_OQ = 2 * DBD_KV;
constexpr int DBD_ODA = DBD_OQ + DBD_QB, DBD_OLO = DBD_ODA + DBD_QB;
constexpr int DBD_LD = DBD_OLO + DBD_QB;      // lse2 [128], then -D [128]
constexpr int DBD_SLOT = DBD_LD + 1024;
constexpr int DBD_SLOTS = 3;
constexpr int DBD_OPS = 3;                    // DMA ops per thread per row

// D = 16 or 32 channels per head (see dma.h for 16; 64 channels use
// db_dma64_kernel below).
template <int D>
__global__ __launch_bounds__(1024) void db_dma_kernel(BwdArgs<bf16> a, int nkb) {
  to_sample(a);
  using M = Mma<bf16>;
  using F = bf16x8;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nqb = (G.n + DBD_Q - 1) / DBD_Q;
  const int kbk = w % nkb;
  const int qb = (w / nkb) % nqb;
  const int rc = (w / (nkb * nqb)) % a.nrc;
  const int h = w / (nkb * nqb * a.nrc);
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qtl = wave & 3, ktl = wave >> 2;
  const int qstart = qb * DBD_Q, kstart = kbk * DBD_K;
  const int q = qstart + qtl * TILE + l32;  // this lane's query
  const int kt = kstart / TILE + ktl;       // this wave's key tile
  const bool active = qstart + qtl * TILE < G.n && kt < G.nkt;
  const bool qok = q < G.n;
  const int nkt = G.nkt;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[DBD_SLOTS * DBD_SLOT];

  f32x16 binit, acc = {};
  {
    const int qt = active ? qstart / TILE + qtl : 0;
    binit = load_frag_tile(frag_tile(a.bt, h, qt, min(kt, nkt - 1), nkt), lane);
  }
  // the bias tile is a plain register load: let it complete before any DMA
  // is issued (with both kinds outstanding the compiler would wait for every
  // DMA at each use of binit)
  wait_vm<0>();

  // ---- DMA lanes (lane offsets fixed, row bases in scalar registers).
  // Op 0: K (waves 0-7) or V (waves 8-15) of the 128 keys, keys
  // 16 (w % 8) + lane / 4.  Op 1: Q (waves 0-7) or dA (waves 8-15) of the
  // 128 queries.  Op 2: the low part of dA (waves 0-7), lse2 (waves 8-11)
  // or -D (waves 12-15), 128 bytes per wave (lanes 0..7).
  const int r0 = rc * a.rpc, r1 = min(G.nr, r0 + a.rpc);
  const int nr = max(r1 - r0, 0);
  // One workgroup per CU: a dispatch round is 256 workgroups.  Alternate
  // rounds walk their chunk's rows in opposite directions, so that a
  // workgroup starts on the rows that the previous round on its XCD ended
  // on, while those are still in the L2.  (The direction depends on the
  // block index only: results stay bitwise reproducible.)
  const bool back = ((blockIdx.x >> 8) & 1u) != 0u;
  const int rfirst = back ? r1 - 1 : r0;
  const int64_t rdir = back ? -1 : 1;
  const int64_t tensor = (int64_t)G.nr * G.n * G.H * D;
  const int hb = h * D;
  const int pp = 16 * (wave & 7) + (lane >> 2);  // position (key or query) of this lane
  const int pc = (lane & 3) ^ swz(pp);
  const bool pok = chunk_exists<D>(pp, lane & 3);  // a chunk to copy for the position ops
  const bf16* src0 = wave < 8 ? a.k : a.v;
  const bf16* src1 = wave < 8 ? a.q : a.da;
  // The first key and query of the block move the 64-bit bases (koff, qoff
  // elements), so a lane's byte offset stays below 2^32 for every accepted
  // size: at most 127 positions x sPos (the ending node's n h 32) x 2 bytes.
  const int64_t koff = (int64_t)kstart * G.sPos, qoff = (int64_t)qstart * G.sPos;
  const uint32_t voff = (uint32_t)(((int64_t)pp * G.sPos + hb + 8 * pc) * 2);
  // op 2: dA low (waves 0-7, same lane offsets as op 1) or lse2 / -D rows
  const bool lo_op = wave < 8;
  const float* lrow = (wave < 12 ? a.lse2 : a.dsum) + (int64_t)h * G.nr * G.np;
  const uint32_t voff2 =
      lo_op ? voff : (uint32_t)((qstart + 32 * (wave & 3) + 4 * lane) * 4);
  char* const dst0 = smem + (wave < 8 ? DBD_OK : DBD_OV) + 1024 * (wave & 7);
  char* const dst1 = smem + (wave < 8 ? DBD_OQ : DBD_ODA) + 1024 * (wave & 7);
  char* const dst2 = lo_op ? smem + DBD_OLO + 1024 * wave
                           : smem + DBD_LD + 128 * (wave - 8);
  // Op bases at row r0, advanced by one row per issue (scalar adds only),
  // with record counts fixed for the loop (see last_row_records; the lse2 /
  // -D rows are whole rows of np floats).
  const int64_t lastr = max(G.nr - 1 - r0, 0);
  const char* const c0 = (const char*)(src0 + (int64_t)r0 * G.sRow + koff);
  const char* const c1r = (const char*)(src1 + (int64_t)r0 * G.sRow + qoff);
  const char* const c2 = lo_op ? (const char*)(a.dalo + (int64_t)r0 * G.sRow + qoff)
                               : (const char*)(lrow + (int64_t)r0 * G.np);
  const int64_t rs = G.sRow * 2, rs2 = lo_op ? rs : (int64_t)G.np * 4;  // bytes per row
  const uint32_t n0 = last_row_records(c0 + lastr * rs, src0 + tensor);
  const uint32_t n1 = last_row_records(c1r + lastr * rs, src1 + tensor);
  const uint32_t n2 = lo_op ? last_row_records(c2 + lastr * rs, a.dalo + tensor)
                            : (uint32_t)G.np * 4;
  const bool op2 = lo_op ? pok : lane < 8;
  // op bases at the walk's first row, moved one row per issue
  const char* b0 = c0 + (int64_t)(rfirst - r0) * rs;
  const char* b1 = c1r + (int64_t)(rfirst - r0) * rs;
  const char* b2 = c2 + (int64_t)(rfirst - r0) * rs2;
  int issued = 0;
  auto issue = [&](int slot) {
    // issues past the chunk's rows copy nothing (empty resources, based on
    // the chunk's first row) but keep the wait counts uniform
    const bool real = issued < nr;
    if (pok) {
      dma16b(real ? buf_rsrc_n(b0, n0) : buf_rsrc_n(c0, 0u), voff, dst0 + slot * DBD_SLOT);
      dma16b(real ? buf_rsrc_n(b1, n1) : buf_rsrc_n(c1r, 0u), voff, dst1 + slot * DBD_SLOT);
    }
    if (op2) dma16b(real ? buf_rsrc_n(b2, n2) : buf_rsrc_n(c2, 0u), voff2, dst2 + slot * DBD_SLOT);
    b0 += rdir * rs;
    b1 += rdir * rs;
    b2 += rdir * rs2;
    ++issued;
  };

  // ---- LDS read addresses (slot 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t qpos = base + (uint32_t)(qtl * TILE + l32) * 64;
  const uint32_t rq0 = qpos + 16 * (g ^ sw), rq1 = qpos + 16 * ((2 + g) ^ sw);
  const uint32_t kpos = base + (uint32_t)(ktl * TILE + l32) * 64;
  const uint32_t rk0 = kpos + 16 * (g ^ sw), rk1 = kpos + 16 * ((2 + g) ^ sw);
  const uint32_t rl = base + DBD_LD + (qtl * TILE + l32) * 4;
  const uint32_t* kbrow = a.kbits + kstart / TILE;

  // FULL: every key < n is valid for every row of the chunk.  The key bits
  // of the wave's tile are then the same for every row, and keys past n
  // read zeros (K, V) through the record counts, so no row needs its V rows
  // cleared.
  bool rows_full = true;
  for (int rr = r0; rr < r1; rr += 64)
    rows_full = rows_full && __all(rr + lane >= r1 || a.rowfull[rr + lane] != 0u);
  const uint32_t wfull = kt < nkt ? in_range_bits(kt, G.n) : 0u;

  auto step = [&](int r, auto slot, auto full_c) {
    constexpr int S = decltype(slot)::value;
    constexpr bool FULL = decltype(full_c)::value;
    const uint32_t wb =
        FULL ? wfull : (kt < nkt ? const_load(kbrow + (int64_t)r * nkt + ktl) : 0u);
    wait_vm<DBD_OPS>();  // row r has landed (only row r + 1 is still in flight)
    lds_barrier();
    if constexpr (!FULL) {
      // key bits of the block's 4 tiles: the same in every wave, so the
      // branch below (it holds a barrier) is uniform across the workgroup
      uint32_t all = 0xffffffffu;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        all &= kstart / TILE + j < nkt ? const_load(kbrow + (int64_t)r * nkt + j) : 0xffffffffu;
      if (all != 0xffffffffu) {
        // zero V rows of keys invalid for the row (P = 0 there, and 0 times
        // a non-finite dP would not be); thread t < 512: key t / 4, 16 bytes
        if (tid < 512) {
          const int j = tid >> 7;
          const uint32_t b = kstart / TILE + j < nkt ? const_load(kbrow + (int64_t)r * nkt + j) : 0u;
          if (!((b >> ((tid >> 2) & 31)) & 1u))
            *(f32x4*)(smem + S * DBD_SLOT + DBD_OV + 16 * tid) = f32x4{};
        }
        __syncthreads();
      }
    }
    // the tile's operand reads first, then the DMA issue, then the products
    const bool act = active && wb != 0u;
    F q0{}, k0{}, q1{}, k1{}, d0{}, e0{}, v0{}, d1{}, e1{}, v1{};
    float l2 = 0.f, nd = 0.f;
    if (act) {
      l2 = *(const TRIATTN_LDS float*)(uintptr_t)(rl + S * DBD_SLOT);
      nd = *(const TRIATTN_LDS float*)(uintptr_t)(rl + S * DBD_SLOT + 512);
      q0 = lds_load16<F>(rq0 + S * DBD_SLOT + DBD_OQ);
      k0 = lds_load16<F>(rk0 + S * DBD_SLOT + DBD_OK);
      d0 = lds_load16<F>(rq0 + S * DBD_SLOT + DBD_ODA);
      e0 = lds_load16<F>(rq0 + S * DBD_SLOT + DBD_OLO);
      v0 = lds_load16<F>(rk0 + S * DBD_SLOT + DBD_OV);
      if constexpr (D == 32) {
        q1 = lds_load16<F>(rq1 + S * DBD_SLOT + DBD_OQ);
        k1 = lds_load16<F>(rk1 + S * DBD_SLOT + DBD_OK);
        d1 = lds_load16<F>(rq1 + S * DBD_SLOT + DBD_ODA);
        e1 = lds_load16<F>(rq1 + S * DBD_SLOT + DBD_OLO);
        v1 = lds_load16<F>(rk1 + S * DBD_SLOT + DBD_OV);
      }
    }
    issue((S + 2) % DBD_SLOTS);  // row r + 2 into the slot of row r - 1
    if (!act) return;
    if (!qok) l2 = pos_inf();
    f32x16 sv = M::mma(k0, q0, binit);  // S^T = bias + K Q^T
    if constexpr (D == 32) sv = M::mma(k1, q1, sv);
    if (wb != 0xffffffffu) mask_rows(sv, wb, g);
    f32x16 dpv = splat16(nd);  // dP^T - D = V dA^T - D (hi and lo parts)
    dpv = M::mma(v0, d0, dpv);
    if constexpr (D == 32) dpv = M::mma(v1, d1, dpv);
    dpv = M::mma(v0, e0, dpv);
    if constexpr (D == 32) dpv = M::mma(v1, e1, dpv);
#pragma unroll
    for (int v = 0; v < 16; ++v)
      acc[v] += __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2)) * dpv[v];
  };

  issue(0);
  issue(1);
  auto run = [&](auto full_c) {
    for (int i = 0; i < nr; i += DBD_SLOTS) {
      step(rfirst + (int)rdir * i, slot_c<0>{}, full_c);
      if (i + 1 >= nr) break;
      step(rfirst + (int)rdir * (i + 1), slot_c<1>{}, full_c);
      if (i + 2 >= nr) break;
      step(rfirst + (int)rdir * (i + 2), slot_c<2>{}, full_c);
    }
  };
  if (rows_full)
    run(std::true_type{});
  else
    run(std::false_type{});
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

// bf16 dB for 64 channels per head.  A position's 128 bytes are staged as
// two 32-channel half-rows (the usual 64-byte block layout each), so a
// 128 x 128 block's row (80 KB) would leave no room for a second ring slot;
// the block is 64 queries x 128 keys instead: 8 waves, wave w owns query
// tile w % 2 and key tile w / 2, one workgroup per CU (two waves per SIMD).
// Per row, K and V of the 128 keys, Q, dA and its low part of the 64
// queries, lse2 and -D (56.5 KB) land in LDS by DMA through a two-slot ring,
// one row ahead.  LDS is laid out by region, each holding both slots, so
// that slot offsets stay small.
constexpr int D6_Q = 64, D6_K = 128, D6_WAVES = 8;
constexpr int D6_KH = D6_K * 64;                 // one channel half of the block's K (or V): 8 KB
constexpr int D6_QH = D6_Q * 64;                 // one channel half of its Q (dA, dA low): 4 KB
constexpr int D6_OK = 0, D6_OV = 2 * 2 * D6_KH;  // [slot][half] regions
constexpr int D6_OQ = 2 * D6_OV, D6_ODA = D6_OQ + 2 * 2 * D6_QH, D6_OLO = D6_ODA + 2 * 2 * D6_QH;
constexpr int D6_OL = D6_OLO + 2 * 2 * D6_QH;    // [slot]: lse2 [64], then -D [64]
constexpr int D6_LDS = D6_OL + 2 * 512;

__global__ __launch_bounds__(64 * D6_WAVES) void db_dma64_kernel(BwdArgs<bf16> a, int nkb) {
  to_sample(a);
  using M = Mma<bf16>;
  using F = bf16x8;
  constexpr int D = 64;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nqb = (G.n + D6_Q - 1) / D6_Q;
  const int kbk = w % nkb;
  const int qb = (w / nkb) % nqb;
  const int rc = (w / (nkb * nqb)) % a.nrc;
  const int h = w / (nkb * nqb * a.nrc);
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qtl = wave & 1, ktl = wave >> 1;
  const int qstart = qb * D6_Q, kstart = kbk * D6_K;
  const int q = qstart + qtl * TILE + l32;  // this lane's query
  const int kt = kstart / TILE + ktl;       // this wave's key tile
  const bool active = qstart + qtl * TILE < G.n && kt < G.nkt;
  const bool qok = q < G.n;
  const int nkt = G.nkt;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[D6_LDS];

  f32x16 binit, acc = {};
  {
    const int qt = active ? qstart / TILE + qtl : 0;
    binit = load_frag_tile(frag_tile(a.bt, h, qt, min(kt, nkt - 1), nkt), lane);
  }
  // the bias tile is a plain register load: let it complete before any DMA
  // is issued
  wait_vm<0>();

  // ---- DMA lanes (lane offsets fixed, row bases in scalar registers).
  // K, V: keys 16 w + lane / 4 of the block, both channel halves (2 ops
  // each).  Q, dA, dA low: queries 16 (w % 4) + lane / 4, channel half w / 4
  // (1 op each).  lse2 (waves 0, 1) or -D (waves 2, 3): queries
  // 32 (w % 2) .. +31, 128 bytes (lanes 0..7).
  const int r0 = rc * a.rpc, r1 = min(G.nr, r0 + a.rpc);
  const int nr = max(r1 - r0, 0);
  const int64_t tensor = (int64_t)G.nr * G.n * G.H * D;
  const int hb = h * D;
  const int pk = 16 * wave + (lane >> 2);        // key position of this lane
  const int pq = 16 * (wave & 3) + (lane >> 2);  // query position of this lane
  const int cq = wave >> 2;                      // channel half of the Q, dA, dA-low ops
  // The first key and query of the block move the 64-bit bases, so a lane's
  // byte offset stays below 2^32 for every accepted size.
  const int64_t koff = (int64_t)kstart * G.sPos, qoff = (int64_t)qstart * G.sPos;
  const uint32_t kvoff = (uint32_t)(((int64_t)pk * G.sPos + hb + 8 * ((lane & 3) ^ swz(pk))) * 2);
  const uint32_t qvoff =
      (uint32_t)(((int64_t)pq * G.sPos + hb + 32 * cq + 8 * ((lane & 3) ^ swz(pq))) * 2);
  const bool l_op = wave < 4;
  const float* lrow = (wave < 2 ? a.lse2 : a.dsum) + (int64_t)h * G.nr * G.np;
  const uint32_t lvoff = (uint32_t)((qstart + 32 * (wave & 1) + 4 * lane) * 4);
  char* const dK = smem + D6_OK + 1024 * wave;  // + slot 2 D6_KH + half D6_KH
  char* const dV = smem + D6_OV + 1024 * wave;
  const int qo = cq * D6_QH + 1024 * (wave & 3);  // + slot 2 D6_QH
  char* const dL = smem + D6_OL + 128 * wave;     // + slot 512
  // Op bases at row r0, advanced by one row per issue, with record counts
  // fixed for the loop (see last_row_records; lse2 / -D rows are whole rows
  // of np floats).
  const int64_t lastr = max(G.nr - 1 - r0, 0);
  const int64_t rs = G.sRow * 2;  // bytes per row
  const char* bk = (const char*)(a.k + (int64_t)r0 * G.sRow + koff);
  const char* bv = (const char*)(a.v + (int64_t)r0 * G.sRow + koff);
  const char* bq = (const char*)(a.q + (int64_t)r0 * G.sRow + qoff);
  const char* ba = (const char*)(a.da + (int64_t)r0 * G.sRow + qoff);
  const char* bl = (const char*)(a.dalo + (int64_t)r0 * G.sRow + qoff);
  const char* b5 = (const char*)(lrow + (int64_t)r0 * G.np);
  const uint32_t nk = last_row_records(bk + lastr * rs, a.k + tensor);
  const uint32_t nv = last_row_records(bv + lastr * rs, a.v + tensor);
  const uint32_t nq = last_row_records(bq + lastr * rs, a.q + tensor);
  const uint32_t na = last_row_records(ba + lastr * rs, a.da + tensor);
  const uint32_t nl = last_row_records(bl + lastr * rs, a.dalo + tensor);
  auto issue = [&](int r, int slot) {
    // rows past the chunk copy nothing (empty resources) but keep the wait
    // counts uniform; rows are issued in order, one per call
    const bool real = r < r1;
    const rsrc_t rk = buf_rsrc_n(bk, real ? nk : 0u);
    const rsrc_t rv = buf_rsrc_n(bv, real ? nv : 0u);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      dma16b(rk, kvoff + 64 * c, dK + (2 * slot + c) * D6_KH);
      dma16b(rv, kvoff + 64 * c, dV + (2 * slot + c) * D6_KH);
    }
    dma16b(buf_rsrc_n(bq, real ? nq : 0u), qvoff, smem + D6_OQ + 2 * slot * D6_QH + qo);
    dma16b(buf_rsrc_n(ba, real ? na : 0u), qvoff, smem + D6_ODA + 2 * slot * D6_QH + qo);
    dma16b(buf_rsrc_n(bl, real ? nl : 0u), qvoff, smem + D6_OLO + 2 * slot * D6_QH + qo);
    if (l_op && lane < 8)
      dma16b(buf_rsrc_n(b5, real ? (uint32_t)G.np * 4 : 0u), lvoff, dL + 512 * slot);
    bk += rs;
    bv += rs;
    bq += rs;
    ba += rs;
    bl += rs;
    b5 += (int64_t)G.np * 4;
  };

  // ---- LDS read addresses (slot 0, channel half 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t qpos = base + (uint32_t)(qtl * TILE + l32) * 64;
  const uint32_t rq0 = qpos + 16 * (g ^ sw), rq1 = qpos + 16 * ((2 + g) ^ sw);
  const uint32_t kpos = base + (uint32_t)(ktl * TILE + l32) * 64;
  const uint32_t rk0 = kpos + 16 * (g ^ sw), rk1 = kpos + 16 * ((2 + g) ^ sw);
  const uint32_t rl = base + D6_OL + (qtl * TILE + l32) * 4;
  const uint32_t* kbrow = a.kbits + kstart / TILE;
  // fragment t (channels 16 t + 8 g .. +7) of this lane's query (q) or key (k) row
  auto qfrag = [&](uint32_t region, int t) {
    return lds_load16<F>((t & 1 ? rq1 : rq0) + (t >> 1) * D6_QH + region);
  };
  auto kfrag = [&](uint32_t region, int t) {
    return lds_load16<F>((t & 1 ? rk1 : rk0) + (t >> 1) * D6_KH + region);
  };

  auto step = [&](int r, auto slot) {
    constexpr int S = decltype(slot)::value;
    const uint32_t wb = kt < nkt ? const_load(kbrow + (int64_t)r * nkt + ktl) : 0u;
    wait_vm<0>();  // row r has landed
    lds_barrier();
    {
      // key bits of the block's 4 tiles: the same in every wave, so the
      // branch below (it holds a barrier) is uniform across the workgroup
      uint32_t all = 0xffffffffu;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        all &= kstart / TILE + j < nkt ? const_load(kbrow + (int64_t)r * nkt + j) : 0xffffffffu;
      if (all != 0xffffffffu) {
        // zero V rows of keys invalid for the row (P = 0 there, and 0 times
        // a non-finite dP would not be); thread t: key t / 4, 16 bytes of
        // each channel half
        const int j = tid >> 7;
        const uint32_t b = kstart / TILE + j < nkt ? const_load(kbrow + (int64_t)r * nkt + j) : 0u;
        if (!((b >> ((tid >> 2) & 31)) & 1u)) {
#pragma unroll
          for (int c = 0; c < 2; ++c)
            *(f32x4*)(smem + D6_OV + (2 * S + c) * D6_KH + 16 * tid) = f32x4{};
        }
        __syncthreads();
      }
    }
    issue(r + 1, S ^ 1);  // row r + 1 into the slot of row r - 1
    if (!active || wb == 0u) return;
    constexpr uint32_t ks = 2 * S * D6_KH, qs = 2 * S * D6_QH;
    float l2 = *(const TRIATTN_LDS float*)(uintptr_t)(rl + 512 * S);
    const float nd = *(const TRIATTN_LDS float*)(uintptr_t)(rl + 512 * S + 256);
    if (!qok) l2 = pos_inf();
    f32x16 sv = binit;  // S^T = bias + K Q^T
#pragma unroll
    for (int t = 0; t < 4; ++t) sv = M::mma(kfrag(D6_OK + ks, t), qfrag(D6_OQ + qs, t), sv);
    if (wb != 0xffffffffu) mask_rows(sv, wb, g);
    f32x16 dpv = splat16(nd);  // dP^T - D = V dA^T - D (hi and lo parts)
#pragma unroll
    for (int t = 0; t < 4; ++t) dpv = M::mma(kfrag(D6_OV + ks, t), qfrag(D6_ODA + qs, t), dpv);
#pragma unroll
    for (int t = 0; t < 4; ++t) dpv = M::mma(kfrag(D6_OV + ks, t), qfrag(D6_OLO + qs, t), dpv);
#pragma unroll
    for (int v = 0; v < 16; ++v)
      acc[v] += __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2)) * dpv[v];
  };

  issue(r0, 0);
  for (int i = 0; i < nr; i += 2) {
    step(r0 + i, slot_c<0>{});
    if (i + 1 >= nr) break;
    step(r0 + i + 1, slot_c<1>{});
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
// starting node stores it at [q][k][h], the ending node at [k][q][h].  One
// workgroup per 32 x 32 block (query tile qa, key tile kb), four heads at a
// time: every slab read is 16 contiguous bytes of a slab row, the sums pass
// through LDS, and the stores run along the output's fastest axes (key, then
// head for the starting node; query, then head for the ending node).
constexpr int DBR_HG = 4;  // heads per pass
template <typename T>
__global__ __launch_bounds__(256) void db_reduce_kernel(Geom G, int node, int nrc,
                                                        const float* slabs, T* dbias) {
  slabs = ws_at_sample(slabs, G.bWs);
  dbias = at_sample(dbias, G.bBias);
  const int nt = G.nkt, n = G.n, tid = threadIdx.x;
  const int qa = blockIdx.x % nt, kb = blockIdx.x / nt;
  const int64_t plane = (int64_t)G.np * G.np;
  __shared__ float tl[DBR_HG][32][33];
  const int r = tid >> 3, c0 = 4 * (tid & 7);  // sums: query 32 qa + r, keys 32 kb + c0 .. +3
  for (int h0 = 0; h0 < G.H; h0 += DBR_HG) {
    const int hn = min(DBR_HG, G.H - h0);
    if (h0 > 0) __syncthreads();  // the previous pass's stores have read the tile
    for (int hh = 0; hh < hn; ++hh) {
      const float* p = slabs + (int64_t)(h0 + hh) * plane + (int64_t)(32 * qa + r) * G.np + 32 * kb + c0;
      f32x4 sum = *(const f32x4*)p;
      for (int c = 1; c < nrc; ++c) sum += *(const f32x4*)(p + (int64_t)c * G.H * plane);
#pragma unroll
      for (int e = 0; e < 4; ++e) tl[hh][r][c0 + e] = sum[e];
    }
    __syncthreads();
    // element e of the block: outer = e / 32, inner = e % 32 (consecutive threads along
    // the output's key axis for the starting node, its query axis for the ending node)
    for (int e = tid; e < 1024; e += 256) {
      const int outer = e >> 5, inner = e & 31;
      const int q = node == 0 ? outer : inner, k = node == 0 ? inner : outer;
      const int qi = 32 * qa + q, ki = 32 * kb + k;
      if (qi >= n || ki >= n) continue;
      const int64_t at = (node == 0 ? ((int64_t)qi * n + ki) : ((int64_t)ki * n + qi)) * G.H + h0;
      if (G.H % DBR_HG == 0) {  // four heads in one aligned store
        store4(dbias + at, f32x4{tl[0][q][k], tl[1][q][k], tl[2][q][k], tl[3][q][k]});
      } else {
        for (int hh = 0; hh < hn; ++hh) dbias[at + hh] = (T)tl[hh][q][k];
      }
    }
  }
}

template <typename T>
hipError_t launch_bwd(const Geom& g, int node, const Prep& p, const BwdWs& ws, const T* q,
                      const T* k, const T* v, const T* gate, const T* out, const float* lse,
                      const T* dout, T* dq, T* dk, T* dv, T* dg, T* dbias, float* dbias_f32,
                      hipStream_t s) {
  T* da = (T*)ws.da;
  T* dalo = (T*)ws.dalo;
  const bool d64 = g.d == 64;  // register-staged kernels with 64 channels per head
  const bool d16 = g.d == 16;  // bf16 only: the DMA kernels with 16 channels per head
  if (d16 && !std::is_same<T, bf16>::value) return hipErrorInvalidValue;
  {
    KernelTimer t(K_BWD_PREP, s);
    const dim3 grid((unsigned)((4 * g.n * g.H + 255) / 256), (unsigned)g.nr, (unsigned)g.batch);
    if (d64)
      hipLaunchKernelGGL((bwd_prep_kernel<T, 64>), grid, dim3(256), 0, s, g, node, out, lse, gate,
                         dout, dg, da, dalo, ws.lse2);
    else if (d16)  // two threads per (pair, head): half the grid
      hipLaunchKernelGGL((bwd_prep_kernel<T, 16>),
                         dim3((unsigned)((2 * g.n * g.H + 255) / 256), (unsigned)g.nr, (unsigned)g.batch),
                         dim3(256), 0, s, g, node, out, lse, gate, dout, dg, da, dalo, ws.lse2);
    else
      hipLaunchKernelGGL((bwd_prep_kernel<T, 32>), grid, dim3(256), 0, s, g, node, out, lse, gate,
                         dout, dg, da, dalo, ws.lse2);
  }
  if (g.np > g.n) {
    const int64_t npad = (int64_t)g.H * g.nr * (g.np - g.n);
    KernelTimer t(K_BWD_PAD, s);
    hipLaunchKernelGGL(bwd_pad_kernel, dim3((unsigned)((npad + 255) / 256), 1, (unsigned)g.batch), dim3(256), 0, s, g,
                       ws.lse2, ws.dsum);
  }
  BwdArgs<T> a{g, p.bt, p.btT, p.kbits, p.rowfull, q, k, v, da, dalo, ws.lse2, ws.dsum, dq, dk, dv, ws.slabs,
               (g.n + BWD_BLK - 1) / BWD_BLK, ws.nrc, (g.nr + ws.nrc - 1) / ws.nrc};
  const int64_t nrow = (int64_t)a.nblk * g.nr * g.H;
  {
    // the dQ kernel first: it produces D for the other two
    KernelTimer t(K_DQ, s);
    if constexpr (std::is_same<T, bf16>::value) {
      const int nqb = (g.n + 32 * QD_QT - 1) / (32 * QD_QT);
      const int64_t nwg = (int64_t)nqb * ((g.nr + QD_ROWS - 1) / QD_ROWS) * g.H;
      if (d64)
        hipLaunchKernelGGL(dq_dma_kernel<64>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * QD_WAVES), 0, s, a, nqb);
      else if (d16)
        hipLaunchKernelGGL(dq_dma_kernel<16>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * QD_WAVES), 0, s, a, nqb);
      else
        hipLaunchKernelGGL(dq_dma_kernel<32>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * QD_WAVES), 0, s, a, nqb);
    } else if (d64) {
      hipLaunchKernelGGL((dq_kernel<T, 64>), dim3((unsigned)nrow, 1, (unsigned)g.batch), dim3(256), 0, s, a);
    } else {
      hipLaunchKernelGGL((dq_kernel<T, 32>), dim3((unsigned)nrow, 1, (unsigned)g.batch), dim3(256), 0, s, a);
    }
  }
  {
    KernelTimer t(K_DKDV, s);
    const hipError_t e = launch_dkdv(a, node, s);
    if (e != hipSuccess) return e;
  }
  {
    const int64_t ndb = (int64_t)a.nblk * a.nblk * ws.nrc * g.H;
    KernelTimer t(K_DB, s);
    if constexpr (std::is_same<T, bf16>::value) {
      if (d64) {
        const int nkb = (g.n + D6_K - 1) / D6_K;
        const int64_t nwg = (int64_t)((g.n + D6_Q - 1) / D6_Q) * nkb * ws.nrc * g.H;
        hipLaunchKernelGGL(db_dma64_kernel, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * D6_WAVES), 0, s, a, nkb);
      } else {
        const int nkb = (g.n + DBD_K - 1) / DBD_K;
        const int64_t nwg = (int64_t)((g.n + DBD_Q - 1) / DBD_Q) * nkb * ws.nrc * g.H;
        if (d16)
          hipLaunchKernelGGL(db_dma_kernel<16>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * DBD_WAVES), 0, s, a, nkb);
        else
          hipLaunchKernelGGL(db_dma_kernel<32>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * DBD_WAVES), 0, s, a, nkb);
      }
    } else if (d64) {
      hipLaunchKernelGGL((db_kernel<T, 64>), dim3((unsigned)ndb, 1, (unsigned)g.batch), dim3(64 * DB_WAVES), 0, s, a);
    } else {
      hipLaunchKernelGGL((db_kernel<T, 32>), dim3((unsigned)ndb, 1, (unsigned)g.batch), dim3(64 * DB_WAVES), 0, s, a);
    }
  }
  {
    const unsigned nblk = (unsigned)(g.nkt * g.nkt);
    KernelTimer t(K_DB_REDUCE, s);
    if (dbias_f32)
      hipLaunchKernelGGL(db_reduce_kernel<float>, dim3(nblk, 1, (unsigned)g.batch), dim3(256), 0, s, g, node,
                         ws.nrc, ws.slabs, dbias_f32);
    else
      hipLaunchKernelGGL(db_reduce_kernel<T>, dim3(nblk, 1, (unsigned)g.batch), dim3(256), 0, s, g, node, ws.nrc,
                         ws.slabs, dbias);
  }
  return hipGetLastError();
}

template hipError_t launch_bwd<bf16>(const Geom&, int, const Prep&, const BwdWs&, const bf16*,
                                     const bf16*, const bf16*, const bf16*, const bf16*,
                                     const float*, const bf16*, bf16*, bf16*, bf16*, bf16*,
                                     bf16*, float*, hipStream_t);
template hipError_t launch_bwd<float>(const Geom&, int, const Prep&, const BwdWs&, const float*,
                                      const float*, const float*, const float*, const float*,
                                      const float*, const float*, float*, float*, float*, float*,
                                      float*, float*, hipStream_t);

}  // namespace triattn
