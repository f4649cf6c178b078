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

#include "kernels.h"
#include "stage.h"
#include "timing.h"

namespace triattn {

template <typename T>
constexpr bool kSplitDA = std::is_same<T, bf16>::value;

// ---- elementwise preparation -------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void bwd_prep_kernel(Geom G, int node, const T* out,
                                                       const float* lse, const T* gate,
                                                       const T* dout, T* dg, T* da,
                                                       T* dalo, float* lse2) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (a, b, h)
  const int64_t total = (int64_t)G.n * G.n * G.H;
  if (idx >= total) return;
  const int h = (int)(idx % G.H);
  const int64_t pair = idx / G.H;
  const int a = (int)(pair / G.n), b = (int)(pair % G.n);
  const int64_t base = idx * HEAD_DIM;
#pragma unroll
  for (int j = 0; j < HEAD_DIM / 4; ++j) {
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
  const int row = node == 0 ? a : b, qi = node == 0 ? b : a;
  const int64_t at = ((int64_t)h * G.n + row) * G.np + qi;
  const float l = lse[idx];
  lse2[at] = l == neg_inf() ? pos_inf() : l * LOG2E;
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

// ---- dK, dV ------------------------------------------------------------------------

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
  float* dsum;  // D per (head, row, query): written by dq_kernel, read after
  T *dq, *dk, *dv;
  float* slabs;
  int nblk;  // 128-wide blocks per axis
  int nrc;   // row chunks (db)
  int rpc;   // rows per chunk (db)
};

template <typename T>
__global__ __launch_bounds__(256) void dkdv_kernel(BwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int kb = w % a.nblk, rh = w / a.nblk;
  const int r = rh % G.n, h = rh / G.n;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int kt = kb * BWD_WAVES + wave;  // this wave's key tile; lane <-> key
  const bool active = kt < G.nkt;
  const uint32_t bits = active ? a.kbits[(int64_t)r * G.nkt + kt] : 0u;
  const int key = kt * TILE + l32;
  const bool kvalid = (bits >> l32) & 1u;

  __shared__ __align__(16) T qs[TILE * LDS_ROW];       // Q tile   [query][channel]
  __shared__ __align__(16) T qT[HEAD_DIM * LDS_ROW];   // Q^T tile [channel][query]
  __shared__ __align__(16) T das[TILE * LDS_ROW];      // dA tile
  __shared__ __align__(16) T daT[HEAD_DIM * LDS_ROW];  // dA^T tile
  __shared__ __align__(16) T dalos[kSplitDA<T> ? TILE * LDS_ROW : 1];  // low part of dA
  __shared__ __align__(16) float l2s[TILE];            // lse2 of the tile's queries
  __shared__ __align__(16) float nds[TILE];            // -D of the tile's queries

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
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
  const float* bk = a.btT + ((int64_t)h * G.np + (active ? key : 0)) * G.np + 4 * g;
  const float* l2row = a.lse2 + ((int64_t)h * G.n + r) * G.np;
  const float* drow = a.dsum + ((int64_t)h * G.n + r) * G.np;

  for (int qt = 0; qt < G.nkt; ++qt) {
    __syncthreads();
    const uint32_t qbits = range_bits(qt * TILE, G.n);
    if (tid < 128) {
      stage_tile<true, true>(a.q + rowbase, G.sPos, qt * TILE, qbits, tid, qs, qT);
      if constexpr (kSplitDA<T>)
        stage_tile<true, false>(a.dalo + rowbase, G.sPos, qt * TILE, qbits, tid, dalos,
                                (T*)nullptr);
    } else {
      stage_tile<true, true>(a.da + rowbase, G.sPos, qt * TILE, qbits, tid - 128, das, daT);
    }
    if (tid < TILE) l2s[tid] = l2row[qt * TILE + tid];
    else if (tid < 2 * TILE) nds[tid - TILE] = -drow[qt * TILE + tid - TILE];
    __syncthreads();
    if (bits == 0u) continue;  // every key of this wave is masked for the row

    // S = bias + Q K^T (lane <-> key, registers <-> queries)
    f32x16 s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 x = *(const f32x4*)(bk + qt * TILE + 8 * j);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[4 * j + e] = kvalid ? x[e] : neg_inf();
    }
    typename M::frag af[M::KCH];
    row_frags(qs + l32 * LDS_ROW, g, af);
#pragma unroll
    for (int t = 0; t < M::KCH; ++t) s = M::mma(af[t], kf[t], s);
    // P = exp2(S * scale * log2 e - lse2[query])
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 l2 = *(const f32x4*)(l2s + 8 * j + 4 * g);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        s[4 * j + e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[4 * j + e], c1, -l2[e]));
    }
    // dP - D = dA V^T - D, then dS = P (dP - D)
    f32x16 dp;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 x = *(const f32x4*)(nds + 8 * j + 4 * g);
#pragma unroll
      for (int e = 0; e < 4; ++e) dp[4 * j + e] = x[e];
    }
    row_frags(das + l32 * LDS_ROW, g, af);
#pragma unroll
    for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], vf[t], dp);
    if constexpr (kSplitDA<T>) {
      row_frags(dalos + l32 * LDS_ROW, g, af);
#pragma unroll
      for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], vf[t], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) dp[v] *= s[v];

    // dV^T += dA^T P,  dK^T += Q^T dS (contraction over the tile's queries)
    typename M::frag pf[M::PCH], xf[M::PCH];
    acc_frags(s, pf);
    quad_frags(daT + l32 * LDS_ROW, g, xf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) dvt = M::mma(xf[t], pf[t], dvt);
    acc_frags(dp, pf);
    quad_frags(qT + l32 * LDS_ROW, g, xf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) dkt = M::mma(xf[t], pf[t], dkt);
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

// ---- dQ ----------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void dq_kernel(BwdArgs<T> a) {
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

  __shared__ __align__(16) T ks[TILE * LDS_ROW];      // K   [key][channel]
  __shared__ __align__(16) T kT[HEAD_DIM * LDS_ROW];  // K^T [channel][key]
  __shared__ __align__(16) T vs[TILE * LDS_ROW];      // V   [key][channel]

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
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
  // dQ = scale sum_k P (dP - D) K = scale (X - D Y) with X = sum_k P dP K,
  // Y = sum_k P K and D = sum_k P dP, all accumulated in this one pass.
  f32x16 xt = {}, yt = {};
  float dpart = 0.f;
  const uint32_t* kb = a.kbits + (int64_t)r * G.nkt;
  const float* bq = a.bt + ((int64_t)h * G.np + (active ? q : 0)) * G.np + 4 * g;

  for (int kt = 0; kt < G.nkt; ++kt) {
    const uint32_t bits = kb[kt];
    if (bits == 0u) continue;
    __syncthreads();
    if (tid < 128)
      stage_tile<true, true>(a.k + rowbase, G.sPos, kt * TILE, bits, tid, ks, kT);
    else
      stage_tile<true, false>(a.v + rowbase, G.sPos, kt * TILE, bits, tid - 128, vs, (T*)nullptr);
    __syncthreads();
    if (!active) continue;

    // S^T = bias + K Q^T (lane <-> query, registers <-> keys)
    f32x16 s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 x = *(const f32x4*)(bq + kt * TILE + 8 * j);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[4 * j + e] = x[e];
    }
    typename M::frag af[M::KCH];
    row_frags(ks + l32 * LDS_ROW, g, af);
#pragma unroll
    for (int t = 0; t < M::KCH; ++t) s = M::mma(af[t], qf[t], s);
    if (bits != 0xffffffffu) {
#pragma unroll
      for (int v = 0; v < 16; ++v)
        if (!((bits >> acc_row(v, g)) & 1u)) s[v] = neg_inf();
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2));
    // dP^T = V dA^T, then P dP and its running sum D
    row_frags(vs + l32 * LDS_ROW, g, af);
    f32x16 dp = {};
#pragma unroll
    for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], daf[t], dp);
    if constexpr (kSplitDA<T>) {
#pragma unroll
      for (int t = 0; t < M::KCH; ++t) dp = M::mma(af[t], dalf[t], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      dp[v] *= s[v];
      dpart += dp[v];
    }
    // X^T += K^T (P dP)^T,  Y^T += K^T P^T (contraction over the tile's keys)
    typename M::frag pf[M::PCH], xf[M::PCH];
    quad_frags(kT + l32 * LDS_ROW, g, xf);
    acc_frags(dp, pf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) xt = M::mma(xf[t], pf[t], xt);
    acc_frags(s, pf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) yt = M::mma(xf[t], pf[t], yt);
  }
  if (!active) return;
  const float dsum = wave_xor32_sum(dpart);
  if (!qok) return;
  if (g == 0) a.dsum[((int64_t)h * G.n + r) * G.np + q] = dsum;
  const int64_t base = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f32x4 x;
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = (xt[4 * j + e] - dsum * yt[4 * j + e]) * G.scale;
    store4(a.dq + base + 8 * j + 4 * g, x);
  }
}

// ---- dBias -------------------------------------------------------------------------

// One workgroup: 128 queries (wave <-> 32 queries, lane <-> query) x 128
// keys (4 tiles) of one head, summed over the rows of one row chunk.
template <typename T>
__global__ __launch_bounds__(256) void db_kernel(BwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int kb = w % a.nblk;
  const int qb = (w / a.nblk) % a.nblk;
  const int rc = (w / (a.nblk * a.nblk)) % a.nrc;
  const int h = w / (a.nblk * a.nblk * a.nrc);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * BWD_BLK + wave * TILE;
  if (q0 >= G.n) return;  // no barriers in this kernel
  const int q = q0 + l32;
  const bool qok = q < G.n;
  const float c1 = G.scale * LOG2E;

  f32x16 binit[BWD_WAVES], acc[BWD_WAVES];
  const float* bq = a.bt + ((int64_t)h * G.np + q) * G.np + 4 * g;
#pragma unroll
  for (int st = 0; st < BWD_WAVES; ++st) {
    acc[st] = f32x16{};
    const int kt = kb * BWD_WAVES + st;
    if (kt < G.nkt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 x = *(const f32x4*)(bq + kt * TILE + 8 * j);
#pragma unroll
        for (int e = 0; e < 4; ++e) binit[st][4 * j + e] = x[e];
      }
    }
  }

  const int r0 = rc * a.rpc, r1 = min(G.n, r0 + a.rpc);
  for (int r = r0; r < r1; ++r) {
    const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
    typename M::frag qf[M::KCH], daf[M::KCH], dalf[M::KCH];
    float l2 = pos_inf(), nd = 0.f;
    zero_frags<T>(dalf);
    if (qok) {
      row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
      row_frags(a.da + rowbase + (int64_t)q * G.sPos, g, daf);
      if constexpr (kSplitDA<T>) row_frags(a.dalo + rowbase + (int64_t)q * G.sPos, g, dalf);
      const int64_t at = ((int64_t)h * G.n + r) * G.np + q;
      l2 = a.lse2[at];
      nd = -a.dsum[at];
    } else {
      zero_frags<T>(qf);
      zero_frags<T>(daf);
    }
    if (__all(l2 == pos_inf())) continue;  // no query of the wave has a valid key
    f32x16 ndv;
#pragma unroll
    for (int v = 0; v < 16; ++v) ndv[v] = nd;
#pragma unroll
    for (int st = 0; st < BWD_WAVES; ++st) {
      const int kt = kb * BWD_WAVES + st;
      if (kt >= G.nkt) continue;
      const uint32_t bits = a.kbits[(int64_t)r * G.nkt + kt];
      if (bits == 0u) continue;
      const int key = kt * TILE + l32;  // A-operand row of this lane
      typename M::frag kf[M::KCH], vf[M::KCH];
      if ((bits >> l32) & 1u) {
        row_frags(a.k + rowbase + (int64_t)key * G.sPos, g, kf);
        row_frags(a.v + rowbase + (int64_t)key * G.sPos, g, vf);
      } else {
        zero_frags<T>(kf);
        zero_frags<T>(vf);
      }
      f32x16 s = binit[st];
#pragma unroll
      for (int t = 0; t < M::KCH; ++t) s = M::mma(kf[t], qf[t], s);
      if (bits != 0xffffffffu) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (!((bits >> acc_row(v, g)) & 1u)) s[v] = neg_inf();
      }
      f32x16 dp = ndv;
#pragma unroll
      for (int t = 0; t < M::KCH; ++t) dp = M::mma(vf[t], daf[t], dp);
      if constexpr (kSplitDA<T>) {
#pragma unroll
        for (int t = 0; t < M::KCH; ++t) dp = M::mma(vf[t], dalf[t], dp);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v)
        acc[st][v] += __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2)) * dp[v];
    }
  }
  float* slab = a.slabs + (((int64_t)rc * G.H + h) * G.np + q) * G.np + 4 * g;
#pragma unroll
  for (int st = 0; st < BWD_WAVES; ++st) {
    const int kt = kb * BWD_WAVES + st;
    if (kt >= G.nkt) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = acc[st][4 * j + e];
      *(f32x4*)(slab + kt * TILE + 8 * j) = x;
    }
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
    hipLaunchKernelGGL(bwd_prep_kernel<T>, dim3((unsigned)((npair + 255) / 256)), dim3(256), 0,
                       s, g, node, out, lse, gate, dout, dg, da, dalo, ws.lse2);
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
    // dq_kernel first: it produces D for the other two
    KernelTimer t(K_DQ, s);
    hipLaunchKernelGGL(dq_kernel<T>, dim3((unsigned)nrow), dim3(256), 0, s, a);
  }
  {
    KernelTimer t(K_DKDV, s);
    hipLaunchKernelGGL(dkdv_kernel<T>, dim3((unsigned)nrow), dim3(256), 0, s, a);
  }
  {
    const int64_t ndb = (int64_t)a.nblk * a.nblk * ws.nrc * g.H;
    KernelTimer t(K_DB, s);
    hipLaunchKernelGGL(db_kernel<T>, dim3((unsigned)ndb), dim3(256), 0, s, a);
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
