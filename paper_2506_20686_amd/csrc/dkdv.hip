// Triangle-attention backward, the paper's first stage (appendix backward
// listing): per (row, head, key block), loop over query tiles:
// dV += P^T dA, dK += scale dS^T Q.  See bwd.hip for the other passes.  The
// file stands alone so that its kernels keep the default instruction
// scheduling while the rest of the backward is built for more
// instruction-level parallelism (which costs the starting node's dK/dV
// time); the ending node's bf16 kernels are in dkdv_end.hip.
#include <type_traits>

#include "bwd.h"
#include "dkdv_dma.h"
#include "dma.h"
#include "kernels.h"
#include "stage.h"

namespace triattn {

// ---- dK, dV --------------------------------------------------------------------------

// Per (row, head, 128 keys; wave <-> 32 keys, lane <-> key): stream the row's
// queries in blocks of 64 (Q, Q^T, dA, dA^T, the low part of dA, lse2 and -D
// staged in LDS, double-buffered).  The paper's first backward stage.
template <typename T, int D>
__global__ __launch_bounds__(256, 2) void dkdv_kernel(BwdArgs<T> a) {
  to_sample(a);
  using M = Mma<T>;
  using TL = Tiles<D>;
  constexpr int KCH = kch<T, D>();
  constexpr int NO = D / 32;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int kbk = w % a.nblk, rh = w / a.nblk;
  const int r = rh % G.nr, h = rh / G.nr;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int kt = kbk * BWD_WAVES + wave;  // this wave's key tile
  const bool active = kt < G.nkt;
  const uint32_t bits = active ? a.kbits[(int64_t)r * G.nkt + kt] : 0u;
  const int key = kt * TILE + l32;
  const bool kvalid = (bits >> l32) & 1u;
  const bool work = bits != 0u;  // some key of this wave is valid for the row

  __shared__ __align__(16) T qs[2 * TL::ROWT];      // Q    [query][channel]
  __shared__ __align__(16) T qT[2 * TL::TRANS];    // Q^T  [channel][query]
  __shared__ __align__(16) T das[2 * TL::ROWT];     // dA
  __shared__ __align__(16) T daT[2 * TL::TRANS];   // dA^T
  __shared__ __align__(16) T dals[kSplitDA<T> ? 2 * TL::ROWT : 1];  // low part of dA
  __shared__ __align__(16) float l2s[2 * SPAN];     // lse2 of the block's queries
  __shared__ __align__(16) float nds[2 * SPAN];     // -D of the block's queries

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * D;
  const T* qr = a.q + rowbase;
  const T* dar = a.da + rowbase;
  const T* dalr = kSplitDA<T> ? a.dalo + rowbase : nullptr;
  const int last = G.n - 1;
  typename M::frag kf[KCH], vf[KCH];
  if (kvalid) {
    row_frags(a.k + rowbase + (int64_t)key * G.sPos, g, kf);
    row_frags(a.v + rowbase + (int64_t)key * G.sPos, g, vf);
  } else {
    zero_frags(kf);
    zero_frags(vf);
  }
  const float c1 = G.scale * LOG2E;
  f32x16 dkt[NO] = {}, dvt[NO] = {};
  const int ktc = active ? kt : 0;  // key tile of the key-major bias (0 for idle waves)
  const float* l2row = a.lse2 + ((int64_t)h * G.nr + r) * G.np;
  const float* drow = a.dsum + ((int64_t)h * G.nr + r) * G.np;
  const int nblk = (G.nkt + 1) >> 1;  // query blocks of 64
  const float kmask = kvalid ? 0.f : neg_inf();
  auto bias_tile = [&](int t) {
    f32x16 x = load_frag_tile(frag_tile(a.btT, h, ktc, min(t, G.nkt - 1), G.nkt), lane);
#pragma unroll
    for (int v = 0; v < 16; ++v) x[v] += kmask;  // -inf for a masked key
    return x;
  };

  PairPiece<T, D> qp, dap;
  RowPiece<T, D> dlp;
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
    qp.store_rows(qs + bf * TL::ROWT, tid);
    qp.store_trans(qT + bf * TL::TRANS, tid);
    dap.store_rows(das + bf * TL::ROWT, tid);
    dap.store_trans(daT + bf * TL::TRANS, tid);
    if constexpr (kSplitDA<T>) dlp.store(dals + bf * TL::ROWT, tid, vb);
    const bool in = b * SPAN + sq < G.np;  // queries n..np-1 carry +inf / 0 already
    if (tid < SPAN)
      l2s[bf * SPAN + sq] = in ? sv : pos_inf();
    else if (tid < 2 * SPAN)
      nds[bf * SPAN + sq] = in ? sv : 0.f;
  };
  auto sub_tile = [&](int bf, const f32x16& bias, int u) {
    const T* qsb = qs + bf * TL::ROWT;
    // S = bias + Q K^T (lane <-> key, registers <-> queries)
    typename M::frag af[KCH];
    row_frags(qsb + (32 * u + l32) * TL::ROW, g, af);
    f32x16 s = M::mma(af[0], kf[0], bias);
#pragma unroll
    for (int t = 1; t < KCH; ++t) s = M::mma(af[t], kf[t], s);
    // P = exp2(S scale log2 e - lse2[query])
    const f32x16 l2 = load_quads(l2s + bf * SPAN + 32 * u + 4 * g);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -l2[v]));
    // dP - D = dA V^T - D, then dS = P (dP - D)
    row_frags(das + bf * TL::ROWT + (32 * u + l32) * TL::ROW, g, af);
    f32x16 dp = M::mma(af[0], vf[0], load_quads(nds + bf * SPAN + 32 * u + 4 * g));
#pragma unroll
    for (int t = 1; t < KCH; ++t) dp = M::mma(af[t], vf[t], dp);
    if constexpr (kSplitDA<T>) {
      row_frags(dals + bf * TL::ROWT + (32 * u + l32) * TL::ROW, g, af);
#pragma unroll
      for (int t = 0; t < KCH; ++t) dp = M::mma(af[t], vf[t], dp);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) dp[v] *= s[v];
    // dV^T += dA^T P,  dK^T += Q^T dS (contraction over the block's queries)
    typename M::frag pf[M::PCH], xf[M::PCH];
    acc_frags(s, pf);
#pragma unroll
    for (int c = 0; c < NO; ++c) {
      quad_frags(daT + bf * TL::TRANS + (32 * c + l32) * LDS_TROW + 32 * u, g, xf);
#pragma unroll
      for (int t = 0; t < M::PCH; ++t) dvt[c] = M::mma(xf[t], pf[t], dvt[c]);
    }
    acc_frags(dp, pf);
#pragma unroll
    for (int c = 0; c < NO; ++c) {
      quad_frags(qT + bf * TL::TRANS + (32 * c + l32) * LDS_TROW + 32 * u, g, xf);
#pragma unroll
      for (int t = 0; t < M::PCH; ++t) dkt[c] = M::mma(xf[t], pf[t], dkt[c]);
    }
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
  for (int c = 0; c < NO; ++c)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c0 = 32 * c + 8 * j + 4 * g;
      f32x4 x, y;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = dvt[c][4 * j + e];
        y[e] = dkt[c][4 * j + e] * G.scale;
      }
      store4(a.dv + base + c0, x);
      store4(a.dk + base + c0, y);
    }
}


template <int D>
__global__ __launch_bounds__(64 * KD_WAVES) void dkdv_dma_kernel(BwdArgs<bf16> a) {
  dkdv_dma_body<D>(a);
}

template <typename T>
hipError_t launch_dkdv(const BwdArgs<T>& a, int node, hipStream_t s) {
  const Geom& g = a.g;
  const bool d64 = g.d == 64, d16 = g.d == 16;
  if constexpr (std::is_same<T, bf16>::value) {
    if (node != 0) return launch_dkdv_dma_end(a, s);
    const int64_t nwg = (int64_t)a.nblk * ((g.nr + KD_ROWS - 1) / KD_ROWS) * g.H;
    if (d64)
      hipLaunchKernelGGL(dkdv_dma_kernel<64>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * KD_WAVES), 0, s, a);
    else if (d16)
      hipLaunchKernelGGL(dkdv_dma_kernel<16>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * KD_WAVES), 0, s, a);
    else
      hipLaunchKernelGGL(dkdv_dma_kernel<32>, dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(64 * KD_WAVES), 0, s, a);
  } else {
    const int64_t nrow = (int64_t)a.nblk * g.nr * g.H;
    if (d64)
      hipLaunchKernelGGL((dkdv_kernel<T, 64>), dim3((unsigned)nrow, 1, (unsigned)g.batch), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((dkdv_kernel<T, 32>), dim3((unsigned)nrow, 1, (unsigned)g.batch), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

template hipError_t launch_dkdv<bf16>(const BwdArgs<bf16>&, int, hipStream_t);
template hipError_t launch_dkdv<float>(const BwdArgs<float>&, int, hipStream_t);

}  // namespace triattn
