// Triangle-attention forward (MegaFold Section IV-A, "EvoFlash-3D" forward):
// per (row, head, block of queries) stream the key tiles of the row, keep a
// running max and sum (online softmax), rescale and accumulate the output,
// and save the log-sum-exp.  Also the per-call preparation kernels.
//
// Differences from the paper's Triton kernel, for gfx950:
//  - one workgroup = 4 waves = 128 queries of one (row, head); the K and V
//    tiles of the row are staged once in LDS and shared by the 4 waves;
//  - logits are formed transposed (S^T = K Q^T) so that each lane owns one
//    query: the running max/sum are per-lane scalars and the output
//    accumulator O^T = V^T P^T is rescaled with one multiply per register;
//  - the bias (pre-divided by the scale, laid out query-major) is the
//    initial MFMA accumulator, so adding it costs no vector instruction, and
//    the softmax runs in base 2 with scale * log2(e) folded into one FMA;
//  - the sigmoid gate is applied in the epilogue;
//  - key tiles that are fully masked for the row are skipped;
//  - keys stream in blocks of 64 through double-buffered LDS: the next
//    block's loads are issued before the current block is computed, one
//    barrier per block;
//  - the running max is only raised when it grows by more than 2^8, so the
//    rescale of the accumulator is rare.
#include "kernels.h"
#include "stage.h"
#include "timing.h"

namespace triattn {

// ---- preparation ------------------------------------------------------------------

// bias / scale over the zero-padded np x np map, in accumulator order (see
// frag_tile): x = 32 t1 + l % 32 is the lane's column, y = 32 t2 + 8 j +
// 4 (l / 32) + e its row.  bt holds bias(query x, key y) for the kernels
// whose lanes own queries; btT holds bias(query y, key x) for the kernel
// whose lanes own keys.  The starting node reads bias[q][k][h], the ending
// node bias[k][q][h].
template <typename T>
__global__ __launch_bounds__(256) void prep_bias_kernel(Geom G, int node, const T* bias,
                                                        float* bt, float* btT) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t np = G.np, total = (int64_t)G.H * np * np;
  if (idx >= total) return;
  const int nt = G.nkt;
  const int e = (int)(idx & 3), l = (int)((idx >> 2) & 63), j = (int)((idx >> 8) & 3);
  const int64_t tt = idx >> 10;
  const int t2 = (int)(tt % nt), t1 = (int)((tt / nt) % nt), h = (int)(tt / ((int64_t)nt * nt));
  const int x = 32 * t1 + (l & 31), y = 32 * t2 + 8 * j + 4 * (l >> 5) + e;
  const int n = G.n;
  auto at = [&](int qi, int ki) -> int64_t {
    return node == 0 ? ((int64_t)qi * n + ki) * G.H + h : ((int64_t)ki * n + qi) * G.H + h;
  };
  const bool in = x < n && y < n;
  bt[idx] = in ? (float)bias[at(x, y)] / G.scale : 0.f;
  if (btT) btT[idx] = in ? (float)bias[at(y, x)] / G.scale : 0.f;
}

// kbits[row][t]: bit e set iff key 32 t + e < n and mask(row, key) != 0.
// The starting node reads mask[row][key], the ending node mask[key][row].
__global__ __launch_bounds__(256) void prep_kbits_kernel(Geom G, int node, const uint8_t* mask,
                                                         uint32_t* kbits) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)G.n * G.nkt) return;
  const int row = (int)(idx / G.nkt), t = (int)(idx % G.nkt), n = G.n;
  uint32_t bits = 0;
  for (int e = 0; e < 32; ++e) {
    const int key = 32 * t + e;
    if (key >= n) break;
    const bool ok = mask == nullptr ||
                    mask[node == 0 ? (int64_t)row * n + key : (int64_t)key * n + row] != 0;
    bits |= (ok ? 1u : 0u) << e;
  }
  kbits[idx] = bits;
}

template <typename T>
hipError_t launch_prep(const Geom& g, int node, const T* bias, const uint8_t* mask, const Prep& p,
                       hipStream_t s) {
  const int64_t nb = ((int64_t)g.H * g.np * g.np + 255) / 256;
  {
    KernelTimer t(K_PREP_BIAS, s);
    hipLaunchKernelGGL(prep_bias_kernel<T>, dim3((unsigned)nb), dim3(256), 0, s, g, node, bias,
                       p.bt, p.btT);
  }
  const int64_t nk = ((int64_t)g.n * g.nkt + 255) / 256;
  {
    KernelTimer t(K_PREP_KBITS, s);
    hipLaunchKernelGGL(prep_kbits_kernel, dim3((unsigned)nk), dim3(256), 0, s, g, node, mask,
                       p.kbits);
  }
  return hipGetLastError();
}

// ---- forward ----------------------------------------------------------------------

constexpr int FWD_WAVES = 4;
constexpr int FWD_QBLK = FWD_WAVES * TILE;  // queries per workgroup
// The running max only moves when a lane's block max exceeds it by more than
// this (log2 units), so unnormalised weights stay <= 2^8 and most blocks skip
// the rescale of the accumulator.  Any stale max gives the same result.
constexpr float STALE_MAX_SLACK = 8.f;

template <typename T>
struct FwdArgs {
  Geom g;
  const float* bt;
  const uint32_t* kbits;
  const T *q, *k, *v, *gate;
  T* out;
  float* lse;
  int nqb;  // query blocks per row
};

template <typename T>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int qb = w % a.nqb, rh = w / a.nqb;
  const int r = rh % G.n, h = rh / G.n;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * FWD_QBLK + wave * TILE;  // first query of this wave
  const bool active = q0 < G.n;
  const int q = q0 + l32;
  const bool qok = q < G.n;

  __shared__ __align__(16) T ks[2 * ROW_TILE];    // K block   [key][channel], 2 buffers
  __shared__ __align__(16) T vt[2 * TRANS_TILE];  // V^T block [channel][key], 2 buffers

  const int64_t rowbase = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
  const T* kr = a.k + rowbase;
  const T* vr = a.v + rowbase;
  const int last = G.n - 1;
  typename M::frag qf[M::KCH];
  if (qok)
    row_frags(a.q + rowbase + (int64_t)q * G.sPos, g, qf);
  else
    zero_frags<T>(qf);

  const float c1 = G.scale * LOG2E;
  float m = neg_inf(), lsum = 0.f;
  f32x16 o = {};
  const uint32_t* kb = a.kbits + (int64_t)r * G.nkt;
  const int nblk = (G.nkt + 1) >> 1;
  // bias tiles of this wave's queries (tile 0 for idle waves: loads stay in bounds)
  const int qt = active ? q0 / TILE : 0;
  auto bias_tile = [&](int kt) {
    return load_frag_tile(frag_tile(a.bt, h, qt, min(kt, G.nkt - 1), G.nkt), lane);
  };

  // one 32-key sub-tile: logits, online softmax (base 2, stale max), P V
  auto sub_tile = [&](const T* ksb, const T* vtb, const f32x16& bias, uint32_t bits, int u) {
    typename M::frag kf[M::KCH];
    row_frags(ksb + (32 * u + l32) * LDS_ROW, g, kf);
    f32x16 s = M::mma(kf[0], qf[0], bias);  // s^T = bias + K Q^T
#pragma unroll
    for (int t = 1; t < M::KCH; ++t) s = M::mma(kf[t], qf[t], s);
    if (bits != 0xffffffffu) mask_rows(s, bits, g);
    const float mx = wave_xor32_max(max16(s)) * c1;
    if (__any(mx > m + STALE_MAX_SLACK)) {
      const float mnew = fmaxf(m, mx);
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      lsum *= alpha;
#pragma unroll
      for (int v = 0; v < 16; ++v) o[v] *= alpha;
      m = mnew;
    }
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -m));
      ps += s[v];
    }
    lsum += ps;
    typename M::frag pf[M::PCH], vf[M::PCH];
    acc_frags(s, pf);
    quad_frags(vtb + l32 * LDS_TROW + 32 * u, g, vf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) o = M::mma(vf[t], pf[t], o);  // O^T += V^T P^T
  };

  RowPiece<T> kp;
  PairPiece<T> vp;
  uint64_t bb = block_bits(kb, G.nkt, 0);
  kp.load(kr, G.sPos, 0, last, tid);
  vp.load(vr, G.sPos, 0, last, tid);
  f32x16 b0 = bias_tile(0), b1 = bias_tile(1);
  kp.store(ks, tid, bb);
  vp.validate(tid, bb);
  vp.store_trans(vt, tid);
  __syncthreads();
  int buf = 0;
  for (int b = 0; b < nblk; ++b) {
    // issue the next block's loads (the last block reloads itself, unused)
    const int bn = min(b + 1, nblk - 1);
    const uint64_t bbn = block_bits(kb, G.nkt, bn);
    kp.load(kr, G.sPos, bn * SPAN, last, tid);
    vp.load(vr, G.sPos, bn * SPAN, last, tid);
    const f32x16 n0 = bias_tile(2 * bn), n1 = bias_tile(2 * bn + 1);
    if (active) {
      const T* ksb = ks + buf * ROW_TILE;
      const T* vtb = vt + buf * TRANS_TILE;
      if ((uint32_t)bb) sub_tile(ksb, vtb, b0, (uint32_t)bb, 0);
      if ((uint32_t)(bb >> 32)) sub_tile(ksb, vtb, b1, (uint32_t)(bb >> 32), 1);
    }
    if (b + 1 < nblk) {
      kp.store(ks + (buf ^ 1) * ROW_TILE, tid, bbn);
      vp.validate(tid, bbn);
      vp.store_trans(vt + (buf ^ 1) * TRANS_TILE, tid);
    }
    __syncthreads();
    b0 = n0;
    b1 = n1;
    bb = bbn;
    buf ^= 1;
  }
  if (!active) return;

  // epilogue: normalise, gate, store; lse = ln(sum exp) = (m + log2 l) ln 2
  const float lt = wave_xor32_sum(lsum);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (!qok) return;
  const int64_t base = rowbase + (int64_t)q * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c0 = 8 * j + 4 * g;
    const f32x4 gv = load4(a.gate + base + c0);
    f32x4 ov;
#pragma unroll
    for (int e = 0; e < 4; ++e) ov[e] = o[4 * j + e] * inv / (1.f + __expf(-gv[e]));
    store4(a.out + base + c0, ov);
  }
  if (g == 0)
    a.lse[(int64_t)r * G.lRow + (int64_t)q * G.lPos + h] =
        lt > 0.f ? (m + log2f(lt)) * LN2 : neg_inf();
}

template <typename T>
hipError_t launch_fwd(const Geom& g, const Prep& p, const T* q, const T* k, const T* v,
                      const T* gate, T* out, float* lse, hipStream_t s) {
  FwdArgs<T> a{g, p.bt, p.kbits, q, k, v, gate, out, lse, (g.n + FWD_QBLK - 1) / FWD_QBLK};
  const int64_t nwg = (int64_t)a.nqb * g.n * g.H;
  {
    KernelTimer t(K_FWD, s);
    hipLaunchKernelGGL(fwd_kernel<T>, dim3((unsigned)nwg), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

template hipError_t launch_prep<bf16>(const Geom&, int, const bf16*, const uint8_t*, const Prep&,
                                      hipStream_t);
template hipError_t launch_prep<float>(const Geom&, int, const float*, const uint8_t*,
                                       const Prep&, hipStream_t);
template hipError_t launch_fwd<bf16>(const Geom&, const Prep&, const bf16*, const bf16*,
                                     const bf16*, const bf16*, bf16*, float*, hipStream_t);
template hipError_t launch_fwd<float>(const Geom&, const Prep&, const float*, const float*,
                                      const float*, const float*, float*, float*, hipStream_t);

}  // namespace triattn
