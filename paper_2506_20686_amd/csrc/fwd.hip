// Triangle-attention forward (MegaFold Section IV-A, "EvoFlash-3D" forward):
// per (row, head, block of queries) stream the key tiles of the row, keep a
// running max and sum (online softmax), rescale and accumulate the output,
// and save the log-sum-exp.  Also the per-call preparation kernels.
//
// Differences from the paper's Triton kernel, for gfx950:
//  - one bf16 workgroup = 8 waves = 128 queries x 4 rows of one head; the
//    K and V tiles of the rows and the bias tiles of the queries (shared by
//    the rows) are copied into LDS by DMA and shared by the waves;
//  - logits are formed transposed (S^T = K Q^T) so that each lane owns one
//    query: the running max/sum are per-lane scalars and the output
//    accumulator O^T = V^T P^T is rescaled with one multiply per register;
//  - the bias (pre-divided by the scale, laid out query-major) is the
//    initial MFMA accumulator, so adding it costs no vector instruction, and
//    the softmax runs in base 2 with scale * log2(e) folded into one FMA;
//  - the sigmoid gate is applied in the epilogue;
//  - key tiles that are fully masked for the row are skipped, and rows with
//    every key valid take a loop without mask steps;
//  - the running max is only raised when it grows by more than 2^8, so the
//    rescale of the accumulator is rare.
#include <type_traits>

#include "dma.h"
#include "kernels.h"
#include "stage.h"
#include "timing.h"

namespace triattn {

// ---- preparation ------------------------------------------------------------------

// bias / scale over the zero-padded np x np map, in accumulator order (see
// frag_tile): in tile (t1, t2), element 256 j + 4 l + e has x = 32 t1 + l % 32
// as the lane's column and y = 32 t2 + 8 j + 4 (l / 32) + e as its row.  bt
// holds bias(query x, key y) for the kernels whose lanes own queries; btT
// holds bias(query y, key x) for the kernel whose lanes own keys.  The
// starting node reads bias[q][k][h], the ending node bias[k][q][h].
//
// One workgroup per 32 x 32 block (query tile qa, key tile kb) of the map,
// one head at a time: the block goes through LDS once and leaves as bt tile
// (qa, kb) and btT tile (kb, qa), both written 16 bytes per thread.
template <typename T>
__device__ inline void load_heads4(const T* p, float (&x)[4]);
template <>
__device__ inline void load_heads4(const bf16* p, float (&x)[4]) {
  const bf16x4 v = *(const bf16x4*)p;
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = (float)v[j];
}
template <>
__device__ inline void load_heads4(const float* p, float (&x)[4]) {
  const f32x4 v = *(const f32x4*)p;
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = v[j];
}

template <typename T>
__global__ __launch_bounds__(256) void prep_bias_kernel(Geom G, int node, const T* bias,
                                                        float* bt, float* btT) {
  bias = at_sample(bias, G.bBias);
  bt = ws_at_sample(bt, G.bWs);
  btT = ws_at_sample(btT, G.bWs);
  const int nt = G.nkt, n = G.n;
  const int qa = blockIdx.x % nt, kb = blockIdx.x / nt;
  const int tid = threadIdx.x;
  constexpr int HG = 4;  // heads per pass through LDS
  __shared__ float tl[HG][32][33];  // [head][query][key] of HG heads: bias / scale
  // loads: query r, keys c0 .. c0 + 3 of the block, HG heads each (one
  // vector load per key when the head count is a multiple of HG)
  const int r = tid >> 3, c0 = 4 * (tid & 7);
  const int q = 32 * qa + r;
  const bool vec = G.H % HG == 0;
  // stores: element 4 tid .. 4 tid + 3 of a tile (j = tid / 64, l = tid % 64)
  const int l = tid & 63, x = l & 31, y0 = 8 * (tid >> 6) + 4 * (l >> 5);
  for (int h0 = 0; h0 < G.H; h0 += HG) {
    const int hn = min(HG, G.H - h0);
    float v[4][HG];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = 32 * kb + c0 + e;
      const int qc = min(q, n - 1), kc = min(k, n - 1);  // in bounds; zero outside the map
      const int64_t at = (node == 0 ? (int64_t)qc * n + kc : (int64_t)kc * n + qc) * G.H + h0;
      if (vec) {
        load_heads4(bias + at, v[e]);
      } else {
#pragma unroll
        for (int j = 0; j < HG; ++j) v[e][j] = j < hn ? (float)bias[at + j] : 0.f;
      }
      if (!(q < n && k < n)) {
#pragma unroll
        for (int j = 0; j < HG; ++j) v[e][j] = 0.f;
      }
    }
    __syncthreads();  // the previous heads' tiles have been read
#pragma unroll
    for (int j = 0; j < HG; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) tl[j][r][c0 + e] = v[e][j] / G.scale;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < HG; ++j) {
      if (j >= hn) break;
      const int h = h0 + j;
      const f32x4 o = {tl[j][x][y0], tl[j][x][y0 + 1], tl[j][x][y0 + 2], tl[j][x][y0 + 3]};
      *(f32x4*)(bt + (((int64_t)h * nt + qa) * nt + kb) * 1024 + 4 * tid) = o;
      if (btT) {
        const f32x4 p = {tl[j][y0][x], tl[j][y0 + 1][x], tl[j][y0 + 2][x], tl[j][y0 + 3][x]};
        *(f32x4*)(btT + (((int64_t)h * nt + kb) * nt + qa) * 1024 + 4 * tid) = p;
      }
    }
  }
}

// kbits[row][t]: bit e set iff key 32 t + e < n and mask(row, key) != 0.
// rowfull[row] = 1 iff every key < n is valid for the row.
//
// Starting node, mask[row][key] (a row's keys contiguous): one workgroup per
// row; each wave reads 64 consecutive keys per load and forms two words with
// a ballot.
__global__ __launch_bounds__(256) void prep_kbits_start_kernel(Geom G, const uint8_t* mask,
                                                               uint32_t* kbits,
                                                               uint32_t* rowfull) {
  mask = at_sample(mask, G.bMask);
  kbits = ws_at_sample(kbits, G.bWs);
  rowfull = ws_at_sample(rowfull, G.bWs);
  const int row = blockIdx.x, n = G.n;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  bool full = true;
  for (int k0 = 64 * wave; k0 < G.np; k0 += 256) {
    const int key = k0 + lane;
    const bool in = key < n;
    const bool ok = in && (mask == nullptr || mask[(int64_t)row * n + min(key, n - 1)] != 0);
    const uint64_t b = __ballot(ok), want = __ballot(in);
    full = full && b == want;
    const int t = k0 >> 5;
    if (lane == 0) kbits[(int64_t)row * G.nkt + t] = (uint32_t)b;
    if (lane == 1 && t + 1 < G.nkt) kbits[(int64_t)row * G.nkt + t + 1] = (uint32_t)(b >> 32);
  }
  const int all = __syncthreads_and(full);
  if (threadIdx.x == 0) rowfull[row] = all ? 1u : 0u;
}

// Ending node, mask[key][row] (consecutive rows contiguous): one workgroup
// per 64 rows, lane <-> row; wave w builds words w, w + 16, ... of the 64
// rows, one 64-byte read of a key's row of the mask per bit.
__global__ __launch_bounds__(1024) void prep_kbits_end_kernel(Geom G, const uint8_t* mask,
                                                              uint32_t* kbits,
                                                              uint32_t* rowfull) {
  mask = at_sample(mask, G.bMask);
  kbits = ws_at_sample(kbits, G.bWs);
  rowfull = ws_at_sample(rowfull, G.bWs);
  const int n = G.n;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = 64 * blockIdx.x + lane;
  const bool rin = row < G.nr;
  const int rowc = min(row, G.nr - 1);  // in-bounds address for lanes past the last row
  bool full = true;
  for (int t = wave; t < G.nkt; t += 16) {
    const uint32_t want = in_range_bits(t, n);
    uint32_t bits = rin ? want : 0u;
    if (mask != nullptr) {
      // every load first (addresses clamped in bounds), then the bits
      uint8_t m[32];
#pragma unroll
      for (int e = 0; e < 32; ++e) m[e] = mask[(int64_t)min(32 * t + e, n - 1) * n + rowc];
#pragma unroll
      for (int e = 0; e < 32; ++e)
        if (m[e] == 0) bits &= ~(1u << e);
    }
    if (rin) kbits[(int64_t)row * G.nkt + t] = bits;
    full = full && bits == want;
  }
  __shared__ uint32_t part[16][64];
  part[wave][lane] = full ? 1u : 0u;
  __syncthreads();
  if (wave == 0 && rin) {
    uint32_t all = 1u;
#pragma unroll
    for (int w = 0; w < 16; ++w) all &= part[w][lane];
    rowfull[row] = all;
  }
}

template <typename T>
hipError_t launch_prep(const Geom& g, int node, const T* bias, const uint8_t* mask, const Prep& p,
                       hipStream_t s) {
  {
    KernelTimer t(K_PREP_BIAS, s);
    hipLaunchKernelGGL(prep_bias_kernel<T>, dim3((unsigned)(g.nkt * g.nkt), 1, (unsigned)g.batch), dim3(256), 0, s,
                       g, node, bias, p.bt, p.btT);
  }
  {
    KernelTimer t(K_PREP_KBITS, s);
    if (node == 0)
      hipLaunchKernelGGL(prep_kbits_start_kernel, dim3((unsigned)g.nr, 1, (unsigned)g.batch), dim3(256), 0, s, g,
                         mask, p.kbits, p.rowfull);
    else
      hipLaunchKernelGGL(prep_kbits_end_kernel, dim3((unsigned)((g.nr + 63) / 64), 1, (unsigned)g.batch), dim3(1024),
                         0, s, g, mask, p.kbits, p.rowfull);
  }
  return hipGetLastError();
}

// ---- forward ----------------------------------------------------------------------

constexpr int FWD_WAVES = 4;
constexpr int FWD_QBLK = FWD_WAVES * TILE;  // queries per workgroup
constexpr int FWD_ROWS = 1;                 // rows per workgroup (they share the bias tiles)
// The running max only moves when a lane's block max exceeds it by more than
// this (log2 units), so unnormalised weights stay <= 2^8 and most blocks skip
// the rescale of the accumulator.  Any stale max gives the same result.
constexpr float STALE_MAX_SLACK = 8.f;
// Starting value of the running max: finite, so that a query whose keys so
// far all have logit -inf (an additive -inf bias) keeps m - mnew = 0 when
// another lane of its wave raises the wave's maxima, and exp2(-inf - m) = 0;
// any finite logit exceeds it by more than the slack.
constexpr float M_FLOOR = -3.4028234663852886e38f;
// Largest per-lane tile sum of weights (32 keys, relative to the running max)
// the bf16 forward accepts without raising the max: weights stay below 2^64,
// so over at most 256 tiles the sums and the weighted values stay finite.
constexpr float WEIGHT_LIMIT = 1.8446744e19f;  // 2^64

template <typename T>
struct FwdArgs {
  Geom g;
  const float* bt;
  const uint32_t* kbits;
  const uint32_t* rowfull;
  const T *q, *k, *v, *gate;
  T* out;
  float* lse;
  int nqb;  // query blocks per row
};

// This block's sample of a batched launch: every tensor and workspace piece
// moved by the sample's strides (no change for sample 0).
template <typename T>
__device__ inline void to_sample(FwdArgs<T>& a) {
  const Geom& G = a.g;
  a.bt = ws_at_sample(a.bt, G.bWs);
  a.kbits = ws_at_sample(a.kbits, G.bWs);
  a.rowfull = ws_at_sample(a.rowfull, G.bWs);
  a.q = at_sample(a.q, G.bPair);
  a.k = at_sample(a.k, G.bPair);
  a.v = at_sample(a.v, G.bPair);
  a.gate = at_sample(a.gate, G.bPair);
  a.out = at_sample(a.out, G.bPair);
  a.lse = at_sample(a.lse, G.bBias);
}

// Online-softmax state of one (row, 32 queries) pair of a wave.  The row
// sums of P accumulate on the MFMA: register 0 of the lanes of half 0 of
// `l` holds sum_k P for the lane's query (see ones_row0).
template <int D>
struct SoftmaxState {
  float m;
  f32x16 l;
  f32x16 o[D / 32];  // O^T accumulators (32 channels each): registers <-> channels, lane <-> query
};

// Forward with register-staged operand blocks (stage.h), for D = 32 or 64
// channels per head.
template <typename T, int D>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdArgs<T> a) {
  to_sample(a);
  using M = Mma<T>;
  using TL = Tiles<D>;
  constexpr int KCH = kch<T, D>();
  constexpr int NO = D / 32;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int qb = w % a.nqb, rh = w / a.nqb;
  const int nrp = (G.nr + FWD_ROWS - 1) / FWD_ROWS;
  const int r0 = (rh % nrp) * FWD_ROWS, h = rh / nrp;
  const bool row1 = FWD_ROWS > 1 && r0 + 1 < G.nr;  // the second row exists
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * FWD_QBLK + wave * TILE;  // first query of this wave
  const bool active = q0 < G.n;
  const int q = q0 + l32;
  const bool qok = q < G.n;

  // K block [key][channel] and V^T block [channel][key] of both rows, 2 buffers
  __shared__ __align__(16) T ks[2 * FWD_ROWS * TL::ROWT];
  __shared__ __align__(16) T vt[2 * FWD_ROWS * TL::TRANS];

  const int last = G.n - 1;  // last key position
  int64_t rowbase[FWD_ROWS];
  typename M::frag qf[FWD_ROWS][KCH];
  const uint32_t* kb[FWD_ROWS];
  SoftmaxState<D> st[FWD_ROWS];
#pragma unroll
  for (int i = 0; i < FWD_ROWS; ++i) {
    const int r = min(r0 + i, G.nr - 1);
    rowbase[i] = (int64_t)r * G.sRow + (int64_t)h * D;
    kb[i] = a.kbits + (int64_t)r * G.nkt;
    if (qok)
      row_frags(a.q + rowbase[i] + (int64_t)q * G.sPos, g, qf[i]);
    else
      zero_frags(qf[i]);
    st[i].m = M_FLOOR;
    st[i].l = f32x16{};
#pragma unroll
    for (int c = 0; c < NO; ++c) st[i].o[c] = f32x16{};
  }

  const float c1 = G.scale * LOG2E;
  const int nblk = (G.nkt + 1) >> 1;
  // bias tiles of this wave's queries (tile 0 for idle waves: loads stay in bounds)
  const int qt = active ? q0 / TILE : 0;
  auto bias_tile = [&](int kt) {
    return load_frag_tile(frag_tile(a.bt, h, qt, min(kt, G.nkt - 1), G.nkt), lane);
  };
  // key bits of block b for both rows (the second row's are zero if it does not exist)
  auto bits_of = [&](int b, uint64_t(&bb)[FWD_ROWS]) {
    bb[0] = block_bits(kb[0], G.nkt, b);
    if constexpr (FWD_ROWS > 1) bb[1] = row1 ? block_bits(kb[1], G.nkt, b) : 0ull;
  };
  const typename M::frag ones = ones_row0<typename M::frag>(l32);

  // raise the running max to include mx (log2 units) and rescale the state
  auto rescale = [&](SoftmaxState<D>& S, float mx) {
    const float mnew = fmaxf(S.m, mx);
    const float alpha = __builtin_amdgcn_exp2f(S.m - mnew);
    S.l[0] *= alpha;  // rows 1..31 of l stay zero
#pragma unroll
    for (int c = 0; c < NO; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) S.o[c][v] *= alpha;
    S.m = mnew;
  };

  // one 32-key sub-tile of one row: logits, online softmax (base 2, stale max), P V
  auto sub_tile = [&](SoftmaxState<D>& S, const typename M::frag(&qfr)[KCH], const T* ksb,
                      const T* vtb, const f32x16& bias, uint32_t bits, int u) {
    typename M::frag kf[KCH];
    row_frags(ksb + (32 * u + l32) * TL::ROW, g, kf);
    f32x16 s = M::mma(kf[0], qfr[0], bias);  // s^T = bias + K Q^T
#pragma unroll
    for (int t = 1; t < KCH; ++t) s = M::mma(kf[t], qfr[t], s);
    if (bits != 0xffffffffu) mask_rows(s, bits, g);
    const float mx = wave_xor32_max(max16(s)) * c1;
    if (__any(mx > S.m + STALE_MAX_SLACK)) rescale(S, mx);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -S.m));
    typename M::frag pf[M::PCH], vf[M::PCH];
    acc_frags(s, pf);
#pragma unroll
    for (int c = 0; c < NO; ++c) {
      quad_frags(vtb + (32 * c + l32) * LDS_TROW + 32 * u, g, vf);
#pragma unroll
      for (int t = 0; t < M::PCH; ++t) S.o[c] = M::mma(vf[t], pf[t], S.o[c]);  // O^T += V^T P^T
    }
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) S.l = M::mma(ones, pf[t], S.l);  // row sums of P
  };

  // A full 64-key block (every key valid in both rows): one straight-line
  // stretch -- all logit MFMAs, then the maxes, one (rare) rescale per row,
  // then exp / sums / bf16 packing interleaved with the P V MFMAs -- so the
  // scheduler can overlap the two rows' and sub-tiles' independent work.
  auto full_block = [&](int buf, const f32x16& c0, const f32x16& c1b) {
    f32x16 s[FWD_ROWS][2];
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) {
      const T* ksb = ks + (buf * FWD_ROWS + i) * TL::ROWT;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        typename M::frag kf[KCH];
        row_frags(ksb + (32 * u + l32) * TL::ROW, g, kf);
        s[i][u] = M::mma(kf[0], qf[i][0], u ? c1b : c0);
#pragma unroll
        for (int t = 1; t < KCH; ++t) s[i][u] = M::mma(kf[t], qf[i][t], s[i][u]);
      }
    }
    float mx[FWD_ROWS];
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) mx[i] = wave_xor32_max(max32(s[i][0], s[i][1])) * c1;
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i)
      if (__any(mx[i] > st[i].m + STALE_MAX_SLACK)) rescale(st[i], mx[i]);
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) {
      SoftmaxState<D>& S = st[i];
      const T* vtb = vt + (buf * FWD_ROWS + i) * TL::TRANS;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          s[i][u][v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[i][u][v], c1, -S.m));
        typename M::frag pf[M::PCH], vf[M::PCH];
        acc_frags(s[i][u], pf);
#pragma unroll
        for (int c = 0; c < NO; ++c) {
          quad_frags(vtb + (32 * c + l32) * LDS_TROW + 32 * u, g, vf);
#pragma unroll
          for (int t = 0; t < M::PCH; ++t) S.o[c] = M::mma(vf[t], pf[t], S.o[c]);
        }
#pragma unroll
        for (int t = 0; t < M::PCH; ++t) S.l = M::mma(ones, pf[t], S.l);
      }
    }
  };

  // staging: each row's block is 256 K pieces and 256 V pieces (64 positions
  // x 32 channels); thread tid moves FWD_ROWS consecutive pieces of row srow
  constexpr int TPR = 256 / FWD_ROWS;  // threads per staged row
  RowPiece<T, D> kp[FWD_ROWS];
  PairPiece<T, D> vp[FWD_ROWS];
  const int srow = tid / TPR;
  const int sp0 = FWD_ROWS * (tid % TPR);
  const T* skr = a.k + rowbase[srow];
  const T* svr = a.v + rowbase[srow];
  auto stage_load = [&](int b) {
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) {
      kp[i].load(skr, G.sPos, b * SPAN, last, sp0 + i);
      vp[i].load(svr, G.sPos, b * SPAN, last, sp0 + i);
    }
  };
  auto stage_store = [&](int buf, const uint64_t(&bb)[FWD_ROWS]) {
    T* kd = ks + (buf * FWD_ROWS + srow) * TL::ROWT;
    T* vd = vt + (buf * FWD_ROWS + srow) * TL::TRANS;
    const uint64_t v = bb[srow];
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) {
      kp[i].store(kd, sp0 + i, v);
      vp[i].validate(sp0 + i, v);
      vp[i].store_trans(vd, sp0 + i);
    }
  };

  uint64_t bb[FWD_ROWS];
  bits_of(0, bb);
  stage_load(0);
  f32x16 bA0 = bias_tile(0), bA1 = bias_tile(1), bB0, bB1;
  stage_store(0, bb);
  __syncthreads();
  auto step = [&](int b, const f32x16& c0, const f32x16& c1b, f32x16& n0, f32x16& n1) {
    const int bn = min(b + 1, nblk - 1);
    uint64_t bbn[FWD_ROWS];
    bits_of(bn, bbn);
    stage_load(bn);
    n0 = bias_tile(2 * bn);
    n1 = bias_tile(2 * bn + 1);
    const int buf = b & 1;
    bool full = bb[0] == ~0ull;
    if constexpr (FWD_ROWS > 1) full = full && (!row1 || bb[1] == ~0ull);
    if (active && full) {
      full_block(buf, c0, c1b);
    } else if (active) {
#pragma unroll
      for (int i = 0; i < FWD_ROWS; ++i) {
        const T* ksb = ks + (buf * FWD_ROWS + i) * TL::ROWT;
        const T* vtb = vt + (buf * FWD_ROWS + i) * TL::TRANS;
        if ((uint32_t)bb[i]) sub_tile(st[i], qf[i], ksb, vtb, c0, (uint32_t)bb[i], 0);
        if ((uint32_t)(bb[i] >> 32))
          sub_tile(st[i], qf[i], ksb, vtb, c1b, (uint32_t)(bb[i] >> 32), 1);
      }
    }
    if (b + 1 < nblk) stage_store(buf ^ 1, bbn);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) bb[i] = bbn[i];
  };
  for (int b = 0; b < nblk; b += 2) {
    step(b, bA0, bA1, bB0, bB1);
    if (b + 1 >= nblk) break;
    step(b + 1, bB0, bB1, bA0, bA1);
  }
  if (!active || !qok) return;

  // epilogue: normalise, gate, store; lse = ln(sum exp) = (m + log2 l) ln 2
#pragma unroll
  for (int i = 0; i < FWD_ROWS; ++i) {
    if (i == 1 && !row1) break;
    const SoftmaxState<D>& S = st[i];
    const float lt = wave_xor32_sum(S.l[0]);  // half 1 holds zeros in register 0
    const float inv = lt > 0.f ? fast_rcp(lt) : 0.f;
    const int64_t base = rowbase[i] + (int64_t)q * G.sPos;
    f32x4 gv[NO][4];  // every gate load before the first store
#pragma unroll
    for (int c = 0; c < NO; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) gv[c][j] = load4(a.gate + base + 32 * c + 8 * j + 4 * g);
#pragma unroll
    for (int c = 0; c < NO; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c0 = 32 * c + 8 * j + 4 * g;
        f32x4 ov;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          ov[e] = S.o[c][4 * j + e] * inv * fast_rcp(1.f + __expf(-gv[c][j][e]));
        store4(a.out + base + c0, ov);
      }
    if (g == 0)
      a.lse[(int64_t)(r0 + i) * G.lRow + (int64_t)q * G.lPos + h] =
          lt > 0.f ? (S.m + log2f(lt)) * LN2 : neg_inf();
  }
}

// bf16 forward with asynchronous LDS staging (see dma.h).  One workgroup =
// 8 waves = 128 queries x 4 rows of one head; wave w owns query tiles
// 2 (w % 2) and 2 (w % 2) + 1 of row r0 + w / 2, so every K and V fragment
// it reads from LDS serves two query tiles.  Keys stream in tiles of 32
// through a double-buffered DMA ring: per slot the K and V tiles of the 4
// rows (16 KB; 32 KB for 64-channel heads) and the bias tiles of the 4 query
// tiles, shared by the rows (16 KB).  With 16 or 32 channels, 64 KB of LDS
// and at most 128 VGPRs let two workgroups share a CU (four waves per SIMD);
// with 64, one workgroup (96 KB) runs per CU at two waves per SIMD.
//
// The loop is unrolled by the ring length, so every LDS read has a constant
// slot offset, and the DMAs go through buffer resources whose base moves
// with the tile: no vector instruction is spent on addresses.  A workgroup
// whose rows have every key valid (every row of an unmasked problem) runs a
// loop without any mask step.
constexpr int FO_QT = 2;                            // query tiles per wave
constexpr int FO_ROWBLK = 32 * 64;                  // one row's K (or V) tile: 32 keys x 64 B
// Workgroup shape and LDS layout.  ROWS rows x 128 queries of one head, two
// waves per row; a ring of SLOTS key tiles.  (8 rows of 16 waves with a
// three-slot ring, 144 KB, measured 15% slower than 4 rows and two slots.)  LDS by region, each region
// holding its piece of every slot (so that slot offsets stay small): K tiles
// [slot][channel half][row], V tiles likewise, then the 4 bias tiles (fp32,
// 4 KB each) [slot].  A 64-channel head keeps each position as two 32-channel
// halves, each a block of the usual layout.
template <int D>
struct FoL {
  static constexpr int NH = D == 64 ? 2 : 1;       // 32-channel halves per position
  static constexpr int ROWS = 4;
  static constexpr int SLOTS = 2;
  static constexpr int WAVES = 2 * ROWS;
  static constexpr int HB = ROWS * FO_ROWBLK;      // one half's K (or V) tiles of the rows
  static constexpr int KS = NH * HB;               // one slot of the K (or V) region
  static constexpr int V0 = SLOTS * KS;            // the V region follows the K region
  static constexpr int BIAS = 2 * SLOTS * KS;      // then the bias region
  static constexpr int BS = 4 * 4096;              // one slot of it
  static constexpr int LDS = BIAS + SLOTS * BS;
  static constexpr int BOPS = 16 / WAVES;          // bias DMA ops (1 KB quarters) per wave per tile
  static constexpr int OPS = 2 * NH + BOPS;        // DMA ops per wave per tile
  static constexpr int WPE = D == 64 ? 2 : 4;      // waves per SIMD
};

//
// D = 16, 32 or 64 channels per head (see dma.h for 16).
template <int D>
__global__ __launch_bounds__(64 * FoL<D>::WAVES) __attribute__((amdgpu_waves_per_eu(FoL<D>::WPE, FoL<D>::WPE)))
void fwd_dma_kernel(FwdArgs<bf16> a) {
  to_sample(a);
  using M = Mma<bf16>;
  using F = bf16x8;
  using L = FoL<D>;
  constexpr int NH = L::NH;
  constexpr int KC = D == 16 ? 1 : D / 16;  // 16-channel MFMA steps of a contraction over channels
  constexpr int KA = D == 64 ? 4 : 2;       // fragment slots per operand row
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  constexpr int FO_ROWS = L::ROWS, FO_SLOTS = L::SLOTS;
  const int nrg = (G.nr + FO_ROWS - 1) / FO_ROWS;
  const int qb = w % a.nqb, rg = (w / a.nqb) % nrg, h = w / (a.nqb * nrg);
  const int r0 = rg * FO_ROWS;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qh = wave & 1, ri = wave >> 1;
  const int row = r0 + ri;  // this wave's row
  const bool rok = row < G.nr;
  const int nkt = G.nkt, last = G.nr - 1;  // last row
  const float c1 = G.scale * LOG2E;
  const int nrows = min(FO_ROWS, G.nr - r0);  // rows of this group that exist

  __shared__ __align__(16) char smem[L::LDS];

  const int64_t hb = (int64_t)h * D;
  const int64_t myrow = (int64_t)min(row, last) * G.sRow + hb;
  // query tiles 2 qh + i of the block: lane <-> query
  int qv[FO_QT];
  bool act[FO_QT];
  F qf[FO_QT][KA];
#pragma unroll
  for (int i = 0; i < FO_QT; ++i) {
    const int q0 = qb * FWD_QBLK + (FO_QT * qh + i) * TILE;
    qv[i] = q0 + l32;
    act[i] = rok && q0 < G.n;
    if (act[i] && qv[i] < G.n) {
      if constexpr (D == 64)
        row_frags(a.q + myrow + (int64_t)qv[i] * G.sPos, g, qf[i]);
      else
        row_frags_d<D>(a.q + myrow + (int64_t)qv[i] * G.sPos, g, qf[i]);
    } else {
      zero_frags(qf[i]);
    }
  }
  const bool active = act[0];  // tile 1 active implies tile 0 active
  bool rows_full = true;
  for (int i = 0; i < nrows; ++i) rows_full = rows_full && const_load(a.rowfull + r0 + i) != 0u;
  // the plain register loads above stay in flight with the first DMAs: the
  // first step's full wait (vmcnt 0) precedes every use of their registers

  // ---- DMA lanes.  Ops 0, 1: K or V tile of one row (wave w: K of row w
  // for w < 4, V of row w - 4 otherwise), keys 16 op + lane / 4.  Ops 2, 3:
  // bias tiles 2 (op - 2) + w / 4, quarter w % 4.  Lane offsets are fixed;
  // the source pointers advance by one tile per issue (scalar registers
  // only).  Tiles past the last are issued with an empty resource: they
  // write zeros into a slot that is never read again and keep the wait
  // counts uniform.
  const int dblk = wave;  // K0..K3, V0..V3
  const int dp = lane >> 2;
  const int64_t tensor = (int64_t)G.nr * G.n * G.H * D;
  const bf16* dsrc = dblk < FO_ROWS ? a.k : a.v;
  const bf16* dptr = dsrc + (int64_t)min(r0 + dblk % FO_ROWS, last) * G.sRow + hb;
  const bf16* const dend = dsrc + tensor;
  uint32_t dvoff[2];
  bool dok[2];  // this lane's chunk exists (always for 32 channels)
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int p = 16 * j + dp;
    dvoff[j] = (uint32_t)(((int64_t)p * G.sPos + 8 * ((lane & 3) ^ swz(p))) * 2);
    dok[j] = chunk_exists<D == 16 ? 16 : 32>(p, lane & 3);
  }
  const int64_t tstep = (int64_t)TILE * G.sPos;
  const float* bptr = a.bt + ((int64_t)h * nkt + (int64_t)qb * 4) * nkt * 1024;
  const float* const bend = a.bt + (int64_t)G.H * nkt * nkt * 1024;
  // bias op j of wave w: quarter u % 4 of tile u / 4, u = BOPS w + j
  uint32_t bvoff[L::BOPS];
  char* bdst[L::BOPS];
#pragma unroll
  for (int j = 0; j < L::BOPS; ++j) {
    const int u = L::BOPS * wave + j, bt = u >> 2;
    bvoff[j] = (uint32_t)(((int64_t)bt * nkt * 1024 + 256 * (u & 3)) * 4 + 16 * lane);
    bdst[j] = smem + L::BIAS + bt * 4096 + 1024 * (u & 3);
  }
  char* const kvdst = smem + (dblk < FO_ROWS ? 0 : L::V0) + (dblk % FO_ROWS) * FO_ROWBLK;
  Walk wkv(dptr, dend, tstep * 2), wbias(bptr, bend, 4096);
  int issued = 0;
  auto issue = [&](int slot) {
    const bool real = issued < nkt;
    const rsrc_t rk = wkv.rsrc(real);
#pragma unroll
    for (int c = 0; c < NH; ++c) {  // channel half c: 32 channels (64 bytes) further on
      if (dok[0]) dma16b(rk, dvoff[0] + 64 * c, kvdst + slot * L::KS + c * L::HB);
      if (dok[1]) dma16b(rk, dvoff[1] + 64 * c, kvdst + slot * L::KS + c * L::HB + 1024);
    }
    const rsrc_t rb = wbias.rsrc(real);
#pragma unroll
    for (int j = 0; j < L::BOPS; ++j) dma16b(rb, bvoff[j], bdst[j] + slot * L::BS);
    wkv.advance();
    wbias.advance();
    ++issued;
  };

  // ---- LDS read addresses (slot 0; the slot adds a constant)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t rk0 = base + ri * FO_ROWBLK + l32 * 64 + 16 * (g ^ sw);
  const uint32_t rk1 = base + ri * FO_ROWBLK + l32 * 64 + 16 * ((2 + g) ^ sw);
  const TrAddr ta(lane);
  const uint32_t rv = base + L::V0 + ri * FO_ROWBLK + ta.off(0);
  const uint32_t rv8 = base + L::V0 + ri * FO_ROWBLK + ta.off(8) - 8 * 64;
  const uint32_t rb = base + L::BIAS + FO_QT * qh * 4096 + lane * 16;
  // K fragment t (channels 16 t + 8 g .. +7) of this wave's row in slot S
  auto kfrag = [&](uint32_t so, int t) {
    return lds_load16<F>((t & 1 ? rk1 : rk0) + (t >> 1) * L::HB + so);
  };

  float m[FO_QT];
  f32x16 o[FO_QT][NH];
  float ls0[FO_QT], ls1[FO_QT];  // this lane's share of sum_k P (its 16 keys of each tile)
#pragma unroll
  for (int i = 0; i < FO_QT; ++i) {
    m[i] = M_FLOOR;
#pragma unroll
    for (int c = 0; c < NH; ++c) o[i][c] = f32x16{};
    ls0[i] = ls1[i] = 0.f;
  }
  const bf16x2 one2 = {(bf16)1.f, (bf16)1.f};

  // zero the V rows of keys invalid for a row in ring slot S (weight 0, and
  // 0 times a non-finite value would not be); thread t < 32 ROWS: row t / 32, key t % 32
  auto zero_invalid_v = [&](auto slot, const uint32_t (&wr)[FO_ROWS]) {
    constexpr int S = decltype(slot)::value;
    if (tid < 32 * FO_ROWS) {
      const int rr = tid >> 5;
      uint32_t wb = 0;
#pragma unroll
      for (int i = 0; i < FO_ROWS; ++i)
        if (rr == i) wb = wr[i];
      if (!((wb >> (tid & 31)) & 1u)) {
        char* z = smem + S * L::KS + L::V0 + rr * FO_ROWBLK + 64 * (tid & 31);
#pragma unroll
        for (int c = 0; c < NH; ++c)
#pragma unroll
          for (int e = 0; e < 4; ++e) *(f32x4*)(z + c * L::HB + 16 * e) = f32x4{};
      }
    }
  };

  // the loop; FULL: every key of every row of the group is valid
  auto run = [&](auto full_c) {
    constexpr bool FULL = decltype(full_c)::value;
    auto step = [&](int t, auto slot) {
      constexpr int S = decltype(slot)::value;
      // key bits of tile t for this wave's row (0 for a row past the end)
      uint32_t wb = 0;
      if constexpr (FULL) {
        wb = rok ? in_range_bits(t, G.n) : 0u;
        wait_vm<(FO_SLOTS - 2) * L::OPS>();  // tile t has landed (tiles after it may be in flight)
        lds_barrier();
      } else {
        uint32_t wr[FO_ROWS];  // per row of the group
#pragma unroll
        for (int i = 0; i < FO_ROWS; ++i)
          wr[i] = i < nrows ? const_load(a.kbits + (int64_t)(r0 + i) * nkt + t) : 0u;
        wait_vm<(FO_SLOTS - 2) * L::OPS>();
        lds_barrier();
        bool full = true;
#pragma unroll
        for (int i = 0; i < FO_ROWS; ++i) full = full && (i >= nrows || wr[i] == 0xffffffffu);
        if (!full) {
          zero_invalid_v(slot, wr);
          __syncthreads();
        }
#pragma unroll
        for (int i = 0; i < FO_ROWS; ++i)
          if (ri == i) wb = wr[i];
      }
      issue((S + FO_SLOTS - 1) % FO_SLOTS);  // tile t + SLOTS - 1 into the slot of tile t - 1
      if (!active || wb == 0u) return;
      F kfr[KA];
#pragma unroll
      for (int t = 0; t < KC; ++t) kfr[t] = kfrag(S * L::KS, t);
      f32x16 s[FO_QT];
#pragma unroll
      for (int i = 0; i < FO_QT; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 y = lds_load16<f32x4>(rb + S * L::BS + i * 4096 + 1024 * j);
#pragma unroll
          for (int e = 0; e < 4; ++e) s[i][4 * j + e] = y[e];
        }
#pragma unroll
        for (int t = 0; t < KC; ++t) s[i] = M::mma(kfr[t], qf[i][t], s[i]);  // S^T = bias + K Q^T
      }
      s16x4 tr[NH][4];
      auto trread = [&](auto cc) {  // V^T fragments of channel half c
        constexpr int c = decltype(cc)::value;
        constexpr uint32_t ho = S * L::KS + c * L::HB;
        tr[c][0] = ds_read_tr<ho>(rv);
        tr[c][1] = ds_read_tr<ho + 8 * 64>(rv8);
        tr[c][2] = ds_read_tr<ho + 16 * 64>(rv);
        tr[c][3] = ds_read_tr<ho + 24 * 64>(rv8);
      };
      trread(std::integral_constant<int, 0>{});
      if constexpr (NH == 2) trread(std::integral_constant<int, 1>{});
      // P = exp2(S c1 - m) against the running max m as it stands (in place of
      // S), and the tile's row sums of the bf16 P the MFMA uses (dot products
      // with (1, 1)).  The max is not formed per tile: a tile whose weights
      // grow past 2^64 (or overflow: the first tile, while m is still the
      // floor) recomputes its logits, raises m to their max, rescales the
      // state and is redone; other tiles only have weights below 2^64, which
      // fp32 sums and bf16 operands hold as exactly as weights below 1.
      F pf[FO_QT][M::PCH];
      float t0[FO_QT], t1[FO_QT];
      auto weights = [&](int i) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          s[i][v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[i][v], c1, -m[i]));
        acc_frags(s[i], pf[i]);
        t0[i] = 0.f;
        t1[i] = 0.f;
#pragma unroll
        for (int u = 0; u < M::PCH; ++u) {
          t0[i] = __builtin_amdgcn_fdot2_f32_bf16(
              __builtin_shufflevector(pf[i][u], pf[i][u], 0, 1), one2, t0[i], false);
          t1[i] = __builtin_amdgcn_fdot2_f32_bf16(
              __builtin_shufflevector(pf[i][u], pf[i][u], 2, 3), one2, t1[i], false);
          t0[i] = __builtin_amdgcn_fdot2_f32_bf16(
              __builtin_shufflevector(pf[i][u], pf[i][u], 4, 5), one2, t0[i], false);
          t1[i] = __builtin_amdgcn_fdot2_f32_bf16(
              __builtin_shufflevector(pf[i][u], pf[i][u], 6, 7), one2, t1[i], false);
        }
      };
#pragma unroll
      for (int i = 0; i < FO_QT; ++i) {
        if (wb != 0xffffffffu) mask_rows(s[i], wb, g);
        weights(i);
        if (__any(!(t0[i] + t1[i] <= WEIGHT_LIMIT))) {
          // the tile's logits again (bias and K from the slot, Q at hand)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const f32x4 y = lds_load16<f32x4>(rb + S * L::BS + i * 4096 + 1024 * j);
#pragma unroll
            for (int e = 0; e < 4; ++e) s[i][4 * j + e] = y[e];
          }
#pragma unroll
          for (int t = 0; t < KC; ++t) s[i] = M::mma(kfrag(S * L::KS, t), qf[i][t], s[i]);
          if (wb != 0xffffffffu) mask_rows(s[i], wb, g);
          const float mx = wave_xor32_max(max16(s[i])) * c1;
          const float mnew = fmaxf(m[i], mx);
          const float alpha = __builtin_amdgcn_exp2f(m[i] - mnew);
          ls0[i] *= alpha;
          ls1[i] *= alpha;
#pragma unroll
          for (int c = 0; c < NH; ++c)
#pragma unroll
            for (int v = 0; v < 16; ++v) o[i][c][v] *= alpha;
          m[i] = mnew;
          weights(i);
        }
      }
#pragma unroll
      for (int c = 0; c < NH; ++c) tr_wait(tr[c]);
#pragma unroll
      for (int i = 0; i < FO_QT; ++i) {
#pragma unroll
        for (int c = 0; c < NH; ++c)
#pragma unroll
          for (int u = 0; u < M::PCH; ++u) o[i][c] = M::mma(tr_frag(tr[c], u), pf[i][u], o[i][c]);
        ls0[i] += t0[i];
        ls1[i] += t1[i];
      }
    };
#pragma unroll
    for (int j = 0; j < FO_SLOTS - 1; ++j) issue(j);
    for (int t = 0; t < nkt; t += FO_SLOTS) {
      step(t, slot_c<0>{});
      if (t + 1 >= nkt) break;
      step(t + 1, slot_c<1 % FO_SLOTS>{});
      if (FO_SLOTS < 3 || t + 2 >= nkt) continue;
      step(t + 2, slot_c<2 % FO_SLOTS>{});
    }
  };
  if (rows_full)
    run(std::true_type{});
  else
    run(std::false_type{});

  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active) return;
  // every gate load is issued before the first store (a store to memory that
  // could alias a later load keeps the compiler from moving the load up)
  constexpr int NQ = D == 16 ? 2 : 4;  // accumulator quads holding channels (32 c + 8 j + 4 g .. +3 < D)
  f32x4 gv[FO_QT][NH][NQ];
#pragma unroll
  for (int i = 0; i < FO_QT; ++i) {
    const bool ok = act[i] && qv[i] < G.n;
    const int64_t gbase = myrow + (int64_t)(ok ? qv[i] : 0) * G.sPos;
#pragma unroll
    for (int c = 0; c < NH; ++c)
#pragma unroll
      for (int j = 0; j < NQ; ++j) gv[i][c][j] = load4(a.gate + gbase + 32 * c + 8 * j + 4 * g);
  }
#pragma unroll
  for (int i = 0; i < FO_QT; ++i) {
    const float lt = wave_xor32_sum(ls0[i] + ls1[i]);  // the lane halves hold 16 keys each
    if (!act[i] || qv[i] >= G.n) continue;
    const float inv = lt > 0.f ? fast_rcp(lt) : 0.f;
    const int64_t gbase = myrow + (int64_t)qv[i] * G.sPos;
#pragma unroll
    for (int c = 0; c < NH; ++c)
#pragma unroll
      for (int j = 0; j < NQ; ++j) {
        const int c0 = 32 * c + 8 * j + 4 * g;
        f32x4 ov;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          ov[e] = o[i][c][4 * j + e] * inv * fast_rcp(1.f + __expf(-gv[i][c][j][e]));
        store4(a.out + gbase + c0, ov);
      }
    if (g == 0)
      a.lse[(int64_t)row * G.lRow + (int64_t)qv[i] * G.lPos + h] =
          lt > 0.f ? (m[i] + log2f(lt)) * LN2 : neg_inf();
  }
}


template <typename T>
hipError_t launch_fwd(const Geom& g, const Prep& p, const T* q, const T* k, const T* v,
                      const T* gate, T* out, float* lse, hipStream_t s) {
  FwdArgs<T> a{g, p.bt, p.kbits, p.rowfull, q, k, v, gate, out, lse, (g.n + FWD_QBLK - 1) / FWD_QBLK};
  const int64_t nwg = (int64_t)a.nqb * ((g.nr + FWD_ROWS - 1) / FWD_ROWS) * g.H;
  if (g.d == 16 && !std::is_same<T, bf16>::value) return hipErrorInvalidValue;  // bf16 only
  if constexpr (std::is_same<T, bf16>::value) {
    KernelTimer t(K_FWD, s);
    auto go = [&](auto kernel, auto lay) {
      using L = decltype(lay);
      const int64_t nwd = (int64_t)a.nqb * ((g.nr + L::ROWS - 1) / L::ROWS) * g.H;
      hipLaunchKernelGGL(kernel, dim3((unsigned)nwd, 1, (unsigned)g.batch), dim3(64 * L::WAVES), 0, s, a);
    };
    if (g.d == 64)
      go(fwd_dma_kernel<64>, FoL<64>{});
    else if (g.d == 16)
      go(fwd_dma_kernel<16>, FoL<16>{});
    else
      go(fwd_dma_kernel<32>, FoL<32>{});
  } else if (g.d == 64) {
    KernelTimer t(K_FWD, s);
    hipLaunchKernelGGL((fwd_kernel<T, 64>), dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(256), 0, s, a);
  } else {
    KernelTimer t(K_FWD, s);
    hipLaunchKernelGGL((fwd_kernel<T, 32>), dim3((unsigned)nwg, 1, (unsigned)g.batch), dim3(256), 0, s, a);
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
