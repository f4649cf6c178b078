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
#include <type_traits>

#include "dma.h"
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
constexpr int FWD_ROWS = 1;                 // rows per workgroup (they share the bias tiles)
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

// Online-softmax state of one (row, 32 queries) pair of a wave.  The row
// sums of P accumulate on the MFMA: register 0 of the lanes of half 0 of
// `l` holds sum_k P for the lane's query (see ones_row0).
struct SoftmaxState {
  float m;
  f32x16 l;
  f32x16 o;  // O^T accumulator: registers <-> channels, lane <-> query
};

template <typename T>
__global__ __launch_bounds__(256, 2) void fwd_kernel(FwdArgs<T> a) {
  using M = Mma<T>;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int qb = w % a.nqb, rh = w / a.nqb;
  const int nrp = (G.n + FWD_ROWS - 1) / FWD_ROWS;
  const int r0 = (rh % nrp) * FWD_ROWS, h = rh / nrp;
  const bool row1 = FWD_ROWS > 1 && r0 + 1 < G.n;  // the second row exists
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int q0 = qb * FWD_QBLK + wave * TILE;  // first query of this wave
  const bool active = q0 < G.n;
  const int q = q0 + l32;
  const bool qok = q < G.n;

  // K block [key][channel] and V^T block [channel][key] of both rows, 2 buffers
  __shared__ __align__(16) T ks[2 * FWD_ROWS * ROW_TILE];
  __shared__ __align__(16) T vt[2 * FWD_ROWS * TRANS_TILE];

  const int last = G.n - 1;
  int64_t rowbase[FWD_ROWS];
  typename M::frag qf[FWD_ROWS][M::KCH];
  const uint32_t* kb[FWD_ROWS];
  SoftmaxState st[FWD_ROWS];
#pragma unroll
  for (int i = 0; i < FWD_ROWS; ++i) {
    const int r = min(r0 + i, last);
    rowbase[i] = (int64_t)r * G.sRow + (int64_t)h * HEAD_DIM;
    kb[i] = a.kbits + (int64_t)r * G.nkt;
    if (qok)
      row_frags(a.q + rowbase[i] + (int64_t)q * G.sPos, g, qf[i]);
    else
      zero_frags<T>(qf[i]);
    st[i].m = neg_inf();
    st[i].l = f32x16{};
    st[i].o = f32x16{};
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
  auto rescale = [&](SoftmaxState& S, float mx) {
    const float mnew = fmaxf(S.m, mx);
    const float alpha = __builtin_amdgcn_exp2f(S.m - mnew);
    S.l[0] *= alpha;  // rows 1..31 of l stay zero
#pragma unroll
    for (int v = 0; v < 16; ++v) S.o[v] *= alpha;
    S.m = mnew;
  };

  // one 32-key sub-tile of one row: logits, online softmax (base 2, stale max), P V
  auto sub_tile = [&](SoftmaxState& S, const typename M::frag(&qfr)[M::KCH], const T* ksb,
                      const T* vtb, const f32x16& bias, uint32_t bits, int u) {
    typename M::frag kf[M::KCH];
    row_frags(ksb + (32 * u + l32) * LDS_ROW, g, kf);
    f32x16 s = M::mma(kf[0], qfr[0], bias);  // s^T = bias + K Q^T
#pragma unroll
    for (int t = 1; t < M::KCH; ++t) s = M::mma(kf[t], qfr[t], s);
    if (bits != 0xffffffffu) mask_rows(s, bits, g);
    const float mx = wave_xor32_max(max16(s)) * c1;
    if (__any(mx > S.m + STALE_MAX_SLACK)) rescale(S, mx);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -S.m));
    typename M::frag pf[M::PCH], vf[M::PCH];
    acc_frags(s, pf);
    quad_frags(vtb + l32 * LDS_TROW + 32 * u, g, vf);
#pragma unroll
    for (int t = 0; t < M::PCH; ++t) {
      S.o = M::mma(vf[t], pf[t], S.o);  // O^T += V^T P^T
      S.l = M::mma(ones, pf[t], S.l);   // row sums of P
    }
  };

  // A full 64-key block (every key valid in both rows): one straight-line
  // stretch -- all logit MFMAs, then the maxes, one (rare) rescale per row,
  // then exp / sums / bf16 packing interleaved with the P V MFMAs -- so the
  // scheduler can overlap the two rows' and sub-tiles' independent work.
  auto full_block = [&](int buf, const f32x16& c0, const f32x16& c1b) {
    f32x16 s[FWD_ROWS][2];
#pragma unroll
    for (int i = 0; i < FWD_ROWS; ++i) {
      const T* ksb = ks + (buf * FWD_ROWS + i) * ROW_TILE;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        typename M::frag kf[M::KCH];
        row_frags(ksb + (32 * u + l32) * LDS_ROW, g, kf);
        s[i][u] = M::mma(kf[0], qf[i][0], u ? c1b : c0);
#pragma unroll
        for (int t = 1; t < M::KCH; ++t) s[i][u] = M::mma(kf[t], qf[i][t], s[i][u]);
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
      SoftmaxState& S = st[i];
      const T* vtb = vt + (buf * FWD_ROWS + i) * TRANS_TILE;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          s[i][u][v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[i][u][v], c1, -S.m));
        typename M::frag pf[M::PCH], vf[M::PCH];
        acc_frags(s[i][u], pf);
        quad_frags(vtb + l32 * LDS_TROW + 32 * u, g, vf);
#pragma unroll
        for (int t = 0; t < M::PCH; ++t) {
          S.o = M::mma(vf[t], pf[t], S.o);
          S.l = M::mma(ones, pf[t], S.l);
        }
      }
    }
  };

  // staging: each row's block is 256 K pieces and 256 V pieces (64 positions
  // x 32 channels); thread tid moves FWD_ROWS consecutive pieces of row srow
  constexpr int TPR = 256 / FWD_ROWS;  // threads per staged row
  RowPiece<T> kp[FWD_ROWS];
  PairPiece<T> vp[FWD_ROWS];
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
    T* kd = ks + (buf * FWD_ROWS + srow) * ROW_TILE;
    T* vd = vt + (buf * FWD_ROWS + srow) * TRANS_TILE;
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
        const T* ksb = ks + (buf * FWD_ROWS + i) * ROW_TILE;
        const T* vtb = vt + (buf * FWD_ROWS + i) * TRANS_TILE;
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
    const SoftmaxState& S = st[i];
    const float lt = wave_xor32_sum(S.l[0]);  // half 1 holds zeros in register 0
    const float inv = lt > 0.f ? fast_rcp(lt) : 0.f;
    const int64_t base = rowbase[i] + (int64_t)q * G.sPos;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c0 = 8 * j + 4 * g;
      const f32x4 gv = load4(a.gate + base + c0);
      f32x4 ov;
#pragma unroll
      for (int e = 0; e < 4; ++e) ov[e] = S.o[4 * j + e] * inv * fast_rcp(1.f + __expf(-gv[e]));
      store4(a.out + base + c0, ov);
    }
    if (g == 0)
      a.lse[(int64_t)(r0 + i) * G.lRow + (int64_t)q * G.lPos + h] =
          lt > 0.f ? (S.m + log2f(lt)) * LN2 : neg_inf();
  }
}

// bf16 forward with asynchronous LDS staging (see dma.h).  One workgroup =
// 8 waves = 128 queries x 2 rows of one head (wave w: query tile w % 4 of
// row r0 + w / 4, one row per wave).  Keys stream in blocks of 32 through a
// three-slot DMA ring (K and V of both rows, the bias tiles of the 128
// queries, shared by the rows: 24 KB per slot), two blocks ahead.  89 VGPRs
// and 72 KB of LDS let two workgroups share a CU: four waves per SIMD hide
// the latency of each wave's dependent MFMA / exp steps (a variant with two
// rows per wave and a software-pipelined loop, at two waves per SIMD, was
// 25% slower).
constexpr int FO_ROWS = 2;
constexpr int FO_ROWBLK = 32 * 64;                     // 2 KB: one row's K (or V) block
constexpr int FO_KV = 2 * FO_ROWS * FO_ROWBLK;         // 8 KB: K0, K1, V0, V1
constexpr int FO_SLOT = FO_KV + 4 * 4096;              // + bias tiles of the 4 query tiles
constexpr int FO_SLOTS = 3;
constexpr int FO_OPS = 3;                              // DMA ops per thread per block

__global__ __launch_bounds__(512, 4) void fwd_dma_kernel(FwdArgs<bf16> a) {
  using M = Mma<bf16>;
  using F = bf16x8;
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nrg = (G.n + FO_ROWS - 1) / FO_ROWS;
  const int qb = w % a.nqb, rg = (w / a.nqb) % nrg, h = w / (a.nqb * nrg);
  const int r0 = rg * FO_ROWS;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qtl = wave & 3, ri = wave >> 2;
  const int row = r0 + ri;                  // this wave's row
  const bool rok = row < G.n;
  const int q0 = qb * FWD_QBLK + qtl * TILE;
  const bool active = rok && q0 < G.n;
  const int q = q0 + l32;
  const bool qok = q < G.n;
  const int nkt = G.nkt, last = G.n - 1;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[FO_SLOTS * FO_SLOT];

  const int64_t hb = (int64_t)h * HEAD_DIM;
  const int64_t myrow = (int64_t)min(row, last) * G.sRow + hb;
  F qf[M::KCH];
  if (active && qok)
    row_frags(a.q + myrow + (int64_t)q * G.sPos, g, qf);
  else
    zero_frags<bf16>(qf);
  // plain register loads: let them complete before any DMA is issued (with
  // both kinds outstanding the compiler would wait for every DMA at each use)
  wait_vm<0>();

  // ---- DMA lanes.  Op 0: K and V of both rows (wave w: block w / 2 of
  // [K0, K1, V0, V1], positions 16 (w % 2) + lane / 4).  Ops 1, 2: bias
  // tiles 2 (op - 1) + w / 4, quarter w % 4.
  const int db = wave >> 1;
  const int dp = 16 * (wave & 1) + (lane >> 2), dc = (lane & 3) ^ swz(dp);
  const bf16* dsrc = db < 2 ? a.k : a.v;
  const int64_t drb = (int64_t)min(r0 + (db & 1), last) * G.sRow + hb + 8 * dc;
  auto issue = [&](int t, int slot) {
    char* sl = smem + slot * FO_SLOT;
    dma16(dsrc + drb + (int64_t)min(t * TILE + dp, last) * G.sPos,
          sl + db * FO_ROWBLK + 1024 * (wave & 1));
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int tile = 2 * j + (wave >> 2);
      const float* src = frag_tile(a.bt, h, min(qb * 4 + tile, nkt - 1), t, nkt);
      dma16((const char*)src + 1024 * (wave & 3) + 16 * lane,
            sl + FO_KV + tile * 4096 + 1024 * (wave & 3));
    }
  };
  // key bits of block t of row r0 + i (zero for a row past the end)
  auto bits = [&](int i, int t) -> uint32_t {
    return r0 + i < G.n ? const_load(a.kbits + (int64_t)(r0 + i) * nkt + t) : 0u;
  };

  // ---- LDS read addresses (slot 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t rk0 = base + ri * FO_ROWBLK + l32 * 64 + 16 * (g ^ sw);
  const uint32_t rk1 = base + ri * FO_ROWBLK + l32 * 64 + 16 * ((2 + g) ^ sw);
  const TrAddr ta(lane);
  const uint32_t rv = base + (2 + ri) * FO_ROWBLK + ta.off(0);
  const uint32_t rv8 = base + (2 + ri) * FO_ROWBLK + ta.off(8) - 8 * 64;
  const uint32_t rb = base + FO_KV + qtl * 4096 + lane * 16;

  float m = neg_inf();
  f32x16 o = {}, lsum = {};  // O^T; row sums of P in accumulator row 0 (see ones_row0)
  const F ones = ones_row0<F>(l32);

#pragma unroll
  for (int j = 0; j < FO_SLOTS - 1; ++j) issue(min(j, nkt - 1), j);
  for (int t = 0; t < nkt; ++t) {
    const uint32_t so = (t % FO_SLOTS) * FO_SLOT;
    wait_vm<(FO_SLOTS - 2) * FO_OPS>();  // block t has landed
    lds_barrier();
    const uint32_t w0 = bits(0, t), w1 = bits(1, t);
    if ((w0 & (r0 + 1 < G.n ? w1 : 0xffffffffu)) != 0xffffffffu) {
      // zero the V rows of keys invalid for a row (weight 0, and 0 times a
      // non-finite value would not be); thread t < 128: row t / 64, key t / 2 % 32
      if (tid < 128) {
        const uint32_t wb = (tid >> 6) ? w1 : w0;
        if (!((wb >> ((tid >> 1) & 31)) & 1u)) {
          char* z = smem + so + 2 * FO_ROWBLK + 32 * tid;
          *(f32x4*)z = f32x4{};
          *(f32x4*)(z + 16) = f32x4{};
        }
      }
      __syncthreads();
    }
    // block t + FO_SLOTS - 1 into the slot of block t - 1 (a copy of the last
    // block past the end keeps the wait counts uniform)
    issue(min(t + FO_SLOTS - 1, nkt - 1), (t + FO_SLOTS - 1) % FO_SLOTS);
    const uint32_t wb = ri ? w1 : w0;
    if (!active || wb == 0u) continue;
    f32x16 s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 y = lds_load16<f32x4>(rb + so + 1024 * j);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[4 * j + e] = y[e];
    }
    {
      const F k0 = lds_load16<F>(rk0 + so), k1 = lds_load16<F>(rk1 + so);
      s = M::mma(k1, qf[1], M::mma(k0, qf[0], s));  // S^T = bias + K Q^T
    }
    if (wb != 0xffffffffu) mask_rows(s, wb, g);
    const float mx = wave_xor32_max(max16(s)) * c1;
    if (__any(mx > m + STALE_MAX_SLACK)) {
      const float mnew = fmaxf(m, mx);
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      lsum[0] *= alpha;
#pragma unroll
      for (int v = 0; v < 16; ++v) o[v] *= alpha;
      m = mnew;
    }
    s16x4 tr[4];
    tr[0] = ds_read_tr<0>(rv + so);
    tr[1] = ds_read_tr<8 * 64>(rv8 + so);
    tr[2] = ds_read_tr<16 * 64>(rv + so);
    tr[3] = ds_read_tr<24 * 64>(rv8 + so);
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c1, -m));
    F pf[M::PCH];
    acc_frags(s, pf);
    tr_wait(tr);
#pragma unroll
    for (int u = 0; u < M::PCH; ++u) {
      o = M::mma(tr_frag(tr, u), pf[u], o);  // O^T += V^T P^T
      lsum = M::mma(ones, pf[u], lsum);      // row sums of P
    }
  }
  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active || !qok) return;
  const float lt = wave_xor32_sum(lsum[0]);  // half 1 holds zero in register 0
  const float inv = lt > 0.f ? fast_rcp(lt) : 0.f;
  const int64_t gbase = myrow + (int64_t)q * G.sPos;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c0 = 8 * j + 4 * g;
    const f32x4 gv = load4(a.gate + gbase + c0);
    f32x4 ov;
#pragma unroll
    for (int e = 0; e < 4; ++e) ov[e] = o[4 * j + e] * inv * fast_rcp(1.f + __expf(-gv[e]));
    store4(a.out + gbase + c0, ov);
  }
  if (g == 0)
    a.lse[(int64_t)row * G.lRow + (int64_t)q * G.lPos + h] =
        lt > 0.f ? (m + log2f(lt)) * LN2 : neg_inf();
}

template <typename T>
hipError_t launch_fwd(const Geom& g, const Prep& p, const T* q, const T* k, const T* v,
                      const T* gate, T* out, float* lse, hipStream_t s) {
  FwdArgs<T> a{g, p.bt, p.kbits, q, k, v, gate, out, lse, (g.n + FWD_QBLK - 1) / FWD_QBLK};
  if constexpr (std::is_same<T, bf16>::value) {
    const int64_t nwg = (int64_t)a.nqb * ((g.n + FO_ROWS - 1) / FO_ROWS) * g.H;
    KernelTimer t(K_FWD, s);
    hipLaunchKernelGGL(fwd_dma_kernel, dim3((unsigned)nwg), dim3(512), 0, s, a);
  } else {
    const int64_t nwg = (int64_t)a.nqb * ((g.n + FWD_ROWS - 1) / FWD_ROWS) * g.H;
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
