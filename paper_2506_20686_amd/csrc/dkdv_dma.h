// The bf16 dK/dV kernel body with asynchronous LDS staging, shared by
// dkdv.hip (the starting node's kernels, default instruction scheduling) and
// dkdv_end.hip (the ending node's, LLVM's max-ilp scheduler at four waves per
// SIMD).  Measured on MI355X at N = 768: max-ilp made the ending node's dK/dV
// 8% faster and the starting node's 3-5% slower, so each node gets its own.
#pragma once

#include <type_traits>

#include "bwd.h"
#include "dma.h"
#include "kernels.h"
#include "stage.h"

namespace triattn {

// bf16 dK, dV with asynchronous LDS staging (see dma.h).  One workgroup =
// 4 KD_ROWS waves = 128 keys x KD_ROWS rows of one head: wave w owns key
// tile w % 4 of the block (lane <-> key) in row r0 + w / 4.  Queries stream
// in tiles of 32; per tile, Q, dA and its low part of the rows, their lse2
// and -D, and the key-major bias tiles of the 128 keys (shared by the rows;
// 16 KB of the 29 KB per tile at KD_ROWS = 2) are copied HBM -> LDS by DMA
// into a ring of KD_SLOTS slots (57 KB of LDS at 2 rows and 2 slots).  Two
// workgroups share a CU at four waves per SIMD.  Q^T and dA^T fragments
// come from the transposing LDS read of the same row-major tiles.  The
// DMAs go through buffer resources advanced in scalar registers, and the
// loop is unrolled by the ring length, so no vector instruction is spent on
// addresses.
#ifndef KD_ROWS_CFG
#define KD_ROWS_CFG 2
#endif
#ifndef KD_SLOTS_CFG
#define KD_SLOTS_CFG 2
#endif
constexpr int KD_ROWS = KD_ROWS_CFG;
constexpr int KD_WAVES = 4 * KD_ROWS;
constexpr int KD_HALF = KD_WAVES / 2;              // waves per half of the DMA lanes
constexpr int KD_BLK = 32 * 64;                        // 2 KB: 32 positions x 32 channels
constexpr int KD_SLOTS = KD_SLOTS_CFG;
constexpr int KD_BOPS = 16 / KD_WAVES;                 // bias DMA ops per wave per tile
// LDS regions, each holding its piece of every ring slot (so that slot
// offsets stay small enough for the immediate field of LDS instructions):
// Q, dA and dA low [slot][channel half][row] tiles, bias [slot][key tile]
// (4 KB each), lse2 / -D [slot][2][row][32].  A 64-channel head keeps each
// position as two 32-channel halves, each a block of the usual layout; 16-
// and 32-channel heads have one.
template <int D>
struct KdL {
  static constexpr int NH = D == 64 ? 2 : 1;         // 32-channel halves per position
  static constexpr int HT = KD_ROWS * KD_BLK;        // one half's tiles of the rows
  static constexpr int TS = NH * HT;                 // one slot of a tile region
  static constexpr int Q = 0, DA = KD_SLOTS * TS, LO = 2 * KD_SLOTS * TS;
  static constexpr int BIAS = 3 * KD_SLOTS * TS, BS = 4 * 4096;
  static constexpr int L2 = BIAS + KD_SLOTS * BS, LS = 2 * KD_ROWS * 128;
  static constexpr int LDS = L2 + KD_SLOTS * LS;     // 57 KB (D <= 32) or 81 KB (D = 64)
  static constexpr int WPE = D == 64 ? 2 : 4;        // waves per SIMD
};

// D = 16, 32 or 64 channels per head (see dma.h for 16).  At 64 the LDS
// ring (81 KB) leaves one workgroup per CU, two waves per SIMD.  The body of
// the kernels: dkdv.hip and dkdv_end.hip wrap it in kernels of their own,
// compiled with different instruction scheduling.
template <int D>
__device__ __forceinline__ void dkdv_dma_body(BwdArgs<bf16> a) {
  to_sample(a);
  using M = Mma<bf16>;
  using F = bf16x8;
  using L = KdL<D>;
  constexpr int NH = L::NH;
  constexpr int KC = D == 16 ? 1 : D / 16;     // 16-channel MFMA steps of a contraction over channels
  constexpr int KA = D == 64 ? 4 : 2;          // fragment slots held per operand row
  const Geom& G = a.g;
  const int w = xcd_swizzle(blockIdx.x, gridDim.x);
  const int nrg = (G.nr + KD_ROWS - 1) / KD_ROWS;
  const int kbk = w % a.nblk, rg = (w / a.nblk) % nrg, h = w / (a.nblk * nrg);
  const int r0 = rg * KD_ROWS;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ri = wave >> 2;                 // row of this wave (0..3)
  const int last = G.nr - 1;  // last row
  const int r = min(r0 + ri, last);
  const bool rok = r0 + ri < G.nr;
  const int kt = kbk * 4 + (wave & 3);      // this wave's key tile
  const int nkt = G.nkt;
  const bool active = rok && kt < nkt;
  const uint32_t bits = active ? const_load(a.kbits + (int64_t)r * nkt + kt) : 0u;
  const int key = kt * TILE + l32;
  const bool kvalid = (bits >> l32) & 1u;
  const bool work = bits != 0u;
  const float c1 = G.scale * LOG2E;

  __shared__ __align__(16) char smem[L::LDS];

  // ---- the wave's keys: K and V fragments (zero for invalid keys, so that
  // non-finite values there cannot reach the products)
  const int64_t hb = (int64_t)h * D;
  const int64_t rowbase = (int64_t)r * G.sRow + hb;
  F kf[KA], vf[KA];
  if (kvalid) {
    if constexpr (D == 64) {
      row_frags(a.k + rowbase + (int64_t)key * G.sPos, g, kf);
      row_frags(a.v + rowbase + (int64_t)key * G.sPos, g, vf);
    } else {
      row_frags_d<D>(a.k + rowbase + (int64_t)key * G.sPos, g, kf);
      row_frags_d<D>(a.v + rowbase + (int64_t)key * G.sPos, g, vf);
    }
  } else {
    zero_frags(kf);
    zero_frags(vf);
  }
  // the plain register loads above stay in flight with the first DMAs: the
  // first step's full wait (vmcnt 0) precedes every use of their registers

  // ---- DMA lanes (lane offsets fixed, bases advanced per tile in scalar
  // registers).  Op 0: Q (waves 0-7) or dA (waves 8-15) of row (w % 8) / 2,
  // positions 16 (w % 2) + lane / 4, one op per 32-channel half.  Op 1: the
  // low part of dA of row w / 2 (waves 0-7, per half), or lse2 (waves 8-11)
  // / -D (waves 12-15) of row w % 4, 128 bytes (lanes 0..7).  Op 2: bias tile
  // w / 4, quarter w % 4.
  const int64_t tensor = (int64_t)G.nr * G.n * G.H * D;
  const int p16 = 16 * (wave & 1) + (lane >> 2);
  const uint32_t pvoff = (uint32_t)(((int64_t)p16 * G.sPos + hb + 8 * ((lane & 3) ^ swz(p16))) * 2);
  const bool pok = chunk_exists<D == 16 ? 16 : 32>(p16, lane & 3);  // a chunk to copy for ops 0 and 1 (dA low)
  const int64_t tstep = (int64_t)TILE * G.sPos;  // elements per query tile
  const int orow = (wave % KD_HALF) >> 1;       // op 0 / op 1 (dA low) row
  const bf16* src0 = wave < KD_HALF ? a.q : a.da;
  const bf16* p0 = src0 + (int64_t)min(r0 + orow, last) * G.sRow;
  const bf16* p1 = a.dalo + (int64_t)min(r0 + orow, last) * G.sRow;
  char* const dst0 = smem + (wave < KD_HALF ? L::Q : L::DA) + orow * KD_BLK + 1024 * (wave & 1);
  const bool lo_op = wave < KD_HALF;
  const int lidx = wave - KD_HALF;                 // lse2 rows, then -D rows
  const float* pl = (lidx < KD_ROWS ? a.lse2 : a.dsum) +
                    ((int64_t)h * G.nr + min(r0 + lidx % KD_ROWS, last)) * G.np;
  const float* const plend = pl + G.np;
  char* const dst1 = lo_op ? smem + L::LO + orow * KD_BLK + 1024 * (wave & 1)
                           : smem + L::L2 + 128 * lidx;
  const int dst1_stride = lo_op ? L::TS : L::LS;
  const uint32_t lvoff = 16u * (uint32_t)lane;
  // bias op j of wave w: quarter (KD_BOPS w + j) % 4 of key tile (KD_BOPS w + j) / 4
  const float* pb = a.btT + ((int64_t)h * nkt + kbk * 4) * nkt * 1024;
  const float* const pbend = a.btT + (int64_t)G.H * nkt * nkt * 1024;
  uint32_t bvoff[KD_BOPS];
  char* dst2[KD_BOPS];
#pragma unroll
  for (int j = 0; j < KD_BOPS; ++j) {
    const int u = KD_BOPS * wave + j, tl = u >> 2;
    bvoff[j] = (uint32_t)(((int64_t)tl * nkt * 1024 + 256 * (u & 3)) * 4 + 16 * lane);
    dst2[j] = smem + L::BIAS + tl * 4096 + 1024 * (u & 3);
  }
  Walk w0(p0, src0 + tensor, tstep * 2);
  Walk w1 = lo_op ? Walk(p1, a.dalo + tensor, tstep * 2) : Walk(pl, plend, TILE * 4);
  Walk wb(pb, pbend, 4096);
  int issued = 0;
  auto issue = [&](int slot) {
    // tiles past the last copy nothing (empty resources) but keep the wait
    // counts uniform
    const bool real = issued < nkt;
    const rsrc_t r0s = w0.rsrc(real);
#pragma unroll
    for (int c = 0; c < NH; ++c)  // channel half c: 32 channels (64 bytes) further on
      if (pok) dma16b(r0s, pvoff + 64 * c, dst0 + slot * L::TS + c * L::HT);
    const rsrc_t r1s = w1.rsrc(real);
    if (lo_op) {
#pragma unroll
      for (int c = 0; c < NH; ++c)
        if (pok) dma16b(r1s, pvoff + 64 * c, dst1 + slot * dst1_stride + c * L::HT);
    } else if (lane < 8) {
      dma16b(r1s, lvoff, dst1 + slot * dst1_stride);
    }
    const rsrc_t rbias = wb.rsrc(real);
#pragma unroll
    for (int j = 0; j < KD_BOPS; ++j) dma16b(rbias, bvoff[j], dst2[j] + slot * L::BS);
    w0.advance();
    w1.advance();
    wb.advance();
    ++issued;
  };

  // ---- LDS read addresses (slot 0, channel half 0)
  const uint32_t base = lds_addr(smem);
  const int sw = swz(l32);
  const uint32_t rq0 = base + ri * KD_BLK + l32 * 64 + 16 * (g ^ sw);
  const uint32_t rq1 = base + ri * KD_BLK + l32 * 64 + 16 * ((2 + g) ^ sw);
  const TrAddr ta(lane);
  const uint32_t rtr = base + ri * KD_BLK + ta.off(0);
  const uint32_t rtr8 = base + ri * KD_BLK + ta.off(8) - 8 * 64;
  const uint32_t rta = rtr + L::DA, rta8 = rtr8 + L::DA;
  const uint32_t rb = base + L::BIAS + (wave & 3) * 4096 + lane * 16;
  const uint32_t rl = base + L::L2 + ri * 128 + 16 * g;  // + 32 j: lse2 quad j; + 512: -D

  f32x16 dkt[NH] = {}, dvt[NH] = {};
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
  // row fragment t (channels 16 t + 8 g .. +7) of this wave's row in a tile region
  auto rfrag = [&](uint32_t region, int t) {
    return lds_load16<F>((t & 1 ? rq1 : rq0) + (t >> 1) * L::HT + region);
  };

  auto step = [&](auto slot) {
    constexpr int S = decltype(slot)::value;
    constexpr uint32_t so = S * L::TS;  // slot offset inside the Q, dA and dA-low regions
    // tile t has landed (the tiles after it may be in flight: each wave issues
    // the same number of DMA ops per tile when NH = 1)
    if constexpr (NH == 1)
      wait_vm<(KD_SLOTS - 2) * (2 + KD_BOPS)>();
    else
      wait_vm<0>();
    lds_barrier();
    issue((S + KD_SLOTS - 1) % KD_SLOTS);  // tile t + KD_SLOTS - 1 into the slot of tile t - 1
    if (!work) return;
    // S = bias + Q K^T (registers <-> queries, lane <-> key)
    f32x16 sv;
    {
      f32x16 bias;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 y = lds_load16<f32x4>(rb + S * L::BS + 1024 * j);
#pragma unroll
        for (int e = 0; e < 4; ++e) bias[4 * j + e] = y[e];
      }
      if (bits != 0xffffffffu) {
#pragma unroll
        for (int v = 0; v < 16; ++v) bias[v] += kmask;  // -inf for an invalid key
      }
      sv = M::mma(rfrag(so + L::Q, 0), kf[0], bias);
#pragma unroll
      for (int t = 1; t < KC; ++t) sv = M::mma(rfrag(so + L::Q, t), kf[t], sv);
    }
    // P = exp2(S c1 - lse2[query])
    const f32x16 l2 = quads(rl + S * L::LS);
#pragma unroll
    for (int v = 0; v < 16; ++v) sv[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], c1, -l2[v]));
    // dP - D = dA V^T - D (hi and lo parts of dA), then dS = P (dP - D)
    f32x16 dp = quads(rl + S * L::LS + KD_ROWS * 128);  // -D
#pragma unroll
    for (int t = 0; t < KC; ++t) dp = M::mma(rfrag(so + L::DA, t), vf[t], dp);
#pragma unroll
    for (int t = 0; t < KC; ++t) dp = M::mma(rfrag(so + L::LO, t), vf[t], dp);
#pragma unroll
    for (int v = 0; v < 16; ++v) dp[v] *= sv[v];
    // dV^T += dA^T P,  dK^T += Q^T dS (contraction over the tile's queries),
    // one 32-channel half at a time
    F pf[M::PCH], sf[M::PCH];
    acc_frags(sv, pf);
    acc_frags(dp, sf);
    auto half = [&](auto cc) {
      constexpr int c = decltype(cc)::value;
      constexpr uint32_t ho = so + c * L::HT;
      s16x4 xa[4], xq[4];
      xa[0] = ds_read_tr<ho>(rta);
      xa[1] = ds_read_tr<ho + 8 * 64>(rta8);
      xa[2] = ds_read_tr<ho + 16 * 64>(rta);
      xa[3] = ds_read_tr<ho + 24 * 64>(rta8);
      xq[0] = ds_read_tr<ho + L::Q>(rtr);
      xq[1] = ds_read_tr<ho + L::Q + 8 * 64>(rtr8);
      xq[2] = ds_read_tr<ho + L::Q + 16 * 64>(rtr);
      xq[3] = ds_read_tr<ho + L::Q + 24 * 64>(rtr8);
      tr_wait(xa);
      tr_wait(xq);
#pragma unroll
      for (int u = 0; u < M::PCH; ++u) {
        dvt[c] = M::mma(tr_frag(xa, u), pf[u], dvt[c]);
        dkt[c] = M::mma(tr_frag(xq, u), sf[u], dkt[c]);
      }
    };
    half(std::integral_constant<int, 0>{});
    if constexpr (NH == 2) half(std::integral_constant<int, 1>{});
  };

#pragma unroll
  for (int j = 0; j < KD_SLOTS - 1; ++j) issue(j);
  for (int t = 0; t < nkt; t += KD_SLOTS) {
    step(slot_c<0>{});
    if (t + 1 >= nkt) break;
    step(slot_c<1 % KD_SLOTS>{});
    if (KD_SLOTS < 3 || t + 2 >= nkt) continue;
    step(slot_c<2 % KD_SLOTS>{});
  }
  wait_vm<0>();  // the copies past the end must land before the workgroup ends
  if (!active || key >= G.n) return;
  const int64_t gb = rowbase + (int64_t)key * G.sPos;
#pragma unroll
  for (int c = 0; c < NH; ++c)
#pragma unroll
    for (int j = 0; j < (D == 16 ? 2 : 4); ++j) {  // the quads of channels 32 c + 8 j + 4 g .. +3 < D
      const int c0 = 32 * c + 8 * j + 4 * g;
      f32x4 x, y;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = dvt[c][4 * j + e];
        y[e] = dkt[c][4 * j + e] * G.scale;
      }
      store4(a.dv + gb + c0, x);
      store4(a.dk + gb + c0, y);
    }
}

}  // namespace triattn
