// Arguments shared by the backward kernels (bwd.hip, and the dK/dV kernels in
// dkdv.hip, a file of its own so that it can be compiled with its own
// scheduling options).
#pragma once

#include <type_traits>

#include "kernels.h"

namespace triattn {

template <typename T>
constexpr bool kSplitDA = std::is_same<T, bf16>::value;

constexpr int BWD_WAVES = 4;
constexpr int BWD_BLK = BWD_WAVES * TILE;

template <typename T>
struct BwdArgs {
  Geom g;
  const float *bt, *btT;
  const uint32_t* kbits;
  const uint32_t* rowfull;
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

// This block's sample of a batched launch: every tensor and workspace piece
// moved by the sample's strides (no change for sample 0).
template <typename T>
__device__ inline void to_sample(BwdArgs<T>& a) {
  const Geom& G = a.g;
  a.bt = ws_at_sample(a.bt, G.bWs);
  a.btT = ws_at_sample(a.btT, G.bWs);
  a.kbits = ws_at_sample(a.kbits, G.bWs);
  a.rowfull = ws_at_sample(a.rowfull, G.bWs);
  a.da = ws_at_sample(a.da, G.bWs);
  a.dalo = ws_at_sample(a.dalo, G.bWs);
  a.lse2 = ws_at_sample(a.lse2, G.bWs);
  a.dsum = ws_at_sample(a.dsum, G.bWs);
  a.slabs = ws_at_sample(a.slabs, G.bWs);
  a.q = at_sample(a.q, G.bPair);
  a.k = at_sample(a.k, G.bPair);
  a.v = at_sample(a.v, G.bPair);
  a.dq = at_sample(a.dq, G.bPair);
  a.dk = at_sample(a.dk, G.bPair);
  a.dv = at_sample(a.dv, G.bPair);
}

// dK and dV (dkdv.hip): the DMA kernels for bf16 (16, 32 or 64 channels), the
// register-staged ones for fp32.  node: 0 starting, 1 ending (the ending
// node's bf16 kernels are built separately, dkdv_end.hip).
template <typename T>
hipError_t launch_dkdv(const BwdArgs<T>& a, int node, hipStream_t s);
hipError_t launch_dkdv_dma_end(const BwdArgs<bf16>& a, hipStream_t s);

}  // namespace triattn
