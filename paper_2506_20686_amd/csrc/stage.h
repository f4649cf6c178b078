// LDS staging of 32 x 32 operand tiles (one head of 32 consecutive pair
// positions of one row), shared by the waves of a workgroup.
#pragma once

#include "common.h"

namespace triattn {

// Padded LDS row length (elements): 32 data + 8 pad keeps every row 16-byte
// aligned and spreads consecutive rows over different banks.
constexpr int LDS_ROW = HEAD_DIM + 8;

// 128 threads (u = 0..127) copy positions start .. start+31 of one row:
// thread u moves positions p, p+1 (p = 2 (u / 8)) x channels c0 .. c0+3
// (c0 = 4 (u % 8)).  Positions whose bit in `valid` is clear are written as
// zeros.  ROW writes tile[p][c] (row-major), TRANS writes tileT[c][p].
template <bool ROW, bool TRANS, typename T>
__device__ inline void stage_tile(const T* src, int64_t sPos, int start, uint32_t valid, int u,
                                  T* tile, T* tileT);

template <bool ROW, bool TRANS>
__device__ inline void stage_tile(const bf16* src, int64_t sPos, int start, uint32_t valid,
                                  int u, bf16* tile, bf16* tileT) {
  const int p = 2 * (u >> 3), c0 = 4 * (u & 7);
  bf16x4 x0 = {}, x1 = {};
  if ((valid >> p) & 1u) x0 = *(const bf16x4*)(src + (int64_t)(start + p) * sPos + c0);
  if ((valid >> (p + 1)) & 1u) x1 = *(const bf16x4*)(src + (int64_t)(start + p + 1) * sPos + c0);
  if (ROW) {
    *(bf16x4*)(tile + p * LDS_ROW + c0) = x0;
    *(bf16x4*)(tile + (p + 1) * LDS_ROW + c0) = x1;
  }
  if (TRANS) {
#pragma unroll
    for (int j = 0; j < 4; ++j) *(bf16x2*)(tileT + (c0 + j) * LDS_ROW + p) = bf16x2{x0[j], x1[j]};
  }
}

template <bool ROW, bool TRANS>
__device__ inline void stage_tile(const float* src, int64_t sPos, int start, uint32_t valid,
                                  int u, float* tile, float* tileT) {
  const int p = 2 * (u >> 3), c0 = 4 * (u & 7);
  f32x4 x0 = {}, x1 = {};
  if ((valid >> p) & 1u) x0 = *(const f32x4*)(src + (int64_t)(start + p) * sPos + c0);
  if ((valid >> (p + 1)) & 1u) x1 = *(const f32x4*)(src + (int64_t)(start + p + 1) * sPos + c0);
  if (ROW) {
    *(f32x4*)(tile + p * LDS_ROW + c0) = x0;
    *(f32x4*)(tile + (p + 1) * LDS_ROW + c0) = x1;
  }
  if (TRANS) {
#pragma unroll
    for (int j = 0; j < 4; ++j) *(f32x2*)(tileT + (c0 + j) * LDS_ROW + p) = f32x2{x0[j], x1[j]};
  }
}

// Bits of positions start .. start+31 that lie inside [0, n).
__device__ inline uint32_t range_bits(int start, int n) {
  const int m = n - start;
  return m >= 32 ? 0xffffffffu : (m <= 0 ? 0u : ((1u << m) - 1u));
}

}  // namespace triattn
