// Staging of operand blocks (64 consecutive pair positions x 32 channels of
// one row and head) from HBM through registers into LDS.  A workgroup of 256
// threads moves one block per call; loads for the next block are issued
// before the current block is computed and stored to the other LDS buffer
// after it, so HBM latency hides behind the MFMA/VALU work.
//
// Loads never depend on the validity of a position: the position is clamped
// into [0, last] (every address stays in bounds) and invalid positions are
// replaced by zeros only when the piece is stored to LDS.  Conditional loads
// would make the compiler wait for them right away.
#pragma once

#include "common.h"

namespace triattn {

constexpr int SPAN = 64;  // positions per staged block
// Transposed tile [channel][position].  The row stride is an odd multiple of
// 8 bytes (136 bytes for bf16, 272 for fp32), so the quad reads of 32
// consecutive rows fall on 32 different bank pairs.
constexpr int LDS_TROW = SPAN + 4;

// Tile shapes for D channels per position: row-major [position][channel]
// with D + 8 elements per row (80-byte rows for bf16 at D = 32), and the
// transposed [channel][position] tile.
template <int D>
struct Tiles {
  static constexpr int ROW = D + 8;
  static constexpr int ROWT = SPAN * ROW;
  static constexpr int TRANS = D * LDS_TROW;
};
constexpr int LDS_ROW = Tiles<HEAD_DIM>::ROW;
constexpr int ROW_TILE = Tiles<HEAD_DIM>::ROWT;
constexpr int TRANS_TILE = Tiles<HEAD_DIM>::TRANS;

template <typename T>
struct Vec;
template <>
struct Vec<bf16> {
  using v4 = bf16x4;
};
template <>
struct Vec<float> {
  using v4 = f32x4;
};

__device__ inline bool bit64(uint64_t b, int i) { return (b >> i) & 1ull; }

// One position x 8 channels per 32-channel group: thread t holds position
// t / 4, channels 32 i + 8 (t % 4) .. +7 for i < D / 32.  Feeds a row-major
// tile.
template <typename T, int D = HEAD_DIM>
struct RowPiece;

template <int D>
struct RowPiece<bf16, D> {
  bf16x8 x[D / 32];
  __device__ inline void load(const bf16* src, int64_t sPos, int start, int last, int t) {
    const int p = start + SPAN - 1 <= last ? start + (t >> 2) : min(start + (t >> 2), last);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) x[i] = *(const bf16x8*)(src + (int64_t)p * sPos + 32 * i + 8 * (t & 3));
  }
  __device__ inline void store(bf16* tile, int t, uint64_t valid) const {
    const bool ok = valid == ~0ull || bit64(valid, t >> 2);
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
      *(bf16x8*)(tile + (t >> 2) * Tiles<D>::ROW + 32 * i + 8 * (t & 3)) = ok ? x[i] : bf16x8{};
  }
};

template <int D>
struct RowPiece<float, D> {
  f32x4 lo[D / 32], hi[D / 32];
  __device__ inline void load(const float* src, int64_t sPos, int start, int last, int t) {
    const int p = min(start + (t >> 2), last);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
      const float* s = src + (int64_t)p * sPos + 32 * i + 8 * (t & 3);
      lo[i] = *(const f32x4*)s;
      hi[i] = *(const f32x4*)(s + 4);
    }
  }
  __device__ inline void store(float* tile, int t, uint64_t valid) const {
    const bool ok = valid == ~0ull || bit64(valid, t >> 2);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
      float* d = tile + (t >> 2) * Tiles<D>::ROW + 32 * i + 8 * (t & 3);
      *(f32x4*)d = ok ? lo[i] : f32x4{};
      *(f32x4*)(d + 4) = ok ? hi[i] : f32x4{};
    }
  }
};

// Two positions x 4 channels per 32-channel group: thread t holds positions
// p, p + 1 with p = 2 (t / 8) and channels 32 i + 4 (t % 8) .. +3 for
// i < D / 32.  Feeds a row-major tile, a transposed tile, or both.  Call
// validate() before storing.
template <typename T, int D = HEAD_DIM>
struct PairPiece {
  using V4 = typename Vec<T>::v4;
  V4 x0[D / 32], x1[D / 32];
  __device__ inline void load(const T* src, int64_t sPos, int start, int last, int t) {
    const int p = start + 2 * (t >> 3), c0 = 4 * (t & 7);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
      x0[i] = *(const V4*)(src + (int64_t)min(p, last) * sPos + 32 * i + c0);
      x1[i] = *(const V4*)(src + (int64_t)min(p + 1, last) * sPos + 32 * i + c0);
    }
  }
  __device__ inline void validate(int t, uint64_t valid) {
    if (valid == ~0ull) return;  // the common full block: no selects
    const int p = 2 * (t >> 3);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
      if (!bit64(valid, p)) x0[i] = V4{};
      if (!bit64(valid, p + 1)) x1[i] = V4{};
    }
  }
  __device__ inline void store_rows(T* tile, int t) const {
    const int p = 2 * (t >> 3), c0 = 4 * (t & 7);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
      *(V4*)(tile + p * Tiles<D>::ROW + 32 * i + c0) = x0[i];
      *(V4*)(tile + (p + 1) * Tiles<D>::ROW + 32 * i + c0) = x1[i];
    }
  }
  __device__ inline void store_trans(T* tileT, int t) const {
    const int p = 2 * (t >> 3), c0 = 4 * (t & 7);
#pragma unroll
    for (int i = 0; i < D / 32; ++i) store_trans4(tileT + (32 * i + c0) * LDS_TROW + p, x0[i], x1[i]);
  }
  // channel j of the two positions -> row j of the transposed tile
  __device__ static inline void store_trans4(T* d, const V4& a, const V4& b);
};

// Interleave the two positions' bf16 channels into 32-bit words with integer
// ops (channel j of positions p and p + 1 form one word).
template <>
__device__ inline void PairPiece<bf16, 32>::store_trans4(bf16* d, const bf16x4& x0, const bf16x4& x1) {
  const u32x2 a = __builtin_bit_cast(u32x2, x0), b = __builtin_bit_cast(u32x2, x1);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t x = a[j >> 1], y = b[j >> 1];
    const uint32_t w = (j & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
    *(uint32_t*)(d + j * LDS_TROW) = w;
  }
}
template <>
__device__ inline void PairPiece<bf16, 64>::store_trans4(bf16* d, const bf16x4& x0, const bf16x4& x1) {
  PairPiece<bf16, 32>::store_trans4(d, x0, x1);
}
template <>
__device__ inline void PairPiece<float, 32>::store_trans4(float* d, const f32x4& x0, const f32x4& x1) {
#pragma unroll
  for (int j = 0; j < 4; ++j) *(f32x2*)(d + j * LDS_TROW) = f32x2{x0[j], x1[j]};
}
template <>
__device__ inline void PairPiece<float, 64>::store_trans4(float* d, const f32x4& x0, const f32x4& x1) {
  PairPiece<float, 32>::store_trans4(d, x0, x1);
}

// Bits of positions start .. start+63 that lie inside [0, n).
__device__ inline uint64_t range_bits64(int start, int n) {
  const int m = n - start;
  return m >= 64 ? ~0ull : (m <= 0 ? 0ull : ((1ull << m) - 1ull));
}

// Key-valid bits of 64-key block b of a row: words 2 b and 2 b + 1 of the
// row's key bits (a word past the last tile counts as empty; the reads stay
// in bounds).
// The words are read through the constant address space: the key bits are
// written by an earlier kernel and only read here, so the compiler may use
// scalar loads (a vector load of a uniform value would make it wait for
// every outstanding vector load before the value can be moved to a scalar).
__device__ inline uint32_t const_load(const uint32_t* p) {
  return *(const __attribute__((address_space(4))) uint32_t*)p;
}
__device__ inline uint64_t block_bits(const uint32_t* kb, int nkt, int b) {
  const int t = 2 * b;
  const uint32_t lo = const_load(kb + min(t, nkt - 1));
  const uint32_t hi = const_load(kb + min(t + 1, nkt - 1));
  return (t < nkt ? (uint64_t)lo : 0ull) | (t + 1 < nkt ? (uint64_t)hi << 32 : 0ull);
}

// Accumulator registers <- the four quads this lane owns of a 32-wide run of
// fp32 (elements 8 j + 4 g .. +3).  `p` must already point at element 4 g.
__device__ inline f32x16 load_quads(const float* p) {
  f32x16 s;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const f32x4 x = *(const f32x4*)(p + 8 * j);
#pragma unroll
    for (int e = 0; e < 4; ++e) s[4 * j + e] = x[e];
  }
  return s;
}

// Bias maps in accumulator order.  The 32 x 32 values of tile (t1, t2) of a
// head are stored as [j][lane][e] (j, e = 0..3), lane l holding register
// 4 j + e of the accumulator (its column is 32 t1 + l % 32, its row
// 32 t2 + 8 j + 4 (l / 32) + e).  A wave then reads each j as one 1 KB
// contiguous run instead of 32 scattered rows.
__device__ inline const float* frag_tile(const float* map, int h, int t1, int t2, int nt) {
  return map + (((int64_t)h * nt + t1) * nt + t2) * 1024;
}
__device__ inline f32x16 load_frag_tile(const float* tile, int lane) {
  f32x16 s;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const f32x4 x = *(const f32x4*)(tile + (j * 64 + lane) * 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) s[4 * j + e] = x[e];
  }
  return s;
}

__device__ inline f32x16 splat16(float x) {
  f32x16 s;
#pragma unroll
  for (int v = 0; v < 16; ++v) s[v] = x;
  return s;
}

}  // namespace triattn
