// Device-side building blocks shared by the triangle-attention kernels
// (gfx950 / CDNA4, wave64).
//
// Tiles are 32 x 32 and use the 32x32 MFMA family:
//   bf16: v_mfma_f32_32x32x16_bf16  (A, B: 8 bf16 per lane, C: 16 fp32 per lane)
//   fp32: v_mfma_f32_32x32x2_f32    (A, B: 1 fp32 per lane,  C: 16 fp32 per lane)
// Lane l of a wave owns row (A) / column (B) l % 32 of the operand and lane
// half g = l / 32 picks which contraction slots it holds.  The accumulator
// layout is: lane l, register v holds element
//   row = 8 * (v / 4) + 4 * g + (v % 4),   col = l % 32.
// So a lane holds four runs ("quads") of 4 consecutive rows, starting at
// 8 * j + 4 * g for j = 0..3, of one column.
//
// A product whose contraction runs over the ROW index of an accumulator
// (P V from P^T, dQ from dS^T, dV from P, dK from dS) feeds the accumulator
// registers straight back as the B operand.  The other operand then has to
// hold the same contraction indices in the same slots, i.e. the same quads:
// it is read from a transposed LDS tile with quad_frags().  Whatever order
// the hardware assigns to contraction slots, the pairing of slots between A
// and B is the same, so the products are exact.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace triattn {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

constexpr int HEAD_DIM = 32;  // d: channels per head
constexpr int TILE = 32;      // rows / columns of one MFMA tile
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

__device__ inline float neg_inf() { return -__builtin_inff(); }
__device__ inline float pos_inf() { return __builtin_inff(); }

// ---- per-dtype MFMA configuration -------------------------------------------------
template <typename T>
struct Mma;

template <>
struct Mma<bf16> {
  using frag = bf16x8;
  static constexpr int KCH = HEAD_DIM / 16;  // MFMAs per 32-channel contraction
  static constexpr int PCH = TILE / 16;      // MFMAs per 32-row contraction
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mma<float> {
  using frag = float;
  static constexpr int KCH = HEAD_DIM / 2;
  static constexpr int PCH = TILE / 2;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// MFMA steps over the channels of a D-channel row.
template <typename T, int D>
constexpr int kch() {
  return std::is_same<T, bf16>::value ? D / 16 : D / 2;
}

// Operand fragments of one row of N MFMA steps (row-major [.][D] data, the
// row being this lane's A row or B column).  Slot assignment: bf16 chunk t
// holds channels 16 t + 8 g .. +7 (N = D / 16); fp32 chunk t holds channel
// N g + t (N = D / 2).
template <int N>
__device__ inline void row_frags(const bf16* p, int g, bf16x8 (&f)[N]) {
#pragma unroll
  for (int t = 0; t < N; ++t) f[t] = *(const bf16x8*)(p + 16 * t + 8 * g);
}
template <int N>
__device__ inline void row_frags(const float* p, int g, float (&f)[N]) {
#pragma unroll
  for (int i = 0; i < N / 4; ++i) {
    f32x4 x = *(const f32x4*)(p + N * g + 4 * i);
#pragma unroll
    for (int e = 0; e < 4; ++e) f[4 * i + e] = x[e];
  }
}
// bf16 row fragments of a row of D = 16 or 32 channels: slot 1 (channels
// 16..31) is zero when D = 16 (its products are skipped as well).
template <int D>
__device__ inline void row_frags_d(const bf16* p, int g, bf16x8 (&f)[2]) {
  static_assert(D == 16 || D == 32, "16 or 32 channels");
  f[0] = *(const bf16x8*)(p + 8 * g);
  f[1] = D == 32 ? *(const bf16x8*)(p + 16 + 8 * g) : bf16x8{};
}
template <typename F, int N>
__device__ inline void zero_frags(F (&f)[N]) {
#pragma unroll
  for (int t = 0; t < N; ++t) f[t] = F{};
}

// Fragments of a transposed tile row p[0..31] whose index is the contraction
// index of an accumulator-fed product: quad j (elements 8 j + 4 g .. +3)
// pairs with accumulator registers 4 j .. 4 j + 3.
__device__ inline void quad_frags(const bf16* p, int g, bf16x8 (&f)[Mma<bf16>::PCH]) {
#pragma unroll
  for (int t = 0; t < Mma<bf16>::PCH; ++t) {
    bf16x4 lo = *(const bf16x4*)(p + 8 * (2 * t) + 4 * g);
    bf16x4 hi = *(const bf16x4*)(p + 8 * (2 * t + 1) + 4 * g);
    f[t] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  }
}
__device__ inline void quad_frags(const float* p, int g, float (&f)[Mma<float>::PCH]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f32x4 x = *(const f32x4*)(p + 8 * j + 4 * g);
#pragma unroll
    for (int e = 0; e < 4; ++e) f[4 * j + e] = x[e];
  }
}

// Accumulator registers -> B-operand fragments (contraction over the
// accumulator's row index).  bf16 rounds to nearest even.
__device__ inline void acc_frags(const f32x16& a, bf16x8 (&f)[Mma<bf16>::PCH]) {
#pragma unroll
  for (int t = 0; t < Mma<bf16>::PCH; ++t) {
    bf16x8 x;
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = (bf16)a[8 * t + u];
    f[t] = x;
  }
}
__device__ inline void acc_frags(const f32x16& a, float (&f)[Mma<float>::PCH]) {
#pragma unroll
  for (int t = 0; t < Mma<float>::PCH; ++t) f[t] = a[t];
}

// Row index (within the tile) of accumulator register v for lane half g.
__device__ inline int acc_row(int v, int g) { return 8 * (v >> 2) + 4 * g + (v & 3); }

// Set accumulator entries whose row bit in `bits` (bit i = row i of the
// tile) is clear to -inf.  Only used on tiles with some masked row.
__device__ inline void mask_rows(f32x16& s, uint32_t bits, int g) {
  const uint32_t b = bits >> (4 * g);
#pragma unroll
  for (int v = 0; v < 16; ++v)
    if (!((b >> (8 * (v >> 2) + (v & 3))) & 1u)) s[v] = -__builtin_inff();
}

// Maximum of the 16 accumulator entries of a lane (a chain of 3-input maxes).
__device__ inline float max16(const f32x16& s) {
  float m = fmaxf(fmaxf(s[0], s[1]), s[2]);
#pragma unroll
  for (int v = 3; v < 15; v += 2) m = fmaxf(fmaxf(m, s[v]), s[v + 1]);
  return fmaxf(m, s[15]);
}

// Maximum of 32 values (two accumulators) as a tree of 3-input maxes: 16
// instructions, depth 4.
__device__ inline float max3f(float a, float b, float c) { return fmaxf(a, fmaxf(b, c)); }
__device__ inline float max32(const f32x16& a, const f32x16& b) {
  float t[12];
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    t[i] = max3f(a[3 * i], a[3 * i + 1], a[3 * i + 2]);
    t[5 + i] = max3f(b[3 * i], b[3 * i + 1], b[3 * i + 2]);
  }
  t[10] = a[15];
  t[11] = b[15];
  const float u0 = max3f(t[0], t[1], t[2]), u1 = max3f(t[3], t[4], t[5]);
  const float u2 = max3f(t[6], t[7], t[8]), u3 = max3f(t[9], t[10], t[11]);
  return fmaxf(max3f(u0, u1, u2), u3);
}
// Tree sum of the 16 entries of a lane.
__device__ inline float sum16(const f32x16& a) {
  float t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) t[i] = (a[4 * i] + a[4 * i + 1]) + (a[4 * i + 2] + a[4 * i + 3]);
  return (t[0] + t[1]) + (t[2] + t[3]);
}

// A-operand that sums a B operand's contraction slots into accumulator row 0:
// row 0 is all ones, the other rows are zero.  D += ones_row0 * B then adds
// sum_k B[k][n] to register 0 of the lanes of half g = 0 (row 0), and leaves
// the other rows at zero.  Moves a per-lane row sum from the VALU to the MFMA.
template <typename F>
__device__ inline F ones_row0(int l32);
template <>
__device__ inline bf16x8 ones_row0<bf16x8>(int l32) {
  const bf16 v = l32 == 0 ? (bf16)1.f : (bf16)0.f;
  return bf16x8{v, v, v, v, v, v, v, v};
}
template <>
__device__ inline float ones_row0<float>(int l32) {
  return l32 == 0 ? 1.f : 0.f;
}

// Hardware reciprocal (about 1 ulp), for normalisation and the sigmoid.
__device__ inline float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Four consecutive elements <-> fp32.
__device__ inline f32x4 load4(const bf16* p) {
  bf16x4 x = *(const bf16x4*)p;
  return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
}
__device__ inline f32x4 load4(const float* p) { return *(const f32x4*)p; }
__device__ inline void store4(bf16* p, f32x4 x) {
  *(bf16x4*)p = bf16x4{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
}
__device__ inline void store4(float* p, f32x4 x) { *(f32x4*)p = x; }

// Workgroup id -> work item, so that consecutive work items land on one XCD.
// The dispatcher hands workgroup b to XCD b % 8; work items are listed with
// the data they share (same row, same bias block) next to each other, and
// this map gives each XCD a contiguous stretch of that list.  Any bijection
// is correct; this one only improves L2 reuse.
__device__ inline int xcd_swizzle(int b, int total) {
  constexpr int XCD = 8;
  const int per = total / XCD;
  if (b >= per * XCD) return b;
  return (b % XCD) * per + b / XCD;
}

// Combine lane l with lane l ^ 32.  v_permlane32_swap(x, x) leaves
// (x[l], x[l ^ 32]) in the two results, in one order or the other, so a
// symmetric combination of them needs no select.
__device__ inline float wave_xor32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float wave_xor32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

}  // namespace triattn
