// Asynchronous staging of bf16 operand blocks through LDS on gfx950.
//
// A block is consecutive pair positions x 32 channels of one (row, head),
// 64 bytes per position (a 64-channel head is staged as two blocks, one per
// 32-channel half; a 16-channel head fills half of each position's row).  It is copied HBM -> LDS with
// global_load_lds_dwordx4 (each lane moves 16 bytes straight into LDS, no
// registers, no vector instructions) into a ring of slots, one or more
// blocks ahead of the compute.
//
// LDS layout of a block: row-major [position][4 chunks of 8 channels], the
// chunk slots of position p permuted by XOR with swz(p) (below).  The DMA
// writes a wave's 64 lanes to 1 KB of consecutive LDS, so the permutation is
// applied on the global side: the lane that fills slot s of position p loads
// chunk s ^ swz(p).  The permutation keeps both read patterns free of bank
// conflicts whether the LDS serves 128 or 256 bytes per cycle:
//   - row fragments (one 16-byte chunk of one position per lane,
//     ds_read_b128, consecutive lanes on consecutive positions): any 8
//     aligned consecutive positions, and any 16, hit distinct 16-byte bank
//     groups;
//   - transposed fragments (ds_read_b64_tr_b16: 16 lanes read 4 consecutive
//     positions x 2 chunks): positions p and p + 2 put their chunk pairs in
//     different halves of the 64-byte row.
//
// Waits: a DMA counts in vmcnt like any vector load and completes in issue
// order.  Before a block is read the waves wait until at most the ops issued
// after it are outstanding, then meet at a barrier.  The compiler neither
// knows that a DMA writes the LDS a later ds_read reads nor may it wait on
// the DMAs by itself, so the waits are explicit and the transposed reads are
// issued with inline assembly (the builtin makes the compiler wait for every
// outstanding load first).
#pragma once

#include <type_traits>

#include "common.h"

namespace triattn {

#define TRIATTN_LDS __attribute__((address_space(3)))

// Bit 1 of the slot permutation is bit 1 ^ bit 3 of the position, bit 0 is
// bit 2: a bijection of the four chunk slots for positions 8 m + b + 2 k
// (k = 0..3) and for 16 m + b + 4 k, and positions p, p + 2 (p % 4 < 2)
// differ in bit 1.
__device__ inline int swz(int p) { return ((((p >> 1) ^ (p >> 3)) & 1) << 1) | ((p >> 2) & 1); }

// Heads of 16 channels use the same 64-byte LDS rows: the DMA lanes of
// chunks 2 and 3 (channels 16..31) stay idle, so those LDS bytes hold
// whatever was there.  They only ever meet products whose results are
// dropped: every contraction over channels skips its second 16-channel step,
// and output rows (channels) 16..31 are never stored.
//
// Whether the DMA lane that fills slot s of position p has a chunk to copy.
template <int D>
__device__ inline bool chunk_exists(int p, int s) {
  static_assert(D == 16 || D == 32, "16 or 32 channels");
  return D == 32 || ((s ^ swz(p)) < 2);
}

// Byte offset of channels 8 c .. 8 c + 7 of position p in a block.
__device__ inline int blk_off(int p, int c) { return p * 64 + 16 * (c ^ swz(p)); }

// One 16-byte DMA lane: `src` is this lane's global address, `dst_wave` the
// LDS address of the wave's 1 KB destination (lane i lands at + 16 i).
__device__ inline void dma16(const void* src, void* dst_wave) {
  __builtin_amdgcn_global_load_lds(src, (TRIATTN_LDS void*)dst_wave, 16, 0, 0);
}

// Buffer resource over `nrec` bytes from `base` (gfx9 raw buffer, stride 0).
// A lane whose offset falls past the record count reads zeros, so the ragged
// tail of a tensor needs no clamped addresses; nrec = 0 gives an empty
// resource (every lane reads zeros and no memory is touched).  Record counts
// saturate at 4 GiB - 1; callers keep each lane's offset below 2^32 by moving
// `base` with the tile or row.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ inline rsrc_t buf_rsrc_n(const void* base, uint32_t nrec) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)nrec,
                                           0x00020000);
}

// Record count for a resource whose base walks the rows of a pair tensor
// ending at `end`: the bytes from the last row's base to `end`, saturated at
// 4 GiB - 1.  A block reads the same offsets from every row's base.  Those
// of positions below n stay under the count (they do in the last row, whose
// last position ends the tensor); those of positions n and up reach past it
// in either node's layout, so they read zeros in every row.
__device__ inline uint32_t last_row_records(const void* last_base, const void* end) {
  const int64_t len = (const char*)end - (const char*)last_base;
  return len <= 0 ? 0u : (len >= 0xffffffffll ? 0xffffffffu : (uint32_t)len);
}

// A buffer resource that walks a tensor in fixed steps (one tile per
// advance): the base moves by `step` bytes and the record count, the bytes
// left to the tensor's end saturated at 4 GiB - 1, shrinks with it.  All of
// it lives in scalar registers; an advance costs a few scalar adds.
struct Walk {
  const char* base;
  uint64_t rem;  // bytes from base to the end (wraps once the base passes it)
  int64_t step;
  Walk() = default;
  __device__ inline Walk(const void* b, const void* end, int64_t s)
      : base((const char*)b), rem((uint64_t)((const char*)end - (const char*)b)), step(s) {}
  // The resource for the current tile; real = false gives an empty one (the
  // copy writes zeros and reads no memory), for tiles past the last.
  __device__ inline rsrc_t rsrc(bool real) const {
    const u32x2 r = __builtin_bit_cast(u32x2, rem);
    const uint32_t n = r[1] != 0u ? 0xffffffffu : r[0];
    return buf_rsrc_n(base, real ? n : 0u);
  }
  __device__ inline void advance() {
    base += step;
    rem -= (uint64_t)step;
  }
};

// One 16-byte DMA lane through a buffer resource: lane i's 16 bytes at
// `voff` land at dst_wave + 16 i.  The resource (and so the per-tile advance)
// lives in scalar registers; the lane offset is fixed for the whole loop.
__device__ inline void dma16b(rsrc_t r, uint32_t voff, void* dst_wave) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (TRIATTN_LDS void*)dst_wave, 16, (int)voff, 0, 0,
                                           0);
}

// Ring slot index as a compile-time constant (loops unrolled by the ring
// length give every LDS access a constant slot offset).
template <int S>
using slot_c = std::integral_constant<int, S>;

// Bits of the keys of tile t that lie below n (all 32 except in a ragged last tile).
__device__ inline uint32_t in_range_bits(int t, int n) {
  const int m = n - 32 * t;
  return m >= 32 ? 0xffffffffu : (m <= 0 ? 0u : (1u << m) - 1u);
}

// 16-byte LDS load from a 32-bit LDS byte address.
template <typename V>
__device__ inline V lds_load16(uint32_t addr) {
  return *(const TRIATTN_LDS V*)(uintptr_t)addr;
}

// s_waitcnt vmcnt(N) (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// and lgkmcnt left at their maxima).
template <int N>
__device__ inline void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier that orders LDS accesses (the compiler may not move
// memory operations across it) without waiting for outstanding loads.
__device__ inline void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// ds_read_b64_tr_b16: in each group of 16 lanes, lane 4 e + j supplies the
// 8 bytes at its address (4 consecutive channels of one position), and lane
// i receives element i % 4 of lane 4 e + i / 4's data as its element e.
template <int OFF = 0>
__device__ inline s16x4 ds_read_tr(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  s16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

// LDS byte address (32-bit) of a pointer into shared memory.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const TRIATTN_LDS void*)p;
}

// Per-lane address of the transposed fragment reads of a block: lane l
// (16-lane group G = l / 16, index j = l % 4 within its row of 4, e = l % 16
// / 4) supplies channels 16 (G % 2) + 4 j .. +3 of position base + e, where
// base = 4 (G / 2) + 16 t (+ 8 for the second half) + key offset.  The
// result of the pair of reads is the A/B fragment whose lane l holds channel
// l % 32 and positions {16 t + 4 g + 0..3, 16 t + 8 + 4 g + 0..3}, g = l / 32:
// the quad order of an accumulator-fed operand (see quad_frags).
struct TrAddr {
  int pe;    // e + 4 (G / 2): position offset of this lane's source row
  int cch;   // logical chunk 2 (G % 2) + j / 2
  int half;  // byte offset 8 (j % 2) inside the chunk
  __device__ inline explicit TrAddr(int lane) {
    const int G = lane >> 4, i = lane & 15, j = i & 3, e = i >> 2;
    pe = e + 4 * (G >> 1);
    cch = 2 * (G & 1) + (j >> 1);
    half = 8 * (j & 1);
  }
  // byte offset for source position p0 + pe
  __device__ inline int off(int p0) const {
    const int p = p0 + pe;
    return blk_off(p, cch) + half;
  }
  // The slot permutation of p0 + pe depends on bit 3 of p0 and not on its
  // bits 4 and up, so for p0 = 16 k the read is off(0) + 64 p0 and for
  // p0 = 16 k + 8 it is off(8) + 64 (p0 - 8): two base addresses and
  // immediate offsets cover a whole block.
};

// DMA-staged data is read with inline assembly: an ordinary load of an LDS
// array that DMA writes makes the compiler wait for every outstanding vector
// load first (it cannot tell which DMA filled what).
// Four LDS reads and the wait for them in ONE asm statement.  A read issued
// by one statement and waited for by a later one leaves the compiler free to
// copy the destination register in between, before the data has arrived;
// within one statement it cannot.  Early-clobber outputs keep the
// destinations off the address registers.
__device__ inline void tr_read4_wait(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3,
                                     s16x4 (&r)[4]) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %4\n\tds_read_b64_tr_b16 %1, %5\n\t"
      "ds_read_b64_tr_b16 %2, %6\n\tds_read_b64_tr_b16 %3, %7\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
      : "v"(a0), "v"(a1), "v"(a2), "v"(a3));
}
__device__ inline void b128_read4_wait(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3,
                                       f32x4 (&r)[4]) {
  asm volatile(
      "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\t"
      "ds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
      : "v"(a0), "v"(a1), "v"(a2), "v"(a3));
}

// Wait for all outstanding LDS reads, tied to the registers they fill so
// that no use of them is scheduled before the wait.
__device__ inline void tr_wait(s16x4 (&r)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]));
}

__device__ inline bf16x8 tr_frag(const s16x4 (&r)[4], int t) {
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(r[2 * t], r[2 * t + 1], 0, 1, 2, 3,
                                                            4, 5, 6, 7));
}

}  // namespace triattn
