// Pieces shared by the verify-attention kernels: tile constants, the
// XCD-aware grid decode, barriers and waits, and the direct global->LDS copy.
#pragma once

#include <algorithm>

#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kKT = 32;          // keys per tile
constexpr int kMaxChunk = kAttnMaxChunk;  // keys per split (pointer table in LDS)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Decode the XCD-aware block index.  Workgroups are dealt to the 8 XCDs
// round-robin (XCD = blockIdx % 8) and each XCD starts its workgroups in
// order.
//
// With 8 rows or more, rows are dealt to XCDs in the order row_order gives
// (longest first), back and forth: ranks 0..7 go to XCDs 0..7, ranks 8..15 to
// XCDs 7..0, and so on, so that no XCD takes the longest row of every group
// of eight.  Every unit of a row runs on one XCD, where the row's shared HCA,
// window and overlapping CSA entries stay in one L2, and each XCD starts its
// longest rows first.
//
// With fewer rows that would leave XCDs idle, so the (row, node, split) units
// are dealt over all eight: consecutive units go to consecutive XCDs.  When a
// node has 8 splits or more, its split count is padded to a multiple of 8 so
// that split s of every node runs on XCD s % 8: split s covers the same key
// positions in every node's list, which past the CSA selections are the same
// HCA entries, so those stay in one L2.  Padding units return at once.
//
// Returns the rank; the unit is valid when the rank is below B.
__device__ __forceinline__ int unit_of(int blk, int B, int D, int splits, int &i, int &s) {
  if (B < 8) {
    const int sp = attn_padded_splits(B, splits);
    s = blk % sp;
    const int r = blk / sp;
    i = r % D;
    return s < splits ? r / D : B;
  }
  const int x = blk & 7, q = blk >> 3;
  s = q % splits;
  const int r = q / splits;
  i = r % D;
  const int g = r / D;  // group of eight ranks
  return g * 8 + ((g & 1) ? 7 - x : x);
}

// Barrier that waits for this wavefront's LDS traffic only: global loads in
// flight (the next tiles) stay in flight across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
template <int N>
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane l's 16 bytes land at LDS byte address lds + 16 l.  Issued from inline
// assembly so that the compiler's wait-count pass does not order later LDS
// reads of other buffers behind it; completion is awaited explicitly with
// vm_wait<> before the barrier that publishes the tile (both carry memory
// clobbers, the copy itself needs none: nothing reads its destination before
// that barrier).  M0 (the LDS base) is saved and restored around the copy.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds)));
}

typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

}  // namespace tv
