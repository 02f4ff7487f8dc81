// Where the committed state of a row lives: the raw row of a position and
// the slot of a CSA or HCA entry, in either layout.
//
// Flat layout (page_size 0): raw rows in a ring per row (position q in slot
// q mod ring_cap), entries at base[b] + s of pools with cap[b] slots per row.
//
// Paged layout (Sec. 4.2: one logical layer of positions viewed as three
// physical layers with shared page-level pointers): logical page j of row b
// (positions jP .. jP+P-1) has the physical page page_table[b][j], -1 when
// none is allocated, and that one id addresses the three layers: raw rows
// ([pages][P][d_u]), CSA entries (P/ratio_csa per page) and HCA entries
// (P/ratio_hca per page), the entry of logical index s in the page holding
// its first token.
#pragma once

#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

// Physical page of logical page j of row b, -1 when none is allocated.
__device__ __forceinline__ int32_t page_of(const tv_dims &d, const int32_t *table, int b, int64_t j) {
  return (j >= 0 && j < d.page_stride) ? table[(int64_t)b * d.page_stride + j] : -1;
}

// Slot of entry s of row b in the pool of `ratio` (flat: base/cap of that
// pool), -1 when the row has none.
__device__ __forceinline__ int64_t pool_slot(const tv_dims &d, const int32_t *table, const int64_t *base,
                                             const int32_t *cap, int b, int64_t s, int ratio) {
  if (d.page_size == 0) return s < cap[b] ? base[b] + s : -1;
  const int per = d.page_size / ratio;
  const int32_t pg = page_of(d, table, b, s / per);
  return pg < 0 ? -1 : (int64_t)pg * per + s % per;
}

// Index (in d_u-wide rows) of the raw row of position q of row b, -1 when
// its page is not allocated.
__device__ __forceinline__ int64_t raw_index(const tv_dims &d, const int32_t *table, int b, int64_t q) {
  if (d.page_size == 0) return (int64_t)b * d.ring_cap + (q & (d.ring_cap - 1));
  const int32_t pg = page_of(d, table, b, q / d.page_size);
  return pg < 0 ? -1 : (int64_t)pg * d.page_size + q % d.page_size;
}

}  // namespace tv
