// The key set one tree node attends to, enumerated without materialising it.
//
// Node i of row b stands at position p = L + depth[i].  Its keys, in order:
//   [0, nsel)            CSA entries chosen by the indexer top-k (sel list,
//                        ascending logical index; an index >= L/ratio_csa is
//                        an entry closed on i's own root path, held in scratch)
//   [.., + n128)         committed HCA entries
//   [.., + s128)         HCA entries closed on the root path (scratch)
//   [.., + nwin_c)       committed raw rows of positions win_lo..L-1
//   [.., + npath)        raw rows of the path nodes at positions max(L, win_lo)..p
// so a node sees the committed history and its own ancestors only
// (branch-aware causal visibility, Sec. 3.1).
#pragma once

#include "pool_addr.h"

namespace tv {

struct NodeKeys {
  int32_t L, n4, n128, nsel, s128, nwin_c, npath, n_keys;
  int64_t p, win_lo;
};

// Key counts of a node at depth di whose root path closes ncsa CSA and nhca
// HCA blocks.
__device__ inline NodeKeys make_node_keys(const tv_dims &d, int32_t L, int di, int ncsa, int nhca) {
  NodeKeys k;
  k.L = L;
  k.p = (int64_t)L + di;
  k.n4 = L / d.ratio_csa;
  k.n128 = L / d.ratio_hca;
  const int cand = k.n4 + ncsa;
  k.nsel = cand < d.topk ? cand : d.topk;
  k.s128 = nhca;
  const int64_t lo = k.p - d.window + 1;
  k.win_lo = lo > 0 ? lo : 0;
  k.nwin_c = (int32_t)(k.win_lo < L ? L - k.win_lo : 0);
  const int64_t pstart = k.win_lo > L ? k.win_lo : L;
  k.npath = (int32_t)(k.p - pstart + 1);
  k.n_keys = k.nsel + k.n128 + k.s128 + k.nwin_c + k.npath;
  return k;
}

// Root-path structure of node i of row b, computed by every wavefront from
// the ancestor mask m and dl, the depth of the row's node `lane` (lanes below
// D): path[d] (ancestor at depth d) and hca_node[t] (t-th path node closing an
// HCA block) are written to shared memory by wavefront 0 and are visible
// after the caller's next barrier; the returned counts need no barrier.
// csa_mask gets the path nodes closing a CSA block (bit = node index; on one
// root path node index order is depth order).
__device__ inline NodeKeys path_keys(const tv_dims &d, int32_t L, int i, uint64_t m, int dl, int32_t *path,
                                     int32_t *hca_node, uint64_t &csa_mask) {
  const int lane = threadIdx.x & 63;
  const bool onp = lane < d.D && ((m >> lane) & 1ull);
  const int32_t pl = L + dl;  // positions stay below 2^30
  const bool c4c = onp && (pl + 1) % d.ratio_csa == 0;
  const bool hcc = onp && (pl + 1) % d.ratio_hca == 0;
  csa_mask = __ballot(c4c);
  const uint64_t hca_mask = __ballot(hcc);
  if ((threadIdx.x >> 6) == 0) {
    if (onp) path[dl] = lane;
    if (hcc) hca_node[(pl + 1) / d.ratio_hca - 1 - L / d.ratio_hca] = lane;
  }
  return make_node_keys(d, L, __shfl(dl, i, 64), __popcll(csa_mask), __popcll(hca_mask));
}

// Fills path[d] (ancestor at depth d, d <= depth of i) and hca_node[t] (t-th
// path node closing an HCA block) in shared memory; must be called by every
// thread of the block (contains barriers).
__device__ inline NodeKeys node_keys(const tv_dims &d, int32_t L, int b, int i, const uint64_t *anc,
                                     const int32_t *depth, int32_t *path, int32_t *hca_node, int32_t *cnt) {
  const int lane = threadIdx.x & 63;
  const uint64_t m = anc[(int64_t)b * d.D + i];
  const int dl = lane < d.D ? depth[(int64_t)b * d.D + lane] : 0;
  uint64_t csa_mask;
  const NodeKeys k = path_keys(d, L, i, m, dl, path, hca_node, csa_mask);
  (void)cnt;
  __syncthreads();
  return k;
}

// Slot of committed entry s (s below the row's committed count) of the pool
// of `ratio`: base + s flat, through the page table paged.  A page the table
// does not allocate breaks the pool's contract; slot 0 keeps every read
// inside the pool.
__device__ __forceinline__ int64_t committed_slot(const tv_dims &d, const int32_t *page_table, int64_t base, int b,
                                                  int64_t s, int ratio) {
  if (d.page_size == 0) return base + s;
  const int64_t v = pool_slot(d, page_table, nullptr, nullptr, b, s, ratio);
  return v < 0 ? 0 : v;
}

// Pointer to the latent row (first d_row channels) of key t of the node.
// c4_base and c128_base are the row's pool bases (flat layout only).
__device__ inline const uint16_t *key_row(const tv_dims &d, const NodeKeys &k, int b, int t,
                                          const int32_t *sel_node, const int32_t *path, const int32_t *hca_node,
                                          const uint16_t *ring, const uint16_t *c4, const int64_t c4_base,
                                          const uint16_t *c128, const int64_t c128_base, const uint16_t *scr_c4,
                                          const uint16_t *scr_c128, const uint16_t *tree_u,
                                          const int32_t *page_table) {
  const int d_u = d.d_row + d.d_idx;
  if (t < k.nsel) {
    int s = sel_node[t];
    if (s < 0) s = 0;  // defensive: a selection list is never shorter than nsel
    if (s < k.n4) return c4 + committed_slot(d, page_table, c4_base, b, s, d.ratio_csa) * d.d_row;
    int64_t dd = (int64_t)(s + 1) * d.ratio_csa - 1 - k.L;
    if (dd < 0 || dd > k.p - k.L) dd = 0;  // defensive: stay on the node's own path
    return scr_c4 + ((int64_t)b * d.D + path[dd]) * d_u;
  }
  t -= k.nsel;
  if (t < k.n128) return c128 + committed_slot(d, page_table, c128_base, b, t, d.ratio_hca) * d.d_row;
  t -= k.n128;
  if (t < k.s128) return scr_c128 + ((int64_t)b * d.D + hca_node[t]) * d.d_row;
  t -= k.s128;
  if (t < k.nwin_c) {
    const int64_t ri = raw_index(d, page_table, b, k.win_lo + t);  // < 0 only if the page table breaks its contract
    return ri < 0 ? tree_u + (int64_t)b * d.D * d_u : ring + ri * d_u;
  }
  t -= k.nwin_c;
  const int64_t q = (k.win_lo > k.L ? k.win_lo : k.L) + t;
  return tree_u + ((int64_t)b * d.D + path[q - k.L]) * d_u;
}

}  // namespace tv
