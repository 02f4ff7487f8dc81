// Accepted-path refresh of the committed state.
//
// After verification only the accepted root path survives (Sec. 3.2, Sec. 4.2):
// its raw rows enter the window ring, every block it closed becomes a committed
// CSA / HCA entry (copied from the path node's scratch slot), and the committed
// length advances.  Entries compressed on rejected branches are never copied,
// so they leave no trace in the persistent state.
//
// One workgroup per row.  All checks run before the first write, so a failing
// row is left exactly as it was.  Destinations follow the cache layout: the
// ring and per-row pools, or with a paged pool the raw, CSA and HCA layers
// through the row's page table (a page it does not allocate fails the row).
// The row's loads go out together; the copies (ring rows, CSA and HCA
// entries) form one list of 16-byte chunks whose loads a thread issues
// before its stores.
//
// With FP8 indexer keys a CSA entry's indexer channels (E4M3 values held
// in bfloat16 in scratch) are narrowed, exactly, to E4M3 codes in the pool.
//
// Refresh schedule (Sec. 4.3): with a designated chain (the root path of
// primary_last[b]), whose CSA entries the compression already wrote into the
// pool, the CSA copies of accepted nodes on that chain are skipped: a single
// chain, or an accepted path that is the cached chain, needs no CSA refresh.
// HCA entries are always written here, once the path is known, all of a
// round's in one pass.
#include "pool_addr.h"

namespace tv {

struct CommitSmem {
  int32_t path[64];
  int32_t ent[2][64];  // closing path depths: CSA entries to copy, HCA entries
  int nent[2];
  int64_t raw_at[64], slot_at[2][64];  // by path depth: raw-row index, CSA / HCA pool slot
};

// The part of a row's commit that one layer's cache decides: destinations
// (flat: ring slot, base + index below the capacity; paged: through the page
// table), all resolved before any write, then the copies and the new length.
// The accepted path (a nodes, path[] in LDS by depth) and the designated
// chain are the row's.  Returns TV_ROW_OK, or TV_ROW_CAPACITY (written to
// row_status[b]) when a destination is missing.  Uniform over the workgroup;
// ends with the entry lists and slots read out.
__device__ __forceinline__ int32_t commit_layer(const tv_dims &d, const tv_cache &c,
                                                const uint16_t *__restrict__ tree_u,
                                                const uint16_t *__restrict__ scr_c4,
                                                const uint16_t *__restrict__ scr_c128,
                                                int32_t *__restrict__ row_status, int b, int32_t L, int a,
                                                uint64_t chain, int32_t cap4, int32_t cap128, int64_t base4,
                                                int64_t base128, CommitSmem &sm) {
  int32_t *path = sm.path;
  int32_t(*ent)[64] = sm.ent;
  int *nent = sm.nent;
  int64_t *raw_at = sm.raw_at;
  int64_t(*slot_at)[64] = sm.slot_at;
  const int tid = threadIdx.x;
  const int64_t rb = (int64_t)b * d.D;
  const bool flat = d.page_size == 0;
  if (tid < 2) nent[tid] = 0;
  bool bad = false;
  if (tid < a) {
    const int64_t p = (int64_t)L + tid;  // path node at depth tid stands at L + tid
    const int64_t ri = raw_index(d, c.page_table, b, p);
    raw_at[tid] = ri;
    bad |= ri < 0;
    if ((p + 1) % d.ratio_csa == 0) {
      const int64_t s4 = (p + 1) / d.ratio_csa - 1;
      const int64_t sl = flat ? (s4 < cap4 ? base4 + s4 : -1)
                              : pool_slot(d, c.page_table, nullptr, nullptr, b, s4, d.ratio_csa);
      slot_at[0][tid] = sl;
      bad |= sl < 0;
    }
    if ((p + 1) % d.ratio_hca == 0) {
      const int64_t s128 = (p + 1) / d.ratio_hca - 1;
      const int64_t sl = flat ? (s128 < cap128 ? base128 + s128 : -1)
                              : pool_slot(d, c.page_table, nullptr, nullptr, b, s128, d.ratio_hca);
      slot_at[1][tid] = sl;
      bad |= sl < 0;
    }
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) row_status[b] = TV_ROW_CAPACITY;
    return TV_ROW_CAPACITY;
  }
  // the closing path depths, in depth order (wave 0: ballots over lanes t < a)
  if (tid < 64) {
    const int64_t p = (int64_t)L + tid;
    const bool c4 = tid < a && (p + 1) % d.ratio_csa == 0 && !((chain >> path[tid < a ? tid : 0]) & 1ull);
    const bool c128 = tid < a && (p + 1) % d.ratio_hca == 0;
    const uint64_t b4 = __ballot(c4), b128 = __ballot(c128);
    const uint64_t below = (1ull << tid) - 1ull;  // lanes below this one
    if (c4) ent[0][__popcll(b4 & below)] = tid;
    if (c128) ent[1][__popcll(b128 & below)] = tid;
    if (tid == 0) {
      nent[0] = __popcll(b4);
      nent[1] = __popcll(b128);
    }
  }
  __syncthreads();
  // Copies as one list of 16-byte chunks: raw rows of the path into the ring,
  // CSA entries (latent row, then indexer key) and HCA entries into their
  // pool slots.  A thread's loads all go out before its stores.
  const int d_u = d.d_row + d.d_idx;
  const int cpr = d_u / 8, c4c = d_u / 8, c128c = d.d_row / 8;
  const int n_ring = a * cpr, n4 = nent[0] * c4c, n128 = nent[1] * c128c;
  const int total = n_ring + n4 + n128;
  constexpr int kBatch = 4;
  for (int e0 = 0; e0 < total; e0 += kBatch * (int)blockDim.x) {
    uint4 v[kBatch];
    uint16_t *dst[kBatch];
    uint8_t *dst8[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int e = e0 + u * (int)blockDim.x + tid;
      dst[u] = nullptr;
      dst8[u] = nullptr;
      v[u] = make_uint4(0, 0, 0, 0);
      if (e < n_ring) {
        const int t = e / cpr, cc = (e - t * cpr) * 8;
        v[u] = *reinterpret_cast<const uint4 *>(tree_u + (rb + path[t]) * d_u + cc);
        dst[u] = c.ring + raw_at[t] * d_u + cc;
      } else if (e < n_ring + n4) {
        const int x = e - n_ring, k = x / c4c, ch = (x - k * c4c) * 8;
        const int t = ent[0][k];
        const int64_t slot = slot_at[0][t];
        v[u] = *reinterpret_cast<const uint4 *>(scr_c4 + (rb + path[t]) * d_u + ch);
        dst[u] = ch < d.d_row ? c.c4 + slot * d.d_row + ch : c.c4_idx + slot * d.d_idx + (ch - d.d_row);
        if (ch >= d.d_row && d.idx_fmt == TV_IDX_E4M3) {  // eight E4M3 codes: 8 bytes at byte offset slot*d_idx + ...
          dst8[u] = reinterpret_cast<uint8_t *>(c.c4_idx) + slot * d.d_idx + (ch - d.d_row);
          dst[u] = nullptr;
        }
      } else if (e < total) {
        const int x = e - n_ring - n4, k = x / c128c, ch = (x - k * c128c) * 8;
        const int t = ent[1][k];
        const int64_t slot = slot_at[1][t];
        v[u] = *reinterpret_cast<const uint4 *>(scr_c128 + (rb + path[t]) * d.d_row + ch);
        dst[u] = c.c128 + slot * d.d_row + ch;
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (dst[u]) *reinterpret_cast<uint4 *>(dst[u]) = v[u];
      if (dst8[u]) {  // the scratch holds E4M3 values in bfloat16: narrow them exactly
        uint2 w;
        w.x = bf16_to_e4m3(v[u].x & 0xFFFF) | (bf16_to_e4m3(v[u].x >> 16) << 8) |
              (bf16_to_e4m3(v[u].y & 0xFFFF) << 16) | (bf16_to_e4m3(v[u].y >> 16) << 24);
        w.y = bf16_to_e4m3(v[u].z & 0xFFFF) | (bf16_to_e4m3(v[u].z >> 16) << 8) |
              (bf16_to_e4m3(v[u].w & 0xFFFF) << 16) | (bf16_to_e4m3(v[u].w >> 16) << 24);
        *reinterpret_cast<uint2 *>(dst8[u]) = w;
      }
    }
  }
  if (tid == 0) c.len[b] = L + a;
  __syncthreads();  // the entry lists and slots are read out
  return TV_ROW_OK;
}

// The commit of row b of one layer's cache, by the whole workgroup.  `status`
// is the row's status before it (TV_ROW_OK to commit); returns the row's status
// after it, having written row_status[b] where it changed.  Uniform over the
// workgroup; ends with the workgroup's LDS free for the next call.
__device__ __forceinline__ int32_t commit_row(const tv_dims &d, const tv_cache &c, const uint16_t *__restrict__ tree_u,
                                              const uint64_t *__restrict__ anc, const int32_t *__restrict__ depth,
                                              const uint16_t *__restrict__ scr_c4,
                                              const uint16_t *__restrict__ scr_c128,
                                              const int32_t *__restrict__ accepted_last,
                                              int32_t *__restrict__ accept_nodes, int32_t *__restrict__ accept_len,
                                              int32_t *__restrict__ row_status,
                                              const int32_t *__restrict__ primary_last, int b, int32_t status,
                                              CommitSmem &sm) {
  const int tid = threadIdx.x;
  const int64_t rb = (int64_t)b * d.D;
  // every independent load first, one wait for all of them
  const int32_t L = c.len[b];
  const int32_t last = accepted_last[b];
  const int32_t P = primary_last ? primary_last[b] : -1;
  const int32_t dt = tid < d.D ? depth[rb + tid] : 0;
  const bool flat = d.page_size == 0;
  const int32_t cap4 = flat ? c.c4_cap[b] : 0, cap128 = flat ? c.c128_cap[b] : 0;
  const int64_t base4 = flat ? c.c4_base[b] : 0, base128 = flat ? c.c128_base[b] : 0;
  if (status != TV_ROW_OK) return status;
  if (!len_ok(L, d.max_len)) {
    if (tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return TV_ROW_BAD_LEN;
  }
  if (last < 0 || last >= d.D) {
    if (tid == 0) row_status[b] = TV_ROW_BAD_ACCEPT;
    return TV_ROW_BAD_ACCEPT;
  }
  const uint64_t m = anc[rb + last];
  const uint64_t chain = (P >= 0 && P < d.D) ? anc[rb + P] : 0ull;
  const int a = depth[rb + last] + 1;
  if (tid < d.D && ((m >> tid) & 1ull)) sm.path[dt] = tid;
  const int32_t st = commit_layer(d, c, tree_u, scr_c4, scr_c128, row_status, b, L, a, chain, cap4, cap128, base4,
                                  base128, sm);
  if (st != TV_ROW_OK) return st;
  if (tid < d.D) accept_nodes[rb + tid] = tid < a ? sm.path[tid] : -1;
  if (tid == 0) accept_len[b] = a;
  __syncthreads();  // the path is read out
  return TV_ROW_OK;
}

__global__ void __launch_bounds__(256) commit_kernel(tv_dims d, tv_cache c, const uint16_t *__restrict__ tree_u,
                                                     const uint64_t *__restrict__ anc,
                                                     const int32_t *__restrict__ depth,
                                                     const uint16_t *__restrict__ scr_c4,
                                                     const uint16_t *__restrict__ scr_c128,
                                                     const int32_t *__restrict__ accepted_last,
                                                     int32_t *__restrict__ accept_nodes,
                                                     int32_t *__restrict__ accept_len,
                                                     int32_t *__restrict__ row_status,
                                                     const int32_t *__restrict__ primary_last) {
  __shared__ CommitSmem sm;
  const int b = blockIdx.x;
  const int32_t status = row_status[b];
  (void)commit_row(d, c, tree_u, anc, depth, scr_c4, scr_c128, accepted_last, accept_nodes, accept_len, row_status,
                   primary_last, b, status, sm);
}

// The commits of several layers that share a tree, one workgroup per row
// walking the layers in order: a row that fails in one layer is skipped by
// every later one, as with one call per layer, and one launch replaces a
// launch per layer (the graph round's commits).  The accepted path is the
// row's and is resolved once; each layer's length, capacities and pool bases
// are loaded while the layer before it copies.
__global__ void __launch_bounds__(256) commit_layers_kernel(tv_dims d, CommitLayers ls, const uint64_t *__restrict__ anc,
                                                            const int32_t *__restrict__ depth,
                                                            const int32_t *__restrict__ accepted_last,
                                                            int32_t *__restrict__ accept_nodes,
                                                            int32_t *__restrict__ accept_len,
                                                            int32_t *__restrict__ row_status,
                                                            const int32_t *__restrict__ primary_last) {
  __shared__ CommitSmem sm;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int64_t rb = (int64_t)b * d.D;
  const bool flat = d.page_size == 0;
  int32_t status = row_status[b];
  const int32_t last = accepted_last[b];
  const int32_t P = primary_last ? primary_last[b] : -1;
  const int32_t dt = tid < d.D ? depth[rb + tid] : 0;
  auto layer_state = [&](int l, int32_t &L, int32_t &cap4, int32_t &cap128, int64_t &base4, int64_t &base128) {
    const tv_cache &c = ls.l[l].cache;
    L = c.len[b];
    cap4 = flat ? c.c4_cap[b] : 0;
    cap128 = flat ? c.c128_cap[b] : 0;
    base4 = flat ? c.c4_base[b] : 0;
    base128 = flat ? c.c128_base[b] : 0;
  };
  int32_t L, cap4, cap128;
  int64_t base4, base128;
  layer_state(0, L, cap4, cap128, base4, base128);
  if (status != TV_ROW_OK) return;
  const bool last_ok = last >= 0 && last < d.D;
  const uint64_t m = last_ok ? anc[rb + last] : 0ull;
  const uint64_t chain = (P >= 0 && P < d.D) ? anc[rb + P] : 0ull;
  const int a = last_ok ? depth[rb + last] + 1 : 0;
  if (tid < d.D && ((m >> tid) & 1ull)) sm.path[dt] = tid;
  bool committed = false;
  for (int l = 0; l < ls.n; ++l) {
    if (!len_ok(L, d.max_len)) {
      if (tid == 0) row_status[b] = TV_ROW_BAD_LEN;
      return;
    }
    if (!last_ok) {
      if (tid == 0) row_status[b] = TV_ROW_BAD_ACCEPT;
      return;
    }
    const CommitLayer &cl = ls.l[l];
    const int32_t Lc = L;
    const int32_t c4c = cap4, c128c = cap128;
    const int64_t b4c = base4, b128c = base128;
    if (l + 1 < ls.n) layer_state(l + 1, L, cap4, cap128, base4, base128);  // in flight during this layer's copies
    if (commit_layer(d, cl.cache, cl.tree_u, cl.scr_c4, cl.scr_c128, row_status, b, Lc, a, chain, c4c, c128c, b4c,
                     b128c, sm) != TV_ROW_OK)
      return;
    if (!committed) {  // every layer's commit writes the same path
      committed = true;
      if (tid < d.D) accept_nodes[rb + tid] = tid < a ? sm.path[tid] : -1;
      if (tid == 0) accept_len[b] = a;
    }
  }
}

hipError_t launch_commit_layers(const tv_dims &d, const CommitLayers &ls, const uint64_t *anc, const int32_t *depth,
                                const int32_t *accepted_last, int32_t *accept_nodes, int32_t *accept_len,
                                int32_t *row_status, const int32_t *primary_last, hipStream_t s) {
  if (ls.n < 1 || ls.n > kCommitMaxLayers) return hipErrorInvalidValue;
  commit_layers_kernel<<<d.B, 256, 0, s>>>(d, ls, anc, depth, accepted_last, accept_nodes, accept_len, row_status,
                                           primary_last);
  return hipGetLastError();
}

hipError_t launch_commit(const tv_dims &d, const tv_cache &c, const uint16_t *tree_u, const uint64_t *anc,
                         const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128,
                         const int32_t *accepted_last, int32_t *accept_nodes, int32_t *accept_len,
                         int32_t *row_status, const int32_t *primary_last, hipStream_t s) {
  commit_kernel<<<d.B, 256, 0, s>>>(d, c, tree_u, anc, depth, scr_c4, scr_c128, accepted_last, accept_nodes,
                                    accept_len, row_status, primary_last);
  return hipGetLastError();
}

}  // namespace tv
