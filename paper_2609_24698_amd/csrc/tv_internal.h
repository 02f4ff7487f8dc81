// Host-side plumbing shared by the API and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tv.h"

namespace tv {

// Device-resident pointers of one verify call, passed to kernels by value.
struct CacheView {
  const uint16_t *ring, *c4, *c4_idx, *c128;
  const int64_t *c4_base, *c128_base;
  const int32_t *c4_cap, *c128_cap;
  const int32_t *len;
  const int32_t *page_table;  // paged pool only (dims page_size > 0)
};

// Keys one attention workgroup takes per split (its LDS pointer table).
constexpr int kAttnMaxChunk = 1280;

// CSA top-k: committed entries one workgroup selects among (longer nodes are
// cut into segments of this many entries and merged), and the survivors the
// merge holds (512 threads x kTopkMergeKPT keys).
constexpr int kTopkSeg = 512 * 33;
constexpr int kTopkMergeKPT = 68;
constexpr int kTopkMergeCap = 512 * kTopkMergeKPT;
constexpr int kTopkMaxSeg = 64;
int topk_max_segments(const tv_dims &d);
bool topk_supported(const tv_dims &d);

// How the verify attention splits a node's keys across workgroups.
struct SplitPlan {
  int32_t max_keys;   // upper bound of any node's key count
  int32_t chunk;      // keys per split (multiple of the key tile)
  int32_t splits;     // splits per node
};

// Byte offsets of the verify workspace regions.
struct WsLayout {
  size_t scores;      // float [B*D][score_stride]
  size_t sel;         // int32 [B*D][topk], used when the caller passes no sel
  size_t part_o;      // float [B*D][splits][H][d_v]
  size_t part_ml;     // float2 [B*D][splits][H] (running max in log2 units, sum)
  size_t row_order;   // int32 [B]: rows by committed length, longest first
  size_t row_rank;    // int32 [B]: the inverse, rank of every row
  size_t keytab;      // const uint16_t* [B rank][D][plan.max_keys]: latent row of every key of every node, by rank
  size_t nkeys;       // int32 [B*D]: key count of every node
  size_t nkeys_rank;  // int32 [B rank][D]: the same counts by rank (0 for a skipped row)
  size_t surv_idx;    // int32 [B*D][topk segments][topk]: survivors of each top-k segment (segmented nodes only)
  size_t surv_key;    // uint32, same shape: their score keys
  size_t surv_cnt;    // int32 [B*D][topk segments]
  size_t total;
  int32_t score_stride;
  SplitPlan plan;
};

SplitPlan split_plan(const tv_dims &d);

// Compression blocks of at most this many tokens are pooled by one wavefront.
constexpr int kWaveMaxR = 4;
// Split compression applies: a CSA block fits one wavefront's registers, so
// CSA and HCA entries are pooled by separate workgroups.
__host__ __device__ inline bool compress_split(const tv_dims &d) {
  return d.ratio_csa <= kWaveMaxR && (d.d_row + d.d_idx) / 8 <= 128;
}

// Splits per node as the attention grid lays them out: with fewer than 8
// rows and 8 splits or more, padded to a multiple of 8 (split s on XCD s % 8).
__host__ __device__ inline int attn_padded_splits(int B, int splits) {
  return (B < 8 && splits >= 8) ? (splits + 7) & ~7 : splits;
}
// Workgroups of the attention grid (see unit_of).
inline int64_t attn_grid(const tv_dims &d, const SplitPlan &p) {
  if (d.B < 8) return (int64_t)d.B * d.D * attn_padded_splits(d.B, p.splits);
  return (int64_t)((d.B + 7) / 8) * 8 * d.D * p.splits;
}
WsLayout ws_layout(const tv_dims &d);

hipError_t launch_mask(const tv_dims &d, const int32_t *parents, uint64_t *anc, int32_t *depth,
                       int32_t *row_status, hipStream_t s);
hipError_t launch_compress(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                           const int32_t *depth, const uint16_t *gate_w, uint16_t *scr_c4, uint16_t *scr_c128,
                           int32_t *row_status, const int32_t *primary_last, uint16_t *pool_c4,
                           uint16_t *pool_c4_idx, hipStream_t s);
hipError_t launch_score(const tv_dims &d, const CacheView &c, const uint16_t *q_idx, const uint16_t *w_idx,
                        const int32_t *row_status, float *scores, int32_t score_stride, hipStream_t s);
// The scoring's fast path (H_idx = 8, D <= 8), which launch_mask_score
// requires.
bool score_fast_path(const tv_dims &d);
// launch_mask and launch_score (fast path) as one launch: the mask's
// workgroups first, then the scoring chunks, which do not read the masks;
// the mask also fails a valid tree whose length is out of range.  With
// csa_gate_w not NULL (split compression, flat pool), the launch also pools
// every CSA entry the tree closes into csa_scr_c4 (and the designated chain's
// into the pool), as the compression does.  With parents NULL there is no
// mask: anc, depth and row_status are inputs.
hipError_t launch_mask_score(const tv_dims &d, const int32_t *parents, uint64_t *anc, int32_t *depth,
                             int32_t *row_status, const CacheView &c, const uint16_t *q_idx, const uint16_t *w_idx,
                             float *scores, int32_t score_stride, const uint16_t *csa_tree_u,
                             const uint16_t *csa_gate_w, uint16_t *csa_scr_c4, const int32_t *csa_primary_last,
                             uint16_t *csa_pool_c4, uint16_t *csa_pool_c4_idx, hipStream_t s);
// With hca_gate_w not NULL (split compression only), the launch also pools
// every HCA entry the tree closes into hca_out, which must be scr_c128.
hipError_t launch_topk(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                       const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128, const uint16_t *q_idx,
                       const uint16_t *w_idx, const float *scores, int32_t score_stride, int32_t *sel,
                       int32_t *row_status, int32_t *row_order, int32_t *row_rank, const uint16_t **keytab,
                       int32_t keytab_stride, int32_t *nkeys, int32_t *nkeys_rank, int32_t *surv_idx,
                       uint32_t *surv_key, int32_t *surv_cnt, const uint16_t *hca_gate_w, uint16_t *hca_out,
                       hipStream_t s);
hipError_t launch_topk_merge(const tv_dims &d, const CacheView &c, const uint64_t *anc, const int32_t *depth,
                             const uint16_t *scr_c4, int32_t *sel, const int32_t *row_status,
                             const int32_t *row_rank, const uint16_t **keytab, int32_t keytab_stride,
                             const int32_t *surv_idx, const uint32_t *surv_key, const int32_t *surv_cnt,
                             hipStream_t s);
hipError_t launch_attn(const tv_dims &d, const uint16_t *q, const int32_t *row_status, const int32_t *row_order,
                       const uint16_t *const *keytab, const int32_t *nkeys, const SplitPlan &plan, float *part_o,
                       float *part_ml, uint16_t *out, float *lse, hipStream_t s);
hipError_t launch_attn_mla(const tv_dims &d, const uint16_t *q, const int32_t *row_status, const int32_t *row_order,
                           const uint16_t *const *keytab, const int32_t *nkeys, const SplitPlan &plan, float *part_o,
                           float *part_ml, uint16_t *out, float *lse, hipStream_t s);
hipError_t launch_combine(const tv_dims &d, const int32_t *row_status, const int32_t *nkeys, const SplitPlan &plan,
                          const float *part_o, const float *part_ml, uint16_t *out, float *lse, hipStream_t s);
// Per-layer buffers of a multi-layer commit (kernel arguments: at most
// kCommitMaxLayers layers per launch).
struct CommitLayer {
  tv_cache cache;
  const uint16_t *tree_u, *scr_c4, *scr_c128;
};
constexpr int kCommitMaxLayers = 32;
struct CommitLayers {
  CommitLayer l[kCommitMaxLayers];
  int32_t n;
};
hipError_t launch_commit_layers(const tv_dims &d, const CommitLayers &ls, const uint64_t *anc, const int32_t *depth,
                                const int32_t *accepted_last, int32_t *accept_nodes, int32_t *accept_len,
                                int32_t *row_status, const int32_t *primary_last, hipStream_t s);
hipError_t launch_commit(const tv_dims &d, const tv_cache &c, const uint16_t *tree_u, const uint64_t *anc,
                         const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128,
                         const int32_t *accepted_last, int32_t *accept_nodes, int32_t *accept_len,
                         int32_t *row_status, const int32_t *primary_last, hipStream_t s);

// Accepted-path selection: chunk keys of the target argmax, then the greedy path.
int select_chunks(int32_t vocab);
hipError_t launch_argmax(const tv_dims &d, const uint16_t *logits, int32_t vocab, uint64_t *part, hipStream_t s);
hipError_t launch_select(const tv_dims &d, const int32_t *parents, const uint64_t *anc, const int32_t *depth,
                         const int32_t *draft, int32_t vocab, const uint64_t *part, const int32_t *row_status,
                         int32_t *target, int32_t *accepted_last, int32_t *next_token, hipStream_t s);

// Kernel timing hooks (no-ops unless profiling is enabled).
int prof_before(const char *name, hipStream_t s);
void prof_after(int record, hipStream_t s);

}  // namespace tv
