// Verify preprocess: parent array -> ancestor bitmask, depth and row status.
//
// One 64-lane wavefront per row, lane i owns node i (D <= 64).  A row is valid
// when the root has parent -1 and every other node's parent precedes it; the
// ancestor set of node i is i plus the ancestor set of its parent (the tree
// topology that branch-aware verification must respect, Sec. 3.1 and Sec. 4.1).
#include "compress_body.h"
#include "score_h8.h"

namespace tv {

// Workgroup `blk` (256 threads) takes rows 4 blk .. 4 blk + 3, one per
// wavefront.  With `len` (and its bound max_len), a valid tree whose row
// length is out of range gets TV_ROW_BAD_LEN, the status the compression
// would give it next.
__device__ __forceinline__ void mask_rows(int B, int D, const int32_t *__restrict__ parents,
                                          uint64_t *__restrict__ anc, int32_t *__restrict__ depth,
                                          int32_t *__restrict__ row_status, const int32_t *__restrict__ len,
                                          int max_len, int blk, int32_t (*par)[64]) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int b = blk * 4 + w;
  const bool live = b < B;
  const int i = lane;
  int32_t p = (live && i < D) ? parents[(int64_t)b * D + i] : 0;
  bool ok = (i >= D) || (i == 0 ? p == -1 : (p >= 0 && p < i));
  par[w][lane] = p;
  const bool row_ok = __all(ok);
  __syncthreads();
  if (!live) return;
  if (i < D) {
    uint64_t m = 0;
    int32_t dep = 0;
    if (row_ok) {
      m = 1ull << i;
      int j = p;
      while (j >= 0) {  // parents strictly decrease, so at most i steps
        m |= 1ull << j;
        ++dep;
        j = par[w][j];
      }
    }
    anc[(int64_t)b * D + i] = m;
    depth[(int64_t)b * D + i] = dep;
  }
  if (lane == 0)
    row_status[b] = !row_ok ? TV_ROW_BAD_PARENT : (len && !len_ok(len[b], max_len)) ? TV_ROW_BAD_LEN : TV_ROW_OK;
}

__global__ void __launch_bounds__(256) mask_kernel(int B, int D, const int32_t *__restrict__ parents,
                                                   uint64_t *__restrict__ anc, int32_t *__restrict__ depth,
                                                   int32_t *__restrict__ row_status) {
  __shared__ int32_t par[4][64];
  mask_rows(B, D, parents, anc, depth, row_status, nullptr, 0, blockIdx.x, par);
}

// The verify preprocess and the indexer scoring (fast path) in one launch:
// the scoring reads only committed state and the queries, not the masks, so
// its chunk workgroups (the scoring kernel's grid) follow the mask's in the
// same grid.  The scoring skips no row on its status, which the mask writes
// meanwhile; a row the mask fails gets scores that no later step reads.
// With the split compression's CSA entries (csa.gate_w not NULL), a
// wavefront per node pools them between the two, deriving the node's
// ancestors from the parent array itself (csa_wave_node<true>).  Without
// parents the launch has no mask workgroups: the masks and the row status
// are already final (a later layer of the round), and the CSA wavefronts
// read them.
struct CsaArgs {
  const uint16_t *tree_u, *gate_w;
  uint16_t *scr_c4;
  const int32_t *primary_last;
  uint16_t *pool_c4, *pool_c4_idx;
};

template <bool FP8>
__global__ void __launch_bounds__(256) mask_score_kernel(tv_dims d, const int32_t *__restrict__ parents,
                                                         uint64_t *__restrict__ anc, int32_t *__restrict__ depth,
                                                         int32_t *__restrict__ row_status, CacheView c,
                                                         const uint16_t *__restrict__ q_idx,
                                                         const uint16_t *__restrict__ w_idx,
                                                         float *__restrict__ scores, int score_stride,
                                                         int chunks_per_row, CsaArgs csa, int ncsa) {
  __shared__ union {
    int32_t par[4][64];
    int32_t paths[4][64];
    ScoreH8Smem<4> ss;
  } sm;
  const int nmask = parents ? (d.B + 3) / 4 : 0;
  const int blk = blockIdx.x;
  if (blk < nmask) {
    mask_rows(d.B, d.D, parents, anc, depth, row_status, c.len, d.max_len, blk, sm.par);
  } else if (blk < nmask + ncsa) {
    const int wv = threadIdx.x >> 6, n = (blk - nmask) * 4 + wv;
    if (n < d.B * d.D) {
      if (parents)  // beside the mask: ancestors from the parent array
        csa_wave_node<true>(d, c, parents, nullptr, nullptr, csa.tree_u, csa.gate_w, csa.scr_c4, row_status,
                            csa.primary_last, csa.pool_c4, csa.pool_c4_idx, n, sm.paths[wv]);
      else  // the masks and row status are final
        csa_wave_node<false>(d, c, nullptr, anc, depth, csa.tree_u, csa.gate_w, csa.scr_c4, row_status,
                             csa.primary_last, csa.pool_c4, csa.pool_c4_idx, n, sm.paths[wv]);
    }
  } else {
    const int k = blk - nmask - ncsa, b = k / chunks_per_row;
    score_h8_chunk<FP8, 4, false>(d, c, q_idx, w_idx, nullptr, scores, score_stride, b, k - b * chunks_per_row,
                                  sm.ss);
  }
}

hipError_t launch_mask_score(const tv_dims &d, const int32_t *parents, uint64_t *anc, int32_t *depth,
                             int32_t *row_status, const CacheView &c, const uint16_t *q_idx, const uint16_t *w_idx,
                             float *scores, int32_t score_stride, const uint16_t *csa_tree_u,
                             const uint16_t *csa_gate_w, uint16_t *csa_scr_c4, const int32_t *csa_primary_last,
                             uint16_t *csa_pool_c4, uint16_t *csa_pool_c4_idx, hipStream_t s) {
  if (!score_fast_path(d)) return hipErrorInvalidValue;
  const bool with_csa = csa_gate_w != nullptr;
  if (with_csa && (!compress_split(d) || d.page_size != 0)) return hipErrorInvalidValue;
  const int chunks = std::max(1, (d.max_len / d.ratio_csa + 255) / 256);
  const int ncsa = with_csa ? (d.B * d.D + 3) / 4 : 0;
  const int64_t grid = (parents ? (int64_t)(d.B + 3) / 4 : 0) + ncsa + (int64_t)d.B * chunks;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  const CsaArgs csa{csa_tree_u, csa_gate_w, csa_scr_c4, csa_primary_last, csa_pool_c4, csa_pool_c4_idx};
  if (d.idx_fmt == TV_IDX_E4M3)
    mask_score_kernel<true><<<(unsigned)grid, 256, 0, s>>>(d, parents, anc, depth, row_status, c, q_idx, w_idx,
                                                           scores, score_stride, chunks, csa, ncsa);
  else
    mask_score_kernel<false><<<(unsigned)grid, 256, 0, s>>>(d, parents, anc, depth, row_status, c, q_idx, w_idx,
                                                            scores, score_stride, chunks, csa, ncsa);
  return hipGetLastError();
}

hipError_t launch_mask(const tv_dims &d, const int32_t *parents, uint64_t *anc, int32_t *depth,
                       int32_t *row_status, hipStream_t s) {
  dim3 grid((d.B + 3) / 4);
  mask_kernel<<<grid, 256, 0, s>>>(d.B, d.D, parents, anc, depth, row_status);
  return hipGetLastError();
}

}  // namespace tv
