// CSA indexer scores of every committed entry for every node of a row.
//
// score[b][i][s] = sum_h w[b][i][h] * relu(q_idx[b][i][h] . k_s) over the
// committed entries s < len/ratio_csa.  The (node, head) query rows of one
// tree form the M side of a dense contraction against the row's indexer keys,
// so the product runs on MFMA (v_mfma_f32_32x32x16_bf16, float32 accumulate);
// the head reduction runs in a fixed order so scores are bitwise repeatable.
// FP8 indexer keys (E4M3 codes) are widened exactly to bfloat16 as they are
// loaded, so the same bfloat16 products score them.
//
// General path: a persistent grid strides over the (row, 128-entry chunk)
// list of all valid rows, so ragged lengths cost no idle workgroups.  Fast
// path (H_idx = 8, D <= 8): one 4-wavefront workgroup per (row, 256-entry
// chunk), the chunk body shared with the compression-and-scoring kernel.
#include <algorithm>

#include "score_h8.h"

namespace tv {

constexpr int kScoreChunk = 128;  // entries per chunk: 4 wavefronts x 32

// Exclusive prefix sum over a 256-thread block; returns the total.
__device__ int block_excl_scan(int v, int *tmp, int *out_excl) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) tmp[wv] = x;
  __syncthreads();
  int base = 0, total = 0;
  for (int k = 0; k < 4; ++k) {
    if (k < wv) base += tmp[k];
    total += tmp[k];
  }
  *out_excl = base + x - v;
  __syncthreads();
  return total;
}

template <bool FP8>
__global__ void __launch_bounds__(256) score_kernel(tv_dims d, CacheView c, const uint16_t *__restrict__ q_idx,
                                                    const uint16_t *__restrict__ w_idx,
                                                    const int32_t *__restrict__ row_status,
                                                    float *__restrict__ scores, int score_stride) {
  __shared__ int chunk_pref[kMaxB + 1];
  __shared__ int scan_tmp[4];
  __shared__ float P[64][kScoreChunk + 4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

  // chunk counts of every row, scanned
  const int per = (d.B + 255) / 256;
  int mine = 0;
  for (int k = 0; k < per; ++k) {
    const int b = tid * per + k;
    if (b < d.B) {
      const int32_t L = c.len[b];
      const bool ok = row_status[b] == TV_ROW_OK && len_ok(L, d.max_len);
      mine += ok ? (L / d.ratio_csa + kScoreChunk - 1) / kScoreChunk : 0;
    }
  }
  int excl;
  const int total = block_excl_scan(mine, scan_tmp, &excl);
  for (int k = 0, run = excl; k < per; ++k) {
    const int b = tid * per + k;
    if (b < d.B) {
      chunk_pref[b] = run;
      const int32_t L = c.len[b];
      const bool ok = row_status[b] == TV_ROW_OK && len_ok(L, d.max_len);
      run += ok ? (L / d.ratio_csa + kScoreChunk - 1) / kScoreChunk : 0;
    }
  }
  if (tid == 0) chunk_pref[d.B] = total;
  __syncthreads();

  const int M = d.D * d.H_idx;
  const int groups = (M + 63) / 64;
  const int nodes_per_group = 64 / d.H_idx;
  for (int cid = blockIdx.x; cid < total; cid += gridDim.x) {
    // row owning chunk cid: last b with chunk_pref[b] <= cid
    int lo = 0, hi = d.B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (chunk_pref[mid] <= cid) lo = mid; else hi = mid - 1;
    }
    const int b = lo;
    const int n4 = c.len[b] / d.ratio_csa;
    const int e0 = (cid - chunk_pref[b]) * kScoreChunk;
    const int e = e0 + wv * 32 + (lane & 31);
    // B operand: the wavefront's 32 keys, 16 channels per k-step
    bf16x8 kb[4];
    {
      const bool live = e < n4;
      const int64_t entry = d.page_size == 0 ? c.c4_base[b] + (live ? e : 0)
                                             : std::max<int64_t>(0, pool_slot(d, c.page_table, nullptr, nullptr, b,
                                                                              live ? e : 0, d.ratio_csa));
      uint4 raw[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        raw[ks] = live ? key_load<FP8>(c.c4_idx, entry, ks * 2 + (lane >> 5)) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) kb[ks] = __builtin_bit_cast(bf16x8, key_bf16<FP8>(raw[ks]));
    }
    for (int g = 0; g < groups; ++g) {
      f32x16 acc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        acc[t] = f32x16{};
        const int r = g * 64 + t * 32 + (lane & 31);
        const bool live = r < M;
        const int node = live ? r / d.H_idx : 0, head = live ? r - node * d.H_idx : 0;
        const uint4 *src = reinterpret_cast<const uint4 *>(
            q_idx + ((((int64_t)b * d.D + node) * d.H_idx + head) * 64));
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          uint4 v = live ? src[ks * 2 + (lane >> 5)] : make_uint4(0, 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, v), kb[ks], acc[t], 0, 0, 0);
        }
      }
      // relu, head weight, park in LDS as P[row][entry]
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int rl = t * 32 + 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
          const int r = g * 64 + rl;
          float wgt = 0.f;
          if (r < M) {
            const int node = r / d.H_idx, head = r - node * d.H_idx;
            wgt = bf2f(w_idx[((int64_t)b * d.D + node) * d.H_idx + head]);
          }
          P[rl][wv * 32 + (lane & 31)] = wgt * fmaxf(acc[t][j], 0.f);
        }
      }
      __syncthreads();
      // per (node, entry): sum over heads in order
      for (int k = tid; k < nodes_per_group * kScoreChunk; k += 256) {
        const int nl = k / kScoreChunk, col = k - nl * kScoreChunk;
        const int node = g * nodes_per_group + nl;
        const int ee = e0 + col;
        if (node < d.D && ee < n4) {
          float s = 0.f;
          for (int h = 0; h < d.H_idx; ++h) s += P[nl * d.H_idx + h][col];
          scores[((int64_t)b * d.D + node) * score_stride + ee] = s;
        }
      }
      __syncthreads();
    }
  }
}


template <bool FP8>
__global__ void __launch_bounds__(256) score_kernel_h8(tv_dims d, CacheView c, const uint16_t *__restrict__ q_idx,
                                                       const uint16_t *__restrict__ w_idx,
                                                       const int32_t *__restrict__ row_status,
                                                       float *__restrict__ scores, int score_stride,
                                                       int chunks_per_row) {
  __shared__ ScoreH8Smem<4> sm;
  const int b = blockIdx.x / chunks_per_row;
  score_h8_chunk<FP8, 4, true>(d, c, q_idx, w_idx, row_status, scores, score_stride, b,
                               blockIdx.x - b * chunks_per_row, sm);
}

bool score_fast_path(const tv_dims &d) { return d.H_idx == 8 && d.D <= 8; }

hipError_t launch_score(const tv_dims &d, const CacheView &c, const uint16_t *q_idx, const uint16_t *w_idx,
                        const int32_t *row_status, float *scores, int32_t score_stride, hipStream_t s) {
  if (score_fast_path(d)) {
    const int chunks = std::max(1, (d.max_len / d.ratio_csa + 255) / 256);
    const int64_t grid = (int64_t)d.B * chunks;
    if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (d.idx_fmt == TV_IDX_E4M3)
      score_kernel_h8<true><<<(unsigned)grid, 256, 0, s>>>(d, c, q_idx, w_idx, row_status, scores, score_stride, chunks);
    else
      score_kernel_h8<false><<<(unsigned)grid, 256, 0, s>>>(d, c, q_idx, w_idx, row_status, scores, score_stride, chunks);
    return hipGetLastError();
  }
  const int64_t upper = (int64_t)d.B * ((d.max_len / d.ratio_csa + kScoreChunk - 1) / kScoreChunk);
  const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(upper, 2048));
  if (d.idx_fmt == TV_IDX_E4M3)
    score_kernel<true><<<grid, 256, 0, s>>>(d, c, q_idx, w_idx, row_status, scores, score_stride);
  else
    score_kernel<false><<<grid, 256, 0, s>>>(d, c, q_idx, w_idx, row_status, scores, score_stride);
  return hipGetLastError();
}

}  // namespace tv
