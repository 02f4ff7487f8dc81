// CSA top-k: per (row, node), keep the topk candidates with the largest
// indexer score, ties to the lower logical index, and list them ascending.
//
// Candidates of node i are the committed entries (scores from the score
// kernel) and the entries closed on i's own root path (scored here from their
// scratch indexer keys): a node never sees an entry compressed on another
// branch (Sec. 3.1, Sec. 4.1).
//
// Selection is an exact radix select on order-preserving 32-bit keys
// (11 + 11 + 10 bit digits, histograms in LDS), then an ordered compaction:
// every key above the threshold plus the lowest-index keys equal to it.
#include <algorithm>

#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kMaxScratch = 64;

__device__ int block_excl_scan_i(int v, int *tmp, int *total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) tmp[wv] = x;
  __syncthreads();
  int base = 0, tot = 0;
  for (int k = 0; k < 4; ++k) {
    if (k < wv) base += tmp[k];
    tot += tmp[k];
  }
  __syncthreads();
  *total = tot;
  return base + x - v;
}

__global__ void __launch_bounds__(256) topk_kernel(tv_dims d, CacheView c, const uint64_t *__restrict__ anc,
                                                   const int32_t *__restrict__ depth,
                                                   const uint16_t *__restrict__ scr_c4,
                                                   const uint16_t *__restrict__ q_idx,
                                                   const uint16_t *__restrict__ w_idx,
                                                   const float *__restrict__ scores, int score_stride,
                                                   int32_t *__restrict__ sel, int32_t *__restrict__ row_status) {
  __shared__ uint32_t hist[2048];
  __shared__ float scr_score[kMaxScratch];
  __shared__ int32_t scr_node[kMaxScratch];
  __shared__ int scan_tmp[4];
  __shared__ uint32_t found[2];  // digit, count of keys above the digit's bin
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int b = blockIdx.x / d.D;
  const int i = blockIdx.x - b * d.D;
  if (row_status[b] != TV_ROW_OK) return;
  const int32_t L = c.len[b];
  if (!len_ok(L, d.max_len)) {
    if (i == 0 && tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return;
  }
  const int64_t node = (int64_t)b * d.D + i;
  const int n4 = L / d.ratio_csa;
  const uint64_t m = anc[node];
  const int d_u = d.d_row + d.d_idx;

  // Entries closed on the root path, in logical-index order (= depth order).
  if (tid < d.D) scr_node[tid] = -1;
  __syncthreads();
  if (tid < d.D && ((m >> tid) & 1ull)) {
    const int64_t p = (int64_t)L + depth[(int64_t)b * d.D + tid];
    if ((p + 1) % d.ratio_csa == 0) scr_node[(p + 1) / d.ratio_csa - 1 - n4] = tid;
  }
  __syncthreads();
  int nscr = 0;
  while (nscr < d.D && scr_node[nscr] >= 0) ++nscr;
  if (wv == 0) {
    for (int t = 0; t < nscr; ++t) {
      const uint16_t *key = scr_c4 + ((int64_t)b * d.D + scr_node[t]) * d_u + d.d_row;
      float s = 0.f;
      for (int h = 0; h < d.H_idx; ++h) {
        const uint16_t *qh = q_idx + (node * d.H_idx + h) * 64;
        const float dot = wave_sum(bf2f(qh[lane]) * bf2f(key[lane]));
        s += bf2f(w_idx[node * d.H_idx + h]) * fmaxf(dot, 0.f);
      }
      if (lane == 0) scr_score[t] = s;
    }
  }
  __syncthreads();

  const int n = n4 + nscr;
  int32_t *out = sel + node * d.topk;
  const float *sc = scores + node * score_stride;
  if (n <= d.topk) {
    for (int t = tid; t < d.topk; t += 256) out[t] = t < n ? t : -1;
    return;
  }
  auto key_of = [&](int s) -> uint32_t { return score_key(s < n4 ? sc[s] : scr_score[s - n4]); };

  // radix select of the k-th largest key
  uint32_t prefix = 0, pmask = 0;
  int remaining = d.topk;
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass], nb = 1 << widths[pass];
    for (int t = tid; t < 2048; t += 256) hist[t] = 0;
    __syncthreads();
    for (int s = tid; s < n; s += 256) {
      const uint32_t k = key_of(s);
      if ((k & pmask) == prefix) atomicAdd(&hist[(k >> sh) & (nb - 1)], 1u);
    }
    __syncthreads();
    // thread t owns bins [nb - 8(t+1), nb - 8t), scanned from the top bin down
    const int per = nb / 256;
    const int hi = nb - per * tid;
    int local = 0;
    for (int q = 1; q <= per; ++q) local += hist[hi - q];
    int total;
    int above = block_excl_scan_i(local, scan_tmp, &total);
    for (int q = 1; q <= per; ++q) {
      const int bin = hi - q;
      const int h = hist[bin];
      if (above < remaining && remaining <= above + h) {
        found[0] = bin;
        found[1] = above;
      }
      above += h;
    }
    __syncthreads();
    const uint32_t digit = found[0];
    remaining -= (int)found[1];
    prefix |= digit << sh;
    pmask |= uint32_t(nb - 1) << sh;
    __syncthreads();
  }
  const uint32_t T = prefix;  // the k-th largest key; take `remaining` keys equal to it

  // ordered compaction over contiguous per-thread segments
  const int seg = (n + 255) / 256;
  const int s0 = std::min(n, tid * seg), s1 = std::min(n, s0 + seg);
  int eq = 0;
  for (int s = s0; s < s1; ++s) eq += key_of(s) == T;
  int tot;
  int eq_before = block_excl_scan_i(eq, scan_tmp, &tot);
  int take = 0;
  {
    int e = eq_before;
    for (int s = s0; s < s1; ++s) {
      const uint32_t k = key_of(s);
      if (k > T) ++take;
      else if (k == T && e++ < remaining) ++take;
    }
  }
  int pos = block_excl_scan_i(take, scan_tmp, &tot);
  {
    int e = eq_before;
    for (int s = s0; s < s1; ++s) {
      const uint32_t k = key_of(s);
      bool f = k > T;
      if (!f && k == T) f = e++ < remaining;
      if (f) out[pos++] = s;
    }
  }
}

hipError_t launch_topk(const tv_dims &d, const CacheView &c, const uint64_t *anc, const int32_t *depth,
                       const uint16_t *scr_c4, const uint16_t *q_idx, const uint16_t *w_idx, const float *scores,
                       int32_t score_stride, int32_t *sel, int32_t *row_status, hipStream_t s) {
  topk_kernel<<<d.B * d.D, 256, 0, s>>>(d, c, anc, depth, scr_c4, q_idx, w_idx, scores, score_stride, sel,
                                        row_status);
  return hipGetLastError();
}

}  // namespace tv
