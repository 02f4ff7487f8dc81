// CSA top-k: per (row, node), keep the topk candidates with the largest
// indexer score, ties to the lower logical index, and list them ascending.
//
// Candidates of node i are the committed entries (scores from the score
// kernel) and the entries closed on i's own root path (scored here from their
// scratch indexer keys): a node never sees an entry compressed on another
// branch (Sec. 3.1, Sec. 4.1).
//
// Selection is an exact radix select on order-preserving 32-bit keys (four
// 8-bit digits, one LDS histogram per wavefront), followed by an ordered
// compaction in index order: wavefront ballots rank the keys above the
// threshold and the lowest-index keys equal to it.  Keys live in LDS when the
// candidate list fits, otherwise they are re-derived from the global scores
// on every pass.
#include <algorithm>

#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kMaxScratch = 64;
constexpr int kLdsKeys = 16384 + 256;  // candidates held in LDS (65 KiB): rows up to L = 65536 plus a path

__global__ void __launch_bounds__(256) topk_kernel(tv_dims d, CacheView c, const uint64_t *__restrict__ anc,
                                                   const int32_t *__restrict__ depth,
                                                   const uint16_t *__restrict__ scr_c4,
                                                   const uint16_t *__restrict__ q_idx,
                                                   const uint16_t *__restrict__ w_idx,
                                                   const float *__restrict__ scores, int score_stride,
                                                   int32_t *__restrict__ sel, int32_t *__restrict__ row_status) {
  __shared__ uint32_t keys[kLdsKeys];
  __shared__ uint32_t hist[4][256];
  __shared__ float scr_score[kMaxScratch];
  __shared__ int32_t scr_node[kMaxScratch];
  __shared__ int wcnt[2][16];
  __shared__ float hterm[16][64];
  __shared__ uint32_t found[2];
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
  // scores of the path entries: wave w takes heads w, w+4, ..; lane = key channel;
  // every operand is loaded before the first reduction
  for (int t0 = 0; t0 < nscr; t0 += 16) {
    const int nt = std::min(16, nscr - t0);
    float kv[16];
#pragma unroll
    for (int t = 0; t < 16; ++t)
      kv[t] = t < nt ? bf2f(scr_c4[((int64_t)b * d.D + scr_node[t0 + t]) * d_u + d.d_row + lane]) : 0.f;
    for (int h = wv; h < d.H_idx; h += 4) {
      const float qv = bf2f(q_idx[(node * d.H_idx + h) * 64 + lane]);
      const float wh = bf2f(w_idx[node * d.H_idx + h]);
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        if (t < nt) {
          const float dot = wave_sum(qv * kv[t]);
          if (lane == 0) hterm[t][h] = wh * fmaxf(dot, 0.f);
        }
      }
    }
    __syncthreads();
    if (tid < nt) {
      float sum = 0.f;
      for (int h = 0; h < d.H_idx; ++h) sum += hterm[tid][h];  // head order
      scr_score[t0 + tid] = sum;
    }
    __syncthreads();
  }

  const int n = n4 + nscr;
  int32_t *out = sel + node * d.topk;
  const float *sc = scores + node * score_stride;
  if (n <= d.topk) {
    for (int t = tid; t < d.topk; t += 256) out[t] = t < n ? t : -1;
    return;
  }
  const bool in_lds = n <= kLdsKeys;
  if (in_lds) {  // sixteen loads in flight per thread
    for (int s0 = 0; s0 < n; s0 += 256 * 16) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int s = s0 + tid + 256 * u;
        v[u] = s < n4 ? sc[s] : (s < n ? scr_score[s - n4] : 0.f);
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int s = s0 + tid + 256 * u;
        if (s < n) keys[s] = score_key(v[u]);
      }
    }
  }
  __syncthreads();
  auto key_of = [&](int s) -> uint32_t {
    return in_lds ? keys[s] : score_key(s < n4 ? sc[s] : scr_score[s - n4]);
  };

  // radix select of the k-th largest key, 8 bits per pass
  uint32_t prefix = 0, pmask = 0;
  int remaining = d.topk;
  for (int pass = 0; pass < 4; ++pass) {
    const int sh = 24 - 8 * pass;
    for (int t = tid; t < 1024; t += 256) (&hist[0][0])[t] = 0;
    __syncthreads();
    for (int s0 = 0; s0 < n; s0 += 256 * 16) {  // sixteen key reads in flight
      uint32_t kk[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int s = s0 + tid + 256 * u;
        kk[u] = s < n ? key_of(s) : 0u;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int s = s0 + tid + 256 * u;
        if (s < n && (kk[u] & pmask) == prefix) atomicAdd(&hist[wv][(kk[u] >> sh) & 255], 1u);
      }
    }
    __syncthreads();
    if (wv == 0) {  // lane owns bins 255-4l .. 252-4l, scanned from the top bin down
      int cntv[4], local = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int bin = 255 - 4 * lane - u;
        cntv[u] = (int)(hist[0][bin] + hist[1][bin] + hist[2][bin] + hist[3][bin]);
        local += cntv[u];
      }
      int incl = local;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      int above = incl - local;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (above < remaining && remaining <= above + cntv[u]) {
          found[0] = 255 - 4 * lane - u;
          found[1] = above;
        }
        above += cntv[u];
      }
    }
    __syncthreads();
    const uint32_t digit = found[0];
    remaining -= (int)found[1];
    prefix |= digit << sh;
    pmask |= 255u << sh;
    __syncthreads();
  }
  const uint32_t T = prefix;  // the k-th largest key; take `remaining` keys equal to it

  // Ordered compaction in chunks of 1024 consecutive indices (element
  // base + 256 u + tid for u = 0..3): wave ballots give in-wave ranks, the
  // per-(u, wave) counts in LDS give every element's offset.
  int out_before = 0, eq_before = 0;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int base = 0; base < n; base += 1024) {
    bool gt[4], eq[4];
    uint64_t beq[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int s = base + 256 * u + tid;
      const uint32_t k = s < n ? key_of(s) : 0u;
      gt[u] = s < n && k > T;
      eq[u] = s < n && k == T;
      beq[u] = __ballot(eq[u]);
      if (lane == 0) wcnt[0][4 * u + wv] = __popcll(beq[u]);
    }
    __syncthreads();
    // exclusive scan of the 16 (u, wave) counts, redundantly in every wave
    auto scan16 = [&](const int *cnt, int &excl, int &tot) {
      const int v = lane < 16 ? cnt[lane] : 0;
      int inc = v;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const int y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
      }
      excl = inc - v;
      tot = __shfl(inc, 15, 64);
    };
    int eq_excl, eq_tot;
    scan16(wcnt[0], eq_excl, eq_tot);
    bool take[4];
    uint64_t bt[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int off = eq_before + __shfl(eq_excl, 4 * u + wv, 64);
      take[u] = gt[u] || (eq[u] && off + __popcll(beq[u] & lt_mask) < remaining);
      bt[u] = __ballot(take[u]);
      if (lane == 0) wcnt[1][4 * u + wv] = __popcll(bt[u]);
    }
    __syncthreads();
    int o_excl, o_tot;
    scan16(wcnt[1], o_excl, o_tot);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int off = out_before + __shfl(o_excl, 4 * u + wv, 64);
      if (take[u]) out[off + __popcll(bt[u] & lt_mask)] = base + 256 * u + tid;
    }
    out_before += o_tot;
    eq_before += eq_tot;
    __syncthreads();
    if (out_before >= d.topk) break;
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
