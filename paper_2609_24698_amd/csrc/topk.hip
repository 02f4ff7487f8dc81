// CSA top-k: per (row, node), keep the topk candidates with the largest
// indexer score, ties to the lower logical index, and list them ascending.
//
// Candidates of node i are the committed entries (scores from the score
// kernel) and the entries closed on i's own root path (scored here from their
// scratch indexer keys): a node never sees an entry compressed on another
// branch (Sec. 3.1, Sec. 4.1).
//
// Selection is an exact radix select on order-preserving 32-bit keys: digits
// of at most 8 bits, starting below the bits that all keys share, counted in
// an LDS histogram kept in eight interleaved copies so that equal digits in
// one wavefront collide at most eight ways.  An ordered compaction then lists
// the keys above the threshold and the lowest-index keys equal to it.  When a
// node's candidates fit, the keys live in LDS; otherwise every pass re-reads
// the global scores.
//
// Each workgroup finally writes its node's key list (one latent-row pointer
// per key, in attention order) so that the attention kernel starts from a
// table instead of re-deriving it.
#include <algorithm>

#include "node_keys.h"
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kMaxScratch = 64;
constexpr int kLdsKeys = 16384 + 256;  // candidates held in LDS (65 KiB): rows up to L = 65536 plus a path
constexpr int kNT = 512;               // threads per workgroup
constexpr int kNW = kNT / 64;
constexpr int kCopies = 8;             // interleaved histogram copies
static_assert(kLdsKeys % 4 == 0, "LDS keys are staged as 16-byte groups");

__device__ __forceinline__ float dot8_bf16(uint4 a, uint4 b) {
  float s = bf2f_lo(a.x) * bf2f_lo(b.x);
  s = fmaf(bf2f_hi(a.x), bf2f_hi(b.x), s);
  s = fmaf(bf2f_lo(a.y), bf2f_lo(b.y), s);
  s = fmaf(bf2f_hi(a.y), bf2f_hi(b.y), s);
  s = fmaf(bf2f_lo(a.z), bf2f_lo(b.z), s);
  s = fmaf(bf2f_hi(a.z), bf2f_hi(b.z), s);
  s = fmaf(bf2f_lo(a.w), bf2f_lo(b.w), s);
  s = fmaf(bf2f_hi(a.w), bf2f_hi(b.w), s);
  return s;
}

template <bool kLds>
__global__ void __launch_bounds__(kNT) topk_kernel(tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u,
                                                   const uint64_t *__restrict__ anc,
                                                   const int32_t *__restrict__ depth,
                                                   const uint16_t *__restrict__ scr_c4,
                                                   const uint16_t *__restrict__ scr_c128,
                                                   const uint16_t *__restrict__ q_idx,
                                                   const uint16_t *__restrict__ w_idx,
                                                   const float *__restrict__ scores, int score_stride,
                                                   int32_t *__restrict__ sel, int32_t *__restrict__ row_status,
                                                   int32_t *__restrict__ row_order,
                                                   const uint16_t **__restrict__ keytab, int keytab_stride,
                                                   int32_t *__restrict__ nkeys_tab) {
  __shared__ __align__(16) uint32_t keys[kLds ? kLdsKeys : 4];
  __shared__ __align__(16) uint32_t hist[256 * kCopies];
  __shared__ float scr_score[kMaxScratch];
  __shared__ int32_t scr_node[kMaxScratch];
  __shared__ uint32_t mm[2][kNW];
  __shared__ int wcnt[2][kNW];
  __shared__ uint32_t found[3];
  __shared__ int32_t path[64], hca_node[64], cnt[2];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int b = blockIdx.x / d.D;
  const int i = blockIdx.x - b * d.D;
  if (i == 0) {
    // Rank of row b by (committed length descending, row ascending), for every
    // row whatever its status: row_order[rank] = b.  The attention kernel
    // starts the longest rows first.
    const int32_t Lb = c.len[b];
    int cnt = 0;
    for (int r = tid; r < d.B; r += kNT) {
      const int32_t Lr = c.len[r];
      cnt += (Lr > Lb || (Lr == Lb && r < b)) ? 1 : 0;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
    if (lane == 0) wcnt[1][wv] = cnt;
    __syncthreads();
    if (tid == 0) {
      int rank = 0;
      for (int w = 0; w < kNW; ++w) rank += wcnt[1][w];
      row_order[rank] = b;
    }
  }
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

  // Entries closed on the root path take the consecutive logical indices
  // n4, n4+1, ... in depth order.
  bool closes = false;
  if (tid < d.D && ((m >> tid) & 1ull)) {
    const int64_t p = (int64_t)L + depth[(int64_t)b * d.D + tid];
    if ((p + 1) % d.ratio_csa == 0) {
      closes = true;
      scr_node[(p + 1) / d.ratio_csa - 1 - n4] = tid;
    }
  }
  if (wv == 0) {
    const int cnt = __popcll(__ballot(closes));
    if (lane == 0) wcnt[0][0] = cnt;
  }
  __syncthreads();
  const int nscr = wcnt[0][0];
  // Scores of the path entries.  Wave w takes entries w, w + 8, ...; lane
  // (h8, c) holds channels 8c..8c+7 of head h0 + h8, for head groups h0.
  {
    const int hl = lane >> 3, cc = lane & 7;
    for (int t = wv; t < nscr; t += kNW) {
      const uint4 kv = *reinterpret_cast<const uint4 *>(scr_c4 + ((int64_t)b * d.D + scr_node[t]) * d_u + d.d_row +
                                                        8 * cc);
      float sum = 0.f;
      for (int h0 = 0; h0 < d.H_idx; h0 += 8) {
        const int h = h0 + hl;
        float part = 0.f, wh = 0.f;
        if (h < d.H_idx) {
          const uint4 qv = *reinterpret_cast<const uint4 *>(q_idx + (node * d.H_idx + h) * 64 + 8 * cc);
          part = dot8_bf16(qv, kv);
          wh = bf2f(w_idx[node * d.H_idx + h]);
        }
        part += __shfl_xor(part, 1, 64);
        part += __shfl_xor(part, 2, 64);
        part += __shfl_xor(part, 4, 64);
        float term = wh * fmaxf(part, 0.f);
        term += __shfl_xor(term, 8, 64);
        term += __shfl_xor(term, 16, 64);
        term += __shfl_xor(term, 32, 64);
        sum += term;
      }
      if (lane == 0) scr_score[t] = sum;
    }
  }
  __syncthreads();

  const int n = n4 + nscr;
  int32_t *out = sel + node * d.topk;
  const float *sc = scores + node * score_stride;
  if (n <= d.topk) {
    for (int t = tid; t < d.topk; t += kNT) out[t] = t < n ? t : -1;
  } else {
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
    if constexpr (kLds) {
      // Keys into LDS in 16-byte groups, with their extremes.  Score rows are
      // 256-byte aligned and padded to a multiple of 64 entries, so whole
      // float4 groups of the committed part can be read.
      const int n4v = (n4 + 3) >> 2;
      const float4 *sc4 = reinterpret_cast<const float4 *>(sc);
      uint4 *keys4 = reinterpret_cast<uint4 *>(keys);
      for (int j0 = 0; j0 < n4v; j0 += kNT * 8) {  // eight float4 loads in flight per thread
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + tid + kNT * u;
          v[u] = j < n4v ? sc4[j] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + tid + kNT * u;
          if (j < n4v) {
            const float f[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
            uint32_t k[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int s = 4 * j + e;
              k[e] = score_key(s < n4 ? f[e] : (s < n ? scr_score[s - n4] : 0.f));
              if (s < n) {
                kmin = min(kmin, k[e]);
                kmax = max(kmax, k[e]);
              }
            }
            keys4[j] = make_uint4(k[0], k[1], k[2], k[3]);
          }
        }
      }
      // path entries beyond the last group of committed ones
      const int s = 4 * n4v + tid;
      if (s < n) {
        const uint32_t k = score_key(scr_score[s - n4]);
        keys[s] = k;
        kmin = min(kmin, k);
        kmax = max(kmax, k);
      }
    } else {
      for (int s0 = 0; s0 < n; s0 += kNT * 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int s = s0 + tid + kNT * u;
          v[u] = s < n4 ? sc[s] : (s < n ? scr_score[s - n4] : 0.f);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (s0 + tid + kNT * u < n) {
            const uint32_t k = score_key(v[u]);
            kmin = min(kmin, k);
            kmax = max(kmax, k);
          }
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, 64));
      kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, 64));
    }
    if (lane == 0) {
      mm[0][wv] = kmin;
      mm[1][wv] = kmax;
    }
    __syncthreads();
    kmin = mm[0][0];
    kmax = mm[1][0];
#pragma unroll
    for (int w = 1; w < kNW; ++w) {
      kmin = min(kmin, mm[0][w]);
      kmax = max(kmax, mm[1][w]);
    }

    // Radix select of the topk-th largest key.  After it, keys whose masked
    // bits exceed `prefix` are taken, and of those equal to it the `remaining`
    // lowest-index ones.  A pass whose chosen bin holds exactly `remaining`
    // keys ends the search: all of them are taken.
    uint32_t prefix = kmin, pmask = 0xFFFFFFFFu;
    int remaining = d.topk;
    if (kmin != kmax) {
      const int hb = 31 - __clz(kmin ^ kmax);
      const uint32_t low = (hb == 31) ? 0xFFFFFFFFu : ((2u << hb) - 1u);
      pmask = ~low;
      prefix = kmin & pmask;
      const int slot = lane & (kCopies - 1);
      for (int top = hb; top >= 0;) {
        const int nb = top + 1 < 8 ? top + 1 : 8;
        const int sh = top + 1 - nb;
        const uint32_t dmask = (1u << nb) - 1u;
        for (int t = tid; t < 256 * kCopies / 4; t += kNT) reinterpret_cast<uint4 *>(hist)[t] = make_uint4(0, 0, 0, 0);
        __syncthreads();
        auto count = [&](uint32_t k, bool ok) {
          if (ok && (k & pmask) == prefix) atomicAdd(&hist[((k >> sh) & dmask) * kCopies + slot], 1u);
        };
        if constexpr (kLds) {
          const int nv = (n + 3) >> 2;
          const uint4 *keys4 = reinterpret_cast<const uint4 *>(keys);
          for (int j0 = 0; j0 < nv; j0 += kNT * 8) {
            uint4 kk[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) kk[u] = keys4[min(j0 + tid + kNT * u, nv - 1)];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const int s = 4 * (j0 + tid + kNT * u);
              count(kk[u].x, s + 0 < n);
              count(kk[u].y, s + 1 < n);
              count(kk[u].z, s + 2 < n);
              count(kk[u].w, s + 3 < n);
            }
          }
        } else {
          for (int s0 = 0; s0 < n; s0 += kNT * 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const int s = s0 + tid + kNT * u;
              v[u] = s < n4 ? sc[s] : (s < n ? scr_score[s - n4] : 0.f);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) count(score_key(v[u]), s0 + tid + kNT * u < n);
          }
        }
        __syncthreads();
        if (wv == 0) {  // lane owns bins 255-4l .. 252-4l, scanned from the top bin down
          const uint4 *h4 = reinterpret_cast<const uint4 *>(hist) + (252 - 4 * lane) * (kCopies / 4);
          int cntv[4], local = 0;
#pragma unroll
          for (int u = 0; u < 4; ++u) {  // bin 255 - 4l - u
            const uint4 a = h4[(3 - u) * 2], bq = h4[(3 - u) * 2 + 1];
            cntv[u] = (int)(a.x + a.y + a.z + a.w + bq.x + bq.y + bq.z + bq.w);
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
              found[2] = cntv[u];
            }
            above += cntv[u];
          }
        }
        __syncthreads();
        prefix |= found[0] << sh;
        pmask |= dmask << sh;
        remaining -= (int)found[1];
        if ((int)found[2] == remaining) break;
        top -= nb;
      }
    }

    // Ordered compaction: wave w owns a contiguous index range.  A counting
    // sweep gives every wave the numbers of greater and equal keys before its
    // range; a second sweep writes each taken index at (greater before it) +
    // min(equal before it, remaining).
    auto key_at = [&](int s) -> uint32_t {  // 0 <= s < n
      if constexpr (kLds) return keys[s];
      else return score_key(s < n4 ? sc[s] : scr_score[s - n4]);
    };
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int seg = (n + kNT - 1) / kNT * 64;
    const int lo = wv * seg, hi = std::min(n, lo + seg);
    int cgt = 0, ceq = 0;
    for (int s0 = lo; s0 < hi; s0 += 256) {
      uint32_t kk[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) kk[u] = key_at(min(s0 + 64 * u + lane, n - 1));
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool ok = s0 + 64 * u + lane < hi;
        const uint32_t km = kk[u] & pmask;
        cgt += __popcll(__ballot(ok && km > prefix));
        ceq += __popcll(__ballot(ok && km == prefix));
      }
    }
    if (lane == 0) {
      wcnt[0][wv] = cgt;
      wcnt[1][wv] = ceq;
    }
    __syncthreads();
    int gt_before = 0, eq_before = 0;
    for (int w = 0; w < wv; ++w) {
      gt_before += wcnt[0][w];
      eq_before += wcnt[1][w];
    }
    for (int s0 = lo; s0 < hi; s0 += 256) {
      uint32_t kk[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) kk[u] = key_at(min(s0 + 64 * u + lane, n - 1));
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int s = s0 + 64 * u + lane;
        const bool ok = s < hi;
        const uint32_t km = kk[u] & pmask;
        const bool gt = ok && km > prefix, eq = ok && km == prefix;
        const uint64_t bgt = __ballot(gt), beq = __ballot(eq);
        const int g = gt_before + __popcll(bgt & lt_mask);
        const int e = eq_before + __popcll(beq & lt_mask);
        if (gt) out[g + std::min(e, remaining)] = s;
        else if (eq && e < remaining) out[g + e] = s;
        gt_before += __popcll(bgt);
        eq_before += __popcll(beq);
      }
    }
  }

  // The node's key list for the attention kernel: latent-row pointers of its
  // selected CSA entries, HCA entries, window rows and path rows, in the
  // order the attention enumerates them.  The selection list written above is
  // read back by this workgroup after the barrier.
  __syncthreads();
  const NodeKeys nk = node_keys(d, L, b, i, anc, depth, path, hca_node, cnt);
  {
    const uint16_t **tab = keytab + node * keytab_stride;
    const int64_t c4b = c.c4_base[b], c128b = c.c128_base[b];
    for (int t = tid; t < nk.n_keys; t += kNT)
      tab[t] = key_row(d, nk, b, t, out, path, hca_node, c.ring, c.c4, c4b, c.c128, c128b, scr_c4, scr_c128, tree_u);
    if (tid == 0) nkeys_tab[node] = nk.n_keys;
  }
}

hipError_t launch_topk(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                       const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128, const uint16_t *q_idx,
                       const uint16_t *w_idx, const float *scores, int32_t score_stride, int32_t *sel,
                       int32_t *row_status, int32_t *row_order, const uint16_t **keytab, int32_t keytab_stride,
                       int32_t *nkeys, hipStream_t s) {
  if (d.D > kMaxScratch) return hipErrorInvalidValue;
  // the LDS variant serves every node when the longest candidate list fits
  const int64_t max_n = (int64_t)d.max_len / d.ratio_csa + d.D;
  if (max_n <= kLdsKeys)
    topk_kernel<true><<<d.B * d.D, kNT, 0, s>>>(d, c, tree_u, anc, depth, scr_c4, scr_c128, q_idx, w_idx, scores,
                                                score_stride, sel, row_status, row_order, keytab, keytab_stride,
                                                nkeys);
  else
    topk_kernel<false><<<d.B * d.D, kNT, 0, s>>>(d, c, tree_u, anc, depth, scr_c4, scr_c128, q_idx, w_idx, scores,
                                                 score_stride, sel, row_status, row_order, keytab, keytab_stride,
                                                 nkeys);
  return hipGetLastError();
}

}  // namespace tv
