// CSA top-k: per (row, node), keep the topk candidates with the largest
// indexer score, ties to the lower logical index, and list them ascending.
//
// Candidates of node i are the committed entries (scores from the score
// kernel) and the entries closed on i's own root path (scored here from their
// scratch indexer keys): a node never sees an entry compressed on another
// branch (Sec. 3.1, Sec. 4.1).
//
// Selection is an exact radix select on order-preserving 32-bit keys held in
// registers (element e of an NT-thread workgroup in slot e / NT of thread
// e % NT; NT is 512 for a segment and 1024 for a merge):
// 13-bit digits counted in an LDS histogram, each pass restricted to the keys
// that share the digits found so far, until the bin holding the topk-th key
// holds exactly the keys still needed or every bit is fixed.  An ordered
// compaction then lists the keys above the threshold and the lowest-index
// keys equal to it, from the registers.
//
// A node with up to kTopkSeg committed entries is selected by one workgroup.
// A longer node is cut into segments of kTopkSeg entries: each segment's
// workgroup keeps its own topk (a superset of its share of the node's topk),
// and a merge kernel selects the node's topk among the survivors of all its
// segments, which are already in index order.
//
// The selecting workgroup also writes its node's key list (one latent-row
// pointer per key, in attention order) so that the attention kernel starts
// from a table instead of re-deriving it; the table and a copy of the key
// count are kept by (row rank, node), the attention's own order.
#include <algorithm>

#include "compress_body.h"
#include "node_keys.h"
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kMaxScratch = 64;
constexpr int kTkNT = 512;  // threads of a selecting workgroup
constexpr int kMergeNT = 1024;  // threads of a merging workgroup (one per node: the more, the fewer keys each)
constexpr int kTkNW = kTkNT / 64;
constexpr int kTkKPT = 34;  // keys per thread of a segment: kTopkSeg committed entries plus up to 64 path entries
constexpr int kTkBits = 13, kTkBins = 1 << kTkBits;
static_assert(kTkNT * kTkKPT >= kTopkSeg + kMaxScratch, "segment plus path entries fit the registers");
static_assert(kTkNT * kTopkMergeKPT == kTopkMergeCap, "merge capacity");

struct __align__(16) SelShared {
  uint32_t hist[kTkBins];
  int wsum[16];  // one per wavefront of the largest workgroup (1024 threads)
  int found[3];
  uint32_t bits[2][16 * kTopkMergeKPT];  // compaction bitmaps in element order: keys above the threshold, equal to it
};

// Barrier for shared-memory hand-offs only: global loads in flight stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

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

// Threshold of the k largest of the keys the workgroup holds (key[j] is
// element tid + NT j; elements from n on, and any other padding, hold key 0,
// below every real key, and are never counted or taken; n_real keys are
// real, all of them below element n, and k < n_real).  On return
// every thread has prefix, pmask and remaining such that the k largest are the
// keys with (key & pmask) > prefix and the `remaining` lowest elements with
// (key & pmask) == prefix.
template <int KPT, int NT = kTkNT>
__device__ __forceinline__ void radix_threshold(const uint32_t (&key)[KPT], int n, int n_real, int k,
                                                SelShared &sh, uint32_t &prefix, uint32_t &pmask,
                                                int &remaining) {
  static_assert(NT % 64 == 0 && NT / 64 <= 16 && 16 * NT >= kTkBins, "wave sums and the scan's bins fit");
  const int nr = (n + NT - 1) / NT;  // slots that hold any element below n
  // Padding keys (0) match the prefix only while it is 0, and then all fall
  // into bin 0: that bin starts at minus their count instead of each key
  // being tested (a test the compiler would keep as one mask per slot).
  const uint32_t n_pad = (uint32_t)(nr * NT - n_real);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  prefix = 0;
  pmask = 0;
  remaining = k;
  // 13, 13 and 6 bits: every pass has at least the 16 bins per thread the scan reads
  static_assert(32 % kTkBits >= 4, "no pass narrower than four bits");
  for (int shift = 32; shift > 0;) {
    const int nb = shift < kTkBits ? shift : kTkBits;
    const int sft = shift - nb;
    const int nbins = 1 << nb;
    const uint32_t dmask = (uint32_t)nbins - 1u;
    for (int t = tid; t < nbins / 4; t += NT)
      reinterpret_cast<uint4 *>(sh.hist)[t] = make_uint4(t == 0 && prefix == 0u ? 0u - n_pad : 0u, 0u, 0u, 0u);
    lds_barrier();
    // The slot bound, laundered through a scalar move each pass: a bound known
    // across passes becomes one lane mask per slot, kept for every pass.
    int nr_p;
    asm volatile("s_mov_b32 %0, %1" : "=s"(nr_p) : "s"(nr));
#pragma unroll
    for (int j = 0; j < KPT; ++j)
      if (j < nr_p && (key[j] & pmask) == prefix) atomicAdd(&sh.hist[(key[j] >> sft) & dmask], 1u);
    lds_barrier();
    // Thread t owns the 16 bins from nbins - 16 (t + 1) up (threads 0.. hold
    // the top bins), read as four 16-byte groups; counts scan from the top.
    const int hb = nbins - 16 * (tid + 1);
    uint32_t h[16];
    if (hb >= 0) {
      const uint4 *g4 = reinterpret_cast<const uint4 *>(sh.hist + hb);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 x = g4[u];
        h[4 * u] = x.x;
        h[4 * u + 1] = x.y;
        h[4 * u + 2] = x.z;
        h[4 * u + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 16; ++u) h[u] = 0u;
    }
    int local = 0;
#pragma unroll
    for (int u = 0; u < 16; ++u) local += (int)h[u];
    const int incl = (int)wave_prefix_sum((uint32_t)local);
    if (lane == 63) sh.wsum[wv] = incl;
    lds_barrier();
    int above = incl - local;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) above += w < wv ? sh.wsum[w] : 0;
    if (above < remaining && remaining <= above + local) {
#pragma unroll
      for (int u = 15; u >= 0; --u) {
        const int c = (int)h[u];
        if (above < remaining && remaining <= above + c) {
          sh.found[0] = hb + u;
          sh.found[1] = above;
          sh.found[2] = c;
        }
        above += c;
      }
    }
    lds_barrier();
    prefix |= (uint32_t)sh.found[0] << sft;
    pmask |= dmask << sft;
    remaining -= sh.found[1];
    const int c = sh.found[2];
    shift = sft;
    if (c == remaining) break;  // every key of the bin is taken
  }
}

// Ordered compaction of the keys the threshold takes: the element index of
// the pos-th taken key (in element order) goes to list[pos], pos < k.  The
// list aliases the histogram, which the threshold search no longer needs.
// Each wave's ballots of a slot are two words of a bitmap in element order
// (keys above the threshold, keys equal to it); one scan over the words gives
// every word the number of taken elements before it (all the keys above,
// the first `remaining` equal ones), and each thread writes the taken
// elements of its words.
template <int KPT, int NT = kTkNT>
__device__ __forceinline__ void compact_taken(const uint32_t (&key)[KPT], int n, uint32_t prefix, uint32_t pmask,
                                              int remaining, SelShared &sh) {
  constexpr int W = NT / 32;  // bitmap words per register slot
  static_assert(W * KPT <= 16 * kTopkMergeKPT, "the bitmaps fit");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int nr = (n + NT - 1) / NT;
  uint32_t *bg = sh.bits[0], *be = sh.bits[1];
  // word W j + 2 wv + h holds the elements NT j + 64 wv + 32 h + bit
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    if (j < nr) {
      const uint32_t km = key[j] & pmask;
      const uint64_t g = __ballot(km > prefix);
      const uint64_t q = __ballot(km == prefix && key[j] != 0u);
      if (lane == 0) {
        *reinterpret_cast<uint2 *>(&bg[W * j + 2 * wv]) = make_uint2((uint32_t)g, (uint32_t)(g >> 32));
        *reinterpret_cast<uint2 *>(&be[W * j + 2 * wv]) = make_uint2((uint32_t)q, (uint32_t)(q >> 32));
      }
    }
  }
  lds_barrier();
  // thread t takes the words t * per .. t * per + per - 1
  const int nw = W * nr;
  constexpr int kPerMax = (W * KPT + NT - 1) / NT;
  const int per = (nw + NT - 1) / NT;
  uint32_t wg[kPerMax], wq[kPerMax];
  uint32_t cnt = 0u;  // above-threshold count | equal count << 16 (each total below 2^16)
#pragma unroll
  for (int u = 0; u < kPerMax; ++u) {
    const int w = tid * per + u;
    const bool ok = u < per && w < nw;
    wg[u] = ok ? bg[w] : 0u;
    wq[u] = ok ? be[w] : 0u;
    cnt += (uint32_t)__popc(wg[u]) | ((uint32_t)__popc(wq[u]) << 16);
  }
  const uint32_t incl = wave_prefix_sum(cnt);
  if (lane == 63) sh.wsum[wv] = (int)incl;
  lds_barrier();
  uint32_t before = incl - cnt;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) before += w < wv ? (uint32_t)sh.wsum[w] : 0u;
  int gb = (int)(before & 0xFFFFu), qb = (int)(before >> 16);  // keys above / equal to the threshold before this thread's words
  int32_t *list = reinterpret_cast<int32_t *>(sh.hist);
#pragma unroll
  for (int u = 0; u < kPerMax; ++u) {
    const int w = tid * per + u;
    if (u < per && w < nw) {
      const int nq = __popc(wq[u]);
      const int r = std::min(std::max(remaining - qb, 0), nq);  // equal keys of this word that are taken
      uint32_t eqt = 0u;
      if (r == nq) {
        eqt = wq[u];
      } else if (r > 0) {
        uint32_t y = wq[u];
        for (int c = 0; c < r; ++c) y &= y - 1u;  // drop the lowest r
        eqt = wq[u] ^ y;
      }
      uint32_t t = wg[u] | eqt;
      int pos = gb + std::min(qb, remaining);
      while (t) {
        list[pos++] = 32 * w + (__ffs(t) - 1);
        t &= t - 1u;
      }
      gb += __popc(wg[u]);
      qb += nq;
    }
  }
  lds_barrier();
}

// Latent row of CSA entry s of node (b, i): committed entries from the pool,
// path entries from the scratch slot of the path node that closed them.
__device__ __forceinline__ const uint16_t *csa_row(const tv_dims &d, const NodeKeys &nk, int b, int s,
                                                   const int32_t *path, const uint16_t *c4, int64_t c4b,
                                                   const int32_t *page_table,
                                                   const uint16_t *scr_c4) {
  if (s < nk.n4) return c4 + committed_slot(d, page_table, c4b, b, s, d.ratio_csa) * d.d_row;
  int64_t dd = (int64_t)(s + 1) * d.ratio_csa - 1 - nk.L;
  if (dd < 0 || dd > nk.p - nk.L) dd = 0;  // defensive: stay on the node's own path
  return scr_c4 + ((int64_t)b * d.D + path[dd]) * (d.d_row + d.d_idx);
}

// Key of a real candidate: the order-preserving key, at least 1, so that the
// padding key 0 sorts below every candidate (only the two all-ones negative
// NaN patterns share key 1).
__device__ __forceinline__ uint32_t live_key(float s) { return max(score_key(s), 1u); }

__device__ __forceinline__ int topk_segments(int n4) { return n4 <= kTopkSeg ? 1 : (n4 + kTopkSeg - 1) / kTopkSeg; }

// One workgroup per (node, segment).  Segment 0 of node 0 of a row also ranks
// the row by length for the attention's row order, and segment 0 of every
// node writes the node's non-CSA keys into its key table.
struct TopkSmem {
  SelShared sh;
  float scr_score[kMaxScratch];
  int wcnt[kTkNW];
  int32_t path[64], hca_nd[64];
};

__device__ __forceinline__ void topk_node(const tv_dims &d, const CacheView &c, const uint16_t *__restrict__ tree_u,
                                          const uint64_t *__restrict__ anc, const int32_t *__restrict__ depth,
                                          const uint16_t *__restrict__ scr_c4, const uint16_t *__restrict__ scr_c128,
                                          const uint16_t *__restrict__ q_idx, const uint16_t *__restrict__ w_idx,
                                          const float *__restrict__ scores, int score_stride,
                                          int32_t *__restrict__ sel, int32_t *__restrict__ row_status,
                                          int32_t *__restrict__ row_order, int32_t *__restrict__ row_rank,
                                          const uint16_t **__restrict__ keytab, int keytab_stride,
                                          int32_t *__restrict__ nkeys_tab, int32_t *__restrict__ nkeys_rank,
                                          int max_seg, int32_t *__restrict__ surv_idx,
                                          uint32_t *__restrict__ surv_key, int32_t *__restrict__ surv_cnt, int blk,
                                          TopkSmem &sm) {
  SelShared &sh = sm.sh;
  float *scr_score = sm.scr_score;
  int *wcnt = sm.wcnt;
  int32_t *path = sm.path, *hca_nd = sm.hca_nd;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t node = blk / max_seg;
  const int seg = blk - (int)node * max_seg;
  const int b = (int)(node / d.D);
  const int i = (int)(node - (int64_t)b * d.D);
  // one round trip: everything whose address is known from (row, node, lane)
  const int32_t status = row_status[b];
  const int32_t L = c.len[b];
  const uint64_t m = anc[node];
  const bool flat = d.page_size == 0;
  const int64_t c4b = flat ? c.c4_base[b] : 0, c128b = flat ? c.c128_base[b] : 0;
  const int dl = lane < d.D ? depth[(int64_t)b * d.D + lane] : 0;  // depth of the row's node `lane`
  const int hl = lane >> 3, cc = lane & 7;  // path-entry scoring: head h0 + hl, channels 8cc..8cc+7
  uint4 qv0 = make_uint4(0, 0, 0, 0);
  float wh0 = 0.f;
  if (hl < d.H_idx) {
    qv0 = *reinterpret_cast<const uint4 *>(q_idx + (node * d.H_idx + hl) * 64 + 8 * cc);
    wh0 = bf2f(w_idx[node * d.H_idx + hl]);
  }
  // Rank of row b by (committed length descending, row ascending), for every
  // row whatever its status: row_order[rank] = b, row_rank[b] = rank.  The
  // key table and a copy of the key count are kept by (rank, node), so the
  // attention reads them from its workgroup index without the row first.
  // Each wave's count goes to LDS now; the rank is summed after the next
  // barrier the workgroup passes anyway.
  int nb = 0;
  for (int r = tid; r < d.B; r += kTkNT) {
    const int32_t Lr = c.len[r];
    nb += (Lr > L || (Lr == L && r < b)) ? 1 : 0;
  }
  nb = (int)wave_total((uint32_t)nb);
  if (lane == 0) wcnt[wv] = nb;
  auto rank_of_row = [&]() {  // after a barrier
    int rk = 0;
#pragma unroll
    for (int w = 0; w < kTkNW; ++w) rk += wcnt[w];
    if (i == 0 && seg == 0 && tid == 0) {
      row_order[rk] = b;
      row_rank[b] = rk;
    }
    return rk;
  };
  const bool bad_len = !len_ok(L, d.max_len);
  if (status != TV_ROW_OK || bad_len) {  // the attention skips the node
    __syncthreads();
    const int rk = rank_of_row();
    if (seg == 0 && tid == 0) nkeys_rank[(int64_t)rk * d.D + i] = 0;
    if (status == TV_ROW_OK && i == 0 && seg == 0 && tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return;
  }
  const int n4 = L / d.ratio_csa;
  const int nseg = topk_segments(n4);
  if (seg >= nseg) return;
  const bool last = seg == nseg - 1;
  const int c0 = seg * kTopkSeg;
  const int cn = std::min(n4, c0 + kTopkSeg) - c0;  // committed candidates of this segment
  const float *sc = scores + node * score_stride + c0;
  // committed scores in flight while the path entries are scored (loads of
  // slots past the segment re-read its last entry, or entry 0 of the row)
  uint32_t key[kTkKPT];  // score bits first, converted to keys below
#pragma unroll
  for (int j = 0; j < kTkKPT; ++j)
    key[j] = __float_as_uint(sc[std::max(std::min(tid + kTkNT * j, cn - 1), 0)]);
  const int d_u = d.d_row + d.d_idx;

  // The node's root path (its key layout) from the ancestor mask, no barrier.
  uint64_t csa_mask;
  const NodeKeys nk = path_keys(d, L, i, m, dl, path, hca_nd, csa_mask);

  // Entries closed on the root path take the consecutive logical indices
  // n4, n4+1, ... in depth (= node index) order; the last segment scores them.
  const int nscr = last ? __popcll(csa_mask) : 0;
  if (last) {
    // Wave w takes entries w, w + 8, ...; lane (h8, c) holds channels
    // 8c..8c+7 of head h0 + h8, for head groups h0.
    for (int t = wv; t < nscr; t += kTkNW) {
      uint64_t x = csa_mask;
      for (int u = 0; u < t; ++u) x &= x - 1;
      const int nd = __ffsll((unsigned long long)x) - 1;  // the t-th path node closing a CSA block
      const uint4 kv = *reinterpret_cast<const uint4 *>(scr_c4 + ((int64_t)b * d.D + nd) * d_u + d.d_row + 8 * cc);
      float sum = 0.f;
      for (int h0 = 0; h0 < d.H_idx; h0 += 8) {
        const int h = h0 + hl;
        float part = 0.f, wh = 0.f;
        if (h < d.H_idx) {
          const uint4 qv =
              h0 == 0 ? qv0 : *reinterpret_cast<const uint4 *>(q_idx + (node * d.H_idx + h) * 64 + 8 * cc);
          part = dot8_bf16(qv, kv);
          wh = h0 == 0 ? wh0 : bf2f(w_idx[node * d.H_idx + h]);
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
  lds_barrier();  // path, hca_nd, the path-entry scores and the wave counts of the rank are visible
  const int64_t rnode = (int64_t)rank_of_row() * d.D + i;
  const int seg_n = cn + nscr;  // path entries follow the committed ones of the last segment
#pragma unroll
  for (int j = 0; j < kTkKPT; ++j) {
    const int e = tid + kTkNT * j;
    const float sv =
        e < cn ? __uint_as_float(key[j]) : scr_score[std::min(std::max(e - cn, 0), kMaxScratch - 1)];
    key[j] = e < seg_n ? live_key(sv) : 0u;
  }

  // The node's key table: non-CSA keys here, selected CSA entries below.
  const uint16_t **tab = keytab + rnode * keytab_stride;
  if (seg == 0) {
    for (int t = nk.nsel + tid; t < nk.n_keys; t += kTkNT)
      tab[t] = key_row(d, nk, b, t, nullptr, path, hca_nd, c.ring, c.c4, c4b, c.c128, c128b, scr_c4, scr_c128,
                       tree_u, c.page_table);
    if (tid == 0) {
      nkeys_tab[node] = nk.n_keys;
      nkeys_rank[rnode] = nk.n_keys;
    }
  }

  // Select: the taken elements in element order, list[t] (t < taken) in LDS,
  // or every element when the segment holds at most k.
  const int k = d.topk;
  const bool all = seg_n <= k;
  const int taken = all ? seg_n : k;
  if (!all) {
    uint32_t prefix, pmask;
    int remaining;
    radix_threshold<kTkKPT>(key, seg_n, seg_n, k, sh, prefix, pmask, remaining);
    compact_taken<kTkKPT>(key, seg_n, prefix, pmask, remaining, sh);
  }
  const int32_t *list = reinterpret_cast<const int32_t *>(sh.hist);
  if (nseg == 1) {
    // the node's selection (ascending, -1 padded) and its CSA key pointers
    int32_t *out = sel + node * k;
    for (int t = tid; t < k; t += kTkNT) {
      // one segment: element index = logical index (a list entry stays inside the segment whatever it holds)
      const int s = t < taken ? (all ? t : std::min(std::max(list[t], 0), seg_n - 1)) : -1;
      out[t] = s;
      if (s >= 0) tab[t] = csa_row(d, nk, b, s, path, c.c4, c4b, c.page_table, scr_c4);
    }
  } else {
    // survivors of this segment, in index order, then padding, for the merge
    const int64_t sv = ((int64_t)node * max_seg + seg) * k;
    for (int t = tid; t < k; t += kTkNT) {
      const int e = t < taken ? (all ? t : std::min(std::max(list[t], 0), seg_n - 1)) : -1;
      surv_idx[sv + t] = e < 0 ? -1 : (e < cn ? c0 + e : n4 + (e - cn));
      surv_key[sv + t] = e < 0 ? 0u : live_key(e < cn ? sc[e] : scr_score[e - cn]);
    }
    if (tid == 0) surv_cnt[node * max_seg + seg] = taken;
  }
}


__global__ void __launch_bounds__(kTkNT) __attribute__((amdgpu_waves_per_eu(4))) topk_kernel(
    tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u, const uint64_t *__restrict__ anc,
    const int32_t *__restrict__ depth, const uint16_t *__restrict__ scr_c4, const uint16_t *__restrict__ scr_c128,
    const uint16_t *__restrict__ q_idx, const uint16_t *__restrict__ w_idx, const float *__restrict__ scores,
    int score_stride, int32_t *__restrict__ sel, int32_t *__restrict__ row_status, int32_t *__restrict__ row_order,
    int32_t *__restrict__ row_rank, const uint16_t **__restrict__ keytab, int keytab_stride,
    int32_t *__restrict__ nkeys_tab, int32_t *__restrict__ nkeys_rank, int max_seg, int32_t *__restrict__ surv_idx,
    uint32_t *__restrict__ surv_key, int32_t *__restrict__ surv_cnt) {
  __shared__ TopkSmem sm;
  topk_node(d, c, tree_u, anc, depth, scr_c4, scr_c128, q_idx, w_idx, scores, score_stride, sel, row_status,
            row_order, row_rank, keytab, keytab_stride, nkeys_tab, nkeys_rank, max_seg, surv_idx, surv_key, surv_cnt,
            blockIdx.x, sm);
}

// The top-k and, in the same grid after its workgroups, the HCA entries of
// the split compression (one workgroup per node; nodes that close no HCA
// block exit at once).  The top-k reads no HCA scratch entry (it only lists
// their addresses), so the two are independent; the HCA workgroups start as
// the short nodes' selections finish.
__global__ void __launch_bounds__(kTkNT) __attribute__((amdgpu_waves_per_eu(4))) topk_hca_kernel(
    tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u, const uint64_t *__restrict__ anc,
    const int32_t *__restrict__ depth, const uint16_t *__restrict__ scr_c4, uint16_t *__restrict__ scr_c128,
    const uint16_t *__restrict__ q_idx, const uint16_t *__restrict__ w_idx, const float *__restrict__ scores,
    int score_stride, int32_t *__restrict__ sel, int32_t *__restrict__ row_status, int32_t *__restrict__ row_order,
    int32_t *__restrict__ row_rank, const uint16_t **__restrict__ keytab, int keytab_stride,
    int32_t *__restrict__ nkeys_tab, int32_t *__restrict__ nkeys_rank, int max_seg, int32_t *__restrict__ surv_idx,
    uint32_t *__restrict__ surv_key, int32_t *__restrict__ surv_cnt, const uint16_t *__restrict__ gate_w) {
  static_assert(kTkNT == kHcaNT, "one workgroup size for both roles");
  __shared__ union {
    TopkSmem t;
    HcaSmem h;
  } sm;
  const int ntk = d.B * d.D * max_seg;
  if ((int)blockIdx.x < ntk)
    topk_node(d, c, tree_u, anc, depth, scr_c4, scr_c128, q_idx, w_idx, scores, score_stride, sel, row_status,
              row_order, row_rank, keytab, keytab_stride, nkeys_tab, nkeys_rank, max_seg, surv_idx, surv_key,
              surv_cnt, blockIdx.x, sm.t);
  else
    hca_node(d, c, tree_u, anc, depth, gate_w, scr_c128, row_status, false, blockIdx.x - ntk, sm.h);
}

// Merge of a segmented node: the topk of the survivors of all its segments.
// Segment s holds k slots (survivors in index order, then padding key 0), so
// the slots of all segments in order list the survivors in index order.
template <int NT>
__global__ void __launch_bounds__(NT, 1) topk_merge_kernel(tv_dims d, CacheView c, const uint64_t *__restrict__ anc,
                                                           const int32_t *__restrict__ depth,
                                                           const uint16_t *__restrict__ scr_c4,
                                                           int32_t *__restrict__ sel,
                                                           const int32_t *__restrict__ row_status,
                                                           const int32_t *__restrict__ row_rank,
                                                           const uint16_t **__restrict__ keytab, int keytab_stride,
                                                           int max_seg, const int32_t *__restrict__ surv_idx,
                                                           const uint32_t *__restrict__ surv_key,
                                                           const int32_t *__restrict__ surv_cnt) {
  __shared__ SelShared sh;
  __shared__ int real_cnt;
  __shared__ int32_t path[64], hca_node[64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t node = blockIdx.x;
  const int b = (int)(node / d.D);
  const int i = (int)(node - (int64_t)b * d.D);
  const int k = d.topk;
  // One round trip for everything whose address is known from (row, node,
  // lane): the row's state, the node's path, and all of the node's survivor
  // slots and counts (those of segments the row does not have are dropped
  // once its length is known).
  const int32_t status = row_status[b];
  const int32_t L = c.len[b];
  const int32_t rank = row_rank[b];
  const int64_t c4b = d.page_size == 0 ? c.c4_base[b] : 0;
  const uint64_t m = anc[node];
  const int dl = lane < d.D ? depth[(int64_t)b * d.D + lane] : 0;
  const int64_t sv = (int64_t)node * max_seg * k;
  const int cnt_s = tid < max_seg ? surv_cnt[node * max_seg + tid] : 0;  // max_seg <= 64: wave 0
  const int all_slots = max_seg * k;
  constexpr int KPT = kTopkMergeCap / NT;
  static_assert(KPT * NT == kTopkMergeCap, "merge capacity");
  const int nr_all = (all_slots + NT - 1) / NT;
  uint32_t key[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j)
    key[j] = j < nr_all ? surv_key[sv + std::min(tid + NT * j, all_slots - 1)] : 0u;
  if (status != TV_ROW_OK || !len_ok(L, d.max_len)) return;
  const int n4 = L / d.ratio_csa;
  const int nseg = topk_segments(n4);
  if (nseg <= 1) return;
  const int slots = nseg * k;
#pragma unroll
  for (int j = 0; j < KPT; ++j)
    if (tid + NT * j >= slots) key[j] = 0u;
  if (tid < 64) {
    const int run = (int)wave_total(tid < nseg ? (uint32_t)cnt_s : 0u);
    if (tid == 0) real_cnt = run;
  }
  uint64_t csa_mask;
  const NodeKeys nk = path_keys(d, L, i, m, dl, path, hca_node, csa_mask);
  __syncthreads();  // the survivor total and the node's path are visible
  const int total = real_cnt;
  const uint16_t **tab = keytab + ((int64_t)rank * d.D + i) * keytab_stride;  // kept by (rank, node)
  int32_t *out = sel + node * k;
  const bool all = total <= k;  // every real survivor (key above 0) is taken
  uint32_t prefix = 0u, pmask = 0xFFFFFFFFu;
  int remaining = 0;
  if (!all) radix_threshold<KPT, NT>(key, slots, total, k, sh, prefix, pmask, remaining);
  compact_taken<KPT, NT>(key, slots, prefix, pmask, remaining, sh);
  const int32_t *list = reinterpret_cast<const int32_t *>(sh.hist);
  const int taken = all ? total : k;
  for (int t = tid; t < k; t += NT) {
    const int s = t < taken ? surv_idx[sv + std::min(std::max(list[t], 0), slots - 1)] : -1;
    out[t] = s;
    if (s >= 0) tab[t] = csa_row(d, nk, b, s, path, c.c4, c4b, c.page_table, scr_c4);
  }
}

int topk_max_segments(const tv_dims &d) {
  const int64_t n4 = (int64_t)d.max_len / d.ratio_csa;
  return n4 <= kTopkSeg ? 1 : (int)((n4 + kTopkSeg - 1) / kTopkSeg);
}

bool topk_supported(const tv_dims &d) {
  const int s = topk_max_segments(d);
  return d.topk <= kTkBins && (s == 1 || (s <= kTopkMaxSeg && (int64_t)s * d.topk <= kTopkMergeCap));
}

hipError_t launch_topk(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                       const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128, const uint16_t *q_idx,
                       const uint16_t *w_idx, const float *scores, int32_t score_stride, int32_t *sel,
                       int32_t *row_status, int32_t *row_order, int32_t *row_rank, const uint16_t **keytab,
                       int32_t keytab_stride, int32_t *nkeys, int32_t *nkeys_rank, int32_t *surv_idx,
                       uint32_t *surv_key, int32_t *surv_cnt, const uint16_t *hca_gate_w, uint16_t *hca_out,
                       hipStream_t s) {
  if (d.D > kMaxScratch || !topk_supported(d)) return hipErrorInvalidValue;
  const int max_seg = topk_max_segments(d);
  const int64_t ntk = (int64_t)d.B * d.D * max_seg;
  if (hca_gate_w) {  // with the HCA entries of the split compression, into hca_out (the scr_c128 buffer)
    if (!compress_split(d) || d.d_row + d.d_idx > kMaxDu || hca_out != scr_c128 ||
        ntk + (int64_t)d.B * d.D > 0x7FFFFFFF)
      return hipErrorInvalidValue;
    topk_hca_kernel<<<(unsigned)(ntk + (int64_t)d.B * d.D), kTkNT, 0, s>>>(
        d, c, tree_u, anc, depth, scr_c4, hca_out, q_idx, w_idx, scores, score_stride, sel,
        row_status, row_order, row_rank, keytab, keytab_stride, nkeys, nkeys_rank, max_seg, surv_idx, surv_key,
        surv_cnt, hca_gate_w);
    return hipGetLastError();
  }
  topk_kernel<<<(unsigned)ntk, kTkNT, 0, s>>>(
      d, c, tree_u, anc, depth, scr_c4, scr_c128, q_idx, w_idx, scores, score_stride, sel, row_status, row_order,
      row_rank, keytab, keytab_stride, nkeys, nkeys_rank, max_seg, surv_idx, surv_key, surv_cnt);
  return hipGetLastError();
}

hipError_t launch_topk_merge(const tv_dims &d, const CacheView &c, const uint64_t *anc, const int32_t *depth,
                             const uint16_t *scr_c4, int32_t *sel, const int32_t *row_status,
                             const int32_t *row_rank, const uint16_t **keytab, int32_t keytab_stride,
                             const int32_t *surv_idx, const uint32_t *surv_key, const int32_t *surv_cnt,
                             hipStream_t s) {
  const int max_seg = topk_max_segments(d);
  if (max_seg <= 1) return hipSuccess;
  topk_merge_kernel<kMergeNT><<<(unsigned)((int64_t)d.B * d.D), kMergeNT, 0, s>>>(d, c, anc, depth, scr_c4, sel,
                                                                                 row_status,
                                                                     row_rank, keytab, keytab_stride, max_seg,
                                                                     surv_idx, surv_key, surv_cnt);
  return hipGetLastError();
}

}  // namespace tv
