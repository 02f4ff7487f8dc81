// Per-branch compression of the block each node closes, into scratch.
//
// Branches that share a prefix share its committed entries, but the block that
// is still open when the tree starts is finished differently on every branch;
// each node therefore pools the tokens of its own root path and writes the
// entry to its own scratch slot, which the persistent cache never sees before
// acceptance (Sec. 4.1 chains compressed independently after branching;
// Sec. 4.2 scratch pad for temporary branch state).
//
// When a CSA block fits one wavefront (ratio_csa <= kWaveMaxR, the supported
// shapes' CSA ratio 4), compression is split (compress_body.h): a
// wavefront per node pools the node's CSA entry (lane k holds channel chunk k
// and k + 64 of every token, so the gate logits are one butterfly per token
// and the weighted sums stay in the lane, with no barrier and no second read),
// and a 512-thread workgroup per node pools its HCA entry, if it closes one;
// the one-call layer step runs the two parts in the launches of the verify
// preprocess and of the top-k.  Otherwise one 1024-thread workgroup per
// (row, node) pools both blocks (nodes that close nothing exit at once): they
// are suffixes of the same token range (both end at the node's position), so
// each token row is read once for the gate logits of both and once for both
// weighted sums.  The rows (committed ones from the ring, path ones from
// tree_u) are resolved once into an LDS pointer table; gate logits (8 lanes
// per token) and the weighted sums (token groups per 16-byte channel chunk)
// stream them with 16-byte loads, all of a thread's loads in flight together.
//
// Committed rows come from the ring or, with a paged pool, from the raw
// layer through the row's page table; a block whose committed rows lie in a
// page the table does not allocate fails the row (TV_ROW_CAPACITY).
//
// With FP8 indexer keys the indexer channels of a CSA entry are rounded to
// E4M3 (held in scratch as the same values in bfloat16, written to a pool
// slot as E4M3 codes).
//
// Refresh schedule (Sec. 4.3): when the caller designates a chain (the root
// path of primary_last[b]), the CSA entries its nodes close are also written
// straight into their persistent pool slots.  Those slots lie past the
// committed entries, so nothing reads them before the commit makes them
// committed, and the commit then skips their copies.
#include "compress_body.h"

namespace tv {

constexpr int kNT = 1024;           // threads per workgroup

__global__ void __launch_bounds__(kNT) compress_kernel(tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u,
                                                       const uint64_t *__restrict__ anc,
                                                       const int32_t *__restrict__ depth,
                                                       const uint16_t *__restrict__ gate_w,
                                                       uint16_t *__restrict__ scr_c4, uint16_t *__restrict__ scr_c128,
                                                       int32_t *__restrict__ row_status,
                                                       const int32_t *__restrict__ primary_last,
                                                       uint16_t *__restrict__ pool_c4, uint16_t *__restrict__ pool_c4_idx) {
  __shared__ int32_t path[64];
  __shared__ const uint16_t *tok[kMaxRatio];
  __shared__ float wgt[2][kMaxRatio];
  __shared__ float gate[2][kMaxDu];
  __shared__ float part[2][kMaxGroups][kMaxDu];
  __shared__ float red[2][2];
  __shared__ uint64_t chain_sh;
  const int b = blockIdx.x / d.D;
  const int i = blockIdx.x - b * d.D;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d_u = d.d_row + d.d_idx;
  const int64_t node = (int64_t)b * d.D + i;
  // every independent load first, one wait for all of them
  const int32_t status = row_status[b];
  const int32_t L = c.len[b];
  const int32_t dep = depth[node];
  const uint64_t m = anc[node];
  const int32_t dj = tid < d.D ? depth[(int64_t)b * d.D + tid] : 0;
  const uint64_t aj = (primary_last && tid < d.D) ? anc[(int64_t)b * d.D + tid] : 0ull;
  const int32_t P = primary_last ? primary_last[b] : -1;
  const bool flat = d.page_size == 0;
  const int32_t cap4 = (primary_last && flat) ? c.c4_cap[b] : 0;
  const int64_t base4 = (primary_last && flat) ? c.c4_base[b] : 0;
  asm volatile("" ::"s"(cap4), "s"(base4));  // issued with the other loads
  const float g0 = tid < d_u ? bf2f(gate_w[tid]) : 0.f;
  const float g1 = tid < d_u ? bf2f(gate_w[d_u + tid]) : 0.f;
  asm volatile("" ::"v"(g0), "v"(g1));  // gate loads issued with the others, not after the checks
  if (status != TV_ROW_OK) return;
  if (!len_ok(L, d.max_len)) {
    if (i == 0 && tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return;
  }
  const int64_t p = (int64_t)L + dep;
  const bool cl[2] = {((p + 1) % d.ratio_csa) == 0, ((p + 1) % d.ratio_hca) == 0};
  if (!cl[0] && !cl[1]) return;
  const int rat[2] = {d.ratio_csa, d.ratio_hca};
  const int keep[2] = {d_u, d.d_row};  // CSA entries keep the indexer key, HCA entries the latent row
  // Both closed blocks end at p: the tokens are positions p-R+1..p of the
  // larger one, and ratio ri pools the last rat[ri] of them.
  const int R = std::max(cl[0] ? rat[0] : 0, cl[1] ? rat[1] : 0);
  const int first[2] = {R - rat[0], R - rat[1]};
  const int64_t slot4 = (p + 1) / d.ratio_csa - 1;
  if (tid < d.D && ((m >> tid) & 1ull)) path[dj] = tid;
  if (wv == 0) {  // the designated chain: ancestor mask of node P (lane P holds it), empty if none
    const uint64_t ap = __shfl(aj, (P >= 0 && P < d.D) ? P : 0, 64);
    if (tid == 0) chain_sh = (P >= 0 && P < d.D) ? ap : 0ull;
  }
  if (tid < d_u) {
    gate[0][tid] = g0;
    gate[1][tid] = g1;
  }
  __syncthreads();
  const int64_t q0 = p - R + 1;
  bool lost = false;  // a committed row of the block whose page is not allocated
  for (int t = tid; t < R; t += kNT) {
    const int64_t qq = q0 + t;
    const int64_t ri = qq < L ? raw_index(d, c.page_table, b, qq) : 0;
    lost |= ri < 0;
    tok[t] = qq < L ? c.ring + (ri < 0 ? 0 : ri) * d_u : tree_u + ((int64_t)b * d.D + path[qq - L]) * d_u;
  }
  if (__syncthreads_or(lost)) {
    if (tid == 0) row_status[b] = TV_ROW_CAPACITY;
    return;
  }

  // Gate logits of every token for every ratio that pools it: 8 lanes per
  // token, 128 tokens per pass, all loads of a lane issued before their use.
  const int nch = d_u / 8;
  for (int t0 = 0; t0 < R; t0 += kNT / 8) {
    const int t = t0 + (tid >> 3), sub = tid & 7;
    float acc[2] = {0.f, 0.f};
    if (t < R) {
      const uint4 *row = reinterpret_cast<const uint4 *>(tok[t]);
      constexpr int U = (kMaxCh + 7) / 8;
      uint4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = sub + 8 * u;
        v[u] = k < nch ? row[k] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int ri = 0; ri < 2; ++ri) {
        if (!cl[ri] || t < first[ri]) continue;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = sub + 8 * u;
          if (k < nch) acc[ri] += dot8(gate[ri] + 8 * k, v[u]);
        }
      }
    }
#pragma unroll
    for (int ri = 0; ri < 2; ++ri) {
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) acc[ri] += __shfl_xor(acc[ri], o, 64);
      if (t < R && sub == 0 && cl[ri] && t >= first[ri]) wgt[ri][t - first[ri]] = acc[ri];
    }
  }
  __syncthreads();
  // softmax over each pooled block: wave ri
  if (wv < 2 && cl[wv]) {
    const int ri = wv, r = rat[ri];
    float mx = -INFINITY;
    for (int t = lane; t < r; t += 64) mx = fmaxf(mx, wgt[ri][t]);
    mx = wave_max(mx);
    float s = 0.f;
    for (int t = lane; t < r; t += 64) s += __expf(wgt[ri][t] - mx);
    s = wave_sum(s);
    if (lane == 0) {
      red[ri][0] = mx;
      red[ri][1] = s;
    }
  }
  __syncthreads();
#pragma unroll
  for (int ri = 0; ri < 2; ++ri) {
    if (!cl[ri]) continue;
    const float mx = red[ri][0], inv = 1.0f / red[ri][1];
    for (int t = tid; t < rat[ri]; t += kNT) wgt[ri][t] = __expf(wgt[ri][t] - mx) * inv;
  }
  __syncthreads();

  // Weighted sums: thread (token group g, chunk k) sums 8 channels over the
  // tokens g, g + G, ... of the block, each read once and added to every
  // ratio that pools it; a thread's token loads (at most twelve for the
  // supported shapes and ratios) are in flight together.
  const int kc = std::max(cl[0] ? keep[0] / 8 : 0, cl[1] ? keep[1] / 8 : 0);
  const int G = std::min(kMaxGroups, kNT / kc);
  {
    const int g = tid / kc, k = tid - g * kc;
    float acc[2][8];
#pragma unroll
    for (int ri = 0; ri < 2; ++ri)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[ri][e] = 0.f;
    if (g < G) {
      for (int tb = g; tb < R; tb += 12 * G) {
        uint4 v[12];
#pragma unroll
        for (int u = 0; u < 12; ++u) {
          const int t = tb + G * u;
          v[u] = t < R ? reinterpret_cast<const uint4 *>(tok[t])[k] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 12; ++u) {
          const int t = tb + G * u;
#pragma unroll
          for (int ri = 0; ri < 2; ++ri) {
            if (!(cl[ri] && t < R && t >= first[ri] && k < keep[ri] / 8)) continue;
            const float w = wgt[ri][t - first[ri]];
            acc[ri][0] += w * bf2f_lo(v[u].x);
            acc[ri][1] += w * bf2f_hi(v[u].x);
            acc[ri][2] += w * bf2f_lo(v[u].y);
            acc[ri][3] += w * bf2f_hi(v[u].y);
            acc[ri][4] += w * bf2f_lo(v[u].z);
            acc[ri][5] += w * bf2f_hi(v[u].z);
            acc[ri][6] += w * bf2f_lo(v[u].w);
            acc[ri][7] += w * bf2f_hi(v[u].w);
          }
        }
      }
#pragma unroll
      for (int ri = 0; ri < 2; ++ri)
        if (cl[ri] && k < keep[ri] / 8)
#pragma unroll
          for (int e = 0; e < 8; ++e) part[ri][g][8 * k + e] = acc[ri][e];
    }
  }
  __syncthreads();
  // a CSA entry closed on the designated chain also goes to its pool slot, capacity permitting
  int64_t pslot = -1;
  if (cl[0] && ((chain_sh >> i) & 1ull))
    pslot = flat ? (slot4 < cap4 ? base4 + slot4 : -1)
                 : pool_slot(d, c.page_table, nullptr, nullptr, b, slot4, d.ratio_csa);
  const bool through = pslot >= 0;
#pragma unroll
  for (int ri = 0; ri < 2; ++ri) {
    if (!cl[ri]) continue;
    uint16_t *dst = ri == 0 ? scr_c4 + node * d_u : scr_c128 + node * d.d_row;
    for (int ch = tid; ch < keep[ri]; ch += kNT) {
      float sum = 0.f;
#pragma unroll
      for (int gg = 0; gg < G; ++gg) sum += part[ri][gg][ch];  // group order
      // FP8 indexer keys: the indexer channels of a CSA entry are E4M3 values
      const bool fp8 = ri == 0 && ch >= d.d_row && d.idx_fmt == TV_IDX_E4M3;
      const uint32_t code = fp8 ? f32_to_e4m3(sum) : 0u;
      const uint16_t v = fp8 ? (uint16_t)e4m3_to_bf16(code) : f2bf(sum);
      dst[ch] = v;
      if (ri == 0 && through) {
        if (ch < d.d_row)
          pool_c4[pslot * d.d_row + ch] = v;
        else if (fp8)
          reinterpret_cast<uint8_t *>(pool_c4_idx)[pslot * d.d_idx + (ch - d.d_row)] = (uint8_t)code;
        else
          pool_c4_idx[pslot * d.d_idx + (ch - d.d_row)] = v;
      }
    }
  }
}

// Split compression (compress_split(d)): one kHcaNT-thread workgroup per
// node for its HCA entry (the rest exit at once), then one workgroup per
// eight nodes, a wavefront per node, for the CSA entries.
constexpr int kSplitWaves = kHcaNT / 64;
__global__ void __launch_bounds__(kHcaNT) compress_split_kernel(
    tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u, const uint64_t *__restrict__ anc,
    const int32_t *__restrict__ depth, const uint16_t *__restrict__ gate_w, uint16_t *__restrict__ scr_c4,
    uint16_t *__restrict__ scr_c128, int32_t *__restrict__ row_status, const int32_t *__restrict__ primary_last,
    uint16_t *__restrict__ pool_c4, uint16_t *__restrict__ pool_c4_idx) {
  __shared__ union {
    HcaSmem h;
    int32_t paths[kSplitWaves][64];
  } sm;
  const int nodes = d.B * d.D;
  const int blk = blockIdx.x;
  if (blk < nodes) {
    hca_node(d, c, tree_u, anc, depth, gate_w, scr_c128, row_status, true, blk, sm.h);
  } else {
    const int wv = threadIdx.x >> 6, n = (blk - nodes) * kSplitWaves + wv;
    if (n < nodes)
      csa_wave_node<false>(d, c, nullptr, anc, depth, tree_u, gate_w, scr_c4, row_status, primary_last, pool_c4,
                           pool_c4_idx, n, sm.paths[wv]);
  }
}

hipError_t launch_compress(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                           const int32_t *depth, const uint16_t *gate_w, uint16_t *scr_c4, uint16_t *scr_c128,
                           int32_t *row_status, const int32_t *primary_last, uint16_t *pool_c4,
                           uint16_t *pool_c4_idx, hipStream_t s) {
  if (d.d_row + d.d_idx > kMaxDu) return hipErrorInvalidValue;
  if (compress_split(d)) {
    const int nodes = d.B * d.D;
    compress_split_kernel<<<nodes + (nodes + kSplitWaves - 1) / kSplitWaves, kHcaNT, 0, s>>>(
        d, c, tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status, primary_last, pool_c4, pool_c4_idx);
    return hipGetLastError();
  }
  dim3 grid(d.B * d.D);
  compress_kernel<<<grid, kNT, 0, s>>>(d, c, tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status, primary_last,
                                       pool_c4, pool_c4_idx);
  return hipGetLastError();
}

}  // namespace tv
