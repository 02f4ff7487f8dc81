// Branch compression, pieces shared by the compression kernels and by the
// kernels of the one-call layer step that run the compression's parts beside
// other work: the short-block path of one wavefront, the HCA-block path of
// one 512-thread workgroup, and the node facts either needs.
//
// Split compression (compress_split): when a CSA block has at most kWaveMaxR
// tokens, every CSA entry is pooled by one wavefront (compress_short) and
// every HCA entry by a workgroup of its own (hca_node), so the two never wait
// for each other; a node closing both gets one of each.  Otherwise one
// workgroup per node pools both (the compression kernel's general path).
#pragma once

#include "pool_addr.h"

namespace tv {

constexpr int kMaxRatio = 1024;
constexpr int kMaxDu = 640;       // raw row width bound (d_row + d_idx): the supported shapes' 640 and 320
constexpr int kMaxCh = kMaxDu / 8;  // 16-byte chunks of the widest row
constexpr int kMaxGroups = 16;      // token groups of the weighted sums

__device__ __forceinline__ float dot8(const float *g, uint4 v) {
  return g[0] * bf2f_lo(v.x) + g[1] * bf2f_hi(v.x) + g[2] * bf2f_lo(v.y) + g[3] * bf2f_hi(v.y) +
         g[4] * bf2f_lo(v.z) + g[5] * bf2f_hi(v.z) + g[6] * bf2f_lo(v.w) + g[7] * bf2f_hi(v.w);
}

// The short-block path, run by one wavefront per node (see above); it uses
// no workgroup barrier.  q0 is the block's first position, R its token count,
// m the node's ancestor mask, dj the depth of node `lane`, path an LDS array
// of the wavefront's own.
__device__ void compress_short(const tv_dims &d, const CacheView &c, const uint16_t *__restrict__ tree_u,
                               const uint16_t *__restrict__ gate_w, int b, int64_t node, int32_t L, int64_t q0, int R,
                               uint64_t m, int32_t dj, int32_t *path, uint16_t *__restrict__ scr_c4,
                               int32_t *__restrict__ row_status, int64_t pslot, uint16_t *__restrict__ pool_c4,
                               uint16_t *__restrict__ pool_c4_idx) {
  const int lane = threadIdx.x & 63;
  const int d_u = d.d_row + d.d_idx, nch = d_u / 8;
  if (lane < d.D && ((m >> lane) & 1ull)) path[dj] = lane;
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the path is in LDS for the whole wave
  __builtin_amdgcn_wave_barrier();
  // token rows: lane t < R resolves token t, then every lane takes them by shuffle
  const int64_t qt = q0 + (lane < R ? lane : 0);
  int64_t ri = 0;
  const uint16_t *rp = nullptr;
  if (qt < L) {
    ri = raw_index(d, c.page_table, b, qt);
    rp = c.ring + (ri < 0 ? 0 : ri) * d_u;
  } else {
    rp = tree_u + ((int64_t)b * d.D + path[qt - L]) * d_u;
  }
  if (__any(lane < R && ri < 0)) {  // a committed row whose page is not allocated
    if (lane == 0) row_status[b] = TV_ROW_CAPACITY;
    return;
  }
  const uintptr_t rpi = reinterpret_cast<uintptr_t>(rp);
  uint4 v[kWaveMaxR][2], g[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int k = lane + 64 * u;
    g[u] = k < nch ? reinterpret_cast<const uint4 *>(gate_w)[k] : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int t = 0; t < kWaveMaxR; ++t) {
    const uintptr_t rt = (uintptr_t)__shfl((unsigned long long)rpi, t < R ? t : 0, 64);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = lane + 64 * u;
      v[t][u] = (t < R && k < nch) ? reinterpret_cast<const uint4 *>(rt)[k] : make_uint4(0, 0, 0, 0);
    }
  }
  // gate logits: the lane's chunks of every token, then a butterfly per token
  float gf[2][8];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    gf[u][0] = bf2f_lo(g[u].x); gf[u][1] = bf2f_hi(g[u].x);
    gf[u][2] = bf2f_lo(g[u].y); gf[u][3] = bf2f_hi(g[u].y);
    gf[u][4] = bf2f_lo(g[u].z); gf[u][5] = bf2f_hi(g[u].z);
    gf[u][6] = bf2f_lo(g[u].w); gf[u][7] = bf2f_hi(g[u].w);
  }
  float w[kWaveMaxR];
  float mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < kWaveMaxR; ++t) {
    float a = 0.f;
#pragma unroll
    for (int u = 0; u < 2; ++u) a += dot8(gf[u], v[t][u]);
    a = wave_sum(a);
    w[t] = t < R ? a : -INFINITY;
    mx = fmaxf(mx, w[t]);
  }
  float sum = 0.f;
#pragma unroll
  for (int t = 0; t < kWaveMaxR; ++t) {
    w[t] = t < R ? __expf(w[t] - mx) : 0.f;
    sum += w[t];
  }
  const float inv = 1.0f / sum;
  // weighted sums of the lane's chunks, in token order
  uint16_t *dst = scr_c4 + node * d_u;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int k = lane + 64 * u;
    if (k >= nch) continue;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < kWaveMaxR; ++t) {
      if (t >= R) continue;
      const float wt = w[t] * inv;
      acc[0] += wt * bf2f_lo(v[t][u].x);
      acc[1] += wt * bf2f_hi(v[t][u].x);
      acc[2] += wt * bf2f_lo(v[t][u].y);
      acc[3] += wt * bf2f_hi(v[t][u].y);
      acc[4] += wt * bf2f_lo(v[t][u].z);
      acc[5] += wt * bf2f_hi(v[t][u].z);
      acc[6] += wt * bf2f_lo(v[t][u].w);
      acc[7] += wt * bf2f_hi(v[t][u].w);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ch = 8 * k + e;
      // FP8 indexer keys: the indexer channels of a CSA entry are E4M3 values
      const bool fp8 = ch >= d.d_row && d.idx_fmt == TV_IDX_E4M3;
      const uint32_t code = fp8 ? f32_to_e4m3(acc[e]) : 0u;
      const uint16_t val = fp8 ? (uint16_t)e4m3_to_bf16(code) : f2bf(acc[e]);
      dst[ch] = val;
      if (pslot >= 0) {
        if (ch < d.d_row)
          pool_c4[pslot * d.d_row + ch] = val;
        else if (fp8)
          reinterpret_cast<uint8_t *>(pool_c4_idx)[pslot * d.d_idx + (ch - d.d_row)] = (uint8_t)code;
        else
          pool_c4_idx[pslot * d.d_idx + (ch - d.d_row)] = val;
      }
    }
  }
}

// The CSA entry node `blk` (row blk / D) closes, if it closes one, pooled by
// the calling wavefront alone (compress_split(d) holds).  kSelfMask: the
// node's ancestor mask and depths come from the parent array (the row checked
// as the verify preprocess checks it) and the row status is not read, so the
// wavefront can run beside the preprocess, which writes them; a row with bad
// parents or a bad length is skipped.  Otherwise they are read from anc,
// depth and row_status.  The wavefront writes a row status only to fail a row
// of a paged pool (a committed row of the block in no allocated page), which
// kSelfMask callers do not use.  `path` is the wavefront's own 64-entry LDS
// array.
template <bool kSelfMask>
__device__ __forceinline__ void csa_wave_node(const tv_dims &d, const CacheView &c, const int32_t *__restrict__ parents,
                                              const uint64_t *__restrict__ anc, const int32_t *__restrict__ depth,
                                              const uint16_t *__restrict__ tree_u, const uint16_t *__restrict__ gate_w,
                                              uint16_t *__restrict__ scr_c4, int32_t *__restrict__ row_status,
                                              const int32_t *__restrict__ primary_last,
                                              uint16_t *__restrict__ pool_c4, uint16_t *__restrict__ pool_c4_idx,
                                              int blk, int32_t *path) {
  const int b = blk / d.D;
  const int i = blk - b * d.D;
  const int lane = threadIdx.x & 63;
  const int64_t rb = (int64_t)b * d.D, node = rb + i;
  const int32_t L = c.len[b];
  const int32_t P = primary_last ? primary_last[b] : -1;
  const bool flat = d.page_size == 0;
  const int32_t cap4 = (primary_last && flat) ? c.c4_cap[b] : 0;
  const int64_t base4 = (primary_last && flat) ? c.c4_base[b] : 0;
  int32_t dep, dj;
  uint64_t m, aj;
  if (kSelfMask) {
    // lane j holds node j: its parent, then (row valid) its ancestor mask and
    // depth by walking up the parents, every lane active at every step
    const int32_t pj = lane < d.D ? parents[rb + lane] : 0;
    const bool okj = lane >= d.D || (lane == 0 ? pj == -1 : (pj >= 0 && pj < lane));
    if (!__all(okj) || !len_ok(L, d.max_len)) return;
    uint64_t mm = lane < d.D ? 1ull << lane : 0ull;
    int32_t dd = 0;
    int j = lane < d.D ? pj : -1;
    for (int step = 0; step < d.D; ++step) {  // parents strictly decrease: at most D - 1 steps
      const bool live = j >= 0;
      if (live) {
        mm |= 1ull << j;
        ++dd;
      }
      const int jn = __shfl(pj, live ? j : 0, 64);
      j = live ? jn : -1;
    }
    dj = dd;
    aj = mm;
    dep = __shfl(dd, i, 64);
    m = __shfl(mm, i, 64);
  } else {
    const int32_t status = row_status[b];
    dep = depth[node];
    m = anc[node];
    dj = lane < d.D ? depth[rb + lane] : 0;
    aj = lane < d.D ? anc[rb + lane] : 0ull;
    if (status != TV_ROW_OK || !len_ok(L, d.max_len)) return;
  }
  const int64_t p = (int64_t)L + dep;
  if (((p + 1) % d.ratio_csa) != 0) return;
  const int R = d.ratio_csa;
  const int64_t slot4 = (p + 1) / d.ratio_csa - 1;
  // a CSA entry closed on the designated chain also goes to its pool slot, capacity permitting
  const uint64_t chain = (P >= 0 && P < d.D) ? __shfl(aj, P, 64) : 0ull;
  int64_t pslot = -1;
  if ((chain >> i) & 1ull)
    pslot = flat ? (slot4 < cap4 ? base4 + slot4 : -1)
                 : pool_slot(d, c.page_table, nullptr, nullptr, b, slot4, d.ratio_csa);
  compress_short(d, c, tree_u, gate_w, b, node, L, p - R + 1, R, m, dj, path, scr_c4, row_status, pslot, pool_c4,
                 pool_c4_idx);
}

// The HCA entry node `blk` closes, if it closes one, pooled by a workgroup of
// kHcaNT threads (compress_split(d) holds; the node's CSA entry is
// csa_wave_node's).  Reads anc, depth and row_status (the verify preprocess
// has run).  With bad_len_writer, the workgroup of node 0 of a row whose
// status is TV_ROW_OK and whose length is out of range writes TV_ROW_BAD_LEN.
// Every exit before a barrier is workgroup-uniform.
constexpr int kHcaNT = 512;
constexpr int kHcaGroups = 16;  // token groups of the weighted sums (at most)
struct HcaSmem {
  int32_t path[64];
  const uint16_t *tok[kMaxRatio];
  float wgt[kMaxRatio];
  float gate[kMaxDu];
  float part[8 * kHcaNT];  // [group][channel]: at most kHcaNT / chunks groups of 8 * chunks channels
  float red[2];
};

__device__ __forceinline__ void hca_node(const tv_dims &d, const CacheView &c, const uint16_t *__restrict__ tree_u,
                                         const uint64_t *__restrict__ anc, const int32_t *__restrict__ depth,
                                         const uint16_t *__restrict__ gate_w, uint16_t *__restrict__ scr_c128,
                                         int32_t *__restrict__ row_status, bool bad_len_writer, int blk, HcaSmem &sm) {
  const int b = blk / d.D;
  const int i = blk - b * d.D;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int d_u = d.d_row + d.d_idx;
  const int64_t node = (int64_t)b * d.D + i;
  // every independent load first, one wait for all of them
  const int32_t status = row_status[b];
  const int32_t L = c.len[b];
  const int32_t dep = depth[node];
  const uint64_t m = anc[node];
  const int32_t dj = tid < d.D ? depth[(int64_t)b * d.D + tid] : 0;
  const float g0 = tid < d_u ? bf2f(gate_w[d_u + tid]) : 0.f;  // the HCA gate is the second row of gate_w
  const float g1 = tid + kHcaNT < d_u ? bf2f(gate_w[d_u + kHcaNT + tid]) : 0.f;
  asm volatile("" ::"v"(g0), "v"(g1));  // gate loads issued with the others, not after the checks
  if (status != TV_ROW_OK) return;
  if (!len_ok(L, d.max_len)) {
    if (bad_len_writer && i == 0 && tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return;
  }
  const int64_t p = (int64_t)L + dep;
  if (((p + 1) % d.ratio_hca) != 0) return;
  const int R = d.ratio_hca;
  if (tid < d.D && ((m >> tid) & 1ull)) sm.path[dj] = tid;
  if (tid < d_u) sm.gate[tid] = g0;
  if (tid + kHcaNT < d_u) sm.gate[tid + kHcaNT] = g1;
  __syncthreads();
  const int64_t q0 = p - R + 1;
  bool lost = false;  // a committed row of the block whose page is not allocated
  for (int t = tid; t < R; t += kHcaNT) {
    const int64_t qq = q0 + t;
    const int64_t ri = qq < L ? raw_index(d, c.page_table, b, qq) : 0;
    lost |= ri < 0;
    sm.tok[t] = qq < L ? c.ring + (ri < 0 ? 0 : ri) * d_u : tree_u + ((int64_t)b * d.D + sm.path[qq - L]) * d_u;
  }
  if (__syncthreads_or(lost)) {
    if (tid == 0) row_status[b] = TV_ROW_CAPACITY;
    return;
  }
  // gate logits: 8 lanes per token, kHcaNT / 8 tokens per pass, a lane's
  // loads of a token issued before their use
  const int nch = d_u / 8;
  for (int t0 = 0; t0 < R; t0 += kHcaNT / 8) {
    const int t = t0 + (tid >> 3), sub = tid & 7;
    float acc = 0.f;
    if (t < R) {
      const uint4 *row = reinterpret_cast<const uint4 *>(sm.tok[t]);
      constexpr int U = (kMaxCh + 7) / 8;
      uint4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = sub + 8 * u;
        v[u] = k < nch ? row[k] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = sub + 8 * u;
        if (k < nch) acc += dot8(sm.gate + 8 * k, v[u]);
      }
    }
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) acc += __shfl_xor(acc, o, 64);
    if (t < R && sub == 0) sm.wgt[t] = acc;
  }
  __syncthreads();
  // softmax over the block: wave 0
  if (wv == 0) {
    float mx = -INFINITY;
    for (int t = lane; t < R; t += 64) mx = fmaxf(mx, sm.wgt[t]);
    mx = wave_max(mx);
    float s = 0.f;
    for (int t = lane; t < R; t += 64) s += __expf(sm.wgt[t] - mx);
    s = wave_sum(s);
    if (lane == 0) {
      sm.red[0] = mx;
      sm.red[1] = s;
    }
  }
  __syncthreads();
  {
    const float mx = sm.red[0], inv = 1.0f / sm.red[1];
    for (int t = tid; t < R; t += kHcaNT) sm.wgt[t] = __expf(sm.wgt[t] - mx) * inv;
  }
  __syncthreads();
  // weighted sums: thread (token group g, chunk k) sums 8 latent channels over
  // the tokens g, g + G, ..., twelve token loads in flight
  const int kc = d.d_row / 8;
  const int G = std::min(kHcaGroups, kHcaNT / kc);
  {
    const int g = tid / kc, k = tid - g * kc;
    if (g < G) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int tb = g; tb < R; tb += 12 * G) {
        uint4 v[12];
#pragma unroll
        for (int u = 0; u < 12; ++u) {
          const int t = tb + G * u;
          v[u] = t < R ? reinterpret_cast<const uint4 *>(sm.tok[t])[k] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 12; ++u) {
          const int t = tb + G * u;
          if (t >= R) continue;
          const float w = sm.wgt[t];
          acc[0] += w * bf2f_lo(v[u].x);
          acc[1] += w * bf2f_hi(v[u].x);
          acc[2] += w * bf2f_lo(v[u].y);
          acc[3] += w * bf2f_hi(v[u].y);
          acc[4] += w * bf2f_lo(v[u].z);
          acc[5] += w * bf2f_hi(v[u].z);
          acc[6] += w * bf2f_lo(v[u].w);
          acc[7] += w * bf2f_hi(v[u].w);
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) sm.part[g * (8 * kc) + 8 * k + e] = acc[e];
    }
  }
  __syncthreads();
  uint16_t *dst = scr_c128 + node * d.d_row;
  for (int ch = tid; ch < d.d_row; ch += kHcaNT) {
    float sum = 0.f;
    for (int gg = 0; gg < G; ++gg) sum += sm.part[gg * (8 * kc) + ch];  // group order
    dst[ch] = f2bf(sum);
  }
}

}  // namespace tv
