// CSA indexer scoring, shared pieces: key loads and the fast-path chunk body
// (H_idx = 8, D <= 8), used by the scoring kernel and by the kernel that runs
// the scoring beside the verify preprocess.
//
// score[b][i][s] = sum_h w[b][i][h] * relu(q_idx[b][i][h] . k_s) over the
// committed entries s < len/ratio_csa, on MFMA (v_mfma_f32_32x32x16_bf16,
// float32 accumulate), head reduction in a fixed order: the bits of a score do
// not depend on how entries are grouped into workgroups.
#pragma once

#include <algorithm>

#include "pool_addr.h"

namespace tv {

// Eight indexer-key channels (chunk = channel / 8) of pool entry `entry` as
// loaded: a 16-byte chunk of bfloat16, or with FP8 keys an 8-byte chunk of
// E4M3 codes (in .x, .y).  key_bf16 widens a loaded chunk to bfloat16; the
// loads of a thread all go out before any chunk is widened.
template <bool FP8>
__device__ __forceinline__ uint4 key_load(const uint16_t *c4_idx, int64_t entry, int chunk) {
  if (FP8) {
    const uint2 w = reinterpret_cast<const uint2 *>(reinterpret_cast<const uint8_t *>(c4_idx) + entry * 64)[chunk];
    return make_uint4(w.x, w.y, 0u, 0u);
  }
  return reinterpret_cast<const uint4 *>(c4_idx + entry * 64)[chunk];
}
template <bool FP8>
__device__ __forceinline__ uint4 key_bf16(uint4 v) {
  return FP8 ? e4m3x8_to_bf16x8(make_uint2(v.x, v.y)) : v;
}

constexpr int kMaxB = 4096;  // rows of one call

// LDS of one fast-path chunk of NW wavefronts.
template <int NW>
struct ScoreH8Smem {
  float wsh[64];
  uint4 qtile[64 * 8];
  uint4 ktile[NW][32 * 8];
};

// Fast path for H_idx = 8 and D <= 8: the (node, head) rows of one tree form
// exactly two 32-row MFMA tiles (row 8 node + head), so in the 32x32 output
// layout a lane holds, for entry column l32, heads 4 hi + 0..3 of nodes
// 4 tile + 0..3.  The weighted ReLU sum over a node's 8 heads is four
// in-lane terms plus the other half-wave's four (one shuffle), in fixed order.
// The workgroup scores chunk ch of row b: NW wavefronts x 64 entries.  The
// loads a chunk needs (row status, length, pool base, indexer weights, then
// queries and keys) are issued as early as their addresses are known, so a
// chunk costs two memory round trips.  kStatus: a row whose status is not
// TV_ROW_OK is skipped (only where nothing writes the status meanwhile, so the
// exit is workgroup-uniform; the length exits always are).
template <bool FP8, int NW, bool kStatus>
__device__ __forceinline__ void score_h8_chunk(const tv_dims &d, const CacheView &c,
                                               const uint16_t *__restrict__ q_idx,
                                               const uint16_t *__restrict__ w_idx,
                                               const int32_t *__restrict__ row_status, float *__restrict__ scores,
                                               int score_stride, int b, int ch, ScoreH8Smem<NW> &sm) {
  constexpr int kChunk = NW * 64;
  constexpr int kQU = (512 + 64 * NW - 1) / (64 * NW);  // 16-byte query pieces per thread (64 rows x 8)
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const int M = d.D * 8;
  const int32_t status = kStatus ? row_status[b] : TV_ROW_OK;
  const int32_t L = c.len[b];
  const bool flat = d.page_size == 0;
  const int64_t c4b = flat ? c.c4_base[b] : 0;
  const float wv_ = tid < M ? bf2f(w_idx[(int64_t)b * M + tid]) : 0.f;
  if (status != TV_ROW_OK || !len_ok(L, d.max_len)) return;
  const int n4 = L / d.ratio_csa;
  const int e0 = ch * kChunk + wv * 64;
  if (ch * kChunk >= n4) return;
  // Operands are read as whole 128-byte rows (eight lanes a row, eight rows a
  // load) and turned into the MFMA layout through LDS: lane l32 + 32 hi holds
  // channels 16 ks + 8 hi of its row.  In a tile, 16-byte slot c of row r sits
  // at slot c ^ (r & 7), so the row writes and the column reads are free of
  // bank conflicts.
  // A: the tree's 64 (node, head) query rows, loaded once for the workgroup
  // (piece t: row t / 8, slot t % 8) into a shared tile.
  uint4 qr[kQU];
#pragma unroll
  for (int u = 0; u < kQU; ++u) {
    const int t = tid + u * 64 * NW, r = t >> 3;
    qr[u] = (t < 512 && r < M) ? reinterpret_cast<const uint4 *>(q_idx + ((int64_t)b * M + r) * 64)[t & 7]
                               : make_uint4(0, 0, 0, 0);
  }
  // B: the wavefront's 64 keys, through its own 32-row tile in two halves.
  // Every load is issued (entries past the row re-read its last one, which
  // exists: n4 > 0 here) and dead lanes are zeroed afterwards, so no branch
  // separates the loads and all of them are in flight together.
  // With a paged pool each entry's slot comes from the row's page table
  // first (a slot of a page the table lacks is clamped to slot 0).
  int64_t ent[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int e = std::min(e0 + 8 * u + (lane >> 3), n4 - 1);
    ent[u] = flat ? c4b + e : std::max<int64_t>(0, pool_slot(d, c.page_table, nullptr, nullptr, b, e, d.ratio_csa));
  }
  uint4 kr[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) kr[u] = key_load<FP8>(c.c4_idx, ent[u], lane & 7);
#pragma unroll
  for (int u = 0; u < 8; ++u)
    if (e0 + 8 * u + (lane >> 3) >= n4) kr[u] = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int u = 0; u < kQU; ++u) {
    const int t = tid + u * 64 * NW, r = t >> 3;
    if (t < 512) sm.qtile[r * 8 + ((t & 7) ^ (r & 7))] = qr[u];
  }
  bf16x8 kb[2][4];
#pragma unroll
  for (int cc = 0; cc < 2; ++cc) {
    if (cc == 1) asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the first half is read out
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 8 * u + (lane >> 3);
      sm.ktile[wv][r * 8 + ((lane & 7) ^ (r & 7))] = key_bf16<FP8>(kr[4 * cc + u]);
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      kb[cc][ks] = __builtin_bit_cast(bf16x8, sm.ktile[wv][l32 * 8 + ((2 * ks + hi) ^ (l32 & 7))]);
  }
  if (tid < 64) sm.wsh[tid] = wv_;
  __syncthreads();
  bf16x8 qa[2][4];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int r = t * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qa[t][ks] = __builtin_bit_cast(bf16x8, sm.qtile[r * 8 + ((2 * ks + hi) ^ (r & 7))]);
  }
#pragma unroll
  for (int cc = 0; cc < 2; ++cc) {
    const int e = e0 + cc * 32 + l32;
    const bool live = e < n4;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      f32x16 acc = f32x16{};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[t][ks], kb[cc][ks], acc, 0, 0, 0);
      // head reduction of node 4t + J: rows 8J + 4hi + r of the tile, the
      // two halves combined in a fixed order
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        const int nd = 4 * t + J;
        float sp = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) sp += sm.wsh[8 * nd + 4 * hi + r] * fmaxf(acc[4 * J + r], 0.f);
        const float other = __shfl_xor(sp, 32, 64);
        const float sfull = hi == 0 ? sp + other : other + sp;
        if (hi == (J & 1) && nd < d.D && live) scores[((int64_t)b * d.D + nd) * score_stride + e] = sfull;
      }
    }
  }
}

}  // namespace tv
