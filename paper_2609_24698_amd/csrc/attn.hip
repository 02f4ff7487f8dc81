// Branch-aware verify attention over CSA / HCA / window keys.
//
// One workgroup (8 wavefronts, two per SIMD) takes one (row, node, key
// split).  Every query head of the node reads the same single KV row per key,
// so a 32-key tile is gathered once into LDS (direct global->LDS copies, two
// tiles ahead of the math) and feeds two MFMA contractions
// (v_mfma_f32_32x32x16_bf16, float32 accumulation):
//   S^T = K Q^T     keys x heads.  Wave (head tile ht, part p) holds the
//                   queries of 32 heads for a quarter of the key channels and
//                   computes a partial S^T; wave p then owns key rows
//                   8p + 4hi + 0..3 of the tile: it adds the four partials in
//                   part order, exponentiates and publishes bf16 P to LDS.
//   O^T += V^T P^T  value channels x heads.  Wave w owns value channels
//                   w*DV/8.. for all heads, so each value element crosses the
//                   slow LDS transpose path (ds_read_b64_tr_b16) exactly once
//                   per tile; P comes back from LDS with plain 8-byte reads.
// Keys on the rows of S^T give each lane one head column, so the softmax
// statistics are per lane.  The loop is software-pipelined: the P V of tile t
// and the logits of tile t+1 form one MFMA phase, the probabilities of tile
// t+1 the next, with one barrier between phases.
//
// A node whose keys fit one split writes its normalised output; otherwise each
// split writes an unnormalised partial (O, reference max, sum) that the
// combine kernel merges in split order.
#include <algorithm>

#include "attn_common.h"

namespace tv {

template <int NW, int HT, int DK, int DV, int VOFF, int DROW>
struct AttnShape {
  static constexpr int NP = NW / HT;            // wavefronts sharing a head tile
  static constexpr int KSP = DK / 16 / NP;      // logit k-steps per wavefront
  static constexpr int DVW = DV / NW;           // value channels per wavefront (all heads)
  static constexpr int CT = DVW / 32;           // 32-row output tiles per wavefront and head tile
  static constexpr int CPR = DROW / 8;          // 16-byte chunks per key row
  static constexpr int NINS = kKT * CPR / 64;   // 1 KiB LDS-copy instructions per tile
  static constexpr int NPW = (NINS + NW - 1) / NW;  // ... per wavefront (the last ones may have one less)
  static constexpr int TILE_BYTES = kKT * DROW * 2;
  static_assert(NP == 4, "the k-step interleave assumes four channel parts per head tile");
  static_assert((DK / 16) % NP == 0, "key width must split over the wavefronts");
  static_assert(DVW % 32 == 0, "value width must split into 32-wide tiles");
  static_assert(CPR % 8 == 0, "rows must be whole 128-byte groups");
  // Own-copy layout: when each wave's value channels are exactly one
  // 128-byte column group of the rows (and one group of rope channels is
  // left), the tile is stored group-major (group g of all 32 rows, then group
  // g+1, ...).  Wave w then copies column group w of the next tile itself, as
  // soon as its own P V reads of the buffer are done, with no barrier.
  static constexpr bool OWN = VOFF == 0 && DVW == 64 && CPR == 8 * (NW + 1);
  static constexpr int GROUP_BYTES = kKT * 128;     // one column group of the tile (OWN)
  static constexpr int KSTRIDE = OWN ? GROUP_BYTES : 128;  // bytes between logit k-steps 4m and 4m+4
  // XOR swizzle of the low three bits of a row's 16-byte chunk index: one
  // chunk column of 16 consecutive rows lands on all 16 four-bank groups of
  // the 64 LDS banks (the row stride is 8 chunks mod 16 in both layouts).
  __device__ static constexpr int swz(int r) { return (OWN || CPR % 16 == 8) ? ((r >> 1) & 7) : (r & 7); }
  // byte offset in a tile of element `col` of row `r`
  __device__ static constexpr int off(int r, int col) {
    const int c = col >> 3;
    if (OWN) return (c >> 3) * GROUP_BYTES + r * 128 + ((c & 7) ^ swz(r)) * 16 + (col & 7) * 2;
    return (r * CPR + (c & ~7) + ((c & 7) ^ swz(r))) * 16 + (col & 7) * 2;
  }
};

template <int NW, int HT, int DK, int DV, int VOFF, int DROW>
__global__ void __launch_bounds__(NW * 64, 1)
attn_kernel(tv_dims d, const uint16_t *__restrict__ q, const int32_t *__restrict__ row_status,
            const int32_t *__restrict__ row_order, const uint16_t *const *__restrict__ keytab, int keytab_stride,
            const int32_t *__restrict__ nkeys_tab, int chunk, int splits, float *__restrict__ part_o,
            float *__restrict__ part_ml, uint16_t *__restrict__ out, float *__restrict__ lse) {
  using S = AttnShape<NW, HT, DK, DV, VOFF, DROW>;
  constexpr int NT = NW * 64;
  constexpr int NBUF = 3;
  __shared__ __attribute__((aligned(1024))) unsigned char sK[NBUF][S::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) float sX[HT][S::NP][64][16];
  __shared__ const uint16_t *sPtr[kMaxChunk];
  __shared__ int sFlag[NW];
  __shared__ uint2 sP[HT][S::NP][64];
  __shared__ float sMx[HT][S::NP][32];
  __shared__ float sRef[HT][32];

  int i, split;
  const int rank = unit_of(blockIdx.x, d.B, d.D, splits, i, split);
  if (rank >= d.B) return;
  const int64_t rnode = (int64_t)rank * d.D + i;  // key table and key count are kept by (rank, node)
  const int b = row_order[rank];
  const int64_t node = (int64_t)b * d.D + i;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const int ht = wv % HT, part = wv / HT;
  const int k0 = split * chunk;
  // Everything the prologue needs is loaded at once: key count (0 for a row
  // the earlier steps skipped), this thread's entries of the node's key table
  // (the top-k kernel wrote it; entries past the count are never used) and
  // the queries.  The table loads come first so that storing them waits for
  // them only.
  (void)row_status;
  const int n_keys = nkeys_tab[rnode];
  constexpr int kPer = (kMaxChunk + NT - 1) / NT;
  const uint16_t *tp[kPer];
  {
    const uint16_t *const *tab = keytab + rnode * keytab_stride + k0;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int t = tid + NT * u;
      tp[u] = (t < chunk && k0 + t < keytab_stride) ? tab[t] : nullptr;
    }
  }
  // This wave's logit k-steps are ks = 4m + part: channels 16 ks + 8 hi of
  // the key row (A, from LDS) and of the query (B, kept in registers).  The
  // key chunk 8m + 2 part + hi keeps its low three bits across m, so the A
  // address is one per-lane base plus the immediate 128 m.
  bf16x8 qf[S::KSP];
  {
    const int h = ht * 32 + l32;
    const uint16_t *qrow = q + (node * d.H + (h < d.H ? h : 0)) * DK + hi * 8;
#pragma unroll
    for (int m = 0; m < S::KSP; ++m) {
      const int ks = S::NP * m + part;
      uint4 v = h < d.H ? *reinterpret_cast<const uint4 *>(qrow + ks * 16) : make_uint4(0, 0, 0, 0);
      qf[m] = __builtin_bit_cast(bf16x8, v);
    }
  }
  if (k0 >= n_keys) return;
  const int k1 = std::min(n_keys, k0 + chunk);
  const int nkeys = k1 - k0;
  const int ntiles = (nkeys + kKT - 1) / kKT;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int t = tid + NT * u;
    if (t < nkeys) sPtr[t] = tp[u];
  }

  const int aoff = S::off(l32, (2 * part + hi) * 8);
  // Value-operand offsets for the transpose reads: rows 16 ks + 8 s + 4 hi + jj/4,
  // columns VOFF + wv*DVW + 16 (g&1) + 4 (jj&3) + 32 ct.
  const int g = lane >> 4, jj = lane & 15;
  int voff[4][S::CT];
#pragma unroll
  for (int rr = 0; rr < 4; ++rr)
#pragma unroll
    for (int ct = 0; ct < S::CT; ++ct)
      voff[rr][ct] = S::off(16 * (rr >> 1) + 8 * (rr & 1) + 4 * hi + (jj >> 2),
                            VOFF + wv * S::DVW + 16 * (g & 1) + 4 * (jj & 3) + 32 * ct);
  // partial-logit exchange slots: chunk u of lane l sits at u ^ ((l >> 2) & 3)
  const int xsw = (lane >> 2) & 3;
  __builtin_amdgcn_s_waitcnt(0x0F70);  // queries are in registers before the loop
  __syncthreads();                     // pointer table ready

  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)&sK[0][0];
  // Source addresses of this wave's copies of the next tile to issue, read
  // from the pointer table one phase ahead of the copies.  Rows past the
  // split's end re-read its last key (finite data, probability forced to 0).
  //   own-copy layout: instruction k < 4 fills rows 8k..8k+7 of column group
  //   wv (lane = row-in-8 * 8 + slot); instruction 4 fills rows 4wv..4wv+3 of
  //   the rope group (lanes 0..31).  Slot s of row r holds logical chunk
  //   s ^ swz(r) of the group.
  //   row-major layout: instruction k fills physical chunk P = (wv + NW k)*64
  //   + lane, which holds logical chunk (P % CPR) ^ swz(row) of row P / CPR.
  const unsigned char *nsrc[S::NPW];
  auto load_srcs = [&](int tile) {
#pragma unroll
    for (int k = 0; k < S::NPW; ++k) {
      int r, c;
      if constexpr (S::OWN) {
        const int s8 = lane & 7;
        if (k < S::NPW - 1) {
          r = 8 * k + (lane >> 3);
          c = 8 * wv + (s8 ^ S::swz(r));
        } else {
          r = 4 * wv + ((lane & 31) >> 3);
          c = 8 * NW + (s8 ^ S::swz(r));
        }
      } else {
        const int P = (wv + NW * k) * 64 + lane;
        r = P / S::CPR;
        c = (P - r * S::CPR) ^ S::swz(r);
      }
      const int t = std::min(tile * kKT + r, nkeys - 1);
      nsrc[k] = reinterpret_cast<const unsigned char *>(sPtr[t]) + c * 16;
    }
  };
  auto issue_tile = [&](int buf) {
#pragma unroll
    for (int k = 0; k < S::NPW; ++k) {
      if constexpr (S::OWN) {
        if (k < S::NPW - 1)
          dma16(nsrc[k], lds_base + buf * S::TILE_BYTES + wv * S::GROUP_BYTES + k * 1024);
        else if (lane < 32)
          dma16(nsrc[k], lds_base + buf * S::TILE_BYTES + NW * S::GROUP_BYTES + wv * 512);
      } else {
        const int ins = wv + NW * k;
        if (S::NINS % NW == 0 || ins < S::NINS) dma16(nsrc[k], lds_base + buf * S::TILE_BYTES + ins * 1024);
      }
    }
  };
  // vmcnt bound that leaves this wave's copies of the newest tile in flight
  const bool full_share = S::OWN || S::NINS % NW == 0 || wv + NW * (S::NPW - 1) < S::NINS;

  f32x16 acc_o[HT][S::CT];
  float m_ref = -INFINITY, m_seen = -INFINITY, l_run = 0.f;
  const float sl2 = d.scale * kLog2e;

  // Softmax reference: each head's probabilities are exp2(s*scale*log2e - m_ref)
  // with m_ref fixed for the whole split (the first tile's maximum), so the
  // output accumulators are never rescaled inside the loop.  Probabilities may
  // reach 2^64 (exact in the float32 sums, relative precision kept in bf16).
  // If, at the end of the split, some head saw a logit more than 64 above its
  // reference, the workgroup runs the split again from the largest logit
  // seen (one verdict per attempt, at most kMaxRestarts).
  //
  // Work split of one tile: every wave of a head tile computes a partial S^T
  // over its k-steps; wave `part` then owns key rows 8 part + 4 hi + 0..3 (its
  // quarter of the C-layout registers): it adds the four partials of that
  // quarter in part order, exponentiates, and publishes the bf16 probabilities.
  // The P V contraction of every wave reads all four quarters as its B operand.
  constexpr float kSlack = 64.0f;
  constexpr int kMaxRestarts = 8;

  // Logits of tile `it` (buffer it % 3): this wave's partial S^T, published for the reduce-scatter.
  auto qk_tile = [&](int it) {
    const unsigned char *kt = sK[it % NBUF];
    bf16x8 a[S::KSP];
#pragma unroll
    for (int m = 0; m < S::KSP; ++m) a[m] = *reinterpret_cast<const bf16x8 *>(kt + aoff + S::KSTRIDE * m);
    f32x16 sacc = f32x16{};
#pragma unroll
    for (int m = 0; m < S::KSP; ++m) sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[m], qf[m], sacc, 0, 0, 0);
    // schedule: key reads kept four ahead of the products
    constexpr int kAhead = S::KSP < 4 ? S::KSP : 4;
    __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
    for (int r = 0; r < S::KSP - kAhead; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);
    float4 *mine = reinterpret_cast<float4 *>(&sX[ht][part][lane][0]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      mine[u ^ xsw] = make_float4(sacc[4 * u], sacc[4 * u + 1], sacc[4 * u + 2], sacc[4 * u + 3]);
  };
  // Probabilities of tile `it` for this wave's quarter (key rows 8 part + 4 hi + 0..3):
  // sum the four partials in part order, exponentiate against the reference,
  // publish bf16 P and the overflow flag.
  auto softmax_tile = [&](int it, bool set_ref) {
    float4 t4[S::NP];
#pragma unroll
    for (int p = 0; p < S::NP; ++p) t4[p] = reinterpret_cast<const float4 *>(&sX[ht][p][lane][0])[part ^ xsw];
    __builtin_amdgcn_sched_group_barrier(0x100, S::NP, 0);  // the partials in flight together
    float4 s4 = t4[0];
#pragma unroll
    for (int p = 1; p < S::NP; ++p) {
      s4.x += t4[p].x;
      s4.y += t4[p].y;
      s4.z += t4[p].z;
      s4.w += t4[p].w;
    }
    float sv[4] = {s4.x, s4.y, s4.z, s4.w};
    const int nvalid = nkeys - it * kKT;
    if (nvalid < kKT) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (8 * part + 4 * hi + r >= nvalid) sv[r] = -INFINITY;
    }
    const float mloc = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])) * sl2;  // this lane's four rows
    m_seen = fmaxf(m_seen, mloc);
    if (set_ref) {  // the reference is the first tile's maximum over all four quarters
      const float mh = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
      if (hi == 0) sMx[ht][part][l32] = mh;
      lds_barrier();
      m_ref = fmaxf(fmaxf(sMx[ht][0][l32], sMx[ht][1][l32]), fmaxf(sMx[ht][2][l32], sMx[ht][3][l32]));
    }
    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[0], sl2, -m_ref));
    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[1], sl2, -m_ref));
    const float p2 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[2], sl2, -m_ref));
    const float p3 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[3], sl2, -m_ref));
    l_run += (p0 + p1) + (p2 + p3);
    uint2 pq;
    pq.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p0, p1}, bf16x2));
    pq.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p2, p3}, bf16x2));
    sP[ht][part][lane] = pq;
  };
  // O^T += V^T P^T for tile `it`, this wave's value channels, every head tile.
  // k-step ks covers key rows {16ks + 4hi + 0..3} (quarter 2ks) and
  // {16ks + 8 + 4hi + 0..3} (quarter 2ks+1).
  auto pv_tile = [&](int it) {
    const unsigned char *kt = sK[it % NBUF];
#pragma unroll
    for (int ks = 0; ks < kKT / 16; ++ks) {
      bf16x8 pb[HT];
#pragma unroll
      for (int t = 0; t < HT; ++t) {
        const uint2 lo = sP[t][2 * ks][lane], hq = sP[t][2 * ks + 1][lane];
        pb[t] = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hq.x, hq.y));
      }
#pragma unroll
      for (int ct = 0; ct < S::CT; ++ct) {
        const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(kt + voff[2 * ks][ct]));
        const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(kt + voff[2 * ks + 1][ct]));
        const bf16x8 va = __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){
                                                         v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]});
#pragma unroll
        for (int t = 0; t < HT; ++t)
          acc_o[t][ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[t], acc_o[t][ct], 0, 0, 0);
      }
    }
  };
  // Y phase of tile t: copy of tile t+2 into the buffer of tile t-1 (read by
  // every wave before this phase), then, after the probabilities, the wait
  // for tile t+1.
  auto issue_next = [&](int t) {
    if constexpr (!S::OWN)
      if (t + 2 < ntiles) issue_tile((t + 2) % NBUF);
  };
  auto wait_next = [&](int t) {
    if (t + 2 < ntiles) {
      if (full_share)
        vm_wait<S::NPW>();
      else
        vm_wait<S::NPW - 1>();
    } else {
      vm_wait<0>();
    }
  };

  // Software pipeline over tiles, two barriers per tile:
  //   X(t): P V of tile t and the logits of tile t+1 (independent MFMA chains)
  //   Y(t+1): probabilities of tile t+1, copy of tile t+3, wait for tile t+2
  // Tiles t and t+1 are resident during X(t); tile t+2 is in flight.
  for (int attempt = 0;; ++attempt) {
#pragma unroll
    for (int t = 0; t < HT; ++t)
#pragma unroll
      for (int ct = 0; ct < S::CT; ++ct) acc_o[t][ct] = f32x16{};
    l_run = 0.f;
    const bool first = attempt == 0;
    bool restart = false;
    load_srcs(0);
    issue_tile(0);
    if (ntiles > 1) {
      load_srcs(1);
      issue_tile(1);
    }
    if (ntiles > 2) load_srcs(2);
    if constexpr (S::OWN) {  // tile 2 goes into the third buffer at once
      if (ntiles > 2) issue_tile(2);
      wait_next(0);
    } else {
      vm_wait<0>();
    }
    __syncthreads();
    qk_tile(0);
    lds_barrier();
    issue_next(0);
    softmax_tile(0, first);
    wait_next(0);
    lds_barrier();

    for (int it = 0; it < ntiles; ++it) {
      const bool more = it + 1 < ntiles;
      // X phase: logits of tile it+1 first (their partials are published at
      // the end of the phase), then P V of tile it, whose products may still
      // be in the matrix pipeline during the next phase.
      if (it + 3 < ntiles) load_srcs(it + 3);  // copied in this phase (own copy) or the next
      if (more) qk_tile(it + 1);
      pv_tile(it);
      if constexpr (S::OWN) {  // this wave's reads of tile it are done: its groups of tile it+3 go there
        if (it + 3 < ntiles) issue_tile(it % NBUF);
      }
      if (!more) break;
      lds_barrier();
      issue_next(it + 1);
      softmax_tile(it + 1, false);
      wait_next(it + 1);
      lds_barrier();
    }
    // One verdict per attempt: the largest logit each head saw, over its four
    // quarters; any head more than kSlack above its reference runs the split
    // again from that maximum.
    vm_wait<0>();
    __syncthreads();
    const float ms = fmaxf(m_seen, __shfl_xor(m_seen, 32, 64));
    if (hi == 0) sMx[ht][part][l32] = ms;
    __syncthreads();
    const float seen = fmaxf(fmaxf(sMx[ht][0][l32], sMx[ht][1][l32]), fmaxf(sMx[ht][2][l32], sMx[ht][3][l32]));
    const bool over = __any(seen > m_ref + kSlack);  // the whole wave votes (not inside the lane-0 branch)
    if (lane == 0) sFlag[wv] = over ? 1 : 0;
    __syncthreads();
    int anyf = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) anyf |= sFlag[w];
    restart = anyf != 0 && attempt < kMaxRestarts;
    __syncthreads();
    if (!restart) break;
    m_ref = seen;
  }
  // Row sums and references per head tile: wave (ht, part) holds the sum over
  // its key quarter for head ht*32 + l32 (halves combined across hi).
  l_run += __shfl_xor(l_run, 32, 64);
  __syncthreads();
  if (hi == 0) {
    sMx[ht][part][l32] = l_run;
    sRef[ht][l32] = m_ref;  // identical across the parts of a head tile
  }
  __syncthreads();
  float lsum[HT], mref[HT];
#pragma unroll
  for (int t = 0; t < HT; ++t) {
    lsum[t] = (sMx[t][0][l32] + sMx[t][1][l32]) + (sMx[t][2][l32] + sMx[t][3][l32]);
    mref[t] = sRef[t][l32];
  }

  // epilogue: lane holds, per head tile t, head t*32 + l32 and value rows
  // wv*DVW + 32ct + 8(j/4) + 4hi + (j%4)
  const bool single = n_keys <= chunk;
#pragma unroll
  for (int t = 0; t < HT; ++t) {
    const int h = t * 32 + l32;
    if (h >= d.H) continue;
    const float inv = single ? 1.0f / lsum[t] : 1.0f;
#pragma unroll
    for (int ct = 0; ct < S::CT; ++ct)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int col = wv * S::DVW + 32 * ct + 8 * jq + 4 * hi;
        const float v0 = acc_o[t][ct][4 * jq] * inv, v1 = acc_o[t][ct][4 * jq + 1] * inv;
        const float v2 = acc_o[t][ct][4 * jq + 2] * inv, v3 = acc_o[t][ct][4 * jq + 3] * inv;
        if (single) {
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v0, v1}, bf16x2));
          w.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v2, v3}, bf16x2));
          *reinterpret_cast<uint2 *>(out + (node * d.H + h) * DV + col) = w;
        } else {
          *reinterpret_cast<float4 *>(part_o + (((node * splits) + split) * d.H + h) * DV + col) =
              make_float4(v0, v1, v2, v3);
        }
      }
    if (wv == 0 && hi == 0) {
      if (single) {
        if (lse) lse[node * d.H + h] = (mref[t] + __log2f(lsum[t])) * kLn2;
      } else {
        part_ml[(((node * splits) + split) * d.H + h) * 2 + 0] = mref[t];
        part_ml[(((node * splits) + split) * d.H + h) * 2 + 1] = lsum[t];
      }
    }
  }
}

// Merge the partials of nodes whose keys spanned several splits.  One
// wavefront per (node, head, 64 CPL value channels), CPL = 4 for 512 value
// channels (two wavefronts a head) and 2 for 128.  Lane s first holds split
// s's running maximum and sum (64 splits at a time), so the merged maximum m
// and sum l are wavefront reductions; split s then weighs exp2(m_s - m) / l
// and the lane's CPL channels of every split's partial are summed in split
// order, kBatch splits' loads in flight at a time (4, 8 or 16: the plan's
// split count rounded up, so that a few splits cost few registers).
template <int DV, int kBatch>
__global__ void __launch_bounds__(256) combine_kernel(tv_dims d, const int32_t *__restrict__ row_status,
                                                      const int32_t *__restrict__ nkeys_tab, int chunk, int splits,
                                                      const float *__restrict__ part_o,
                                                      const float *__restrict__ part_ml, uint16_t *__restrict__ out,
                                                      float *__restrict__ lse) {
  constexpr int kCPL = DV == 512 ? 4 : 2;  // value channels per lane
  constexpr int kWPH = DV / (64 * kCPL);   // wavefronts per head
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (node, head, part)
  const int part = (int)(wid % kWPH);
  const int64_t nh = wid / kWPH;
  const int h = (int)(nh % d.H);
  const int64_t node = nh / d.H;
  if (node >= (int64_t)d.B * d.D) return;
  const int b = (int)(node / d.D);
  const float2 *ml = reinterpret_cast<const float2 *>(part_ml) + node * splits * d.H + h;  // split s at s * H
  const int c0 = (part * 64 + lane) * kCPL;  // first value channel of the lane
  const float *po = part_o + (node * splits * d.H + h) * DV + c0;
  const int64_t pstride = (int64_t)d.H * DV;  // next split, same head and channels
  // One round trip for the row state, the first 64 splits' (maximum, sum)
  // (lane s holds split s's) and the first kBatch splits' partials; splits
  // the node does not use are dropped once its key count is known.
  const int32_t status = row_status[b];
  const int n_keys = nkeys_tab[node];
  const float2 ml0 = lane < splits ? ml[(int64_t)lane * d.H] : make_float2(-INFINITY, 0.f);
  float o[kBatch][kCPL];
  auto load_batch = [&](int s_first, int n_valid) {
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      if (k >= n_valid) {  // the same in every lane
#pragma unroll
        for (int c = 0; c < kCPL; ++c) o[k][c] = 0.f;
        continue;
      }
      const float *src = po + (int64_t)(s_first + k) * pstride;
      if constexpr (kCPL == 4) {
        const float4 v = *reinterpret_cast<const float4 *>(src);
        o[k][0] = v.x;
        o[k][1] = v.y;
        o[k][2] = v.z;
        o[k][3] = v.w;
      } else {
        const float2 v = *reinterpret_cast<const float2 *>(src);
        o[k][0] = v.x;
        o[k][1] = v.y;
      }
    }
  };
  load_batch(0, std::min(kBatch, splits));
  if (status != TV_ROW_OK) return;
  if (n_keys <= chunk) return;  // written by its only split
  const int used = (n_keys + chunk - 1) / chunk;
#pragma unroll
  for (int k = 0; k < kBatch; ++k)  // the prefetched partials of splits past `used` hold anything
    if (k >= used)
#pragma unroll
      for (int c = 0; c < kCPL; ++c) o[k][c] = 0.f;
  auto ml_at = [&](int s0) {  // lane's split s0 + lane, past `used`: (-inf, 0)
    if (s0 + lane >= used) return make_float2(-INFINITY, 0.f);
    return s0 == 0 ? ml0 : ml[(int64_t)(s0 + lane) * d.H];
  };
  float mx = -INFINITY;
  for (int s0 = 0; s0 < used; s0 += 64) mx = fmaxf(mx, ml_at(s0).x);
#pragma unroll
  for (int o_ = 32; o_ > 0; o_ >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o_, 64));
  float l = 0.f;
  for (int s0 = 0; s0 < used; s0 += 64) {
    const float2 v = ml_at(s0);
    float t = s0 + lane < used ? exp2f(v.x - mx) * v.y : 0.f;
#pragma unroll
    for (int o_ = 32; o_ > 0; o_ >>= 1) t += __shfl_xor(t, o_, 64);
    l += t;
  }
  const float inv_l = 1.0f / l;
  float acc[kCPL] = {};
  for (int s0 = 0; s0 < used; s0 += 64) {
    const float2 v = ml_at(s0);
    const float w = s0 + lane < used ? exp2f(v.x - mx) * inv_l : 0.f;  // lane j: weight of split s0 + j
    const int n = std::min(64, used - s0);
    for (int k0 = 0; k0 < n; k0 += kBatch) {
      if (s0 + k0 > 0) load_batch(s0 + k0, std::min(kBatch, n - k0));
#pragma unroll
      for (int k = 0; k < kBatch; ++k) {
        const float wk = k0 + k < n ? __shfl(w, k0 + k, 64) : 0.f;
#pragma unroll
        for (int c = 0; c < kCPL; ++c) acc[c] += wk * o[k][c];
      }
    }
  }
  uint16_t *dst = out + (node * d.H + h) * DV + c0;
  if constexpr (kCPL == 4) {
    uint2 packed;
    packed.x = uint32_t(f2bf(acc[0])) | (uint32_t(f2bf(acc[1])) << 16);
    packed.y = uint32_t(f2bf(acc[2])) | (uint32_t(f2bf(acc[3])) << 16);
    *reinterpret_cast<uint2 *>(dst) = packed;
  } else {
    *reinterpret_cast<uint32_t *>(dst) = uint32_t(f2bf(acc[0])) | (uint32_t(f2bf(acc[1])) << 16);
  }
  if (part == 0 && lane == 0 && lse) lse[node * d.H + h] = (mx + __log2f(l)) * kLn2;
}

template <int NW, int HT, int DK, int DV, int VOFF, int DROW>
static hipError_t launch_attn_t(const tv_dims &d, const uint16_t *q, const int32_t *row_status,
                                const int32_t *row_order, const uint16_t *const *keytab, const int32_t *nkeys,
                                const SplitPlan &plan, float *part_o, float *part_ml, uint16_t *out, float *lse,
                                hipStream_t s) {
  if (plan.chunk > kMaxChunk) return hipErrorInvalidValue;
  const int64_t grid = attn_grid(d, plan);
  attn_kernel<NW, HT, DK, DV, VOFF, DROW><<<dim3((unsigned)grid), NW * 64, 0, s>>>(
      d, q, row_status, row_order, keytab, plan.max_keys, nkeys, plan.chunk, plan.splits, part_o, part_ml, out, lse);
  return hipGetLastError();
}

hipError_t launch_attn(const tv_dims &d, const uint16_t *q, const int32_t *row_status, const int32_t *row_order,
                       const uint16_t *const *keytab, const int32_t *nkeys, const SplitPlan &plan, float *part_o,
                       float *part_ml, uint16_t *out, float *lse, hipStream_t s) {
  if (d.H == 64 && d.d_k == 576 && d.d_v == 512 && d.v_off == 0 && d.d_row == 576)
    return launch_attn_mla(d, q, row_status, row_order, keytab, nkeys, plan, part_o, part_ml, out, lse, s);
  if (d.H == 8 && d.d_k == 128 && d.d_v == 128 && d.v_off == 128 && d.d_row == 256)
    return launch_attn_t<4, 1, 128, 128, 128, 256>(d, q, row_status, row_order, keytab, nkeys, plan, part_o,
                                                   part_ml, out, lse, s);
  return hipErrorInvalidValue;
}

hipError_t launch_combine(const tv_dims &d, const int32_t *row_status, const int32_t *nkeys, const SplitPlan &plan,
                          const float *part_o, const float *part_ml, uint16_t *out, float *lse, hipStream_t s) {
  if (plan.splits <= 1) return hipSuccess;
  const int64_t waves = (int64_t)d.B * d.D * d.H * (d.d_v == 512 ? 2 : 1);
  dim3 grid((unsigned)((waves + 3) / 4));
  auto go = [&](auto kernel) {
    kernel<<<grid, 256, 0, s>>>(d, row_status, nkeys, plan.chunk, plan.splits, part_o, part_ml, out, lse);
  };
  const bool wide = d.d_v == 512;
  if (plan.splits <= 4)
    wide ? go(combine_kernel<512, 4>) : go(combine_kernel<128, 4>);
  else if (plan.splits <= 8)
    wide ? go(combine_kernel<512, 8>) : go(combine_kernel<128, 8>);
  else
    wide ? go(combine_kernel<512, 16>) : go(combine_kernel<128, 16>);
  return hipGetLastError();
}

}  // namespace tv
