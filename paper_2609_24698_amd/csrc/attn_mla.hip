// Branch-aware verify attention for the shared-latent shape: 64 query heads
// over one 576-wide latent row per key; keys are the whole row, values its
// first 512 channels.
//
// One workgroup (8 wavefronts, two per SIMD) takes one (row, node, key
// split).  A 32-key tile is gathered once into LDS (direct global->LDS
// copies) and feeds two contractions on MFMA, float32 accumulation:
//   S^T = K Q^T     keys x heads, v_mfma_f32_16x16x32_bf16.  Wave (head
//                   quarter hq, key half kh) computes the complete logits of
//                   heads 16hq..16hq+15 against keys 16kh..16kh+15 over all
//                   576 channels (its queries stay in registers), so no
//                   partial logits cross LDS.  It exponentiates them in
//                   registers against a fixed per-head reference and
//                   publishes bf16 P.
//   O^T += V^T P^T  value channels x heads, v_mfma_f32_32x32x16_bf16.  Wave w
//                   owns value channels 64w..64w+63 for all heads; V^T comes
//                   from the LDS transpose read (ds_read_b64_tr_b16), each
//                   value element once per tile.
// The tile is stored group-major: column group g (64 channels, 128 bytes) of
// all 32 rows, then group g+1, the 16-byte chunk slot XOR-swizzled by row
// pair, which keeps both the logit reads (16 rows x one chunk) and the
// transpose reads free of bank conflicts.  Wave w reads only group w of a
// tile for its values, and every wave's logit reads of tile t end one barrier
// before tile t's values are read, so wave w copies group w of tile t+3 (and
// a quarter of the rope group, read by the logits only) into the buffer of
// tile t right after its own P V reads: two iterations of lead, no barrier.
//
// One barrier per tile: iteration t computes the logits and probabilities of
// tile t+1 and the P V of tile t.  The probabilities use a fixed reference
// per head (the first tile's maximum), so the output accumulators are never
// rescaled; a logit more than 64 (log2 units) above it restarts the split
// from the largest logit seen, at most kMaxRestarts times.
//
// A node whose keys fit one split writes its normalised output; otherwise each
// split writes an unnormalised partial (O, reference, sum) that the combine
// kernel merges.
#include "attn_common.h"

namespace tv {

namespace mla {

constexpr int kH = 64, kDK = 576, kDV = 512;
constexpr int kNW = 8, kNT = kNW * 64;
constexpr int kKS = kDK / 32;             // logit k-steps of 32 channels
constexpr int kGroups = kDK / 64;         // 128-byte column groups of a row (the last one: rope channels)
constexpr int kGB = kKT * 128;            // bytes of one column group of a tile
constexpr int kTB = kGroups * kGB;        // bytes of a tile
constexpr int kNBUF = 3;
constexpr int kNPW = kKT * 128 / 1024 + 1;  // copy instructions per wave and tile: its group, then a rope quarter
static_assert(kGroups == kNW + 1, "one value group per wave plus one rope group");
static_assert(kDV == 64 * kNW, "wave w owns value channels 64w..64w+63");

// 16-byte chunk slot of logical chunk `c` (0..7 within its group) in row r.
__device__ constexpr int slot(int r, int c) { return c ^ ((r >> 1) & 7); }
// Byte offset in a tile of channel `col` of row r.
__device__ constexpr int off(int r, int col) {
  return (col >> 6) * kGB + r * 128 + slot(r, (col >> 3) & 7) * 16 + (col & 7) * 2;
}

// P^T for the value contraction, per head a 64-byte row of the tile's 32 keys:
// key 16s + 8a + 4h + i (s, a, h in {0,1}, i < 4) sits at 16s + 8h + 4a + i,
// so the eight keys one lane of the value contraction needs (k-step s, lane
// half h: keys 16s + 4h + 0..3, then 16s + 8 + 4h + 0..3) are one 16-byte
// chunk; chunk slots are XOR-swizzled by head so a read of 32 heads spreads
// over all banks.
__device__ constexpr int p_off(int head, int chunk) { return head * 64 + ((chunk ^ ((head >> 2) & 3)) * 16); }

}  // namespace mla

__global__ void __launch_bounds__(mla::kNT, 1)
attn_mla_kernel(tv_dims d, const uint16_t *__restrict__ q, const int32_t *__restrict__ row_status,
                const int32_t *__restrict__ row_order, const uint16_t *const *__restrict__ keytab, int keytab_stride,
                const int32_t *__restrict__ nkeys_tab, int chunk, int splits, float *__restrict__ part_o,
                float *__restrict__ part_ml, uint16_t *__restrict__ out, float *__restrict__ lse) {
  using namespace mla;
  __shared__ __attribute__((aligned(1024))) unsigned char sK[kNBUF][kTB];
  __shared__ __attribute__((aligned(16))) unsigned char sP[2][kH * 64];
  __shared__ const uint16_t *sPtr[kMaxChunk];
  __shared__ int sFlag[2][kNW];
  __shared__ float sMx[2][kH];
  __shared__ float sRef[kH];

  int i, split;
  const int rank = unit_of(blockIdx.x, d.D, splits, i, split);
  if (rank >= d.B) return;
  const int b = row_order[rank];
  const int64_t node = (int64_t)b * d.D + i;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int hq = wv & 3, kh = wv >> 2;      // logit roles: head quarter, key half
  const int l16 = lane & 15, g4 = lane >> 4;
  const int l32 = lane & 31, hi = lane >> 5;
  const int head = 16 * hq + l16;           // this lane's head in the logit roles
  const int k0 = split * chunk;
  // Row status, key count, this thread's entries of the node's key table and
  // the queries are loaded together; the table loads come first so that
  // storing them waits for them only.
  const int32_t status = row_status[b];
  const int n_keys = nkeys_tab[node];
  constexpr int kPer = (kMaxChunk + kNT - 1) / kNT;
  const uint16_t *tp[kPer];
  {
    const uint16_t *const *tab = keytab + node * keytab_stride + k0;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int t = tid + kNT * u;
      tp[u] = (t < chunk && k0 + t < keytab_stride) ? tab[t] : nullptr;
    }
  }
  // Queries as the B operand of the logits: lane holds head `head`, channels
  // 32 ks + 8 g4 .. +7 of k-step ks.
  bf16x8 qf[kKS];
  {
    const uint16_t *qrow = q + (node * kH + head) * kDK + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(qrow + 32 * ks));
  }
  if (status != TV_ROW_OK || k0 >= n_keys) return;
  const int k1 = std::min(n_keys, k0 + chunk);
  const int nkeys = k1 - k0;
  const int ntiles = (nkeys + kKT - 1) / kKT;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int t = tid + kNT * u;
    if (t < nkeys) sPtr[t] = tp[u];
  }
  // Logit A operand: lane reads row 16 kh + l16, chunk 4 ks + g4, i.e. group
  // ks/2, logical chunk 4 (ks & 1) + g4 of that group.
  const int krow = 16 * kh + l16;
  const int kbase[2] = {krow * 128 + slot(krow, g4) * 16, krow * 128 + slot(krow, 4 + g4) * 16};
  // Value-operand offsets for the transpose reads: rows 16 ks + 8 s + 4 hi + jj/4,
  // columns 64 wv + 16 (g & 1) + 4 (jj & 3) + 32 ct.
  const int g = lane >> 4, jj = lane & 15;
  int voff[4][2];
#pragma unroll
  for (int rr = 0; rr < 4; ++rr)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
      voff[rr][ct] = off(16 * (rr >> 1) + 8 * (rr & 1) + 4 * hi + (jj >> 2), 64 * wv + 16 * (g & 1) + 4 * (jj & 3) + 32 * ct);
  // P^T writes of this lane: keys 16 kh + 4 g4 + 0..3 of head `head`
  const int pw = p_off(head, 2 * kh + (g4 & 1)) + (g4 >> 1) * 8;
  __builtin_amdgcn_s_waitcnt(0x0F70);  // queries are in registers before the loop
  __syncthreads();                     // pointer table ready

  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)&sK[0][0];
  // Source addresses of this wave's copies of a tile, read from the pointer
  // table one phase ahead of the copies.  Instruction k < 4 fills rows
  // 8k..8k+7 of group wv (lane = row-in-8 * 8 + slot); instruction 4 fills rows
  // 4wv..4wv+3 of the rope group (lanes 0..31).  Slot s of row r holds logical
  // chunk slot(r, s) of the group.  Rows past the split's end re-read its last
  // key (finite data; their probabilities are forced to 0).
  const unsigned char *nsrc[kNPW];
  auto load_srcs = [&](int tile) {
#pragma unroll
    for (int k = 0; k < kNPW; ++k) {
      const int s8 = lane & 7;
      int r, c;
      if (k < kNPW - 1) {
        r = 8 * k + (lane >> 3);
        c = 8 * wv + slot(r, s8);
      } else {
        r = 4 * wv + ((lane & 31) >> 3);
        c = 8 * kNW + slot(r, s8);
      }
      const int t = std::min(tile * kKT + r, nkeys - 1);
      nsrc[k] = reinterpret_cast<const unsigned char *>(sPtr[t]) + c * 16;
    }
  };
  auto issue_tile = [&](int buf) {
#pragma unroll
    for (int k = 0; k < kNPW; ++k) {
      if (k < kNPW - 1)
        dma16(nsrc[k], lds_base + buf * kTB + wv * kGB + k * 1024);
      else if (lane < 32)
        dma16(nsrc[k], lds_base + buf * kTB + kNW * kGB + wv * 512);
    }
  };

  f32x16 acc_o[2][2];
  float m_ref = -INFINITY, m_seen = -INFINITY, l_run = 0.f;
  const float sl2 = d.scale * kLog2e;
  constexpr float kSlack = 64.0f;
  constexpr int kMaxRestarts = 8;

  // Complete logits of this wave's 16 keys x 16 heads of tile `it`, two
  // accumulator chains (even and odd k-steps), key reads kept four ahead.
  auto qk_tile = [&](int it) {
    const unsigned char *kt = sK[it % kNBUF];
    f32x4 s0 = f32x4{}, s1 = f32x4{};
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kt + (ks >> 1) * kGB + kbase[ks & 1]);
      if (ks & 1)
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], s1, 0, 0, 0);
      else
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], s0, 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int r = 0; r < kKS - 4; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    return f32x4{s0[0] + s1[0], s0[1] + s1[1], s0[2] + s1[2], s0[3] + s1[3]};
  };
  // Lane holds keys 16 kh + 4 g4 + 0..3 of head `head`; keys past the split are -inf.
  auto masked = [&](int it, f32x4 s) {
    const int nvalid = nkeys - it * kKT;
    float sv[4] = {s[0], s[1], s[2], s[3]};
    if (nvalid < kKT) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (16 * kh + 4 * g4 + r >= nvalid) sv[r] = -INFINITY;
    }
    return f32x4{sv[0], sv[1], sv[2], sv[3]};
  };
  // Probabilities against the reference, published as bf16 P^T with the
  // overflow flag of this wave.
  auto softmax_tile = [&](int it, f32x4 sv) {
    const float mloc = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])) * sl2;
    m_seen = fmaxf(m_seen, mloc);
    const bool over = mloc > m_ref + kSlack;
    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[0], sl2, -m_ref));
    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[1], sl2, -m_ref));
    const float p2 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[2], sl2, -m_ref));
    const float p3 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[3], sl2, -m_ref));
    l_run += (p0 + p1) + (p2 + p3);
    uint2 pq;
    pq.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p0, p1}, bf16x2));
    pq.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p2, p3}, bf16x2));
    *reinterpret_cast<uint2 *>(&sP[it & 1][pw]) = pq;
    const bool anyo = __any(over);
    if (lane == 0) sFlag[it & 1][wv] = anyo ? 1 : 0;
  };
  // O^T += V^T P^T for tile `it`, this wave's value channels, both head tiles.
  auto pv_tile = [&](int it) {
    const unsigned char *kt = sK[it % kNBUF];
    const unsigned char *pt = sP[it & 1];
#pragma unroll
    for (int ks = 0; ks < kKT / 16; ++ks) {
      bf16x8 pb[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) pb[t] = *reinterpret_cast<const bf16x8 *>(pt + p_off(32 * t + l32, 2 * ks + hi));
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(kt + voff[2 * ks][ct]));
        const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(kt + voff[2 * ks + 1][ct]));
        const bf16x8 va = __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){
                                                         v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]});
#pragma unroll
        for (int t = 0; t < 2; ++t)
          acc_o[t][ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[t], acc_o[t][ct], 0, 0, 0);
      }
    }
  };
  // the largest of v over the lanes holding this lane's head (same l16), then
  // over the two key halves through LDS; every lane gets its head's value
  auto head_max = [&](float v) {
    v = fmaxf(v, __shfl_xor(v, 16, 64));
    v = fmaxf(v, __shfl_xor(v, 32, 64));
    if (g4 == 0) sMx[kh][head] = v;
    lds_barrier();
    return fmaxf(sMx[0][head], sMx[1][head]);
  };

  for (int attempt = 0;; ++attempt) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) acc_o[t][ct] = f32x16{};
    l_run = 0.f;
    bool restart = false;
    // tiles 0, 1, 2 into buffers 0, 1, 2; wait for tile 0
    load_srcs(0);
    issue_tile(0);
    if (ntiles > 1) {
      load_srcs(1);
      issue_tile(1);
    }
    if (ntiles > 2) {
      load_srcs(2);
      issue_tile(2);
      vm_wait<2 * kNPW>();
    } else if (ntiles > 1) {
      vm_wait<kNPW>();
    } else {
      vm_wait<0>();
    }
    __syncthreads();
    const f32x4 s_first = masked(0, qk_tile(0));
    if (attempt == 0)  // the reference: the first tile's maximum per head
      m_ref = head_max(fmaxf(fmaxf(s_first[0], s_first[1]), fmaxf(s_first[2], s_first[3])) * sl2);
    softmax_tile(0, s_first);
    if (ntiles > 2)
      vm_wait<kNPW>();
    else
      vm_wait<0>();
    lds_barrier();

    for (int it = 0; it < ntiles; ++it) {
      const bool more = it + 1 < ntiles;
      int anyf = 0;  // overflow flags of the probabilities of tile it
#pragma unroll
      for (int w = 0; w < kNW; ++w) anyf |= sFlag[it & 1][w];
      if (it + 3 < ntiles) load_srcs(it + 3);
      if (more) softmax_tile(it + 1, masked(it + 1, qk_tile(it + 1)));
      pv_tile(it);
      if (anyf) {  // probabilities of tile it overflowed the reference
        restart = attempt < kMaxRestarts;
        if (restart) break;
      }
      if (it + 3 < ntiles) issue_tile(it % kNBUF);  // this wave's reads of buffer it % 3 are done
      if (!more) break;
      // this wave's copies of tile it+2 have landed (those of tile it+3 may still fly)
      if (it + 3 < ntiles)
        vm_wait<kNPW>();
      else
        vm_wait<0>();
      lds_barrier();
    }
    if (!restart) break;
    // restart from the largest logit any lane has seen, per head
    vm_wait<0>();
    __syncthreads();
    m_ref = head_max(m_seen);
    __syncthreads();
  }

  // Row sums per head: the four lanes of a head in a wave (fixed order), then
  // the two key halves; references per head.
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  __syncthreads();
  if (g4 == 0) {
    sMx[kh][head] = l_run;
    if (kh == 0) sRef[head] = m_ref;
  }
  __syncthreads();
  float lsum[2], mref[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    lsum[t] = sMx[0][32 * t + l32] + sMx[1][32 * t + l32];
    mref[t] = sRef[32 * t + l32];
  }

  // epilogue: lane holds, per head tile t, head 32t + l32 and value rows
  // 64wv + 32ct + 8(j/4) + 4hi + (j%4)
  const bool single = n_keys <= chunk;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int h = t * 32 + l32;
    const float inv = single ? 1.0f / lsum[t] : 1.0f;
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int col = wv * 64 + 32 * ct + 8 * jq + 4 * hi;
        const float v0 = acc_o[t][ct][4 * jq] * inv, v1 = acc_o[t][ct][4 * jq + 1] * inv;
        const float v2 = acc_o[t][ct][4 * jq + 2] * inv, v3 = acc_o[t][ct][4 * jq + 3] * inv;
        if (single) {
          uint2 w;
          w.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v0, v1}, bf16x2));
          w.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v2, v3}, bf16x2));
          *reinterpret_cast<uint2 *>(out + (node * kH + h) * kDV + col) = w;
        } else {
          *reinterpret_cast<float4 *>(part_o + (((node * splits) + split) * kH + h) * kDV + col) =
              make_float4(v0, v1, v2, v3);
        }
      }
    if (wv == 0 && hi == 0) {
      if (single) {
        if (lse) lse[node * kH + h] = (mref[t] + __log2f(lsum[t])) * kLn2;
      } else {
        part_ml[(((node * splits) + split) * kH + h) * 2 + 0] = mref[t];
        part_ml[(((node * splits) + split) * kH + h) * 2 + 1] = lsum[t];
      }
    }
  }
}

hipError_t launch_attn_mla(const tv_dims &d, const uint16_t *q, const int32_t *row_status, const int32_t *row_order,
                           const uint16_t *const *keytab, const int32_t *nkeys, const SplitPlan &plan, float *part_o,
                           float *part_ml, uint16_t *out, float *lse, hipStream_t s) {
  if (plan.chunk > kMaxChunk || d.H != mla::kH || d.d_k != mla::kDK || d.d_v != mla::kDV || d.v_off != 0 ||
      d.d_row != mla::kDK)
    return hipErrorInvalidValue;
  const int64_t grid = (int64_t)((d.B + 7) / 8) * 8 * d.D * plan.splits;
  attn_mla_kernel<<<dim3((unsigned)grid), mla::kNT, 0, s>>>(d, q, row_status, row_order, keytab, plan.max_keys, nkeys,
                                                           plan.chunk, plan.splits, part_o, part_ml, out, lse);
  return hipGetLastError();
}

}  // namespace tv
