// Branch-aware verify attention for the shared-latent shape: 64 query heads
// over one 576-wide latent row per key; keys are the whole row, values its
// first 512 channels.
//
// One workgroup (8 wavefronts) takes one (row, node, key split).  Wavefronts
// w and w+4 share a SIMD, and w0..w3 occupy the four SIMDs, so the roles are:
//   w0, w1  logit waves: S^T = K Q^T for 32 keys x 32 heads (head half w)
//           over all 576 channels on v_mfma_f32_32x32x16_bf16, the queries of
//           their 32 heads held in registers; they exponentiate against a
//           fixed per-head reference and publish bf16 P^T.
//   w2, w3, w6, w7  value waves: O^T += V^T P^T, 128 value channels each for
//           all 64 heads (32x32x16, V^T from the LDS transpose read).
//   w4, w5  copy waves: gather the key rows of tile t+3 into LDS with direct
//           global->LDS copies (w4 also copies the key-pointer table of tile
//           t+6), so a tile lands two iterations before its logits.
// Per tile a logit SIMD issues 36 products and a value SIMD 32; nothing is
// recomputed and no partial logits cross LDS.
//
// Iteration it (one barrier each, it = -1 .. T-1) computes the logits and
// probabilities of tile it+1 and the P V of tile it.  K tiles live in four
// LDS buffers (tile u in buffer u % 4), stored group-major: column group g
// (64 channels, 128 bytes) of all 32 rows, then group g+1, the 16-byte chunk
// slot XOR-swizzled per row (slot()) so that both the logit reads (32 rows x
// one chunk, 16-byte reads) and the value transpose reads (8 rows x four
// chunks) are free of bank conflicts.
//
// The probabilities use a fixed reference per head (the first tile's
// maximum), so the output accumulators are never rescaled; if any logit of
// the split ends up more than 64 (log2 units) above it, the split runs again
// from the largest logit seen, at most kMaxRestarts times.  Each head's
// probability sum is the product of P^T with a value operand of ones (one
// value wave, four products per tile), so the sums cover exactly the bf16
// probabilities the value contraction uses.  A node whose keys fit one split writes its
// normalised output; otherwise each split writes an unnormalised partial
// (O, reference, sum) that the combine kernel merges.
#include "attn_common.h"

namespace tv {

namespace mla {

constexpr int kH = 64, kDK = 576, kDV = 512;
constexpr int kNW = 8, kNT = kNW * 64;
constexpr int kKS = kDK / 16;             // logit k-steps of 16 channels
constexpr int kGroups = kDK / 64;         // 128-byte column groups of a row (the last one: rope channels)
constexpr int kGB = kKT * 128;            // bytes of one column group of a tile
constexpr int kTB = kGroups * kGB;        // bytes of a tile
constexpr int kNBUF = 4;                  // K tile buffers
constexpr int kPSlots = 8;                // key-pointer table slots (one tile each)
// Column groups each wave copies: w4 groups 0..2, w5 3..5, w3 6..7, w2 8 (the
// rope group); the value waves w2, w3 have the most idle time per tile.
constexpr float kSlack = 64.0f;
constexpr int kMaxRestarts = 8;
static_assert(kDV == 128 * 4, "four value waves of 128 channels");
static_assert(kGroups == 9, "eight value groups and one rope group");

// 16-byte chunk slot of logical chunk `c` (0..7 within its group) in row r.
// Chosen by measurement (the LDS bank-conflict counter on gfx950, seven
// swizzles of these two access patterns): the 16-byte reads were free of
// conflicts when rows of one parity within 16 rows took distinct XOR values,
// the 8-byte transpose reads when rows r and r + 2 of each group of four fell
// in different 64-byte halves (bit 2).  This XOR (bit 1 of r into bit 2, bits
// 2-3 of r into bits 0-1) was free of conflicts for both; XOR by the row pair
// alone left the transpose reads 2-way conflicted.
__device__ constexpr int slot(int r, int c) { return c ^ ((((r >> 1) & 1) << 2) | ((r >> 2) & 3)); }
// Byte offset in a tile of channel `col` of row r.
__device__ constexpr int off(int r, int col) {
  return (col >> 6) * kGB + r * 128 + slot(r, (col >> 3) & 7) * 16 + (col & 7) * 2;
}

// P^T for the value contraction, per head a 64-byte row of the tile's 32 keys:
// key 16s + 8a + 4h + i (s, a, h in {0,1}, i < 4) sits at 16s + 8h + 4a + i,
// so the eight keys one lane of the value contraction needs (k-step s, lane
// half h: keys 16s + 4h + 0..3, then 16s + 8 + 4h + 0..3) are one 16-byte
// chunk, and so are the eight logits one lane of the logit product holds for
// that k-step.  Chunk slots are XOR-swizzled by head so that a read or write
// of 32 heads spreads over all banks.
__device__ constexpr int p_off(int head, int chunk) { return head * 64 + ((chunk ^ ((head >> 2) & 3)) * 16); }

}  // namespace mla

// Direct global -> LDS copy of 4 bytes per lane (global_load_lds_dword): lane
// l's 4 bytes land at LDS byte address lds + 4 l.  Same protocol as dma16.
__device__ __forceinline__ void dma4(const void *g, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds)));
}

// Wait until at most n of this wavefront's vector-memory operations are in
// flight (n is one of the counts a copy wave issues per iteration).
__device__ __forceinline__ void vm_wait_n(int n) {
  switch (n) {
    case 0: vm_wait<0>(); break;
    case 1: vm_wait<1>(); break;
    case 4: vm_wait<4>(); break;
    case 8: vm_wait<8>(); break;
    case 12: vm_wait<12>(); break;
    case 13: vm_wait<13>(); break;
    default: vm_wait<0>(); break;
  }
}

__global__ void __launch_bounds__(mla::kNT, 1)
attn_mla_kernel(tv_dims d, const uint16_t *__restrict__ q, const int32_t *__restrict__ row_status,
                const int32_t *__restrict__ row_order, const uint16_t *const *__restrict__ keytab, int keytab_stride,
                const int32_t *__restrict__ nkeys_tab, int chunk, int splits, float *__restrict__ part_o,
                float *__restrict__ part_ml, uint16_t *__restrict__ out, float *__restrict__ lse) {
  using namespace mla;
  __shared__ __attribute__((aligned(1024))) unsigned char sK[kNBUF][kTB];
  __shared__ __attribute__((aligned(16))) unsigned char sP[2][kH * 64];
  __shared__ __attribute__((aligned(16))) const uint16_t *sPtr[kPSlots][kKT];
  __shared__ int sOver[2];
  __shared__ float sSum[kH];

  int i, split;
  const int rank = unit_of(blockIdx.x, d.B, d.D, splits, i, split);
  if (rank >= d.B) return;
  const int64_t rnode = (int64_t)rank * d.D + i;  // key table and key count are kept by (rank, node)
  const int b = row_order[rank];
  const int64_t node = (int64_t)b * d.D + i;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform role index
  const int l32 = lane & 31, hi = lane >> 5;
  const int k0 = split * chunk;
  (void)row_status;  // a row the earlier steps skipped has key count 0 here
  const int n_keys = nkeys_tab[rnode];
  // Pointer table of tile u (w4 only): lane l copies 4 bytes (half l & 1) of
  // the pointer of key 32 u + l / 2, within the node's table row, so it needs
  // no key count: the tiles 0..4 of the first attempt go out with the key
  // count and the row index, in the workgroup's first round trip.
  const uint16_t *const *tab = keytab + rnode * keytab_stride + k0;
  const int tab_len = keytab_stride - k0;  // >= 1: every split starts inside the table row
  const uint32_t lds_p = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)&sPtr[0][0];
  auto copy_ptrs = [&](int u) {
    const int r = std::min(u * kKT + (lane >> 1), tab_len - 1);
    dma4(reinterpret_cast<const unsigned char *>(tab + r) + 4 * (lane & 1), lds_p + (u % kPSlots) * (kKT * 8));
  };
  if (wv == 4)
    for (int u = 0; u < 5; ++u) copy_ptrs(u);
  if (k0 >= n_keys) {
    vm_wait<0>();  // no copy into LDS outlives the workgroup
    return;
  }
  const int nkeys = std::min(n_keys, k0 + chunk) - k0;
  const int T = (nkeys + kKT - 1) / kKT;
  const bool single = n_keys <= chunk;
  const float sl2 = d.scale * kLog2e;
  // Every role runs the same barrier sequence per attempt: two in the
  // prologue, one per iteration but the last, one at the end (E: overflow
  // verdicts and probability sums published, both written right after the
  // loop), and one more before a restart.  A restart is decided once per attempt, from the largest logit
  // each logit wave saw: any head more than kSlack above its reference.
  auto restart_now = [&](int attempt) { return (sOver[0] | sOver[1]) != 0 && attempt < kMaxRestarts; };

  // Direct copies of key rows into the tile buffers.  The copying waves and
  // their column groups: w4 0..2, w5 3..5, w3 6..7, w2 8.
  const int g_lo = wv == 4 ? 0 : wv == 5 ? 3 : wv == 3 ? 6 : wv == 2 ? 8 : 0;
  const int g_hi = wv == 4 ? 3 : wv == 5 ? 6 : wv == 3 ? 8 : wv == 2 ? 9 : 0;
  const int n_g = 4 * (g_hi - g_lo);
  const uint32_t lds_k = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)&sK[0][0];
  // Rows of tile u into buffer u % 4: instruction (g, k) fills rows 8k ..
  // 8k+7 of group g (lane = row-in-8 * 8 + slot); slot s of row r holds
  // logical chunk slot(r, s) of the group.  Rows past the split's end repeat
  // its last key (finite data; their probabilities are 0).  All source
  // addresses are formed before the first copy is issued.
  auto copy_tile = [&](int u) {
    const unsigned char *src[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int r = 8 * k + (lane >> 3);
      const int rv = std::min(r, nkeys - 1 - u * kKT);
      src[k] = reinterpret_cast<const unsigned char *>(sPtr[u % kPSlots][rv]) + slot(r, lane & 7) * 16;
    }
    const uint32_t dst = lds_k + (u % kNBUF) * kTB;
    const unsigned char *a[3][4];
#pragma unroll
    for (int gg = 0; gg < 3; ++gg)
#pragma unroll
      for (int k = 0; k < 4; ++k) a[gg][k] = src[k] + (g_lo + gg) * 128;
#pragma unroll
    for (int gg = 0; gg < 3; ++gg)
      if (g_lo + gg < g_hi)
#pragma unroll
        for (int k = 0; k < 4; ++k) dma16(a[gg][k], dst + (g_lo + gg) * kGB + k * 1024);
  };
  // The copying waves' share of an attempt's prologue and of iteration it.
  auto copy_prologue = [&](int attempt) {
    if (wv == 4) {
      if (attempt > 0)  // the first attempt's tables went out with the row status
        for (int u = 0; u < std::min(T, 5); ++u) copy_ptrs(u);
      vm_wait<0>();
    }
    lds_barrier();  // pointer tables of tiles 0..4 copied
    if (n_g) {
      copy_tile(0);
      if (T > 1) copy_tile(1);
    }
    vm_wait_n(T > 1 ? n_g : 0);
  };
  auto copy_step = [&](int it) {  // issue tile it+3 (and pointers of tile it+6); returns copies issued
    int n = 0;
    if (wv == 4 && it + 6 < T) {
      copy_ptrs(it + 6);
      n += 1;
    }
    if (n_g && it + 3 < T) {
      copy_tile(it + 3);  // buffer (it+3) % 4 held tile it-1, read before the last barrier
      n += n_g;
    }
    return n;
  };

  if (wv == 0 || wv == 1) {
    // ---- logit wave: heads 32 hh .. 32 hh + 31 ------------------------------
    const int hh = wv;
    const int head = 32 * hh + l32;
    // Queries as the B operand: lane holds head `head`, channels 16 ks + 8 hi .. +7.
    bf16x8 qf[kKS];
    {
      const uint16_t *qrow = q + (node * kH + head) * kDK + 8 * hi;
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks)
        qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(qrow + 16 * ks));
    }
    // A operand: lane reads row l32, chunk 2 (ks & 3) + hi of group ks / 4.
    int kofs[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) kofs[c] = l32 * 128 + slot(l32, 2 * c + hi) * 16;
    const int pw0 = p_off(head, hi), pw1 = p_off(head, 2 + hi);

    float m_ref = -INFINITY, m_seen = -INFINITY;
    // Complete logits of the tile's 32 keys x this wave's 32 heads: two
    // accumulator chains (even and odd k-steps), key reads six ahead.
    auto qk_tile = [&](int tile) {
      const unsigned char *kt = sK[tile % kNBUF];
      f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kt + (ks >> 2) * kGB + kofs[ks & 3]);
        if (ks & 1)
          s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s1, 0, 0, 0);
        else
          s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s0, 0, 0, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
      for (int r = 0; r < kKS - 6; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
      return s0 + s1;
    };
    // Element v of a lane's logits is key 8 (v / 4) + 4 hi + v % 4 of the
    // tile; keys past the split are -inf.  Probabilities against the reference
    // go to LDS as bf16 P^T; their sums come from the value contraction.
    auto process = [&](int tile, f32x16 s, bool first) {
      const int nvalid = nkeys - tile * kKT;
      if (nvalid < kKT) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (8 * (v >> 2) + 4 * hi + (v & 3) >= nvalid) s[v] = -INFINITY;
      }
      float mx = s[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[v]);
      mx *= sl2;
      if (first) m_ref = fmaxf(mx, __shfl_xor(mx, 32, 64));  // the reference: the first tile's maximum
      m_seen = fmaxf(m_seen, mx);
      float p[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) p[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], sl2, -m_ref));
      uint4 c0, c1;
      c0.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[0], p[1]}, bf16x2));
      c0.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[2], p[3]}, bf16x2));
      c0.z = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[4], p[5]}, bf16x2));
      c0.w = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[6], p[7]}, bf16x2));
      c1.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[8], p[9]}, bf16x2));
      c1.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[10], p[11]}, bf16x2));
      c1.z = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[12], p[13]}, bf16x2));
      c1.w = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){p[14], p[15]}, bf16x2));
      unsigned char *pt = sP[tile & 1];
      *reinterpret_cast<uint4 *>(pt + pw0) = c0;
      *reinterpret_cast<uint4 *>(pt + pw1) = c1;
    };

    for (int attempt = 0;; ++attempt) {
      lds_barrier();  // pointer tables of the first tiles copied
      __builtin_amdgcn_s_waitcnt(0x0F70);  // queries are in registers
      lds_barrier();  // tile 0 landed
      for (int it = -1; it < T; ++it) {
        if (it + 1 < T) process(it + 1, qk_tile(it + 1), it + 1 == 0 && attempt == 0);
        if (it == T - 1) break;
        lds_barrier();
      }
      const float seen = fmaxf(m_seen, __shfl_xor(m_seen, 32, 64));
      const bool over = __any(seen > m_ref + kSlack);
      if (lane == 0) sOver[hh] = over ? 1 : 0;
      lds_barrier();  // E: the overflow verdicts and the sums are published
      if (!restart_now(attempt)) break;
      m_ref = seen;  // restart from the largest logit seen
      lds_barrier();
    }
    if (hi == 0) {
      const float lsum = sSum[head];
      if (single) {
        if (lse) lse[node * kH + head] = (m_ref + __log2f(lsum)) * kLn2;
      } else {
        part_ml[(((node * splits) + split) * kH + head) * 2 + 0] = m_ref;
        part_ml[(((node * splits) + split) * kH + head) * 2 + 1] = lsum;
      }
    }
  } else if (wv == 4 || wv == 5) {
    // ---- copy wave ------------------------------------------------------------
    for (int attempt = 0;; ++attempt) {
      copy_prologue(attempt);
      lds_barrier();  // tile 0 landed
      for (int it = -1; it < T; ++it) {
        const int n = copy_step(it);
        if (it == T - 1) break;
        vm_wait_n(n);  // tile it+2 has landed (tile it+3 and the pointer table may still fly)
        lds_barrier();
      }
      vm_wait<0>();
      lds_barrier();  // E
      if (!restart_now(attempt)) break;
      lds_barrier();
    }
  } else {
    // ---- value wave: channels 128 pq .. 128 pq + 127 for all heads -------------
    // Wave pq == 0 also accumulates each head's probability sum, as the
    // product of P^T with a value operand of ones.
    const int pq = (wv & 1) | ((wv >> 2) << 1);
    const int g = lane >> 4, jj = lane & 15;
    // Transpose-read offsets: rows 16 ks + 8 s + 4 hi + jj/4, columns
    // 128 pq + 32 ct + 16 (g & 1) + 4 (jj & 3).
    int voff[4][4];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
        voff[rr][ct] = off(16 * (rr >> 1) + 8 * (rr & 1) + 4 * hi + (jj >> 2),
                           128 * pq + 32 * ct + 16 * (g & 1) + 4 * (jj & 3));
    const bf16x8 ones = __builtin_bit_cast(bf16x8, make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));
    f32x16 acc_o[2][4], acc_l[2];
    auto pv_tile = [&](int it) {
      const unsigned char *kt = sK[it % kNBUF];
      const unsigned char *pt = sP[it & 1];
      bf16x8 pb[2][2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int t = 0; t < 2; ++t) pb[ks][t] = *reinterpret_cast<const bf16x8 *>(pt + p_off(32 * t + l32, 2 * ks + hi));
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(kt + voff[2 * ks][ct]));
          const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(kt + voff[2 * ks + 1][ct]));
          const bf16x8 va = __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){
                                                           v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]});
#pragma unroll
          for (int t = 0; t < 2; ++t)
            acc_o[t][ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[ks][t], acc_o[t][ct], 0, 0, 0);
        }
        if (pq == 0)
#pragma unroll
          for (int t = 0; t < 2; ++t) acc_l[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ones, pb[ks][t], acc_l[t], 0, 0, 0);
      }
    };

    for (int attempt = 0;; ++attempt) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        acc_l[t] = f32x16{};
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) acc_o[t][ct] = f32x16{};
      }
      copy_prologue(attempt);
      lds_barrier();  // tile 0 landed
      for (int it = -1; it < T; ++it) {
        const int n = copy_step(it);
        if (it >= 0) pv_tile(it);
        if (it == T - 1) break;
        vm_wait_n(n);
        lds_barrier();
      }
      vm_wait<0>();
      if (pq == 0 && hi == 0) {  // every row of the sums' accumulator holds the sum of its lane's head
        sSum[l32] = acc_l[0][0];
        sSum[32 + l32] = acc_l[1][0];
      }
      lds_barrier();  // E
      if (!restart_now(attempt)) break;
      lds_barrier();
    }
    // Epilogue through LDS (the K buffers are free): lane holds, per head
    // tile t, head 32 t + l32 and value channels 128 pq + 32 ct + 8 (j / 4) +
    // 4 hi + (j % 4).  The wave writes its block as rows [head][128 channels]
    // (bf16, 256-byte rows; float32, 512-byte rows for a split's partial),
    // 16-byte chunks XOR-swizzled by head, then stores each row contiguously.
    unsigned char *ob = &sK[0][0] + pq * (single ? 64 * 256 : 64 * 512);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int h = t * 32 + l32;
      const float inv = single ? 1.0f / sSum[h] : 1.0f;
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int jq = 0; jq < 4; ++jq) {
          const int c = 32 * ct + 8 * jq + 4 * hi;  // channel within this wave's 128
          const float v0 = acc_o[t][ct][4 * jq] * inv, v1 = acc_o[t][ct][4 * jq + 1] * inv;
          const float v2 = acc_o[t][ct][4 * jq + 2] * inv, v3 = acc_o[t][ct][4 * jq + 3] * inv;
          if (single) {
            uint2 w;
            w.x = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v0, v1}, bf16x2));
            w.y = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v2, v3}, bf16x2));
            *reinterpret_cast<uint2 *>(ob + h * 256 + (((c >> 3) ^ (h & 15)) << 4) + ((c >> 2) & 1) * 8) = w;
          } else {
            *reinterpret_cast<float4 *>(ob + h * 512 + (((c >> 2) ^ (h & 31)) << 4)) = make_float4(v0, v1, v2, v3);
          }
        }
    }
    if (single) {
#pragma unroll
      for (int u = 0; u < 16; ++u) {  // rows 4u .. 4u+3, sixteen 16-byte chunks each
        const int r = 4 * u + (lane >> 4), ch = lane & 15;
        const uint4 v = *reinterpret_cast<const uint4 *>(ob + r * 256 + ((ch ^ (r & 15)) << 4));
        *reinterpret_cast<uint4 *>(out + (node * kH + r) * kDV + 128 * pq + 8 * ch) = v;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 32; ++u) {  // rows 2u, 2u+1, thirty-two 16-byte chunks each
        const int r = 2 * u + (lane >> 5), ch = lane & 31;
        const float4 v = *reinterpret_cast<const float4 *>(ob + r * 512 + ((ch ^ (r & 31)) << 4));
        *reinterpret_cast<float4 *>(part_o + (((node * splits) + split) * kH + r) * kDV + 128 * pq + 4 * ch) = v;
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
  const int64_t grid = attn_grid(d, plan);
  attn_mla_kernel<<<dim3((unsigned)grid), mla::kNT, 0, s>>>(d, q, row_status, row_order, keytab, plan.max_keys, nkeys,
                                                           plan.chunk, plan.splits, part_o, part_ml, out, lse);
  return hipGetLastError();
}

}  // namespace tv
