// Branch-aware verify attention over CSA / HCA / window keys.
//
// One workgroup (4 wavefronts) takes one (row, node, key split).  All query
// heads of the node share every key (one KV row per token), so a 32-key tile
// staged in LDS feeds an MFMA contraction heads x keys for the logits and
// heads x values for the output:
//   S = Q K^T   v_mfma_f32_32x32x16_bf16, head tiles x dimension parts over waves
//   online softmax in float32 (base-2 exponent), probabilities rounded to bf16
//   O += P V    v_mfma_f32_32x32x16_bf16, value columns split over waves
// A node whose keys fit one split writes its normalised output directly;
// otherwise the split writes an unnormalised partial (O, running max, sum)
// that the combine kernel merges in split order.
#include <algorithm>

#include "node_keys.h"
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kKT = 32;         // keys per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int HT, int DK, int DV, int VOFF, int DROW>
struct AttnShape {
  static constexpr int NP = 4 / HT;            // dimension parts of the logit contraction
  static constexpr int KS = DK / 16;           // k-steps over the key channels
  static constexpr int KSP = KS / NP;          // k-steps per wave
  static constexpr int CT = DV / 4 / 32;       // 32-column output tiles per wave
  static constexpr int QS = DK + 8;            // padded LDS row strides (elements)
  static constexpr int KRS = DROW + 8;
  static constexpr int PS = kKT + 8;
  static_assert(KS % NP == 0, "key width must split over the waves");
  static_assert(DV % 128 == 0, "value width must be a multiple of 128");
};

template <int HT, int DK, int DV, int VOFF, int DROW>
__global__ void __launch_bounds__(256, 1)
attn_kernel(tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u, const uint64_t *__restrict__ anc,
            const int32_t *__restrict__ depth, const uint16_t *__restrict__ scr_c4,
            const uint16_t *__restrict__ scr_c128, const uint16_t *__restrict__ q, const int32_t *__restrict__ sel,
            const int32_t *__restrict__ row_status, int chunk, int splits, float *__restrict__ part_o,
            float *__restrict__ part_ml, uint16_t *__restrict__ out, float *__restrict__ lse) {
  using S = AttnShape<HT, DK, DV, VOFF, DROW>;
  constexpr int R = HT * 32;  // padded head rows
  __shared__ __attribute__((aligned(16))) uint16_t sQ[R * S::QS];
  __shared__ __attribute__((aligned(16))) uint16_t sK[kKT * S::KRS];
  __shared__ float sS[S::NP][R][kKT + 1];
  __shared__ __attribute__((aligned(16))) uint16_t sP[R * S::PS];
  __shared__ float sAlpha[R], sM[R], sL[R];
  __shared__ const uint16_t *sPtr[kKT];
  __shared__ int32_t path[64], hca_node[64], cnt[2];

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int split = blockIdx.x % splits;
  const int nodeg = blockIdx.x / splits;
  const int b = nodeg / d.D, i = nodeg - b * d.D;
  if (row_status[b] != TV_ROW_OK) return;
  const int32_t L = c.len[b];
  if (!len_ok(L, d.max_len)) return;
  const NodeKeys nk = node_keys(d, L, b, i, anc, depth, path, hca_node, cnt);
  const int k0 = split * chunk;
  if (k0 >= nk.n_keys) return;
  const int k1 = std::min(nk.n_keys, k0 + chunk);
  const int64_t node = (int64_t)b * d.D + i;
  const int32_t *sel_node = sel + node * d.topk;
  const int64_t c4b = c.c4_base[b], c128b = c.c128_base[b];

  // queries -> LDS (rows >= H are zero)
  const uint16_t *qn = q + node * d.H * DK;
  for (int e = tid; e < R * (DK / 8); e += 256) {
    const int r = e / (DK / 8), cc = (e - r * (DK / 8)) * 8;
    uint4 v = r < d.H ? *reinterpret_cast<const uint4 *>(qn + (int64_t)r * DK + cc) : make_uint4(0, 0, 0, 0);
    *reinterpret_cast<uint4 *>(sQ + r * S::QS + cc) = v;
  }
  if (tid < R) { sM[tid] = -INFINITY; sL[tid] = 0.f; }

  f32x16 acc_o[HT][S::CT];
#pragma unroll
  for (int h = 0; h < HT; ++h)
#pragma unroll
    for (int ct = 0; ct < S::CT; ++ct) acc_o[h][ct] = f32x16{};

  const float sl2 = d.scale * kLog2e;
  const int ht_qk = wv % HT, dp = wv / HT;
  const int l32 = lane & 31, hi = lane >> 5;

  for (int t0 = k0; t0 < k1; t0 += kKT) {
    if (tid < kKT) {
      const int t = t0 + tid;
      sPtr[tid] = t < k1 ? key_row(d, nk, b, t, sel_node, path, hca_node, c.ring, c.c4, c4b, c.c128, c128b,
                                   scr_c4, scr_c128, tree_u)
                         : nullptr;
    }
    __syncthreads();
    for (int e = tid; e < kKT * (DROW / 8); e += 256) {
      const int r = e / (DROW / 8), cc = (e - r * (DROW / 8)) * 8;
      const uint16_t *src = sPtr[r];
      uint4 v = src ? *reinterpret_cast<const uint4 *>(src + cc) : make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sK + r * S::KRS + cc) = v;
    }
    __syncthreads();

    // logits: wave (head tile, dimension part)
    {
      f32x16 acc = f32x16{};
      const uint16_t *qa = sQ + (ht_qk * 32 + l32) * S::QS + hi * 8;
      const uint16_t *kb = sK + l32 * S::KRS + hi * 8;
#pragma unroll 6
      for (int ks = dp * S::KSP; ks < (dp + 1) * S::KSP; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(qa + ks * 16);
        const bf16x8 bb = *reinterpret_cast<const bf16x8 *>(kb + ks * 16);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb, acc, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) sS[dp][ht_qk * 32 + 8 * (j >> 2) + 4 * hi + (j & 3)][l32] = acc[j];
    }
    __syncthreads();

    // online softmax, one thread per head row
    if (tid < R) {
      const int h = tid;
      const int nv = k1 - t0 < kKT ? k1 - t0 : kKT;
      if (h < d.H) {
        float sv[kKT];
        float mx = sM[h];
#pragma unroll
        for (int t = 0; t < kKT; ++t) {
          float s = 0.f;
#pragma unroll
          for (int pp = 0; pp < S::NP; ++pp) s += sS[pp][h][t];
          s = t < nv ? s * sl2 : -INFINITY;
          sv[t] = s;
          mx = fmaxf(mx, s);
        }
        const float alpha = exp2f(sM[h] - mx);
        float lsum = 0.f;
#pragma unroll
        for (int t = 0; t < kKT; ++t) {
          const uint16_t pb = f2bf(exp2f(sv[t] - mx));
          sP[h * S::PS + t] = pb;
          lsum += bf2f(pb);
        }
        sL[h] = sL[h] * alpha + lsum;
        sM[h] = mx;
        sAlpha[h] = alpha;
      } else {
#pragma unroll
        for (int t = 0; t < kKT; ++t) sP[h * S::PS + t] = 0;
        sAlpha[h] = 1.f;
      }
    }
    __syncthreads();

    // O = O * alpha + P V ; wave owns value columns [wv*DV/4, (wv+1)*DV/4)
#pragma unroll
    for (int h = 0; h < HT; ++h)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float al = sAlpha[h * 32 + 8 * (j >> 2) + 4 * hi + (j & 3)];
#pragma unroll
        for (int ct = 0; ct < S::CT; ++ct) acc_o[h][ct][j] *= al;
      }
#pragma unroll
    for (int ks = 0; ks < kKT / 16; ++ks) {
      bf16x8 pa[HT];
#pragma unroll
      for (int h = 0; h < HT; ++h)
        pa[h] = *reinterpret_cast<const bf16x8 *>(sP + (h * 32 + l32) * S::PS + ks * 16 + hi * 8);
#pragma unroll
      for (int ct = 0; ct < S::CT; ++ct) {
        const int col = VOFF + wv * (DV / 4) + ct * 32 + l32;
        const uint16_t *vb = sK + (ks * 16 + hi * 8) * S::KRS + col;
        uint32_t w4[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) w4[u] = uint32_t(vb[(2 * u) * S::KRS]) | (uint32_t(vb[(2 * u + 1) * S::KRS]) << 16);
        const bf16x8 vv = __builtin_bit_cast(bf16x8, make_uint4(w4[0], w4[1], w4[2], w4[3]));
#pragma unroll
        for (int h = 0; h < HT; ++h)
          acc_o[h][ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa[h], vv, acc_o[h][ct], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // epilogue
  const bool single = nk.n_keys <= chunk;
#pragma unroll
  for (int h = 0; h < HT; ++h)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int r = h * 32 + 8 * (j >> 2) + 4 * hi + (j & 3);
      if (r >= d.H) continue;
      const float inv = single ? 1.0f / sL[r] : 1.0f;
#pragma unroll
      for (int ct = 0; ct < S::CT; ++ct) {
        const int col = wv * (DV / 4) + ct * 32 + l32;
        const float v = acc_o[h][ct][j];
        if (single)
          out[(node * d.H + r) * DV + col] = f2bf(v * inv);
        else
          part_o[(((node * splits) + split) * d.H + r) * DV + col] = v;
      }
    }
  if (tid < d.H) {
    if (single) {
      if (lse) lse[node * d.H + tid] = (sM[tid] + __log2f(sL[tid])) * kLn2;
    } else {
      part_ml[(((node * splits) + split) * d.H + tid) * 2 + 0] = sM[tid];
      part_ml[(((node * splits) + split) * d.H + tid) * 2 + 1] = sL[tid];
    }
  }
}

// Merge the partials of nodes whose keys spanned several splits.
template <int DV>
__global__ void __launch_bounds__(256) combine_kernel(tv_dims d, CacheView c, const uint64_t *__restrict__ anc,
                                                      const int32_t *__restrict__ depth,
                                                      const int32_t *__restrict__ row_status, int chunk, int splits,
                                                      const float *__restrict__ part_o,
                                                      const float *__restrict__ part_ml, uint16_t *__restrict__ out,
                                                      float *__restrict__ lse) {
  __shared__ int32_t path[64], hca_node[64], cnt[2];
  __shared__ float sW[64][64];  // per (split, head) weight exp2(m_s - m*) / l*
  const int nodeg = blockIdx.x;
  const int b = nodeg / d.D, i = nodeg - b * d.D;
  if (row_status[b] != TV_ROW_OK) return;
  const int32_t L = c.len[b];
  if (!len_ok(L, d.max_len)) return;
  const NodeKeys nk = node_keys(d, L, b, i, anc, depth, path, hca_node, cnt);
  if (nk.n_keys <= chunk) return;
  const int used = (nk.n_keys + chunk - 1) / chunk;
  const int64_t node = nodeg;
  const int tid = threadIdx.x;
  for (int h0 = 0; h0 < d.H; h0 += 64) {
    const int h = h0 + tid;
    if (tid < 64 && h < d.H) {
      float mx = -INFINITY;
      for (int s = 0; s < used; ++s) mx = fmaxf(mx, part_ml[((node * splits + s) * d.H + h) * 2]);
      float l = 0.f;
      for (int s = 0; s < used; ++s) {
        const float* ml = part_ml + ((node * splits + s) * d.H + h) * 2;
        l += exp2f(ml[0] - mx) * ml[1];
      }
      for (int s = 0; s < used; ++s) {
        const float* ml = part_ml + ((node * splits + s) * d.H + h) * 2;
        if (s < 64) sW[s][tid] = exp2f(ml[0] - mx) / l;
      }
      if (lse) lse[node * d.H + h] = (mx + __log2f(l)) * kLn2;
    }
    __syncthreads();
    const int hn = std::min(64, d.H - h0);
    for (int e = tid; e < hn * DV; e += 256) {
      const int hh = e / DV, col = e - hh * DV;
      float v = 0.f;
      for (int s = 0; s < used; ++s) v += sW[s][hh] * part_o[((node * splits + s) * d.H + h0 + hh) * DV + col];
      out[(node * d.H + h0 + hh) * DV + col] = f2bf(v);
    }
    __syncthreads();
  }
}

template <int HT, int DK, int DV, int VOFF, int DROW>
static hipError_t launch_attn_t(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                                const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128,
                                const uint16_t *q, const int32_t *sel, const int32_t *row_status,
                                const SplitPlan &plan, float *part_o, float *part_ml, uint16_t *out, float *lse,
                                hipStream_t s) {
  const int64_t grid = (int64_t)d.B * d.D * plan.splits;
  attn_kernel<HT, DK, DV, VOFF, DROW><<<dim3((unsigned)grid), 256, 0, s>>>(
      d, c, tree_u, anc, depth, scr_c4, scr_c128, q, sel, row_status, plan.chunk, plan.splits, part_o, part_ml,
      out, lse);
  return hipGetLastError();
}

hipError_t launch_attn(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                       const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128, const uint16_t *q,
                       const int32_t *sel, const int32_t *row_status, const SplitPlan &plan, float *part_o,
                       float *part_ml, uint16_t *out, float *lse, hipStream_t s) {
  if (d.H == 64 && d.d_k == 576 && d.d_v == 512 && d.v_off == 0 && d.d_row == 576)
    return launch_attn_t<2, 576, 512, 0, 576>(d, c, tree_u, anc, depth, scr_c4, scr_c128, q, sel, row_status, plan,
                                              part_o, part_ml, out, lse, s);
  if (d.H == 8 && d.d_k == 128 && d.d_v == 128 && d.v_off == 128 && d.d_row == 256)
    return launch_attn_t<1, 128, 128, 128, 256>(d, c, tree_u, anc, depth, scr_c4, scr_c128, q, sel, row_status,
                                                plan, part_o, part_ml, out, lse, s);
  return hipErrorInvalidValue;
}

hipError_t launch_combine(const tv_dims &d, const CacheView &c, const uint64_t *anc, const int32_t *depth,
                          const int32_t *sel, const int32_t *row_status, const SplitPlan &plan,
                          const float *part_o, const float *part_ml, uint16_t *out, float *lse, hipStream_t s) {
  (void)sel;
  if (plan.splits <= 1) return hipSuccess;
  dim3 grid(d.B * d.D);
  if (d.d_v == 512)
    combine_kernel<512><<<grid, 256, 0, s>>>(d, c, anc, depth, row_status, plan.chunk, plan.splits, part_o, part_ml,
                                             out, lse);
  else
    combine_kernel<128><<<grid, 256, 0, s>>>(d, c, anc, depth, row_status, plan.chunk, plan.splits, part_o, part_ml,
                                             out, lse);
  return hipGetLastError();
}

}  // namespace tv
