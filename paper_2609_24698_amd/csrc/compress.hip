// Per-branch compression of the block each node closes, into scratch.
//
// Branches that share a prefix share its committed entries, but the block that
// is still open when the tree starts is finished differently on every branch;
// each node therefore pools the tokens of its own root path and writes the
// entry to its own scratch slot, which the persistent cache never sees before
// acceptance (Sec. 4.1 chains compressed independently after branching;
// Sec. 4.2 scratch pad for temporary branch state).
//
// One workgroup per (row, node); nodes that close no block exit at once.
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kMaxRatio = 1024;

__global__ void __launch_bounds__(256) compress_kernel(tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u,
                                                       const uint64_t *__restrict__ anc,
                                                       const int32_t *__restrict__ depth,
                                                       const uint16_t *__restrict__ gate_w,
                                                       uint16_t *__restrict__ scr_c4, uint16_t *__restrict__ scr_c128,
                                                       int32_t *__restrict__ row_status) {
  __shared__ int32_t path[64];
  __shared__ float wgt[kMaxRatio];
  __shared__ float red[2];
  const int b = blockIdx.x / d.D;
  const int i = blockIdx.x - b * d.D;
  const int tid = threadIdx.x;
  const int d_u = d.d_row + d.d_idx;
  if (row_status[b] != TV_ROW_OK) return;
  const int32_t L = c.len[b];
  if (!len_ok(L, d.max_len)) {
    if (i == 0 && tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return;
  }
  const int64_t node = (int64_t)b * d.D + i;
  const int32_t dep = depth[node];
  const int64_t p = (int64_t)L + dep;
  const bool close4 = ((p + 1) % d.ratio_csa) == 0;
  const bool close128 = ((p + 1) % d.ratio_hca) == 0;
  if (!close4 && !close128) return;
  const uint64_t m = anc[node];
  for (int j = tid; j < d.D; j += blockDim.x)
    if ((m >> j) & 1ull) path[depth[(int64_t)b * d.D + j]] = j;
  __syncthreads();

  const int lane = tid & 63, wv = tid >> 6;
  for (int ri = 0; ri < 2; ++ri) {
    if (ri == 0 && !close4) continue;
    if (ri == 1 && !close128) continue;
    const int r = ri == 0 ? d.ratio_csa : d.ratio_hca;
    const int keep = ri == 0 ? d_u : d.d_row;
    const uint16_t *g = gate_w + (int64_t)ri * d_u;
    const int64_t q0 = p - r + 1;
    auto tok = [&](int64_t q) -> const uint16_t * {
      if (q < L) return ring_row(c.ring, b, d.ring_cap, d_u, q);
      return tree_u + ((int64_t)b * d.D + path[q - L]) * d_u;
    };
    // gate logits, one wavefront per token
    for (int t = wv; t < r; t += 4) {
      const uint16_t *u = tok(q0 + t);
      float acc = 0.f;
      for (int ch = lane; ch < d_u; ch += 64) acc += bf2f(g[ch]) * bf2f(u[ch]);
      acc = wave_sum(acc);
      if (lane == 0) wgt[t] = acc;
    }
    __syncthreads();
    if (wv == 0) {
      float mx = -INFINITY;
      for (int t = lane; t < r; t += 64) mx = fmaxf(mx, wgt[t]);
      mx = wave_max(mx);
      float s = 0.f;
      for (int t = lane; t < r; t += 64) s += __expf(wgt[t] - mx);
      s = wave_sum(s);
      if (lane == 0) { red[0] = mx; red[1] = s; }
    }
    __syncthreads();
    const float mx = red[0], inv = 1.0f / red[1];
    for (int t = tid; t < r; t += blockDim.x) wgt[t] = __expf(wgt[t] - mx) * inv;
    __syncthreads();
    uint16_t *dst = ri == 0 ? scr_c4 + node * d_u : scr_c128 + node * d.d_row;
    for (int ch = tid; ch < keep; ch += blockDim.x) {
      float acc = 0.f;
      for (int t = 0; t < r; ++t) acc += wgt[t] * bf2f(tok(q0 + t)[ch]);
      dst[ch] = f2bf(acc);
    }
    __syncthreads();
  }
}

hipError_t launch_compress(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                           const int32_t *depth, const uint16_t *gate_w, uint16_t *scr_c4, uint16_t *scr_c128,
                           int32_t *row_status, hipStream_t s) {
  dim3 grid(d.B * d.D);
  compress_kernel<<<grid, 256, 0, s>>>(d, c, tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status);
  return hipGetLastError();
}

}  // namespace tv
