// Per-branch compression of the block each node closes, into scratch.
//
// Branches that share a prefix share its committed entries, but the block that
// is still open when the tree starts is finished differently on every branch;
// each node therefore pools the tokens of its own root path and writes the
// entry to its own scratch slot, which the persistent cache never sees before
// acceptance (Sec. 4.1 chains compressed independently after branching;
// Sec. 4.2 scratch pad for temporary branch state).
//
// One workgroup per (row, node); nodes that close no block exit at once.  The
// block's token rows (committed ones from the ring, path ones from tree_u) are
// resolved once into an LDS pointer table; gate logits and the weighted sum
// then stream the rows with 16-byte loads.
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kMaxRatio = 1024;
constexpr int kMaxDu = 1024;  // raw row width bound (d_row + d_idx), 128 chunks of 16 bytes

__global__ void __launch_bounds__(256) compress_kernel(tv_dims d, CacheView c, const uint16_t *__restrict__ tree_u,
                                                       const uint64_t *__restrict__ anc,
                                                       const int32_t *__restrict__ depth,
                                                       const uint16_t *__restrict__ gate_w,
                                                       uint16_t *__restrict__ scr_c4, uint16_t *__restrict__ scr_c128,
                                                       int32_t *__restrict__ row_status) {
  __shared__ int32_t path[64];
  __shared__ const uint16_t *tok[kMaxRatio];
  __shared__ float wgt[kMaxRatio];
  __shared__ float gate[kMaxDu];
  __shared__ float part[4][kMaxDu];
  __shared__ float red[2];
  const int b = blockIdx.x / d.D;
  const int i = blockIdx.x - b * d.D;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
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

  const int nch = d_u / 8;  // 16-byte chunks per raw row
  for (int ri = 0; ri < 2; ++ri) {
    if (ri == 0 && !close4) continue;
    if (ri == 1 && !close128) continue;
    const int r = ri == 0 ? d.ratio_csa : d.ratio_hca;
    const int keep = ri == 0 ? d_u : d.d_row;
    const int64_t q0 = p - r + 1;
    for (int t = tid; t < r; t += blockDim.x) {
      const int64_t qq = q0 + t;
      tok[t] = qq < L ? ring_row(c.ring, b, d.ring_cap, d_u, qq) : tree_u + ((int64_t)b * d.D + path[qq - L]) * d_u;
    }
    for (int ch = tid; ch < d_u; ch += blockDim.x) gate[ch] = bf2f(gate_w[(int64_t)ri * d_u + ch]);
    __syncthreads();
    // gate logits: 8 lanes per token, each a strided set of 16-byte chunks
    // (all loads of a lane issued before their use; rows hold at most 128 chunks)
    for (int t0 = 0; t0 < r; t0 += 32) {
      const int t = t0 + (tid >> 3), sub = tid & 7;
      float acc = 0.f;
      if (t < r) {
        const uint4 *row = reinterpret_cast<const uint4 *>(tok[t]);
        uint4 v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int k = sub + 8 * u;
          v[u] = k < nch ? row[k] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int k = sub + 8 * u;
          if (k < nch) {
            const float *gk = gate + 8 * k;
            acc += gk[0] * bf2f_lo(v[u].x) + gk[1] * bf2f_hi(v[u].x) + gk[2] * bf2f_lo(v[u].y) +
                   gk[3] * bf2f_hi(v[u].y) + gk[4] * bf2f_lo(v[u].z) + gk[5] * bf2f_hi(v[u].z) +
                   gk[6] * bf2f_lo(v[u].w) + gk[7] * bf2f_hi(v[u].w);
          }
        }
      }
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) acc += __shfl_xor(acc, o, 64);
      if (t < r && sub == 0) wgt[t] = acc;
    }
    __syncthreads();
    if (wv == 0) {
      float mx = -INFINITY;
      for (int t = lane; t < r; t += 64) mx = fmaxf(mx, wgt[t]);
      mx = wave_max(mx);
      float s = 0.f;
      for (int t = lane; t < r; t += 64) s += __expf(wgt[t] - mx);
      s = wave_sum(s);
      if (lane == 0) {
        red[0] = mx;
        red[1] = s;
      }
    }
    __syncthreads();
    const float mx = red[0], inv = 1.0f / red[1];
    for (int t = tid; t < r; t += blockDim.x) wgt[t] = __expf(wgt[t] - mx) * inv;
    __syncthreads();
    // weighted sum: thread (token group wv of 4, chunk k) sums 8 channels over
    // tokens wv, wv+4, ...; loads are issued eight tokens at a time
    const int kch = keep / 8;
    for (int k0 = 0; k0 < kch; k0 += 64) {
      const int k = k0 + lane;
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (k < kch) {
        for (int tb = wv; tb < r; tb += 32) {
          uint4 v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int t = tb + 4 * u;
            v[u] = t < r ? reinterpret_cast<const uint4 *>(tok[t])[k] : make_uint4(0, 0, 0, 0);
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int t = tb + 4 * u;
            const float w = t < r ? wgt[t] : 0.f;
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
        for (int e = 0; e < 8; ++e) part[wv][8 * k + e] = acc[e];
      }
    }
    __syncthreads();
    uint16_t *dst = ri == 0 ? scr_c4 + node * d_u : scr_c128 + node * d.d_row;
    for (int ch = tid; ch < keep; ch += blockDim.x)
      dst[ch] = f2bf((part[0][ch] + part[1][ch]) + (part[2][ch] + part[3][ch]));
    __syncthreads();
  }
}

hipError_t launch_compress(const tv_dims &d, const CacheView &c, const uint16_t *tree_u, const uint64_t *anc,
                           const int32_t *depth, const uint16_t *gate_w, uint16_t *scr_c4, uint16_t *scr_c128,
                           int32_t *row_status, hipStream_t s) {
  if (d.d_row + d.d_idx > kMaxDu) return hipErrorInvalidValue;
  dim3 grid(d.B * d.D);
  compress_kernel<<<grid, 256, 0, s>>>(d, c, tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status);
  return hipGetLastError();
}

}  // namespace tv
