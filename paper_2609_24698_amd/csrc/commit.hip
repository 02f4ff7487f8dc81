// Accepted-path refresh of the committed state.
//
// After verification only the accepted root path survives (Sec. 3.2, Sec. 4.2):
// its raw rows enter the window ring, every block it closed becomes a committed
// CSA / HCA entry (copied from the path node's scratch slot), and the committed
// length advances.  Entries compressed on rejected branches are never copied,
// so they leave no trace in the persistent state.
//
// One workgroup per row.  All checks run before the first write, so a failing
// row is left exactly as it was.
//
// Refresh schedule (Sec. 4.3): with a designated chain (the root path of
// primary_last[b]), whose CSA entries the compression already wrote into the
// pool, the CSA copies of accepted nodes on that chain are skipped: a single
// chain, or an accepted path that is the cached chain, needs no CSA refresh.
// HCA entries are always written here, once the path is known, all of a
// round's in one pass.
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

__global__ void __launch_bounds__(256) commit_kernel(tv_dims d, tv_cache c, const uint16_t *__restrict__ tree_u,
                                                     const uint64_t *__restrict__ anc,
                                                     const int32_t *__restrict__ depth,
                                                     const uint16_t *__restrict__ scr_c4,
                                                     const uint16_t *__restrict__ scr_c128,
                                                     const int32_t *__restrict__ accepted_last,
                                                     int32_t *__restrict__ accept_nodes,
                                                     int32_t *__restrict__ accept_len,
                                                     int32_t *__restrict__ row_status,
                                                     const int32_t *__restrict__ primary_last) {
  __shared__ int32_t path[64];
  const int b = blockIdx.x, tid = threadIdx.x;
  if (row_status[b] != TV_ROW_OK) return;
  const int32_t L = c.len[b];
  if (!len_ok(L, d.max_len)) {
    if (tid == 0) row_status[b] = TV_ROW_BAD_LEN;
    return;
  }
  const int32_t last = accepted_last[b];
  const int32_t P = primary_last ? primary_last[b] : -1;
  if (last < 0 || last >= d.D) {
    if (tid == 0) row_status[b] = TV_ROW_BAD_ACCEPT;
    return;
  }
  const uint64_t m = anc[(int64_t)b * d.D + last];
  const uint64_t chain = (P >= 0 && P < d.D) ? anc[(int64_t)b * d.D + P] : 0ull;
  const int a = depth[(int64_t)b * d.D + last] + 1;
  if (tid < d.D && ((m >> tid) & 1ull)) path[depth[(int64_t)b * d.D + tid]] = tid;
  bool bad = false;
  if (tid < a) {
    const int64_t p = (int64_t)L + tid;  // path node at depth tid stands at L + tid
    if ((p + 1) % d.ratio_csa == 0 && (p + 1) / d.ratio_csa - 1 >= c.c4_cap[b]) bad = true;
    if ((p + 1) % d.ratio_hca == 0 && (p + 1) / d.ratio_hca - 1 >= c.c128_cap[b]) bad = true;
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) row_status[b] = TV_ROW_CAPACITY;
    return;
  }
  const int d_u = d.d_row + d.d_idx;
  // raw rows -> ring (16-byte chunks)
  const int cpr = d_u / 8;
  for (int e = tid; e < a * cpr; e += blockDim.x) {
    const int t = e / cpr, cc = (e - t * cpr) * 8;
    const uint4 v = *reinterpret_cast<const uint4 *>(tree_u + ((int64_t)b * d.D + path[t]) * d_u + cc);
    uint16_t *dst = c.ring + ((int64_t)b * d.ring_cap + ((L + t) & (d.ring_cap - 1))) * d_u + cc;
    *reinterpret_cast<uint4 *>(dst) = v;
  }
  // scratch entries of the closing path nodes -> pools
  for (int t = 0; t < a; ++t) {
    const int64_t p = (int64_t)L + t;
    const int j = path[t];
    if ((p + 1) % d.ratio_csa == 0 && !((chain >> j) & 1ull)) {
      const int64_t slot = c.c4_base[b] + (p + 1) / d.ratio_csa - 1;
      const uint16_t *src = scr_c4 + ((int64_t)b * d.D + j) * d_u;
      for (int e = tid; e < d_u / 8; e += blockDim.x) {
        const uint4 v = *reinterpret_cast<const uint4 *>(src + e * 8);
        if (e * 8 < d.d_row)
          *reinterpret_cast<uint4 *>(c.c4 + slot * d.d_row + e * 8) = v;
        else
          *reinterpret_cast<uint4 *>(c.c4_idx + slot * d.d_idx + (e * 8 - d.d_row)) = v;
      }
    }
    if ((p + 1) % d.ratio_hca == 0) {
      const int64_t slot = c.c128_base[b] + (p + 1) / d.ratio_hca - 1;
      const uint16_t *src = scr_c128 + ((int64_t)b * d.D + j) * d.d_row;
      for (int e = tid; e < d.d_row / 8; e += blockDim.x)
        *reinterpret_cast<uint4 *>(c.c128 + slot * d.d_row + e * 8) = *reinterpret_cast<const uint4 *>(src + e * 8);
    }
  }
  __syncthreads();
  if (tid < d.D) accept_nodes[(int64_t)b * d.D + tid] = tid < a ? path[tid] : -1;
  if (tid == 0) {
    accept_len[b] = a;
    c.len[b] = L + a;
  }
}

hipError_t launch_commit(const tv_dims &d, const tv_cache &c, const uint16_t *tree_u, const uint64_t *anc,
                         const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128,
                         const int32_t *accepted_last, int32_t *accept_nodes, int32_t *accept_len,
                         int32_t *row_status, const int32_t *primary_last, hipStream_t s) {
  commit_kernel<<<d.B, 256, 0, s>>>(d, c, tree_u, anc, depth, scr_c4, scr_c128, accepted_last, accept_nodes,
                                    accept_len, row_status, primary_last);
  return hipGetLastError();
}

}  // namespace tv
