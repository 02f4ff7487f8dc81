// Verify preprocess: parent array -> ancestor bitmask, depth and row status.
//
// One 64-lane wavefront per row, lane i owns node i (D <= 64).  A row is valid
// when the root has parent -1 and every other node's parent precedes it; the
// ancestor set of node i is i plus the ancestor set of its parent (the tree
// topology that branch-aware verification must respect, Sec. 3.1 and Sec. 4.1).
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

__global__ void __launch_bounds__(256) mask_kernel(int B, int D, const int32_t *__restrict__ parents,
                                                   uint64_t *__restrict__ anc, int32_t *__restrict__ depth,
                                                   int32_t *__restrict__ row_status) {
  __shared__ int32_t par[4][64];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int b = blockIdx.x * 4 + w;
  const bool live = b < B;
  const int i = lane;
  int32_t p = (live && i < D) ? parents[(int64_t)b * D + i] : 0;
  bool ok = (i >= D) || (i == 0 ? p == -1 : (p >= 0 && p < i));
  par[w][lane] = p;
  const bool row_ok = __all(ok);
  __syncthreads();
  if (!live) return;
  if (i < D) {
    uint64_t m = 0;
    int32_t dep = 0;
    if (row_ok) {
      m = 1ull << i;
      int j = p;
      while (j >= 0) {  // parents strictly decrease, so at most i steps
        m |= 1ull << j;
        ++dep;
        j = par[w][j];
      }
    }
    anc[(int64_t)b * D + i] = m;
    depth[(int64_t)b * D + i] = dep;
  }
  if (lane == 0) row_status[b] = row_ok ? TV_ROW_OK : TV_ROW_BAD_PARENT;
}

hipError_t launch_mask(const tv_dims &d, const int32_t *parents, uint64_t *anc, int32_t *depth,
                       int32_t *row_status, hipStream_t s) {
  dim3 grid((d.B + 3) / 4);
  mask_kernel<<<grid, 256, 0, s>>>(d.B, d.D, parents, anc, depth, row_status);
  return hipGetLastError();
}

}  // namespace tv
