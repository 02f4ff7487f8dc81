// Accepted-path selection after verification (Sec. 4.1 target verify ends by
// selecting the accepted path; Sec. 3.1 the result is one path through the
// tree; Sec. 4.3 metadata work kept on the device).
//
// Greedy verification: the target token of a node is the argmax of the
// target's next-token logits there; a node is accepted when every non-root
// node on its root path drafted its parent's target token, and the path ends
// at the deepest accepted node (smallest index among equally deep ones).
//
// Two launches.  The argmax streams the logits once (B*D*vocab bfloat16, the
// only sizeable traffic): one workgroup per (node, 8192-entry chunk), each
// thread with all of its 16-byte loads in flight, reduced to one sortable
// 64-bit key (value, then lowest index) per chunk.  (A grid-stride loop with
// the next chunk's loads issued early measured slower: more registers, fewer
// resident workgroups.)  The selection then runs
// one wavefront per row: lane i folds node i's chunk keys into its target
// token, a ballot marks the matching nodes, and the ancestor masks of the
// verify preprocess decide every node's acceptance at once (no walk).
#include "tv_common.h"
#include "tv_internal.h"

namespace tv {

constexpr int kSelNT = 256;                        // threads per argmax workgroup
constexpr int kSelLoads = 4;                       // 16-byte loads per thread
constexpr int kSelChunk = kSelNT * 8 * kSelLoads;  // logits per workgroup

int select_chunks(int32_t vocab) { return (vocab + kSelChunk - 1) / kSelChunk; }

// Order of bfloat16 logits as an unsigned key: larger value -> larger key,
// -0 equal to +0, every NaN above +inf.
__device__ __forceinline__ uint32_t logit_key(uint32_t x) {
  x &= 0xFFFFu;
  if ((x & 0x7FFFu) > 0x7F80u) return 0xFFFFu;
  if (x == 0x8000u) x = 0;
  return (x & 0x8000u) ? (~x & 0xFFFFu) : (x | 0x8000u);
}

// Key of (logit, index): the larger logit wins, then the smaller index.
__device__ __forceinline__ uint64_t pack(uint32_t key, uint32_t idx) {
  return (uint64_t(key) << 32) | uint64_t(0xFFFFFFFFu - idx);
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Two passes over registers.  The first keeps a float maximum (bfloat16 is
// exact in float32; fmaxf ignores NaN, which is tracked on the side), about
// three vector operations per logit.  Only the wavefronts holding the
// workgroup maximum then look for its first index, so the search costs one
// wavefront.
// kVec: vocab % 8 == 0, so every node's logits start on a 16-byte boundary.
template <bool kVec>
__global__ void __launch_bounds__(kSelNT) argmax_kernel(const uint16_t *__restrict__ logits, int32_t vocab,
                                                        int chunks, uint64_t *__restrict__ part) {
  constexpr int kWaves = kSelNT / 64;
  constexpr int kWords = kVec ? 4 * kSelLoads : kSelChunk / kSelNT / 2;  // 32-bit words (logit pairs) per thread
  constexpr uint32_t kNegInfPair = 0xFF80FF80u;  // out-of-range logits never beat an in-range one
  __shared__ float red_max[kWaves];
  __shared__ int red_nan[kWaves];
  __shared__ int red_idx[kWaves];
  const int64_t node = blockIdx.x / chunks;
  const int ch = blockIdx.x - (int)node * chunks;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const uint16_t *row = logits + node * vocab;
  const int c0 = ch * kSelChunk;
  // index of the logit in the low half of word j of this thread
  auto first_of = [&](int j) {
    if constexpr (kVec)
      return c0 + ((j >> 2) * kSelNT + tid) * 8 + 2 * (j & 3);
    else
      return c0 + 2 * (j * kSelNT + tid);
  };
  uint32_t w[kWords];
  if constexpr (kVec) {
#pragma unroll
    for (int u = 0; u < kSelLoads; ++u) {
      const int e = first_of(4 * u);
      const uint4 v = e < vocab ? *reinterpret_cast<const uint4 *>(row + e)
                                : make_uint4(kNegInfPair, kNegInfPair, kNegInfPair, kNegInfPair);
      w[4 * u] = v.x;
      w[4 * u + 1] = v.y;
      w[4 * u + 2] = v.z;
      w[4 * u + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kWords; ++j) {
      const int e = first_of(j);
      const uint32_t lo = e < vocab ? row[e] : 0xFF80u, hi = e + 1 < vocab ? row[e + 1] : 0xFF80u;
      w[j] = lo | (hi << 16);
    }
  }
  float m = -INFINITY;
  bool nan = false;
#pragma unroll
  for (int j = 0; j < kWords; ++j) {
    const float lo = __uint_as_float(w[j] << 16), hi = __uint_as_float(w[j] & 0xFFFF0000u);
    m = fmaxf(m, fmaxf(lo, hi));
    nan |= (lo != lo) | (hi != hi);
  }
  const float wm = wave_max(m);
  const bool wnan = __any(nan);
  if (lane == 0) {
    red_max[wv] = wm;
    red_nan[wv] = wnan;
  }
  __syncthreads();
  float M = red_max[0];
  bool any_nan = red_nan[0];
#pragma unroll
  for (int k = 1; k < kWaves; ++k) {
    M = fmaxf(M, red_max[k]);
    any_nan = any_nan || red_nan[k];
  }
  // the first index holding the maximum (a NaN when there is one), wavefronts that hold it only
  int idx = 0x7FFFFFFF;
  if (any_nan ? wnan : wm == M) {
#pragma unroll
    for (int j = kWords - 1; j >= 0; --j) {  // backwards: the last hit is the first index
      const float lo = __uint_as_float(w[j] << 16), hi = __uint_as_float(w[j] & 0xFFFF0000u);
      const int e = first_of(j);
      if (any_nan ? (hi != hi) : (hi == M)) idx = e + 1 < vocab ? e + 1 : idx;
      if (any_nan ? (lo != lo) : (lo == M)) idx = e < vocab ? e : idx;
    }
    idx = wave_min_i32(idx);  // the wavefront's condition is uniform: every lane is here
  }
  if (lane == 0) red_idx[wv] = idx;
  __syncthreads();
  if (tid == 0) {
    int best = red_idx[0];
#pragma unroll
    for (int k = 1; k < kWaves; ++k) best = min(best, red_idx[k]);
    const uint32_t key = any_nan ? 0xFFFFu : logit_key(__float_as_uint(M) >> 16);
    part[blockIdx.x] = pack(key, (uint32_t)best);
  }
}

// One wavefront per row, lane i owns node i (D <= 64).
__global__ void __launch_bounds__(256) select_kernel(int B, int D, int chunks, const int32_t *__restrict__ parents,
                                                     const uint64_t *__restrict__ anc,
                                                     const int32_t *__restrict__ depth,
                                                     const int32_t *__restrict__ draft,
                                                     const uint64_t *__restrict__ part,
                                                     const int32_t *__restrict__ row_status,
                                                     int32_t *__restrict__ target, int32_t *__restrict__ accepted_last,
                                                     int32_t *__restrict__ next_token) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const int i = lane;
  const bool live = i < D;
  const int64_t node = (int64_t)b * D + (live ? i : 0);
  const int32_t status = row_status[b];
  const int32_t p = parents[node];
  const int32_t dr = draft[node];
  const uint64_t m = anc[node];
  const int32_t dep = depth[node];
  uint64_t best = 0;
  for (int c = 0; c < chunks; ++c) best = umax64(best, part[node * chunks + c]);
  if (status != TV_ROW_OK) return;  // wave-uniform
  const int32_t t = (int32_t)(0xFFFFFFFFu - (uint32_t)best);
  if (live) target[node] = t;
  const int32_t tp = __shfl(t, p < 0 ? 0 : p, 64);  // target token of the parent
  const bool match = live && i > 0 && dr == tp;
  const uint64_t M = __ballot(match);
  // accepted: every non-root node of the root path (bits of anc) matches
  const bool ok = live && (i == 0 || ((m & ~1ull & ~M) == 0));
  uint32_t key = ok ? (uint32_t(dep) << 8) | uint32_t(255 - i) : 0u;
  key = wave_max_u32(key);
  const int last = 255 - int(key & 255u);
  const int32_t t_last = __shfl(t, last, 64);
  if (lane == 0) {
    accepted_last[b] = last;
    if (next_token) next_token[b] = t_last;
  }
}

hipError_t launch_argmax(const tv_dims &d, const uint16_t *logits, int32_t vocab, uint64_t *part, hipStream_t s) {
  const int chunks = select_chunks(vocab);
  const int64_t grid = (int64_t)d.B * d.D * chunks;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  if (vocab % 8 == 0)
    argmax_kernel<true><<<(unsigned)grid, kSelNT, 0, s>>>(logits, vocab, chunks, part);
  else
    argmax_kernel<false><<<(unsigned)grid, kSelNT, 0, s>>>(logits, vocab, chunks, part);
  return hipGetLastError();
}

hipError_t launch_select(const tv_dims &d, const int32_t *parents, const uint64_t *anc, const int32_t *depth,
                         const int32_t *draft, int32_t vocab, const uint64_t *part, const int32_t *row_status,
                         int32_t *target, int32_t *accepted_last, int32_t *next_token, hipStream_t s) {
  select_kernel<<<(d.B + 3) / 4, 256, 0, s>>>(d.B, d.D, select_chunks(vocab), parents, anc, depth, draft, part,
                                             row_status, target, accepted_last, next_token);
  return hipGetLastError();
}

}  // namespace tv
