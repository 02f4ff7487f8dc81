// C ABI of the tree-verify library: argument checks, workspace layout,
// launch sequencing and optional kernel timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "tv_internal.h"

namespace tv {

static bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

static bool shape_supported(const tv_dims &d) {
  const bool mla = d.H == 64 && d.d_row == 576 && d.d_k == 576 && d.v_off == 0 && d.d_v == 512;
  const bool mha = d.H == 8 && d.d_row == 256 && d.d_k == 128 && d.v_off == 128 && d.d_v == 128;
  return (mla || mha) && d.d_idx == 64 && pow2(d.H_idx) && d.H_idx <= 64 && d.d_row + d.d_idx <= 1024;
}

// Dimension checks shared by every entry point.
static tv_status check_dims(const tv_dims *dp) {
  if (!dp) return TV_ERR_INVALID_ARG;
  const tv_dims &d = *dp;
  if (d.B < 1 || d.D < 1 || d.D > 64) return TV_ERR_INVALID_ARG;
  if (d.H < 1 || d.d_row < 1 || d.d_k < 1 || d.d_v < 1 || d.v_off < 0 || d.d_idx < 1 || d.H_idx < 1)
    return TV_ERR_INVALID_ARG;
  if (d.d_k > d.d_row || d.v_off + d.d_v > d.d_row || d.d_row % 8 || d.d_idx % 8) return TV_ERR_INVALID_ARG;
  if (d.ratio_csa < 1 || d.ratio_hca < 1 || d.ratio_csa > 1024 || d.ratio_hca > 1024) return TV_ERR_INVALID_ARG;
  if (d.window < 1 || d.topk < 1) return TV_ERR_INVALID_ARG;
  // The ring must hold the window, a block's committed tail and, on top of
  // the window, a whole accepted path: a commit of up to D rows then never
  // writes two of its rows to one slot.
  if (d.page_size < 0 || d.page_stride < 0) return TV_ERR_INVALID_ARG;
  if (d.page_size > 0) {  // paged pool: pages hold whole CSA and HCA blocks
    if (!pow2(d.page_size) || d.page_size > (1 << 20) || d.page_size % d.ratio_csa || d.page_size % d.ratio_hca ||
        d.page_stride < 1)
      return TV_ERR_INVALID_ARG;
  } else if (!pow2(d.ring_cap) || d.ring_cap < std::max({d.window + d.D, d.ratio_csa, d.ratio_hca})) {
    return TV_ERR_INVALID_ARG;
  }
  if (d.max_len < 0 || (int64_t)d.max_len + d.D + 1 >= (int64_t(1) << 30)) return TV_ERR_INVALID_ARG;
  if (!std::isfinite(d.scale) || !(d.scale > 0.f)) return TV_ERR_INVALID_ARG;
  if (d.idx_fmt != TV_IDX_BF16 && d.idx_fmt != TV_IDX_E4M3) return TV_ERR_INVALID_ARG;
  if (d.B > 4096 || !shape_supported(d) || !topk_supported(d)) return TV_ERR_UNSUPPORTED;
  return TV_OK;
}

static bool cache_complete(const tv_dims &d, const tv_cache *c) {
  if (!c || !c->ring || !c->c4 || !c->c4_idx || !c->c128 || !c->len) return false;
  if (d.page_size > 0) return c->page_table != nullptr;
  return c->c4_base && c->c4_cap && c->c128_base && c->c128_cap;
}

// Kernels move rows with 16-byte loads and stores; every buffer must allow them.
static bool a16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
template <typename... P>
static bool all_a16(const P *...p) {
  return (a16(p) && ...);
}
static bool cache_a16(const tv_cache *c) {
  auto ok = [](const void *p) { return !p || a16(p); };  // pointers a layout does not use may be NULL
  return all_a16(c->ring, c->c4, c->c4_idx, c->c128, c->len) && ok(c->c4_base) && ok(c->c4_cap) &&
         ok(c->c128_base) && ok(c->c128_cap) && ok(c->page_table);
}

// The library only runs on gfx950; the answer is cached per device.
static tv_status check_device() {
  static std::mutex mu;
  static std::vector<int> verdict;  // -1 unknown, 0 bad, 1 good
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TV_ERR_DEVICE;
  std::lock_guard<std::mutex> lk(mu);
  if ((int)verdict.size() <= dev) verdict.resize(dev + 1, -1);
  if (verdict[dev] < 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return TV_ERR_DEVICE;
    verdict[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 0;
  }
  return verdict[dev] == 1 ? TV_OK : TV_ERR_DEVICE;
}

// Attention workgroups the split plan aims for, and the fewest keys a split
// takes when splitting is optional.  Every split pays a prologue (key table,
// first tiles, queries), an epilogue and a partial-output round trip through
// memory, so nodes are split only while there are fewer workgroups than
// compute units to fill.
#ifndef TV_ATTN_TARGET_WG
#define TV_ATTN_TARGET_WG 256
#endif
#ifndef TV_ATTN_MIN_CHUNK
#define TV_ATTN_MIN_CHUNK 256
#endif

SplitPlan split_plan(const tv_dims &d) {
  SplitPlan p;
  const int64_t mk = (int64_t)d.topk + d.max_len / d.ratio_hca + d.D + d.window;
  p.max_keys = (int32_t)mk;
  const int64_t nodes = (int64_t)d.B * d.D;
  int64_t splits = std::max<int64_t>(1, (TV_ATTN_TARGET_WG + nodes - 1) / nodes);
  splits = std::min<int64_t>(splits, std::max<int64_t>(1, mk / TV_ATTN_MIN_CHUNK));
  splits = std::max<int64_t>(splits, (mk + kAttnMaxChunk - 1) / kAttnMaxChunk);  // pointer table bound
  const int64_t chunk = ((mk + splits - 1) / splits + 31) / 32 * 32;
  p.chunk = (int32_t)chunk;
  p.splits = (int32_t)((mk + chunk - 1) / chunk);
  return p;
}

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

WsLayout ws_layout(const tv_dims &d) {
  WsLayout w;
  w.plan = split_plan(d);
  const int64_t nodes = (int64_t)d.B * d.D;
  w.score_stride = (int32_t)((d.max_len / d.ratio_csa + 63) / 64 * 64);
  size_t off = 0;
  w.scores = off;
  off = align256(off + sizeof(float) * nodes * std::max(w.score_stride, 1));
  w.sel = off;
  off = align256(off + sizeof(int32_t) * nodes * d.topk);
  w.part_o = off;
  if (w.plan.splits > 1) off = align256(off + sizeof(float) * nodes * w.plan.splits * d.H * d.d_v);
  w.part_ml = off;
  if (w.plan.splits > 1) off = align256(off + sizeof(float) * 2 * nodes * w.plan.splits * d.H);
  w.row_order = off;
  off = align256(off + sizeof(int32_t) * d.B);
  w.row_rank = off;
  off = align256(off + sizeof(int32_t) * d.B);
  w.keytab = off;
  off = align256(off + sizeof(void *) * nodes * w.plan.max_keys);
  w.nkeys = off;
  off = align256(off + sizeof(int32_t) * nodes);
  w.nkeys_rank = off;
  off = align256(off + sizeof(int32_t) * nodes);
  const int tseg = topk_max_segments(d);
  const int64_t surv = tseg > 1 ? nodes * tseg * d.topk : 0;
  w.surv_idx = off;
  off = align256(off + sizeof(int32_t) * surv);
  w.surv_key = off;
  off = align256(off + sizeof(uint32_t) * surv);
  w.surv_cnt = off;
  off = align256(off + sizeof(int32_t) * (tseg > 1 ? nodes * tseg : 0));
  w.total = off;
  return w;
}

// ---- kernel timing -------------------------------------------------------
namespace {
struct ProfRec {
  const char *name;
  hipEvent_t start, stop;
};
struct Prof {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> pool;
  std::vector<ProfRec> recs;
  size_t cap = 0;
} g_prof;
}  // namespace

// Kernels recorded by the round-graph capture running on this thread (-1: none).
thread_local int t_capture_kernels = -1;

// Starts the timing of one launch; returns its record index (-1: not timed).
int prof_before(const char *name, hipStream_t s) {
  if (t_capture_kernels >= 0) {  // inside a graph capture: count, never time
    ++t_capture_kernels;
    return -1;
  }
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || g_prof.recs.size() >= g_prof.cap) return -1;
  const int k = (int)g_prof.recs.size();
  ProfRec r{name, g_prof.pool[2 * k], g_prof.pool[2 * k + 1]};
  hipEventRecord(r.start, s);
  g_prof.recs.push_back(r);
  return k;
}

void prof_after(int k, hipStream_t s) {
  if (k < 0) return;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (k < (int)g_prof.recs.size()) hipEventRecord(g_prof.recs[k].stop, s);
}

static CacheView view(const tv_cache &c) {
  return CacheView{c.ring, c.c4, c.c4_idx, c.c128, c.c4_base, c.c128_base, c.c4_cap, c.c128_cap, c.len,
                   c.page_table};
}

#define TV_LAUNCH_ON(name, call, strm)    \
  do {                                    \
    const int k_ = prof_before(name, strm); \
    hipError_t e_ = (call);               \
    prof_after(k_, strm);                 \
    if (e_ != hipSuccess) return TV_ERR_LAUNCH; \
  } while (0)
#define TV_LAUNCH(name, call) TV_LAUNCH_ON(name, call, stream)

}  // namespace tv

using namespace tv;

// Workspace of tv_verify_attention_noalloc: one array per device, loaded with
// the library's code object and held until the process ends.  Host code must
// never pass the array's name to a kernel (on the host it is a stand-in, not
// a device address): its device address is looked up once per device and
// cached below.
static __device__ __align__(256) unsigned char scratch[TV_NOALLOC_SCRATCH_BYTES];

namespace tv {

// Device address of the current device's scratch array (first call on a
// device: hipGetSymbolAddress with that device current).
static tv_status noalloc_scratch(void **ptr) {
  static std::mutex mu;
  static std::vector<void *> addr;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TV_ERR_DEVICE;
  std::lock_guard<std::mutex> lk(mu);
  if ((int)addr.size() <= dev) addr.resize(dev + 1, nullptr);
  if (!addr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TV_ERR_DEVICE;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return TV_OK;
}

// Argument checks of the mask and compression calls (no launch).
static tv_status mask_check(const tv_dims *dims, const int32_t *parents, const uint64_t *anc, const int32_t *depth,
                            const int32_t *row_status) {
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (!parents || !anc || !depth || !row_status) return TV_ERR_INVALID_ARG;
  if (!all_a16(parents, anc, depth, row_status)) return TV_ERR_INVALID_ARG;
  return check_device();
}
static tv_status compress_check(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                                const uint64_t *anc, const int32_t *depth, const uint16_t *gate_w,
                                const uint16_t *scr_c4, const uint16_t *scr_c128, const int32_t *row_status,
                                const int32_t *primary_last) {
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (!cache_complete(*dims, cache) || !tree_u || !anc || !depth || !gate_w || !scr_c4 || !scr_c128 || !row_status)
    return TV_ERR_INVALID_ARG;
  if (!cache_a16(cache) || !all_a16(tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status) ||
      (primary_last && !a16(primary_last)))
    return TV_ERR_INVALID_ARG;
  return check_device();
}

// Argument checks of the verify call (no launch).
static tv_status verify_check(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                              const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                              const uint16_t *scr_c128, const uint16_t *q, const uint16_t *q_idx,
                              const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel, int32_t *row_status,
                              void *workspace, size_t workspace_bytes) {
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (!cache_complete(*dims, cache) || !tree_u || !anc || !depth || !scr_c4 || !scr_c128 || !q || !q_idx || !w_idx ||
      !out || !row_status)
    return TV_ERR_INVALID_ARG;
  if (!cache_a16(cache) || !all_a16(tree_u, anc, depth, scr_c4, scr_c128, q, q_idx, w_idx, out, row_status) ||
      (lse && !a16(lse)) || (sel && !a16(sel)))
    return TV_ERR_INVALID_ARG;
  const WsLayout w = ws_layout(*dims);
  if (!workspace || workspace_bytes < w.total) return TV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) & 255) return TV_ERR_INVALID_ARG;
  return check_device();
}

// The verify call's first kernel, the indexer scoring: it reads the committed
// state and the indexer queries only, not the compression's scratch.
static tv_status verify_score(const tv_dims &d, const tv_cache *cache, const uint16_t *q_idx, const uint16_t *w_idx,
                              int32_t *row_status, void *workspace, hipStream_t stream) {
  const WsLayout w = ws_layout(d);
  float *scores = reinterpret_cast<float *>(static_cast<char *>(workspace) + w.scores);
  TV_LAUNCH("indexer_score", launch_score(d, view(*cache), q_idx, w_idx, row_status, scores, w.score_stride, stream));
  return TV_OK;
}

// The rest of the verify call: selection (and merge), attention (and combine).
// With hca_gate_w (the split compression's gate rows), the top-k launch also
// pools the HCA entries into hca_out (the scr_c128 buffer).
static tv_status verify_rest(const tv_dims &d, const tv_cache *cache, const uint16_t *tree_u, const uint64_t *anc,
                             const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128, const uint16_t *q,
                             const uint16_t *q_idx, const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel,
                             int32_t *row_status, void *workspace, hipStream_t stream,
                             const uint16_t *hca_gate_w = nullptr, uint16_t *hca_out = nullptr) {
  const WsLayout w = ws_layout(d);
  char *ws = static_cast<char *>(workspace);
  float *scores = reinterpret_cast<float *>(ws + w.scores);
  int32_t *selp = sel ? sel : reinterpret_cast<int32_t *>(ws + w.sel);
  float *part_o = reinterpret_cast<float *>(ws + w.part_o);
  float *part_ml = reinterpret_cast<float *>(ws + w.part_ml);
  const CacheView cv = view(*cache);
  int32_t *row_order = reinterpret_cast<int32_t *>(ws + w.row_order);
  int32_t *row_rank = reinterpret_cast<int32_t *>(ws + w.row_rank);
  const uint16_t **keytab = reinterpret_cast<const uint16_t **>(ws + w.keytab);
  int32_t *nkeys = reinterpret_cast<int32_t *>(ws + w.nkeys);
  int32_t *nkeys_rank = reinterpret_cast<int32_t *>(ws + w.nkeys_rank);
  int32_t *surv_idx = reinterpret_cast<int32_t *>(ws + w.surv_idx);
  uint32_t *surv_key = reinterpret_cast<uint32_t *>(ws + w.surv_key);
  int32_t *surv_cnt = reinterpret_cast<int32_t *>(ws + w.surv_cnt);
  TV_LAUNCH("topk_select", launch_topk(d, cv, tree_u, anc, depth, scr_c4, scr_c128, q_idx, w_idx, scores,
                                       w.score_stride, selp, row_status, row_order, row_rank, keytab, w.plan.max_keys,
                                       nkeys, nkeys_rank, surv_idx, surv_key, surv_cnt, hca_gate_w, hca_out,
                                       stream));
  if (topk_max_segments(d) > 1)
    TV_LAUNCH("topk_merge", launch_topk_merge(d, cv, anc, depth, scr_c4, selp, row_status, row_rank, keytab,
                                              w.plan.max_keys, surv_idx, surv_key, surv_cnt, stream));
  TV_LAUNCH("verify_attn", launch_attn(d, q, row_status, row_order, keytab, nkeys_rank, w.plan, part_o, part_ml, out,
                                       lse, stream));
  if (w.plan.splits > 1)
    TV_LAUNCH("attn_combine", launch_combine(d, row_status, nkeys, w.plan, part_o, part_ml, out, lse, stream));
  return TV_OK;
}

static tv_status verify_impl(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                              const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                              const uint16_t *scr_c128, const uint16_t *q, const uint16_t *q_idx,
                              const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel, int32_t *row_status,
                              void *workspace, size_t workspace_bytes, hipStream_t stream) {
  tv_status st = verify_check(dims, cache, tree_u, anc, depth, scr_c4, scr_c128, q, q_idx, w_idx, out, lse, sel,
                              row_status, workspace, workspace_bytes);
  if (st != TV_OK) return st;
  if ((st = verify_score(*dims, cache, q_idx, w_idx, row_status, workspace, stream)) != TV_OK) return st;
  return verify_rest(*dims, cache, tree_u, anc, depth, scr_c4, scr_c128, q, q_idx, w_idx, out, lse, sel, row_status,
                     workspace, stream);
}

// One layer's verify preprocess (with_mask), compression and verification.
// With the scoring's fast path, a flat pool and the split compression, no
// kernel of its own is left for the compression: the first launch runs the
// mask (with_mask), the CSA entries (a wavefront per node; beside the mask
// from the parent array) and the indexer scoring (it reads neither the masks
// nor the scratch), and the top-k's launch also runs the HCA entries (the
// top-k only lists their addresses).  With the mask and the scoring's fast
// path otherwise, the mask and the scoring share a launch before the
// compression.  Otherwise the calls' kernels in the calls' order.  Every part computes what it computes
// in the separate calls, so the results are the same bits.  Arguments already
// checked.
static tv_status layer_step(const tv_dims *d, const tv_round &r, const tv_layer &L, bool with_mask,
                            hipStream_t stream) {
  const bool split = score_fast_path(*d) && d->page_size == 0 && compress_split(*d);
  const bool fused = (with_mask && score_fast_path(*d)) || split;
  if (fused) {
    const WsLayout w = ws_layout(*d);
    float *scores = reinterpret_cast<float *>(static_cast<char *>(L.workspace) + w.scores);
    TV_LAUNCH("mask_score", launch_mask_score(*d, with_mask ? r.parents : nullptr, r.anc, r.depth, r.row_status,
                                              view(L.cache), L.q_idx,
                                              L.w_idx, scores, w.score_stride, split ? L.tree_u : nullptr,
                                              split ? L.gate_w : nullptr, split ? L.scr_c4 : nullptr,
                                              split ? r.primary_last : nullptr, split ? L.cache.c4 : nullptr,
                                              split ? L.cache.c4_idx : nullptr, stream));
  } else if (with_mask) {
    TV_LAUNCH("tree_mask", launch_mask(*d, r.parents, r.anc, r.depth, r.row_status, stream));
  }
  if (!split)
    TV_LAUNCH("branch_compress", launch_compress(*d, view(L.cache), L.tree_u, r.anc, r.depth, L.gate_w, L.scr_c4,
                                                 L.scr_c128, r.row_status, r.primary_last, L.cache.c4,
                                                 L.cache.c4_idx, stream));
  if (!fused) {
    const tv_status st = verify_score(*d, &L.cache, L.q_idx, L.w_idx, r.row_status, L.workspace, stream);
    if (st != TV_OK) return st;
  }
  return verify_rest(*d, &L.cache, L.tree_u, r.anc, r.depth, L.scr_c4, L.scr_c128, L.q, L.q_idx, L.w_idx, L.out,
                     L.lse, L.sel, r.row_status, L.workspace, stream, split ? L.gate_w : nullptr,
                     split ? L.scr_c128 : nullptr);
}

static tv_status commit_check(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                              const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                              const uint16_t *scr_c128, const int32_t *accepted_last, const int32_t *accept_nodes,
                              const int32_t *accept_len, const int32_t *row_status, const int32_t *primary_last) {
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (!cache_complete(*dims, cache) || !tree_u || !anc || !depth || !scr_c4 || !scr_c128 || !accepted_last ||
      !accept_nodes || !accept_len || !row_status)
    return TV_ERR_INVALID_ARG;
  if (!cache_a16(cache) ||
      !all_a16(tree_u, anc, depth, scr_c4, scr_c128, accepted_last, accept_nodes, accept_len, row_status) ||
      (primary_last && !a16(primary_last)))
    return TV_ERR_INVALID_ARG;
  return check_device();
}

static tv_status layer_check(const tv_dims *d, const tv_round &r, const tv_layer &L) {
  tv_status st = compress_check(d, &L.cache, L.tree_u, r.anc, r.depth, L.gate_w, L.scr_c4, L.scr_c128, r.row_status,
                                r.primary_last);
  if (st != TV_OK) return st;
  return verify_check(d, &L.cache, L.tree_u, r.anc, r.depth, L.scr_c4, L.scr_c128, L.q, L.q_idx, L.w_idx, L.out,
                      L.lse, L.sel, r.row_status, L.workspace, L.workspace_bytes);
}

}  // namespace tv

extern "C" {

const char *tv_status_string(int s) {
  switch (s) {
    case TV_OK: return "ok";
    case TV_ERR_INVALID_ARG: return "invalid argument";
    case TV_ERR_UNSUPPORTED: return "unsupported dimensions";
    case TV_ERR_WORKSPACE: return "workspace missing or too small";
    case TV_ERR_LAUNCH: return "kernel launch failed";
    case TV_ERR_DEVICE: return "no gfx950 device";
    default: return "unknown status";
  }
}

tv_status tv_build_tree_mask(const tv_dims *dims, const int32_t *parents, uint64_t *anc, int32_t *depth,
                             int32_t *row_status, hipStream_t stream) {
  const tv_status st = mask_check(dims, parents, anc, depth, row_status);
  if (st != TV_OK) return st;
  TV_LAUNCH("tree_mask", launch_mask(*dims, parents, anc, depth, row_status, stream));
  return TV_OK;
}

tv_status tv_branch_compress(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                             const uint64_t *anc, const int32_t *depth, const uint16_t *gate_w, uint16_t *scr_c4,
                             uint16_t *scr_c128, int32_t *row_status, const int32_t *primary_last,
                             hipStream_t stream) {
  tv_status st = compress_check(dims, cache, tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status, primary_last);
  if (st != TV_OK) return st;
  TV_LAUNCH("branch_compress", launch_compress(*dims, view(*cache), tree_u, anc, depth, gate_w, scr_c4, scr_c128,
                                               row_status, primary_last, cache->c4, cache->c4_idx, stream));
  return TV_OK;
}

tv_status tv_verify_round(const tv_dims *dims, const tv_round *round, const tv_layer *layer, hipStream_t stream) {
  if (!round || !layer) return TV_ERR_INVALID_ARG;
  const bool with_mask = round->parents != nullptr;  // NULL: anc and depth already hold this round's mask
  tv_status st = layer_check(dims, *round, *layer);
  if (st != TV_OK) return st;
  if (with_mask && (st = mask_check(dims, round->parents, round->anc, round->depth, round->row_status)) != TV_OK)
    return st;
  return layer_step(dims, *round, *layer, with_mask, stream);
}

size_t tv_verify_workspace_bytes(const tv_dims *dims) {
  if (check_dims(dims) != TV_OK) return 0;
  return ws_layout(*dims).total;
}

tv_status tv_verify_attention(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                              const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                              const uint16_t *scr_c128, const uint16_t *q, const uint16_t *q_idx,
                              const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel, int32_t *row_status,
                              void *workspace, size_t workspace_bytes, hipStream_t stream) {
  return verify_impl(dims, cache, tree_u, anc, depth, scr_c4, scr_c128, q, q_idx, w_idx, out, lse, sel, row_status,
                     workspace, workspace_bytes, stream);
}

tv_status tv_verify_attention_noalloc(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                                      const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                                      const uint16_t *scr_c128, const uint16_t *q, const uint16_t *q_idx,
                                      const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel,
                                      int32_t *row_status, hipStream_t stream) {
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (ws_layout(*dims).total > TV_NOALLOC_SCRATCH_BYTES) return TV_ERR_WORKSPACE;
  if ((st = check_device()) != TV_OK) return st;
  void *ws = nullptr;
  if ((st = noalloc_scratch(&ws)) != TV_OK) return st;
  return verify_impl(dims, cache, tree_u, anc, depth, scr_c4, scr_c128, q, q_idx, w_idx, out, lse, sel, row_status,
                     ws, TV_NOALLOC_SCRATCH_BYTES, stream);
}

tv_status tv_commit_accepted_path(const tv_dims *dims, tv_cache *cache, const uint16_t *tree_u, const uint64_t *anc,
                                  const int32_t *depth, const uint16_t *scr_c4, const uint16_t *scr_c128,
                                  const int32_t *accepted_last, int32_t *accept_nodes, int32_t *accept_len,
                                  int32_t *row_status, const int32_t *primary_last, hipStream_t stream) {
  const tv_status st = commit_check(dims, cache, tree_u, anc, depth, scr_c4, scr_c128, accepted_last, accept_nodes,
                                    accept_len, row_status, primary_last);
  if (st != TV_OK) return st;
  TV_LAUNCH("commit_path", launch_commit(*dims, *cache, tree_u, anc, depth, scr_c4, scr_c128, accepted_last,
                                         accept_nodes, accept_len, row_status, primary_last, stream));
  return TV_OK;
}

size_t tv_select_workspace_bytes(const tv_dims *dims, int32_t vocab) {
  if (check_dims(dims) != TV_OK || vocab < 1) return 0;
  return align256(sizeof(uint64_t) * (size_t)dims->B * dims->D * select_chunks(vocab));
}

tv_status tv_select_accepted_path(const tv_dims *dims, const int32_t *parents, const uint64_t *anc,
                                  const int32_t *depth, const int32_t *draft_tokens, const uint16_t *target_logits,
                                  int32_t vocab, int32_t *target_tokens, int32_t *accepted_last,
                                  int32_t *next_token, const int32_t *row_status, void *workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (vocab < 1) return TV_ERR_INVALID_ARG;
  if (!parents || !anc || !depth || !draft_tokens || !target_logits || !target_tokens || !accepted_last ||
      !row_status)
    return TV_ERR_INVALID_ARG;
  if (!all_a16(parents, anc, depth, draft_tokens, target_logits, target_tokens, accepted_last, row_status) ||
      (next_token && !a16(next_token)))
    return TV_ERR_INVALID_ARG;
  const size_t need = tv_select_workspace_bytes(dims, vocab);
  if (!workspace || workspace_bytes < need) return TV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) & 255) return TV_ERR_INVALID_ARG;
  if ((int64_t)dims->B * dims->D * select_chunks(vocab) > 0x7FFFFFFF) return TV_ERR_UNSUPPORTED;
  if ((st = check_device()) != TV_OK) return st;
  uint64_t *part = static_cast<uint64_t *>(workspace);
  TV_LAUNCH("target_argmax", launch_argmax(*dims, target_logits, vocab, part, stream));
  TV_LAUNCH("select_path", launch_select(*dims, parents, anc, depth, draft_tokens, vocab, part, row_status,
                                         target_tokens, accepted_last, next_token, stream));
  return TV_OK;
}

}  // extern "C"

struct tv_round_graph {
  hipGraph_t graph;
  hipGraphExec_t exec;
  int32_t kernels;
};

namespace tv {

// The calls of one round, in order, on stream s (argument checks included).
static tv_status record_round(const tv_dims *d, const tv_round &r, const tv_layer *layers, int n, hipStream_t s) {
  tv_status st = mask_check(d, r.parents, r.anc, r.depth, r.row_status);
  for (int l = 0; l < n && st == TV_OK; ++l) {  // each layer as tv_verify_round runs it, the mask with layer 0
    if ((st = layer_check(d, r, layers[l])) == TV_OK) st = layer_step(d, r, layers[l], l == 0, s);
  }
  if (st == TV_OK && r.target_logits)
    st = tv_select_accepted_path(d, r.parents, r.anc, r.depth, r.draft_tokens, r.target_logits, r.vocab,
                                 r.target_tokens, r.accepted_last, r.next_token, r.row_status, r.select_workspace,
                                 r.select_workspace_bytes, s);
  // the commits: one launch per group of up to kCommitMaxLayers layers, each row walking its layers in order
  for (int l0 = 0; l0 < n && st == TV_OK; l0 += kCommitMaxLayers) {
    CommitLayers ls{};
    ls.n = std::min(n - l0, kCommitMaxLayers);
    for (int k = 0; k < ls.n && st == TV_OK; ++k) {
      const tv_layer &L = layers[l0 + k];
      st = commit_check(d, &L.cache, L.tree_u, r.anc, r.depth, L.scr_c4, L.scr_c128, r.accepted_last,
                        r.accept_nodes, r.accept_len, r.row_status, r.primary_last);
      ls.l[k] = CommitLayer{L.cache, L.tree_u, L.scr_c4, L.scr_c128};
    }
    if (st != TV_OK) break;
    hipStream_t stream = s;
    TV_LAUNCH("commit_path", launch_commit_layers(*d, ls, r.anc, r.depth, r.accepted_last, r.accept_nodes,
                                                  r.accept_len, r.row_status, r.primary_last, stream));
  }
  return st;
}

}  // namespace tv

extern "C" {

tv_status tv_round_graph_create(const tv_dims *dims, const tv_round *round, const tv_layer *layers,
                                int32_t n_layers, tv_round_graph **graph) {
  if (!graph) return TV_ERR_INVALID_ARG;
  *graph = nullptr;
  tv_status st = check_dims(dims);
  if (st != TV_OK) return st;
  if (!round || !layers || n_layers < 1 || n_layers > 1024) return TV_ERR_INVALID_ARG;
  if (!round->target_logits && (round->draft_tokens || round->target_tokens)) return TV_ERR_INVALID_ARG;
  if ((st = check_device()) != TV_OK) return st;
  hipStream_t cs = nullptr;
  if (hipStreamCreateWithFlags(&cs, hipStreamNonBlocking) != hipSuccess) return TV_ERR_DEVICE;
  if (hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal) != hipSuccess) {
    (void)hipStreamDestroy(cs);
    return TV_ERR_LAUNCH;
  }
  t_capture_kernels = 0;
  st = record_round(dims, *round, layers, n_layers, cs);
  const int32_t kernels = t_capture_kernels;
  t_capture_kernels = -1;
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(cs, &g);
  (void)hipStreamDestroy(cs);
  if (st != TV_OK || e != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    return st != TV_OK ? st : TV_ERR_LAUNCH;
  }
  hipGraphExec_t x = nullptr;
  if (hipGraphInstantiate(&x, g, nullptr, nullptr, 0) != hipSuccess) {
    (void)hipGraphDestroy(g);
    return TV_ERR_LAUNCH;
  }
  *graph = new tv_round_graph{g, x, kernels};
  return TV_OK;
}

int32_t tv_round_graph_kernels(const tv_round_graph *graph) { return graph ? graph->kernels : 0; }

tv_status tv_round_graph_launch(tv_round_graph *graph, hipStream_t stream) {
  if (!graph) return TV_ERR_INVALID_ARG;
  return hipGraphLaunch(graph->exec, stream) == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

tv_status tv_round_graph_destroy(tv_round_graph *graph) {
  if (!graph) return TV_ERR_INVALID_ARG;
  const bool ok = hipGraphExecDestroy(graph->exec) == hipSuccess && hipGraphDestroy(graph->graph) == hipSuccess;
  delete graph;
  return ok ? TV_OK : TV_ERR_LAUNCH;
}

tv_status tv_profile_enable(int32_t capacity) {
  if (capacity < 1 || capacity > (1 << 20)) return TV_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  for (hipEvent_t e : g_prof.pool) hipEventDestroy(e);
  g_prof.pool.assign(2 * (size_t)capacity, nullptr);
  for (auto &e : g_prof.pool)
    if (hipEventCreate(&e) != hipSuccess) return TV_ERR_DEVICE;
  g_prof.recs.clear();
  g_prof.recs.reserve(capacity);
  g_prof.cap = capacity;
  g_prof.on = true;
  return TV_OK;
}

tv_status tv_profile_disable(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = false;
  return TV_OK;
}

tv_status tv_profile_read(tv_kernel_time *out, int32_t max_entries, int32_t *n_entries) {
  if (!out || !n_entries || max_entries < 1) return TV_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  std::vector<tv_kernel_time> acc;
  for (const ProfRec &r : g_prof.recs) {
    if (hipEventSynchronize(r.stop) != hipSuccess) return TV_ERR_DEVICE;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) return TV_ERR_DEVICE;
    auto it = std::find_if(acc.begin(), acc.end(), [&](const tv_kernel_time &k) { return std::strcmp(k.name, r.name) == 0; });
    if (it == acc.end()) {
      tv_kernel_time k{};
      std::strncpy(k.name, r.name, sizeof(k.name) - 1);
      acc.push_back(k);
      it = acc.end() - 1;
    }
    it->launches += 1;
    it->total_ms += ms;
  }
  g_prof.recs.clear();
  const int n = (int)std::min<size_t>(acc.size(), (size_t)max_entries);
  for (int k = 0; k < n; ++k) out[k] = acc[k];
  *n_entries = n;
  return TV_OK;
}

}  // extern "C"
