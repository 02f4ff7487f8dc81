/*
 * tv.h - tree-structured speculative verification over CSA/HCA compressed
 * attention, for one MI355X (gfx950) GPU.
 *
 * The library implements the target-verify step of tree speculation on a model
 * whose history is compressed online along the sequence (the paper's Sec. 3
 * "Challenges" and Sec. 4 "Our Approach"):
 *
 *   tv_build_tree_mask       verify preprocess: draft tree -> per-node ancestor
 *                            bitmask and depth (Sec. 4.1; device-side metadata,
 *                            Sec. 4.3)
 *   tv_branch_compress       each node compresses the block it closes along its
 *                            own root path into a scratch slot, never mixing
 *                            branches (Sec. 4.1, Sec. 4.2)
 *   tv_verify_attention      branch-aware causal verification: every node
 *                            attends to the committed compressed history plus
 *                            its own ancestors only (Sec. 3.1, Sec. 4.1)
 *   tv_select_accepted_path  greedy accepted-path selection from the target's
 *                            logits at every node (Sec. 4.1, Sec. 4.4)
 *   tv_commit_accepted_path  accepted-path refresh of token window, CSA and HCA
 *                            state; rejected branches leave no trace (Sec. 3.2,
 *                            Sec. 4.2)
 *   tv_verify_round          mask, compression and verification of one layer in
 *                            one call, with fewer launches: the compression and
 *                            the indexer scoring ride in the mask's and the
 *                            top-k's launches (Sec. 4.1, Sec. 4.3)
 *
 * Reading of the compressed-attention arithmetic (the paper cites DeepSeek-V4
 * for it): a ratio-r entry pools the r raw rows of a block with softmax
 * weights of the gate logits g_r . u; the CSA (ratio_csa) entry keeps every
 * channel of the raw row (latent row, then indexer key), the HCA (ratio_hca)
 * entry the latent row.  A node scores every visible CSA entry with
 * sum_h w[h] * relu(q_idx[h] . key), keeps the topk best (score descending,
 * then logical index ascending), and runs one softmax over those entries,
 * every visible HCA entry and the raw window of the last `window` positions
 * up to and including itself.  Keys are row[0:d_k], values row[v_off:v_off+d_v].
 *
 * Conventions shared by every call
 *   - Every pointer is device memory owned by the caller.  The library never
 *     allocates device memory and keeps no state between calls besides device
 *     properties, the array of tv_verify_attention_noalloc and the optional
 *     profiling records.
 *   - Every buffer must start on a 16-byte boundary (the kernels move rows
 *     with 16-byte accesses); a misaligned pointer is TV_ERR_INVALID_ARG.
 *   - The verify workspace must be 256-byte aligned.
 *   - Calls enqueue work on `stream` and return without synchronising the
 *     host.  Issue them in the order mask -> compress -> verify -> select ->
 *     commit (select is optional when the accepted node is known).
 *   - Floating-point buffers hold bfloat16 bit patterns (uint16_t) unless
 *     stated otherwise; arithmetic is float32 on the device.
 *   - A row is the draft tree of one sequence.  Node 0 is the root; node i has
 *     parent parents[i] < i.  The committed length of row b is len[b] = L; the
 *     root stands at position L and node i at L + depth[i].
 *   - Host-checkable problems return a tv_status other than TV_OK and launch
 *     nothing.  Data problems found on the device are written to
 *     row_status[b] (first error wins); a row whose status is not TV_ROW_OK is
 *     skipped by every later call and its outputs and cache are left as they
 *     were.
 */
#ifndef TV_H
#define TV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TV_OK = 0,
  TV_ERR_INVALID_ARG = 1, /* null pointer, bad size or inconsistent dims */
  TV_ERR_UNSUPPORTED = 2, /* valid dims the library has no kernel for */
  TV_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  TV_ERR_LAUNCH = 4,      /* a HIP call failed while enqueuing work */
  TV_ERR_DEVICE = 5       /* no current HIP device, or it is not gfx950 */
} tv_status;

/* Per-row data errors written to row_status[b]. */
enum {
  TV_ROW_OK = 0,
  TV_ROW_BAD_PARENT = 1, /* parents[b][0] != -1 or parents[b][i] outside [0, i) */
  TV_ROW_BAD_ACCEPT = 2, /* accepted_last[b] outside [0, D) */
  TV_ROW_CAPACITY = 3,   /* a committed entry would land beyond c4_cap/c128_cap */
  TV_ROW_BAD_LEN = 4     /* len[b] < 0 or len[b] > max_len */
};

/* Sizes of one verify round.  Supported head shapes:
 *   H=64, d_row=576, d_k=576, v_off=0,   d_v=512  (shared MLA latent row)
 *   H=8,  d_row=256, d_k=128, v_off=128, d_v=128  (one KV head, row = K|V)
 * with d_idx = 64 and H_idx a power of two <= 64. */
typedef struct {
  int32_t B;         /* rows (sequences), 1..4096 */
  int32_t D;         /* tree nodes per row including the root, 1..64 */
  int32_t H;         /* query heads sharing the single KV row */
  int32_t d_row;     /* width of a latent KV row (compressed entries, window keys) */
  int32_t d_k;       /* key channels row[0:d_k] */
  int32_t v_off;     /* value channels row[v_off:v_off+d_v] */
  int32_t d_v;
  int32_t d_idx;     /* indexer key width; a raw token row has d_u = d_row + d_idx channels */
  int32_t H_idx;     /* indexer heads */
  int32_t ratio_csa; /* CSA compression ratio (4) */
  int32_t ratio_hca; /* HCA compression ratio (128) */
  int32_t window;    /* raw sliding window in positions, the query included (128) */
  int32_t topk;      /* CSA entries kept per node, 1..8192; with more than 16,896 candidates a node is
                        selected in segments of that many, at most 64 of them and segments x topk <= 34,816
                        (TV_ERR_UNSUPPORTED otherwise) */
  int32_t ring_cap;  /* raw-token ring slots per row: power of two >= max(window + D, ratio_csa, ratio_hca),
                        so one commit of up to D rows never writes two rows to one slot */
  int32_t max_len;   /* bound on every len[b]; sizes launches and the verify workspace */
  float scale;       /* logit scale, finite and > 0, normally 1/sqrt(d_k) */
  int32_t idx_fmt;   /* number format of stored indexer keys: TV_IDX_BF16, or TV_IDX_E4M3 (FP8 keys, a
                        fidelity reading of the CSA indexer: the c4_idx pool holds one OCP E4M3 code per
                        channel, and the indexer channels of a CSA scratch entry hold E4M3 values widened
                        to bfloat16; compression rounds the pooled key to E4M3, nearest even, saturating
                        at +-448; scoring widens keys exactly and multiplies them with bfloat16 queries) */
  int32_t page_size;   /* 0: flat pools and a ring per row.  > 0: the paged pool (Sec. 4.2: one logical layer
                          of positions over three physical layers sharing page-level pointers), pages of
                          page_size tokens, a power of two and a multiple of ratio_csa and ratio_hca */
  int32_t page_stride; /* paged pool: page-table entries per row (>= 1) */
} tv_dims;

enum { TV_IDX_BF16 = 0, TV_IDX_E4M3 = 1 };

/* Committed (persistent) state of every row.  Only tv_commit_accepted_path
 * writes its committed part; verify only reads it (Sec. 4.2: speculative
 * branch state never touches the persistent cache before acceptance).  The
 * one exception is the refresh schedule of tv_branch_compress with a
 * designated chain, which writes CSA pool slots past the committed entries:
 * slots no call reads until a commit makes them committed. */
typedef struct {
  uint16_t *ring;   /* [B][ring_cap][d_row + d_idx]: raw row of position q in slot q & (ring_cap-1) */
  uint16_t *c4;     /* [*][d_row]: CSA entry s of row b at c4[c4_base[b] + s], s < len/ratio_csa */
  uint16_t *c4_idx; /* [*][d_idx]: indexer key of the same CSA entry (bfloat16 bits, or one byte per
                       channel, E4M3 codes, with idx_fmt TV_IDX_E4M3) */
  uint16_t *c128;   /* [*][d_row]: HCA entry s of row b at c128[c128_base[b] + s] */
  const int64_t *c4_base;   /* [B] first pool slot of each row */
  const int32_t *c4_cap;    /* [B] pool slots owned by each row */
  const int64_t *c128_base; /* [B] */
  const int32_t *c128_cap;  /* [B] */
  int32_t *len;             /* [B] committed tokens L of each row */
  /* Paged pool (dims page_size P > 0): page_table [B][page_stride] gives the physical page of each logical
   * page j (positions jP..jP+P-1) of each row, -1 where none is allocated.  The page id addresses all three
   * layers: ring becomes [pages][P][d_row + d_idx] (position q at [page(q / P)][q % P]); c4 and c4_idx hold
   * P/ratio_csa entries per page (entry s at slot page(s * ratio_csa / P) * (P/ratio_csa) + s % (P/ratio_csa)),
   * c128 likewise with ratio_hca; c4_base, c4_cap, c128_base, c128_cap are not read (may be NULL).  Every
   * page overlapping positions 0..len-1 must be allocated (compression fails a row whose committed rows it
   * cannot find, TV_ROW_CAPACITY); a commit needing a page with no id fails the row, TV_ROW_CAPACITY.  Page
   * ids must lie within the caller's layers.  NULL with page_size 0. */
  const int32_t *page_table;
} tv_cache;

/* Verify preprocess (Sec. 4.1): for every row, validate the parent array and
 * build per node the ancestor bitmask (bit j set iff node j is i or an ancestor
 * of i; bit i set, bit 0 set) and depth (root 0).
 *   parents    int32 [B][D], read
 *   anc        uint64 [B][D], written (0 for a bad row)
 *   depth      int32 [B][D], written (0 for a bad row)
 *   row_status int32 [B], written: TV_ROW_OK or TV_ROW_BAD_PARENT (resets the row) */
tv_status tv_build_tree_mask(const tv_dims *dims, const int32_t *parents, uint64_t *anc,
                             int32_t *depth, int32_t *row_status, hipStream_t stream);

/* Per-branch compression into scratch (Sec. 4.1, Sec. 4.2).  Node i at
 * position p = L + depth[i] closes a ratio-r block when (p + 1) % r == 0; the
 * block is positions p-r+1..p of "committed tokens, then the root path of i"
 * (committed tokens from the ring, path tokens from tree_u).  Its CSA entry
 * (d_row + d_idx channels) goes to scr_c4[b][i], its HCA entry (d_row
 * channels) to scr_c128[b][i]; slots of nodes that close nothing are not
 * written.
 *   tree_u   [B][D][d_row + d_idx] raw rows of the draft tokens, read
 *   gate_w   [2][d_row + d_idx] gate vectors for ratio_csa then ratio_hca, read
 *   row_status in/out: a row with len outside [0, max_len] becomes TV_ROW_BAD_LEN
 *   primary_last  int32 [B] or NULL.  Refresh schedule (Sec. 4.3): the root
 *            path of primary_last[b] is the row's designated chain (say, the
 *            drafter's first choice); the CSA entries its nodes close are also
 *            written to their pool slots c4/c4_idx[c4_base[b] + s], s =
 *            (p+1)/ratio_csa - 1, when s < c4_cap[b].  A value outside [0, D)
 *            designates no chain.  Pass the same array to the commit. */
tv_status tv_branch_compress(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                             const uint64_t *anc, const int32_t *depth, const uint16_t *gate_w,
                             uint16_t *scr_c4, uint16_t *scr_c128, int32_t *row_status,
                             const int32_t *primary_last, hipStream_t stream);

/* Bytes of device workspace tv_verify_attention needs for these dims (the
 * largest row is bounded by dims->max_len).  0 on invalid dims. */
size_t tv_verify_workspace_bytes(const tv_dims *dims);

/* Branch-aware verify attention (Sec. 3.1, Sec. 4.1).  For node i of row b:
 *   CSA candidates: committed entries 0..L/ratio_csa-1 and the scratch entries
 *     closed by i and its ancestors (logical index (p_j+1)/ratio_csa - 1);
 *   HCA keys: committed entries and the scratch entries closed on the path;
 *   window keys: raw rows of positions max(0, p_i-window+1)..p_i (committed
 *     ones from the ring, path ones from tree_u).
 *   q        [B][D][H][d_k], q_idx [B][D][H_idx][d_idx], w_idx [B][D][H_idx], read
 *   out      [B][D][H][d_v] bfloat16, written
 *   lse      float32 [B][D][H] natural-log sum of exp(logits), written if not NULL
 *   sel      int32 [B][D][topk] chosen CSA logical indices ascending, -1 padded,
 *            written if not NULL
 *   workspace  device scratch of at least tv_verify_workspace_bytes(dims),
 *            contents on entry ignored
 * Reads the cache only.  Rows with nonzero status are skipped. */
tv_status tv_verify_attention(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                              const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                              const uint16_t *scr_c128, const uint16_t *q, const uint16_t *q_idx,
                              const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel,
                              int32_t *row_status, void *workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* Size of the device array tv_verify_attention_noalloc works in. */
#define TV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* tv_verify_attention without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments (but workspace), same
 * outputs and errors.  The library allocates nothing either: the workspace is
 * a static device array of TV_NOALLOC_SCRATCH_BYTES (64 MiB), one per device,
 * present from the library's first use on a device until the process ends.
 * Returns TV_ERR_WORKSPACE when tv_verify_workspace_bytes(dims) exceeds it
 * (it holds the B=64, 64K-token and the 1M-token workloads, 38 and 41 MiB).
 * Every call on one device shares that device's array: calls that overlap on
 * one device (on different streams, or from different threads) race on it
 * and must be serialised by the caller.  Nothing in the array has to start at
 * zero; its contents on entry are ignored. */
tv_status tv_verify_attention_noalloc(const tv_dims *dims, const tv_cache *cache, const uint16_t *tree_u,
                                      const uint64_t *anc, const int32_t *depth, const uint16_t *scr_c4,
                                      const uint16_t *scr_c128, const uint16_t *q, const uint16_t *q_idx,
                                      const uint16_t *w_idx, uint16_t *out, float *lse, int32_t *sel,
                                      int32_t *row_status, hipStream_t stream);

/* Accepted-path refresh (Sec. 3.2, Sec. 4.2).  The accepted path is the root
 * path of accepted_last[b], a = depth + 1 nodes.  Writes the raw rows of the
 * path into ring slots of positions L..L+a-1, the scratch entry of every path
 * node that closed a block into the pools at its logical index, len[b] = L + a,
 * accept_nodes[b][0:a] = path (root first, -1 after it) and accept_len[b] = a.
 * A row that fails a check (accept index, pool capacity) is left untouched and
 * gets the row status.
 *   parents, depth, anc: as produced by tv_build_tree_mask (read)
 *   accepted_last int32 [B], accept_nodes int32 [B][D], accept_len int32 [B]
 *   primary_last  int32 [B] or NULL: the designated chains given to
 *            tv_branch_compress.  CSA copies of accepted nodes on a row's
 *            designated chain are skipped (the compression put them in
 *            place): a single chain, or an accepted path that is the cached
 *            chain, needs no CSA refresh (Sec. 4.3).  HCA entries are always
 *            written here, after the path is known (Sec. 4.3: C128 writes
 *            delayed and combined).  The committed state is the same as
 *            without a designated chain. */
tv_status tv_commit_accepted_path(const tv_dims *dims, tv_cache *cache, const uint16_t *tree_u,
                                  const uint64_t *anc, const int32_t *depth,
                                  const uint16_t *scr_c4, const uint16_t *scr_c128,
                                  const int32_t *accepted_last, int32_t *accept_nodes,
                                  int32_t *accept_len, int32_t *row_status,
                                  const int32_t *primary_last, hipStream_t stream);

/* Bytes of device workspace tv_select_accepted_path needs for these dims and
 * vocabulary size.  0 on invalid dims or vocab < 1. */
size_t tv_select_workspace_bytes(const tv_dims *dims, int32_t vocab);

/* Greedy accepted-path selection after verification (Sec. 4.1: target verify
 * ends by selecting the accepted path; Sec. 3.1: the outcome is one path
 * through the tree).  The target token of node i is the index of the largest
 * of its vocab logits (the first one on ties; a NaN counts as the largest, and
 * -0 equals +0).  A non-root node matches when its draft token equals its
 * parent's target token; a node is accepted when every non-root node on its
 * root path matches; the accepted path ends at the deepest accepted node, the
 * smallest index among equally deep ones.  Called between
 * tv_verify_attention and tv_commit_accepted_path, whose accepted_last it
 * produces.
 *   parents, anc, depth  as read and produced by tv_build_tree_mask (read)
 *   draft_tokens   int32 [B][D] token drafted at each node; the root's is not read (read)
 *   target_logits  bfloat16 [B][D][vocab] the target's next-token logits at each node (read)
 *   target_tokens  int32 [B][D] argmax of each node's logits (written)
 *   accepted_last  int32 [B] last node of the accepted path (written)
 *   next_token     int32 [B] target token of accepted_last, the token the next
 *                  round starts from (written if not NULL)
 *   row_status     read only: rows whose status is not TV_ROW_OK are skipped
 *                  and their outputs left as they were
 *   workspace      device scratch of at least tv_select_workspace_bytes(dims,
 *                  vocab) bytes, 256-byte aligned, contents on entry ignored */
tv_status tv_select_accepted_path(const tv_dims *dims, const int32_t *parents, const uint64_t *anc,
                                  const int32_t *depth, const int32_t *draft_tokens,
                                  const uint16_t *target_logits, int32_t vocab, int32_t *target_tokens,
                                  int32_t *accepted_last, int32_t *next_token, const int32_t *row_status,
                                  void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ---- Captured multi-layer round (Sec. 4.3: graph replay needs stable
 * shapes; the tree configuration bounds what one graph covers) -------------
 *
 * A model verifies the same draft tree in every layer.  One round is the
 * verify preprocess once, then per layer the branch compression and verify
 * attention, then (optionally) the greedy path selection, then per layer the
 * commit.  tv_round_graph_create records that whole sequence, with every
 * argument check done once, into one HIP graph (each layer as tv_verify_round
 * runs it); tv_round_graph_launch replays
 * it on any stream.  A graph is bound to its dims (B, D, max_len: the "D
 * bucket") and to the buffer addresses given at creation; the tree shape,
 * token contents and lengths are read from device memory at replay, so new
 * trees need no new graph.  The graph issues no memory sets and allocates
 * nothing at replay.  Kernel timing is not recorded inside graphs. */

/* The buffers of one layer: its committed state, the inputs and outputs of
 * tv_branch_compress and tv_verify_attention for it. */
typedef struct {
  tv_cache cache;
  const uint16_t *tree_u, *gate_w, *q, *q_idx, *w_idx;
  uint16_t *scr_c4, *scr_c128, *out;
  float *lse;   /* may be NULL */
  int32_t *sel; /* may be NULL */
  void *workspace;
  size_t workspace_bytes;
} tv_layer;

/* The buffers every layer of a round shares.  row_status is shared: a row
 * that fails in any call is skipped by every later call of the round (the
 * layers committed before the failure keep their commit).  When
 * target_logits is not NULL the selection runs after the last verify and
 * writes accepted_last, which every commit then reads; otherwise
 * accepted_last is an input. */
typedef struct {
  const int32_t *parents;
  uint64_t *anc;
  int32_t *depth, *row_status, *accepted_last, *accept_nodes, *accept_len;
  const int32_t *primary_last;     /* designated chains, or NULL (see tv_branch_compress) */
  const int32_t *draft_tokens;     /* selection inputs (may be NULL together) */
  const uint16_t *target_logits;
  int32_t vocab;
  int32_t *target_tokens, *next_token;
  void *select_workspace;
  size_t select_workspace_bytes;
} tv_round;

/* Verify preprocess, branch compression and verify attention of one layer
 * (Sec. 4.1: mask, then per-branch compression, then branch-aware causal
 * attention) in one call, with the same results, bit for bit, as
 * tv_build_tree_mask, tv_branch_compress and tv_verify_attention issued in
 * that order on `stream` with the same arguments.  The indexer scoring reads
 * only committed CSA keys and the indexer queries, neither the masks nor the
 * compression's output, so where its fast path applies (H_idx = 8, D <= 8)
 * it runs in the same kernel launch as the mask.  With a flat pool and CSA
 * blocks of at most 4 tokens, the compression needs no launch of its own
 * either: each CSA entry is pooled by one wavefront in the mask's launch
 * (from the parent array, not the masks being written), and each HCA entry,
 * which the top-k does not read, by a workgroup in the top-k's launch
 * (overlap of independent device work, Sec. 4.3).  Everything runs on `stream`, in order
 * with earlier and later work on it.  The selection inputs of `round`
 * (draft_tokens, target_logits, ...) and accepted_last, accept_nodes,
 * accept_len are not used.  With round->parents NULL the mask is not built:
 * anc and depth are inputs that already hold this round's tree (the later
 * layers of a model that share it).  Every check of the three calls runs
 * before anything is launched. */
tv_status tv_verify_round(const tv_dims *dims, const tv_round *round, const tv_layer *layer, hipStream_t stream);

typedef struct tv_round_graph tv_round_graph;

/* Records one round over n_layers layers (1..1024) into a graph.  Returns
 * the first failing check of any call (nothing is kept then).  The graph is
 * owned by the caller until tv_round_graph_destroy. */
tv_status tv_round_graph_create(const tv_dims *dims, const tv_round *round, const tv_layer *layers,
                                int32_t n_layers, tv_round_graph **graph);
/* Kernel launches recorded in the graph. */
int32_t tv_round_graph_kernels(const tv_round_graph *graph);
tv_status tv_round_graph_launch(tv_round_graph *graph, hipStream_t stream);
tv_status tv_round_graph_destroy(tv_round_graph *graph);

/* Human-readable name of a status code (static string). */
const char *tv_status_string(int status);

/* Optional kernel timing.  While enabled, every kernel the library launches is
 * bracketed by HIP events recorded on the caller's stream (at most `capacity`
 * launches are recorded; later ones run untimed).  tv_profile_read waits for
 * the recorded events and returns, per kernel name, the launch count and the
 * summed duration in milliseconds; it resets the records. */
typedef struct {
  char name[32];
  int32_t launches;
  double total_ms;
} tv_kernel_time;

tv_status tv_profile_enable(int32_t capacity);
tv_status tv_profile_disable(void);
tv_status tv_profile_read(tv_kernel_time *out, int32_t max_entries, int32_t *n_entries);

#ifdef __cplusplus
}
#endif

#endif /* TV_H */
