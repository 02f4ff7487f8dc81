"""Float64 CPU oracle of the tree-verify path.

TEST INFRASTRUCTURE ONLY: used by the test suite, the smoke check and the
benchmark's CPU-baseline leg; never by the library.  Shares no code with the
GPU path.

What it computes, with the paper passage each step follows:

* ``build_tree_mask``: the verification plan of the draft tree (Sec. 4.1,
  verify preprocess turns the tree into candidate chains; Sec. 3.1: a candidate sees the
  accepted context plus the ancestors on its own branch).  Bit ``j`` of
  ``anc[i]`` is set iff node ``j`` is ``i`` or an ancestor of ``i``.
* ``branch_compress``: each branch compresses its own not-yet-full block,
  never mixing sibling branches (Sec. 4.1, chains compressed independently
  after branching; Sec. 4.2, isolated compression state per chain kept in a
  scratch pad).
* ``verify_attention``: branch-aware causal verification over the compressed
  history (Sec. 3.1, Sec. 4.1 target verify; Sec. 2.2 multi-resolution
  compressed context).  A node attends to CSA entries chosen by the indexer
  top-k, all HCA entries, and the raw sliding window, restricted to entries
  whose tokens lie on its own root path.
* ``commit_accepted_path``: refresh of token history, window KV and the
  compressed states along the accepted path only (Sec. 3.2 and Sec. 4.2,
  accepted-path refresh; rejected branches leave no trace).
* ``write_through`` and ``commit_accepted_path(primary_last=...)``: the
  refresh schedules of Sec. 4.3.  The CSA entries of one designated chain are
  written into the persistent pool while compressing (timely C4 refresh);
  its entries lie past the committed length, so nothing can see them before
  the commit makes them committed.  The commit then skips the CSA copies of
  accepted nodes on that chain (a single chain, or an accepted chain that is
  already the cached one, needs no CSA refresh), and writes every HCA entry
  of the accepted path in one go once the path is known (delayed, combined
  C128 writes).
* ``select_accepted_path``: accepted-path selection after verification
  (Sec. 4.1: target verify ends by selecting the accepted path; Sec. 3.1: the
  result is one path through the tree, not a prefix length; Sec. 4.4: selection
  precedes the state refresh).  Greedy verification in the EAGLE/MTP setting of
  Sec. 2.1: a draft token is accepted when it equals the target model's
  highest-scoring next token at its parent.

The paper cites DeepSeek-V4 for the CSA/HCA arithmetic without restating it.
The reading taken here (kept identical on the GPU side):

* compression of a ratio-r block is softmax-gated pooling: gate logit
  ``z_q = g_r . u_q`` over the full raw row, ``alpha = softmax(z)`` over the r
  tokens of the block, entry ``sum_q alpha_q u_q``; the CSA entry keeps every
  channel (latent row plus indexer key), the HCA entry the latent row only;
* the CSA indexer score of entry s for a query node is
  ``sum_h w[h] * relu(q_idx[h] . k_s)``; the node keeps the top-k candidates
  by (score descending, logical index ascending);
* one softmax runs over the selected CSA entries, all visible HCA entries and
  the raw window of the last ``window`` positions up to and including the
  node; keys are ``row[:d_k]``, values ``row[v_off:v_off+d_v]``;
* an entry is visible from the query at its closing position onward;
* with ``dims["idx_fmt"] == 1`` (a fidelity reading of DeepSeek-V4's FP8
  indexer keys, which the paper does not restate) every stored indexer key
  holds OCP FP8 E4M3 values: the committed pool ``c4_idx`` as E4M3 codes, a
  CSA scratch entry's indexer channels as the same values widened to
  bfloat16.  The pooled key is rounded to E4M3 (nearest, ties to even,
  saturating at +-448) instead of to bfloat16; scoring widens it exactly;
* with ``dims["page_size"] = P > 0`` (the paged pool of Sec. 4.2: one
  logical layer of positions viewed as three physical layers that share
  page-level pointers) a row's positions form logical pages of P tokens and
  ``page_table[b][j]`` names the physical page of logical page j (-1: not
  allocated).  That one page id addresses all three layers: the raw rows
  (``ring`` becomes ``[pages][P][d_u]``, position q at
  ``[page(q // P)][q % P]``), the CSA entries (``P / ratio_csa`` per page,
  entry s at slot ``page(s * ratio_csa // P) * (P / ratio_csa) + s % (P /
  ratio_csa)``) and the HCA entries likewise.  A commit that needs a page
  the table does not allocate fails the row with CAPACITY.

All arithmetic is float64.  Inputs are bfloat16 bit patterns, widened
exactly; a value the cache stores (a compressed entry) is rounded to
bfloat16, round-to-nearest-even, before anything reads it.
"""
from __future__ import annotations

import numpy as np

ROW_OK, ROW_BAD_PARENT, ROW_BAD_ACCEPT, ROW_CAPACITY, ROW_BAD_LEN = 0, 1, 2, 3, 4


# --------------------------------------------------------------------------
# bfloat16 conversions
# --------------------------------------------------------------------------
def bf16_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) to float64, exactly."""
    b = np.asarray(bits, dtype=np.uint16)
    with np.errstate(invalid="ignore"):  # NaN patterns stay NaN
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def f64_to_bf16(x) -> np.ndarray:
    """float64 to bfloat16 bits, one rounding, to nearest with ties to even.

    bfloat16 keeps 8 significant bits and the float32 exponent range, so the
    spacing of representable values around ``x = f * 2**E`` (0.5 <= f < 1) is
    ``2**(E-8)``, never finer than the subnormal spacing ``2**-133``.
    ``x / spacing`` is an exact power-of-two scaling, ``rint`` rounds it half to
    even, and the product is exactly representable in float32.
    """
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite value")
    _, e = np.frexp(x)
    spacing = np.ldexp(1.0, np.maximum(e - 8, -133))
    y = np.rint(x / spacing) * spacing
    big = np.abs(y) >= 2.0 ** 128
    y = np.where(big, np.copysign(np.inf, x), y)
    return (y.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def round_bf16(x) -> np.ndarray:
    return bf16_to_f64(f64_to_bf16(x))


# --------------------------------------------------------------------------
# FP8 E4M3 (OCP "fn" variant: 1 sign, 4 exponent bits with bias 7, 3 mantissa
# bits; no infinities, codes 0x7F and 0xFF are NaN; largest finite 448)
# --------------------------------------------------------------------------
IDX_BF16, IDX_E4M3 = 0, 1
E4M3_MAX = 448.0


def e4m3_to_f64(codes) -> np.ndarray:
    """E4M3 codes (uint8) to float64, exactly: exponent field 0 holds the
    subnormals m * 2**-9, field e > 0 the normals (1 + m/8) * 2**(e-7)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.ldexp(1.0, e - 7))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return np.where(c & 0x80, -mag, mag)


def f64_to_e4m3(x) -> np.ndarray:
    """float64 to E4M3 codes, one rounding to nearest with ties to even;
    magnitudes beyond 448 saturate to +-448.

    E4M3 keeps 4 significant bits, so around ``|x| = f * 2**E`` (0.5 <= f < 1)
    representable values are ``2**(E-4)`` apart, never closer than the
    subnormal spacing ``2**-9``.  ``|x| / spacing`` is an exact power-of-two
    scaling and ``rint`` rounds it half to even; the rounded magnitude is then
    encoded field by field.
    """
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite value")
    a = np.abs(x)
    _, E = np.frexp(a)
    spacing = np.ldexp(1.0, np.maximum(E - 4, -9))
    y = np.minimum(np.rint(a / spacing) * spacing, E4M3_MAX)
    _, Ey = np.frexp(y)                      # y = fy * 2**Ey, 0.5 <= fy < 1 (Ey = 0 for y = 0)
    normal = y >= 2.0 ** -6
    e_field = np.where(normal, Ey - 1 + 7, 0)
    m_field = np.where(normal, np.rint((y / np.ldexp(1.0, Ey - 1) - 1.0) * 8.0), np.rint(y / 2.0 ** -9))
    code = (e_field.astype(np.int64) << 3) | m_field.astype(np.int64)
    code = np.where(np.signbit(x), code | 0x80, code)
    return code.astype(np.uint8)


def round_e4m3(x) -> np.ndarray:
    return e4m3_to_f64(f64_to_e4m3(x))


def idx_fmt(dims) -> int:
    return int(dims.get("idx_fmt", IDX_BF16))


def stored_idx_to_f64(dims, bits) -> np.ndarray:
    """Committed indexer keys of the pool, widened: bfloat16 or E4M3 codes."""
    return e4m3_to_f64(bits) if idx_fmt(dims) == IDX_E4M3 else bf16_to_f64(bits)


def scratch_idx_to_pool(dims, scr_bits) -> np.ndarray:
    """The pool's form of a scratch entry's indexer channels: the same values,
    as bfloat16 bits or (exactly) as E4M3 codes."""
    if idx_fmt(dims) == IDX_E4M3:
        return f64_to_e4m3(bf16_to_f64(scr_bits))
    return np.asarray(scr_bits, dtype=np.uint16).copy()


# --------------------------------------------------------------------------
# verification plan
# --------------------------------------------------------------------------
def build_tree_mask(parents):
    """Ancestor masks, depths and row status of a batch of draft trees.

    ``parents[b][i]`` is the parent of node i; node 0 is the root (parent -1)
    and every parent precedes its child.  A row breaking this gets status
    BAD_PARENT and zero masks and depths.
    """
    parents = np.asarray(parents, dtype=np.int64)
    B, D = parents.shape
    anc = np.zeros((B, D), dtype=np.uint64)
    depth = np.zeros((B, D), dtype=np.int32)
    status = np.zeros(B, dtype=np.int32)
    for b in range(B):
        p = parents[b]
        ok = p[0] == -1 and all(0 <= p[i] < i for i in range(1, D))
        if not ok:
            status[b] = ROW_BAD_PARENT
            continue
        m = [0] * D
        m[0] = 1
        for i in range(1, D):
            depth[b, i] = depth[b, p[i]] + 1
            m[i] = m[p[i]] | (1 << i)
        anc[b] = np.array(m, dtype=np.uint64)
    return anc, depth, status


def node_path(anc_row, depth_row, i):
    """Nodes on the root path of node i, ordered by depth (root first)."""
    bits = int(anc_row[i])
    path = [j for j in range(len(depth_row)) if (bits >> j) & 1]
    path.sort(key=lambda j: int(depth_row[j]))
    return path


def _len_ok(L, dims):
    return 0 <= L <= dims["max_len"]


def paged(dims) -> bool:
    return int(dims.get("page_size", 0)) > 0


def _page(wl, b, j):
    """Physical page of logical page j of row b, or -1 when not allocated."""
    d = wl.dims
    return int(wl.page_table[b, j]) if 0 <= j < d["page_stride"] else -1


def raw_index(wl, b, q):
    """Index into ``wl.ring`` of the raw row of position q of row b (None
    when its page is not allocated): the ring slot q mod ring_cap, or with a
    paged pool the row's place in its page."""
    d = wl.dims
    if not paged(d):
        return (b, q & (d["ring_cap"] - 1))
    P = d["page_size"]
    pg = _page(wl, b, q // P)
    return None if pg < 0 else (pg, q % P)


def pool_index(wl, b, s, layer):
    """Slot of logical entry s of row b in pool ``layer`` ("c4" for CSA,
    "c128" for HCA), or None when the row has no slot for it: past its
    capacity, or with a paged pool in a page the table does not allocate."""
    d = wl.dims
    ratio = d["ratio_csa"] if layer == "c4" else d["ratio_hca"]
    if not paged(d):
        base, cap = (wl.c4_base, wl.c4_cap) if layer == "c4" else (wl.c128_base, wl.c128_cap)
        return int(base[b]) + s if s < int(cap[b]) else None
    per = d["page_size"] // ratio
    pg = _page(wl, b, s // per)
    return None if pg < 0 else pg * per + s % per


def _token(wl, b, path, L, q):
    """Raw row (float64, all d_u channels) at absolute position q on a branch."""
    if q < L:
        return bf16_to_f64(wl.ring[raw_index(wl, b, q)])
    return bf16_to_f64(wl.tree_u[b, path[q - L]])


def compress_block(tokens, gate):
    """Softmax-gated pooling of the r raw rows of one block (float64)."""
    z = tokens @ gate
    a = np.exp(z - z.max())
    a /= a.sum()
    return a @ tokens


# --------------------------------------------------------------------------
# per-branch compression into scratch
# --------------------------------------------------------------------------
def branch_compress(wl, anc, depth, row_status, scr_c4=None, scr_c128=None, pooled=None):
    """Compressed entries closed by each node along its own branch.

    Node i at position ``p = L + depth[i]`` closes a ratio-r block when
    ``(p + 1) % r == 0``; the block covers positions ``p-r+1 .. p`` of the
    sequence ``committed || root path of i``.  CSA entries (all d_u channels)
    go to ``scr_c4[b][i]``, HCA entries (the d_row latent channels) to
    ``scr_c128[b][i]``; other slots are left as given.  Returns the scratch
    arrays, the written-slot masks and the updated row status.  A dict given
    as ``pooled`` receives each entry's value before it is stored (float64),
    keyed by (b, i, 0 for CSA / 1 for HCA).
    """
    d = wl.dims
    B, D = d["B"], d["D"]
    d_row, d_u = d["d_row"], d["d_row"] + d["d_idx"]
    if scr_c4 is None:
        scr_c4 = np.zeros((B, D, d_u), dtype=np.uint16)
    if scr_c128 is None:
        scr_c128 = np.zeros((B, D, d_row), dtype=np.uint16)
    scr_c4, scr_c128 = scr_c4.copy(), scr_c128.copy()
    status = np.array(row_status, dtype=np.int32).copy()
    w4 = np.zeros((B, D), dtype=bool)
    w128 = np.zeros((B, D), dtype=bool)
    g = bf16_to_f64(wl.gate_w)
    for b in range(B):
        if status[b] != ROW_OK:
            continue
        L = int(wl.lens[b])
        if not _len_ok(L, d):
            status[b] = ROW_BAD_LEN
            continue
        for i in range(D):
            path = node_path(anc[b], depth[b], i)
            p = L + int(depth[b, i])
            for ri, r in enumerate((d["ratio_csa"], d["ratio_hca"])):
                if (p + 1) % r:
                    continue
                toks = np.stack([_token(wl, b, path, L, q) for q in range(p - r + 1, p + 1)])
                e = compress_block(toks, g[ri])
                if pooled is not None:
                    pooled[(b, i, ri)] = e.copy()
                if ri == 0:
                    if idx_fmt(d) == IDX_E4M3:  # the indexer key is stored as E4M3
                        e = np.concatenate([e[:d_row], round_e4m3(e[d_row:])])
                    scr_c4[b, i] = f64_to_bf16(e)
                    w4[b, i] = True
                else:
                    scr_c128[b, i] = f64_to_bf16(e[:d_row])
                    w128[b, i] = True
    return scr_c4, scr_c128, w4, w128, status


# --------------------------------------------------------------------------
# verify attention
# --------------------------------------------------------------------------
class _RowCache:
    """Float64 views of one row's committed state, widened once."""

    def __init__(self, wl, b):
        d = wl.dims
        self.L = L = int(wl.lens[b])
        self.n4 = L // d["ratio_csa"]
        self.n128 = L // d["ratio_hca"]
        s4 = [pool_index(wl, b, s, "c4") for s in range(self.n4)]
        s128 = [pool_index(wl, b, s, "c128") for s in range(self.n128)]
        if None in s4 or None in s128:
            raise ValueError(f"row {b}: a committed entry has no pool slot")
        s4, s128 = np.asarray(s4, dtype=np.int64), np.asarray(s128, dtype=np.int64)
        self.k4 = stored_idx_to_f64(d, wl.c4_idx[s4])
        self.c4_bits = wl.c4[s4]
        self.c128 = bf16_to_f64(wl.c128[s128])


def indexer_scores(keys, q_idx, w_idx):
    """S(s) = sum_h w[h] * relu(q_idx[h] . k_s) for every key row (float64)."""
    return np.maximum(keys @ q_idx.T, 0.0) @ w_idx


def verify_node(wl, b, i, anc, depth, scr_c4, scr_c128, rc=None, chosen=None):
    """Output of node i of row b: the definition written out for one query.

    Returns a dict with ``out`` [H][d_v], ``lse`` [H], ``sel`` (selected CSA
    logical indices, ascending), ``scores`` (logical index -> indexer score of
    every candidate) and ``n_keys`` (size of the attended key set).

    ``chosen`` replaces the top-k by a given set of candidate indices.  Where
    scores tie at the selection boundary several sets are correct; the
    attention over a set another implementation chose is then computed with
    that set (every index must be a visible candidate).
    """
    d = wl.dims
    r4, r128, W, k = d["ratio_csa"], d["ratio_hca"], d["window"], d["topk"]
    d_row, d_k, v_off, d_v = d["d_row"], d["d_k"], d["v_off"], d["d_v"]
    if rc is None:
        rc = _RowCache(wl, b)
    L = rc.L
    path = node_path(anc[b], depth[b], i)
    p = L + int(depth[b, i])
    pos = {j: L + int(depth[b, j]) for j in path}

    # CSA candidates: committed entries, then entries closed on this branch.
    cand_idx = list(range(rc.n4))
    cand_keys = [rc.k4]
    scratch_rows = {}
    for j in path:
        if (pos[j] + 1) % r4 == 0:
            s = (pos[j] + 1) // r4 - 1
            cand_idx.append(s)
            cand_keys.append(bf16_to_f64(scr_c4[b, j, d_row:])[None, :])
            scratch_rows[s] = bf16_to_f64(scr_c4[b, j, :d_row])
    cand_idx = np.asarray(cand_idx, dtype=np.int64)
    keys = np.concatenate(cand_keys, axis=0) if len(cand_idx) else np.zeros((0, d["d_idx"]))
    S = indexer_scores(keys, bf16_to_f64(wl.q_idx[b, i]), bf16_to_f64(wl.w_idx[b, i]))
    if chosen is None:
        order = np.lexsort((cand_idx, -S))  # score descending, then index ascending
        chosen = np.sort(cand_idx[order[:min(k, len(cand_idx))]])
    else:
        chosen = np.sort(np.asarray(chosen, dtype=np.int64))
        assert len(chosen) == min(k, len(cand_idx)) and set(chosen.tolist()) <= set(cand_idx.tolist())

    rows = []
    for s in chosen:
        rows.append(scratch_rows[s] if s >= rc.n4 else bf16_to_f64(rc.c4_bits[s]))
    rows.extend(rc.c128)
    for j in path:
        if (pos[j] + 1) % r128 == 0:
            rows.append(bf16_to_f64(scr_c128[b, j]))
    for qpos in range(max(0, p - W + 1), p + 1):
        rows.append(_token(wl, b, path, L, qpos)[:d_row])
    R = np.stack(rows) if rows else np.zeros((0, d_row))

    Q = bf16_to_f64(wl.q[b, i])                       # [H][d_k]
    scale = float(np.float32(d["scale"]))
    logits = scale * (Q @ R[:, :d_k].T)               # [H][n_keys]
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    s = e.sum(axis=1, keepdims=True)
    out = (e / s) @ R[:, v_off:v_off + d_v]
    lse = (m + np.log(s))[:, 0]
    return dict(out=out, lse=lse, sel=chosen, scores=dict(zip(cand_idx.tolist(), S.tolist())),
                n_keys=R.shape[0])


def verify_attention(wl, anc, depth, scr_c4, scr_c128, row_status, nodes=None):
    """Verify outputs for every node of every valid row (or for ``nodes``).

    Returns ``out`` float64 [B][D][H][d_v], ``lse`` [B][D][H], ``sel`` int32
    [B][D][topk] (ascending, -1 padded), ``status`` and per-node details.
    Rows with a nonzero status are skipped (outputs left NaN, sel -1).
    """
    d = wl.dims
    B, D, H = d["B"], d["D"], d["H"]
    out = np.full((B, D, H, d["d_v"]), np.nan)
    lse = np.full((B, D, H), np.nan)
    sel = np.full((B, D, d["topk"]), -1, dtype=np.int32)
    status = np.array(row_status, dtype=np.int32).copy()
    detail = {}
    want = nodes if nodes is not None else [(b, i) for b in range(B) for i in range(D)]
    rcs = {}
    for b, i in want:
        if status[b] != ROW_OK:
            continue
        if not _len_ok(int(wl.lens[b]), d):
            status[b] = ROW_BAD_LEN
            continue
        if b not in rcs:
            rcs.clear()
            rcs[b] = _RowCache(wl, b)
        r = verify_node(wl, b, i, anc, depth, scr_c4, scr_c128, rcs[b])
        out[b, i], lse[b, i] = r["out"], r["lse"]
        sel[b, i, :len(r["sel"])] = r["sel"]
        detail[(b, i)] = r
    return out, lse, sel, status, detail


# --------------------------------------------------------------------------
# accepted-path commit
# --------------------------------------------------------------------------
def primary_chain(anc_row, primary_last):
    """Nodes of a row's designated chain: the root path of ``primary_last``,
    as a bit set; empty when ``primary_last`` is outside [0, D)."""
    D = len(anc_row)
    return int(anc_row[primary_last]) if 0 <= primary_last < D else 0


def write_through(wl, anc, depth, scr_c4, w4, primary_last, row_status):
    """CSA pools after the compression step writes the entries closed on each
    row's designated chain into their pool slots (logical index
    ``(p+1)/ratio_csa - 1``, past the committed entries), slot capacity
    permitting.  ``w4`` marks the scratch slots the compression wrote; rows
    whose status is not OK write nothing.  Returns new (c4, c4_idx)."""
    d = wl.dims
    c4, c4_idx = wl.c4.copy(), wl.c4_idx.copy()
    d_row = d["d_row"]
    for b in range(d["B"]):
        if row_status[b] != ROW_OK:
            continue
        chain = primary_chain(anc[b], int(primary_last[b]))
        L = int(wl.lens[b])
        for j in range(d["D"]):
            if not (chain >> j) & 1 or not w4[b, j]:
                continue
            s = (L + int(depth[b, j]) + 1) // d["ratio_csa"] - 1
            slot = pool_index(wl, b, s, "c4")
            if slot is not None:
                c4[slot] = scr_c4[b, j, :d_row]
                c4_idx[slot] = scratch_idx_to_pool(d, scr_c4[b, j, d_row:])
    return c4, c4_idx


def commit_accepted_path(wl, anc, depth, scr_c4, scr_c128, accepted_last, row_status,
                         accept_nodes=None, accept_len=None, primary_last=None, pools=None):
    """Refresh the committed state along the accepted path of every valid row.

    The accepted path is the root path of ``accepted_last[b]`` (a = depth + 1
    tokens).  Its raw rows enter the ring (or, paged, their pages) at
    positions L..L+a-1, each of its nodes that closed a block writes its
    scratch entry to the pool at the entry's logical index, and ``len``
    becomes L + a.  A row whose new rows or entries would not fit (pool
    capacity, or a page the table does not allocate) gets status CAPACITY
    and is left intact.
    With ``primary_last``, CSA entries of accepted nodes on the row's
    designated chain are not copied (``write_through`` put them in place);
    ``pools`` = (c4, c4_idx) then gives the pools as the compression left them.
    Returns a dict of new arrays (inputs are not modified).
    """
    d = wl.dims
    B, D = d["B"], d["D"]
    r4, r128 = d["ratio_csa"], d["ratio_hca"]
    d_row = d["d_row"]
    ring, c128 = wl.ring.copy(), wl.c128.copy()
    c4, c4_idx = (wl.c4.copy(), wl.c4_idx.copy()) if pools is None else (pools[0].copy(), pools[1].copy())
    lens = wl.lens.copy()
    status = np.array(row_status, dtype=np.int32).copy()
    an = np.full((B, D), -1, dtype=np.int32) if accept_nodes is None else accept_nodes.copy()
    al = np.zeros(B, dtype=np.int32) if accept_len is None else accept_len.copy()
    for b in range(B):
        if status[b] != ROW_OK:
            continue
        L = int(lens[b])
        if not _len_ok(L, d):
            status[b] = ROW_BAD_LEN
            continue
        last = int(accepted_last[b])
        if not 0 <= last < D:
            status[b] = ROW_BAD_ACCEPT
            continue
        path = node_path(anc[b], depth[b], last)
        chain = 0 if primary_last is None else primary_chain(anc[b], int(primary_last[b]))
        writes4, writes128, skip4 = [], [], set()
        for j in path:
            p = L + int(depth[b, j])
            if (p + 1) % r4 == 0:
                writes4.append(((p + 1) // r4 - 1, j))
                if (chain >> j) & 1:
                    skip4.add(j)
            if (p + 1) % r128 == 0:
                writes128.append(((p + 1) // r128 - 1, j))
        raw_at = [raw_index(wl, b, L + t) for t in range(len(path))]
        at4 = [pool_index(wl, b, s, "c4") for s, _ in writes4]
        at128 = [pool_index(wl, b, s, "c128") for s, _ in writes128]
        if None in raw_at or None in at4 or None in at128:
            status[b] = ROW_CAPACITY
            continue
        for t, j in enumerate(path):
            ring[raw_at[t]] = wl.tree_u[b, j]
        for (s, j), slot in zip(writes4, at4):
            if j in skip4:
                continue
            c4[slot] = scr_c4[b, j, :d_row]
            c4_idx[slot] = scratch_idx_to_pool(d, scr_c4[b, j, d_row:])
        for (s, j), slot in zip(writes128, at128):
            c128[slot] = scr_c128[b, j]
        lens[b] = L + len(path)
        an[b] = -1
        an[b, :len(path)] = path
        al[b] = len(path)
    return dict(ring=ring, c4=c4, c4_idx=c4_idx, c128=c128, lens=lens, status=status,
                accept_nodes=an, accept_len=al)


# --------------------------------------------------------------------------
# accepted-path selection
# --------------------------------------------------------------------------
def target_argmax(logits_bits) -> np.ndarray:
    """Index of the largest logit along the last axis; the first one on ties.

    Logits are bfloat16 bit patterns widened exactly.  A NaN counts as larger
    than every number (the first NaN wins), and -0 equals +0.
    """
    x = bf16_to_f64(logits_bits)
    return np.argmax(x, axis=-1).astype(np.int32)


def select_accepted_path(parents, draft_tokens, target_logits, row_status):
    """Greedy accepted-path selection over each row's draft tree.

    The target token of node i is the argmax of its logits (the target
    model's next token after node i's prefix).  A non-root node matches when
    its draft token equals its parent's target token, and a node is accepted
    when every non-root node on its root path matches (the root is the token
    the previous round already produced).  The accepted path ends at the
    deepest accepted node; among equally deep ones, the smallest index
    (siblings drafted with equal tokens are the only way to get a tie).
    Rows whose status is not OK are skipped: their outputs are -1.

    Returns (target_tokens [B][D], accepted_last [B], next_token [B]), where
    next_token is the target token of the accepted node (the token the next
    round starts from).
    """
    parents = np.asarray(parents, dtype=np.int64)
    draft = np.asarray(draft_tokens, dtype=np.int64)
    B, D = parents.shape
    tgt_all = target_argmax(target_logits)
    tgt = np.full((B, D), -1, dtype=np.int32)
    acc = np.full(B, -1, dtype=np.int32)
    nxt = np.full(B, -1, dtype=np.int32)
    for b in range(B):
        if row_status[b] != ROW_OK:
            continue
        tgt[b] = tgt_all[b]
        best, best_depth = 0, 0
        for i in range(1, D):
            ok, j, dep = True, i, 0
            while j != 0:  # walk the root path of i
                ok = ok and draft[b, j] == tgt[b, parents[b, j]]
                j = int(parents[b, j])
                dep += 1
            if ok and dep > best_depth:
                best, best_depth = i, dep
        acc[b] = best
        nxt[b] = tgt[b, best]
    return tgt, acc, nxt


def run_round(wl, nodes=None):
    """All four steps on one workload; returns every intermediate."""
    anc, depth, st = build_tree_mask(wl.parents)
    pooled = {}
    scr4, scr128, w4, w128, st = branch_compress(wl, anc, depth, st, pooled=pooled)
    out, lse, sel, st_v, det = verify_attention(wl, anc, depth, scr4, scr128, st, nodes)
    com = commit_accepted_path(wl, anc, depth, scr4, scr128, wl.accepted_last, st_v)
    return dict(anc=anc, depth=depth, scr_c4=scr4, scr_c128=scr128, w4=w4, w128=w128, pooled=pooled,
                out=out, lse=lse, sel=sel, status_verify=st_v, detail=det, commit=com)
