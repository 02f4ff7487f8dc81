"""Seeded synthetic workloads for tree verification over CSA/HCA compressed attention.

Every buffer is drawn from ``numpy.random.Generator(PCG64(seed))`` in a fixed
stream order (lengths, tail offsets, parents, accepted path, ring, committed C4
rows, committed C4 indexer keys, committed C128 rows, tree tokens, queries,
indexer queries, indexer weights, gate weights) so that the same seed gives the
same bytes.  Floating-point buffers are drawn as float32 normals and stored as
bfloat16 bit patterns (uint16, round-to-nearest-even), which is the form both
the oracle and the GPU library read.

The workloads follow the paper's experimental setting (a draft tree of D
nodes, counting the root, verified against a long committed context; Sec. 5.1
"Setup and Metrics") with sizes of the five configurations the library is
measured on.  No dataset is used: token contents are i.i.d. N(0, 1), gate
weights N(0, 0.02).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

# Head shapes.  "mla": 64 query heads over one shared 576-wide latent row, keys
# are the full row, values its first 512 channels.  "mha128": 8 query heads over
# one KV head, the row is K(128) followed by V(128).
SHAPES = {
    "mla": dict(H=64, d_row=576, d_k=576, v_off=0, d_v=512),
    "mha128": dict(H=8, d_row=256, d_k=128, v_off=128, d_v=128),
}

_COMMON = dict(d_idx=64, H_idx=8, ratio_csa=4, ratio_hca=128, window=128, ring_cap=256)

# name -> (B, lens spec, D, parents spec, shape, topk)
CONFIGS: Dict[str, dict] = {
    # B=1, L=2048, 8 heads on one KV head of width 128, top-k 64, tree [-1,0,0,1,1].
    "C0": dict(B=1, lens=("fixed", 2048), D=5, parents=("fixed", [-1, 0, 0, 1, 1]), shape="mha128", topk=64),
    # B=8, L=8192, MLA latent shape, top-k 512, D=6 random tree.
    "C1": dict(B=8, lens=("fixed", 8192), D=6, parents=("random",), shape="mla", topk=512),
    # B=32, L=32768, D=8 random tree (a chain twin on identical KV is chain=True).
    "C2": dict(B=32, lens=("fixed", 32768), D=8, parents=("random",), shape="mla", topk=512),
    # B=64 ragged, L log-uniform in [1024, 65536] with a partially filled C128 tail.
    "C3": dict(B=64, lens=("loguniform_tail", 1024, 65536), D=8, parents=("random",), shape="mla", topk=512),
    # B=1, L=2^20, top-k 2048.
    "C4": dict(B=1, lens=("fixed", 1 << 20), D=8, parents=("random",), shape="mla", topk=2048),
}

BF16_NAN = 0x7FC0  # poison for storage the verify path must never read
E4M3_NAN = 0x7F    # the same poison for FP8 E4M3 indexer-key slots


def _f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bits, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _bf16_bits_to_e4m3(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> FP8 E4M3 codes by torch's float8_e4m3fn
    conversion (the generator's values are far inside the E4M3 range)."""
    import torch

    f = torch.from_numpy((bits.astype(np.uint32) << np.uint32(16)).view(np.float32))
    return f.to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0, chunk: int = 1 << 24) -> np.ndarray:
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.uint16)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        v = rng.standard_normal(e - s, dtype=np.float32)
        if std != 1.0:
            v *= np.float32(std)
        out[s:e] = _f32_to_bf16_bits(v)
    return out.reshape(shape)


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    dims: dict                  # tv_dims fields
    lens: np.ndarray            # int32 [B] committed tokens per row
    parents: np.ndarray         # int32 [B][D], node 0 is the root (parent -1)
    accepted_last: np.ndarray   # int32 [B], last node of the accepted root path
    ring: np.ndarray            # uint16 [B][ring_cap][d_u], position q in slot q & (ring_cap-1)
    c4: np.ndarray              # uint16 [c4_total][d_row]
    c4_idx: np.ndarray          # [c4_total][d_idx]: uint16 bfloat16, or uint8 FP8 E4M3 codes when idx_fmt is 1
    c128: np.ndarray            # uint16 [c128_total][d_row]
    c4_base: np.ndarray         # int64 [B]
    c4_cap: np.ndarray          # int32 [B]
    c128_base: np.ndarray       # int64 [B]
    c128_cap: np.ndarray        # int32 [B]
    tree_u: np.ndarray          # uint16 [B][D][d_u]
    q: np.ndarray               # uint16 [B][D][H][d_k]
    q_idx: np.ndarray           # uint16 [B][D][H_idx][d_idx]
    w_idx: np.ndarray           # uint16 [B][D][H_idx]
    gate_w: np.ndarray          # uint16 [2][d_u]; row 0 for the CSA ratio, row 1 for the HCA ratio
    # Paged pool (dims page_size > 0): physical page of each logical page of each row, -1 where not
    # allocated; ring is then [pages][page_size][d_u] and the pools are laid out page by page.
    page_table: Optional[np.ndarray] = None

    @property
    def B(self) -> int:
        return self.dims["B"]

    @property
    def D(self) -> int:
        return self.dims["D"]

    def nbytes(self) -> int:
        return sum(getattr(self, f.name).nbytes for f in dataclasses.fields(self)
                   if isinstance(getattr(self, f.name), np.ndarray))


def config_dims(name: str, **over) -> dict:
    cfg = dict(CONFIGS[name])
    cfg.update({k: v for k, v in over.items() if k in ("B", "D", "topk", "shape")})
    dims = dict(B=cfg["B"], D=cfg["D"], topk=cfg["topk"])
    dims.update(SHAPES[cfg["shape"]])
    dims.update(_COMMON)
    for k in ("d_idx", "H_idx", "ratio_csa", "ratio_hca", "window", "ring_cap", "H", "idx_fmt"):
        if k in over:
            dims[k] = over[k]
    dims.setdefault("idx_fmt", 0)
    dims["scale"] = float(over.get("scale", 1.0 / math.sqrt(dims["d_k"])))
    return dims


def _draw_lens(rng, B, spec):
    kind = spec[0]
    if kind == "fixed":
        return np.full(B, spec[1], dtype=np.int64), np.zeros(B, dtype=np.int64)
    if kind == "list":
        v = np.asarray(spec[1], dtype=np.int64)
        assert v.shape == (B,)
        return v, np.zeros(B, dtype=np.int64)
    if kind == "loguniform_tail":
        # Stratified log-uniform draw: row b takes one point of its own 1/B
        # quantile band (the bands dealt to rows in a random order), so the
        # batch follows the distribution closely (mean ~15.5K for [1K, 64K])
        # instead of depending on how B independent draws happen to fall.
        lo, hi = spec[1], spec[2]
        band = rng.permutation(B)
        u = math.log(lo) + (band + rng.random(size=B)) / B * (math.log(hi) - math.log(lo))
        base = np.floor(np.exp(u)).astype(np.int64)
        off = rng.integers(1, 128, size=B)  # tail offset in 1..127
        # The first eight rows sit 127-(b mod 4) tokens into a 128-block, so a
        # node at depth (b mod 4) closes an HCA block inside the tree.
        for b in range(min(B, 8)):
            off[b] = 127 - (b % 4)
        lens = (base // 128) * 128 + off
        lens = np.where(lens < lo, lens + 128, lens)
        lens = np.where(lens > hi, lens - 128, lens)
        return lens, off
    raise ValueError(kind)


def _draw_parents(rng, B, D, spec, chain: bool):
    # Always consume the same number of draws so that a chain twin shares
    # every later byte with its tree sibling.
    draws = rng.random(size=(B, D))
    if chain:
        return np.tile(np.arange(-1, D - 1, dtype=np.int32), (B, 1))
    if spec[0] == "fixed":
        p = np.asarray(spec[1], dtype=np.int32)
        assert p.shape == (D,)
        return np.tile(p, (B, 1))
    par = np.empty((B, D), dtype=np.int32)
    par[:, 0] = -1
    for i in range(1, D):
        par[:, i] = np.minimum((draws[:, i] * i).astype(np.int32), i - 1)
    return par


def _draw_accepted(rng, parents):
    # Per-row accepted length a uniform in 1..(max depth + 1); the accepted
    # node is then uniform among the nodes at depth a-1.  The depth count here
    # only serves this draw.
    B, D = parents.shape
    u = rng.random(size=(B, 2))
    acc = np.zeros(B, dtype=np.int32)
    for b in range(B):
        dep = [0] * D
        for i in range(1, D):
            dep[i] = dep[parents[b, i]] + 1
        a = 1 + min(int(u[b, 0] * (max(dep) + 1)), max(dep))
        cands = [i for i in range(D) if dep[i] == a - 1]
        acc[b] = cands[min(int(u[b, 1] * len(cands)), len(cands) - 1)]
    return acc


def make_workload(name: str, seed: Optional[int] = None, *, chain: bool = False,
                  tree=None, lens=None, extra_c4: int = 96, extra_c128: int = 8,
                  max_len_margin: int = 0, page_size: int = 0, **over) -> Workload:
    """Draw the workload of configuration ``name`` (C0..C4).

    ``lens`` overrides the committed lengths (an int or a list of B ints);
    ``tree`` overrides the tree shape ("random" or one parent list for every
    row); ``chain=True`` replaces the tree by a chain on identical bytes;
    ``over`` overrides B, D, topk, shape, H_idx, window, ring_cap, scale,
    idx_fmt (1: committed indexer keys as FP8 E4M3 codes).
    ``extra_c4``/``extra_c128`` are the spare pool slots per row that commits
    append into; ``max_len_margin`` is added to the largest length to form the
    ``max_len`` bound that sizes the verify workspace.  ``page_size`` > 0
    lays the same state out in a paged pool (see ``paginate``).
    """
    cfg = dict(CONFIGS[name])
    for k in ("B", "D", "topk", "shape"):
        if k in over:
            cfg[k] = over[k]
    if tree is not None:
        cfg["parents"] = ("random",) if tree == "random" else ("fixed", list(tree))
    if lens is not None:
        cfg["lens"] = ("fixed", int(lens)) if np.isscalar(lens) else ("list", list(lens))
    if seed is None:
        seed = 20260 + int(name[1:])
    dims = config_dims(name, **over)
    B, D = dims["B"], dims["D"]
    d_row, d_idx = dims["d_row"], dims["d_idx"]
    d_u = d_row + d_idx
    cap = dims["ring_cap"]

    rng = np.random.Generator(np.random.PCG64(seed))
    lens_v, _off = _draw_lens(rng, B, cfg["lens"])
    parents = _draw_parents(rng, B, D, cfg["parents"], chain)
    accepted = _draw_accepted(rng, parents)

    ring = _normal_bf16(rng, (B, cap, d_u))
    for b in range(B):
        if lens_v[b] < cap:  # slots of positions that do not exist yet
            ring[b, lens_v[b]:, :] = BF16_NAN

    n4 = lens_v // dims["ratio_csa"]
    n128 = lens_v // dims["ratio_hca"]
    c4_cap = (n4 + extra_c4).astype(np.int32)
    c128_cap = (n128 + extra_c128).astype(np.int32)
    c4_base = np.concatenate([[0], np.cumsum(c4_cap)[:-1]]).astype(np.int64)
    c128_base = np.concatenate([[0], np.cumsum(c128_cap)[:-1]]).astype(np.int64)
    t4, t128 = int(c4_cap.sum()), int(c128_cap.sum())

    c4 = np.full((t4, d_row), BF16_NAN, dtype=np.uint16)
    fp8 = dims["idx_fmt"] == 1
    c4_idx = np.full((t4, d_idx), E4M3_NAN if fp8 else BF16_NAN, dtype=np.uint8 if fp8 else np.uint16)
    c128 = np.full((t128, d_row), BF16_NAN, dtype=np.uint16)
    tot4 = int(n4.sum())
    tot128 = int(n128.sum())
    v4 = _normal_bf16(rng, (tot4, d_row))
    v4i = _normal_bf16(rng, (tot4, d_idx))
    if fp8:  # the same draws, stored as FP8 E4M3 codes (torch's float32 -> e4m3fn conversion)
        v4i = _bf16_bits_to_e4m3(v4i)
    v128 = _normal_bf16(rng, (tot128, d_row))
    s4 = s128 = 0
    for b in range(B):
        c4[c4_base[b]:c4_base[b] + n4[b]] = v4[s4:s4 + n4[b]]
        c4_idx[c4_base[b]:c4_base[b] + n4[b]] = v4i[s4:s4 + n4[b]]
        c128[c128_base[b]:c128_base[b] + n128[b]] = v128[s128:s128 + n128[b]]
        s4 += n4[b]
        s128 += n128[b]
    del v4, v4i, v128

    tree_u = _normal_bf16(rng, (B, D, d_u))
    q = _normal_bf16(rng, (B, D, dims["H"], dims["d_k"]))
    q_idx = _normal_bf16(rng, (B, D, dims["H_idx"], d_idx))
    w_idx = _normal_bf16(rng, (B, D, dims["H_idx"]))
    gate_w = _normal_bf16(rng, (2, d_u), std=0.02)

    dims["max_len"] = int(lens_v.max()) + int(max_len_margin)
    dims["page_size"], dims["page_stride"] = 0, 0
    wl = Workload(
        name=name + ("-chain" if chain else ""), seed=seed, dims=dims,
        lens=lens_v.astype(np.int32), parents=parents, accepted_last=accepted,
        ring=ring, c4=c4, c4_idx=c4_idx, c128=c128,
        c4_base=c4_base, c4_cap=c4_cap, c128_base=c128_base, c128_cap=c128_cap,
        tree_u=tree_u, q=q, q_idx=q_idx, w_idx=w_idx, gate_w=gate_w,
    )
    return paginate(wl, page_size, seed) if page_size else wl


def paginate(wl: Workload, page_size: int, seed: int) -> Workload:
    """The same logical state in a paged pool of ``page_size``-token pages.

    Each row owns the logical pages covering its CSA capacity (c4_cap *
    ratio_csa positions); its page-table row has one more entry, left
    unallocated (-1).  Physical page ids are a random permutation of all
    owned pages, drawn from a generator of its own so that every other byte
    equals the flat workload's.  Raw rows of the last ring_cap committed
    positions are copied from the ring, committed entries from the flat
    pools; every other slot holds the poison pattern.
    """
    d = dict(wl.dims)
    P = int(page_size)
    r4, r128, cap = d["ratio_csa"], d["ratio_hca"], d["ring_cap"]
    assert P % r4 == 0 and P % r128 == 0
    B = d["B"]
    owned = [-(-int(wl.c4_cap[b]) * r4 // P) for b in range(B)]
    stride = max(owned) + 1
    total = int(sum(owned))
    perm = np.random.Generator(np.random.PCG64(seed + 104729)).permutation(total).astype(np.int32)
    table = np.full((B, stride), -1, dtype=np.int32)
    k = 0
    for b in range(B):
        table[b, :owned[b]] = perm[k:k + owned[b]]
        k += owned[b]
    d_u = wl.ring.shape[-1]
    raw = np.full((total, P, d_u), BF16_NAN, dtype=np.uint16)
    per4, per128 = P // r4, P // r128
    c4 = np.full((total * per4, wl.c4.shape[1]), BF16_NAN, dtype=np.uint16)
    c4_idx = np.full((total * per4, wl.c4_idx.shape[1]), E4M3_NAN if wl.c4_idx.dtype == np.uint8 else BF16_NAN,
                     dtype=wl.c4_idx.dtype)
    c128 = np.full((total * per128, wl.c128.shape[1]), BF16_NAN, dtype=np.uint16)
    for b in range(B):
        L = int(wl.lens[b])
        for q in range(max(0, L - cap), L):
            raw[table[b, q // P], q % P] = wl.ring[b, q % cap]
        n4, n128 = L // r4, L // r128
        s = np.arange(n4)
        slots = table[b, s // per4].astype(np.int64) * per4 + s % per4
        c4[slots] = wl.c4[wl.c4_base[b]:wl.c4_base[b] + n4]
        c4_idx[slots] = wl.c4_idx[wl.c4_base[b]:wl.c4_base[b] + n4]
        s = np.arange(n128)
        slots = table[b, s // per128].astype(np.int64) * per128 + s % per128
        c128[slots] = wl.c128[wl.c128_base[b]:wl.c128_base[b] + n128]
    d["page_size"], d["page_stride"] = P, stride
    return dataclasses.replace(wl, name=wl.name + f"-paged{P}", dims=d, ring=raw, c4=c4, c4_idx=c4_idx,
                               c128=c128, page_table=table)


# DeepSeek-V3's vocabulary size; the paper does not state DeepSeek-V4's, so the
# selection workloads take its predecessor's.
VOCAB = 129280


@dataclasses.dataclass
class Selection:
    vocab: int
    draft_tokens: np.ndarray    # int32 [B][D] token drafted at each node (the root's is unused)
    target_logits: np.ndarray   # uint16 [B][D][vocab] bfloat16 next-token logits of the target at each node
    planted_last: np.ndarray    # int32 [B] node whose root path the logits were built to accept


def make_selection(wl: Workload, vocab: int = VOCAB, seed: Optional[int] = None, *, dup_rows: int = 0,
                   peak: float = 16.0, noise_std: float = 1.0) -> Selection:
    """Draft tokens and target logits over the trees of ``wl``.

    Siblings draft distinct tokens (a top-k drafter proposes different tokens
    at one node), except in the first ``dup_rows`` rows, where the second child
    of the first node with two children repeats its elder sibling's token.
    Logits are N(0, noise_std) bfloat16 noise; along the root path of
    ``wl.accepted_last`` the logits of each node peak (value ``peak``) at the
    token drafted by the next node of that path, and at the path's last node
    at a token none of its children drafted, so greedy selection accepts that
    path.  The draw uses its own generator, so the workload's bytes do not
    depend on it.
    """
    B, D = wl.parents.shape
    if seed is None:
        seed = wl.seed + 7919
    rng = np.random.Generator(np.random.PCG64(seed))
    draft = rng.integers(0, vocab, size=(B, D)).astype(np.int32)
    extra = rng.integers(0, vocab, size=(B, D, 8))  # redraws for sibling collisions and the final peak
    logits = _normal_bf16(rng, (B, D, vocab), std=noise_std)
    peak_bits = int(_f32_to_bf16_bits(np.array([peak], dtype=np.float32))[0])
    planted = np.asarray(wl.accepted_last, dtype=np.int32).copy()
    for b in range(B):
        par = wl.parents[b]
        kids = [[c for c in range(1, D) if par[c] == i] for i in range(D)]
        for i in range(D):  # distinct sibling tokens
            seen = set()
            for c in kids[i]:
                k = 0
                while int(draft[b, c]) in seen and vocab > len(kids[i]):
                    draft[b, c] = extra[b, c, k % 8] if k < 8 else (int(draft[b, c]) + 1) % vocab
                    k += 1
                seen.add(int(draft[b, c]))
        if b < dup_rows:
            for i in range(D):
                if len(kids[i]) >= 2:
                    draft[b, kids[i][1]] = draft[b, kids[i][0]]
                    break
        path = [int(planted[b])]
        while par[path[-1]] >= 0 and len(path) <= D:  # bounded: a broken parent array may loop
            path.append(int(par[path[-1]]))
        path.reverse()
        for t in range(len(path) - 1):
            logits[b, path[t], draft[b, path[t + 1]]] = peak_bits
        last = path[-1]
        taken = {int(draft[b, c]) for c in kids[last]}
        y = int(extra[b, last, 7])
        while y in taken and vocab > len(taken):
            y = (y + 1) % vocab
        logits[b, last, y] = peak_bits
    return Selection(vocab=vocab, draft_tokens=draft, target_logits=logits, planted_last=planted)
