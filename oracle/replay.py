"""Brute-force linear replay: every root-to-leaf branch decoded as a plain sequence.

TEST INFRASTRUCTURE ONLY (see the package docstring).  This module is a second,
independent statement of what tree verification must produce: the paper's
method (Sec. 3.1, Sec. 3.2, Sec. 4.1) is correct exactly when each tree node
gets the result a linear decoder would give for the sequence
``committed prefix || root path of the node``, and when the state after
committing the accepted path equals the state of that decoder after decoding
the accepted tokens.

The decoder here keeps an explicit growing sequence: it appends one token,
compresses the block the token closes (if any) into the ratio's entry list,
and attends as an ordinary decoder over "top-k of all CSA entries so far, all
HCA entries so far, the last ``window`` tokens".  It never looks at the tree,
masks, depths or scratch slots, and it has its own bfloat16 and FP8 E4M3 roundings written on
float64 bit fields, so that it also cross-checks the oracle's conversions.
"""
from __future__ import annotations

import copy

import numpy as np


def _widen(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _to_bf16(x):
    """float64 -> bfloat16 bits by rounding the float64 significand field.

    For normal float32-range values: keep the top 7 of the 52 explicit
    significand bits, round to nearest even on the discarded 45 bits (a carry
    may bump the exponent, which is the right result), then narrow the now
    exactly representable value to float32.
    """
    x = np.asarray(x, dtype=np.float64)
    u = x.view(np.uint64)
    tiny = np.abs(x) < 2.0 ** -126
    if np.any(tiny & (x != 0)):
        raise ValueError("subnormal bfloat16 results are outside this replay's range")
    keep = (u >> np.uint64(45)) & np.uint64(1)
    r = (u + np.uint64((1 << 44) - 1) + keep) & ~np.uint64((1 << 45) - 1)
    y = r.view(np.float64).astype(np.float32)
    return (y.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _to_e4m3(x):
    """float64 -> FP8 E4M3 codes (OCP "fn": bias 7, 3 mantissa bits, largest
    finite 448), rounding to nearest even on float64 bit fields.

    Inputs of magnitude >= 2**-6 give normal results: keep the top 3 of the 52
    explicit significand bits, round half to even on the 49 discarded bits (a
    carry may bump the exponent), re-bias the exponent from 1023 to 7, and
    clamp to 448 (code 0x7E).  Smaller inputs round half to even to a multiple
    of 2**-9 (possibly 2**-6 itself).
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape, dtype=np.uint8)
    for idx, v in np.ndenumerate(x):
        sign = 0x80 if np.signbit(v) else 0
        a = abs(float(v))
        if a < 2.0 ** -6:                                 # multiples of 2**-9 (8 of them is 2**-6, code 0x08)
            sub = a * 512.0
            lo = np.floor(sub)
            frac = sub - lo
            m = lo + (1.0 if frac > 0.5 or (frac == 0.5 and int(lo) % 2 == 1) else 0.0)
            out[idx] = sign | int(m)
            continue
        u = int(np.float64(a).view(np.uint64))
        keep = (u >> 49) & 1
        r = (u + (1 << 48) - 1 + keep) & ~((1 << 49) - 1)
        exp = ((r >> 52) & 0x7FF) - 1023 + 7
        man = (r >> 49) & 0x7
        code = 0x7E if exp > 15 or (exp == 15 and man == 7) else (exp << 3) | man
        out[idx] = sign | code
    return out


_E4M3_TABLE = np.array([(-1.0 if c & 0x80 else 1.0) * (((c & 7) / 8.0) * 2.0 ** -6 if (c >> 3) & 15 == 0
                                                      else (1 + (c & 7) / 8.0) * 2.0 ** (((c >> 3) & 15) - 7))
                        for c in range(256)])


def _widen_key(d, bits):
    """A stored indexer key, widened: bfloat16 bits, or E4M3 codes when the
    indexer keys are FP8."""
    if d.get("idx_fmt", 0) == 1:
        return _E4M3_TABLE[np.asarray(bits, dtype=np.uint8)]
    return _widen(bits)


class LinearState:
    """Committed state of one row, held as an explicit sequence."""

    def __init__(self, wl, b):
        d = wl.dims
        self.d = d
        L = int(wl.lens[b])
        self.L = L
        n4, n128 = L // d["ratio_csa"], L // d["ratio_hca"]
        self.raw = {}  # raw rows by absolute position (only the recent ones exist)
        P = d.get("page_size", 0)
        if P:
            # paged pool: position q sits in row q % P of physical page table[q // P];
            # an entry of ratio r is number s % (P / r) of the page holding its first token
            table = [int(x) for x in wl.page_table[b]]
            for q in range(max(0, L - max(d["window"], d["ratio_csa"], d["ratio_hca"])), L):
                self.raw[q] = wl.ring[table[q // P], q % P].copy()

            def slot(s, r):
                per = P // r
                return table[s * r // P] * per + s % per
            self.csa = [(wl.c4[slot(s, d["ratio_csa"])].copy(), wl.c4_idx[slot(s, d["ratio_csa"])].copy())
                        for s in range(n4)]
            self.hca = [wl.c128[slot(s, d["ratio_hca"])].copy() for s in range(n128)]
        else:
            cap = d["ring_cap"]
            for q in range(max(0, L - cap), L):
                self.raw[q] = wl.ring[b, q % cap].copy()
            b4, b128 = int(wl.c4_base[b]), int(wl.c128_base[b])
            # CSA entries as (latent row bits, indexer key bits); HCA entries as latent bits
            self.csa = [(wl.c4[b4 + s].copy(), wl.c4_idx[b4 + s].copy()) for s in range(n4)]
            self.hca = [wl.c128[b128 + s].copy() for s in range(n128)]
        self.gate = {d["ratio_csa"]: _widen(wl.gate_w[0]), d["ratio_hca"]: _widen(wl.gate_w[1])}

    def append(self, token_bits):
        """Append one raw token; compress every block it closes."""
        d = self.d
        pos = self.L
        self.raw[pos] = np.asarray(token_bits, dtype=np.uint16).copy()
        self.L += 1
        for r in (d["ratio_csa"], d["ratio_hca"]):
            if self.L % r != 0:
                continue
            block = np.array([_widen(self.raw[x]) for x in range(self.L - r, self.L)])
            logit = np.array([float(np.dot(self.gate[r], t)) for t in block])
            wgt = np.exp(logit - np.max(logit))
            wgt = wgt / np.sum(wgt)
            pooled = np.zeros(block.shape[1])
            for t in range(r):
                pooled += wgt[t] * block[t]
            bits = _to_bf16(pooled)
            if r == d["ratio_csa"]:
                key = _to_e4m3(pooled[d["d_row"]:]) if d.get("idx_fmt", 0) == 1 else bits[d["d_row"]:]
                self.csa.append((bits[:d["d_row"]], key))
            else:
                self.hca.append(bits[:d["d_row"]])

    def attend(self, q_bits, qi_bits, w_bits):
        """Attention output of a query standing at the last appended position."""
        d = self.d
        k = d["topk"]
        qi = _widen(qi_bits)
        w = _widen(w_bits)
        scored = []
        for s, (_, key) in enumerate(self.csa):
            kk = _widen_key(d, key)
            sc = 0.0
            for h in range(qi.shape[0]):
                sc += w[h] * max(0.0, float(np.dot(qi[h], kk)))
            scored.append((-sc, s))
        scored.sort()
        chosen = sorted(s for _, s in scored[:k])
        keys = [_widen(self.csa[s][0]) for s in chosen]
        keys += [_widen(e) for e in self.hca]
        last = self.L - 1
        for x in range(max(0, last - d["window"] + 1), last + 1):
            keys.append(_widen(self.raw[x])[:d["d_row"]])
        R = np.array(keys)
        Q = _widen(q_bits)
        sc = np.float64(np.float32(d["scale"]))
        out = np.zeros((Q.shape[0], d["d_v"]))
        lse = np.zeros(Q.shape[0])
        for h in range(Q.shape[0]):
            lg = sc * (R[:, :d["d_k"]] @ Q[h])
            mx = lg.max()
            e = np.exp(lg - mx)
            out[h] = (e @ R[:, d["v_off"]:d["v_off"] + d["d_v"]]) / e.sum()
            lse[h] = mx + np.log(e.sum())
        return out, lse, chosen

    def clone(self):
        return copy.deepcopy(self)


def branch_paths(parents_row):
    """Every root-to-leaf node sequence of one tree (walking parent links)."""
    D = len(parents_row)
    children = [[] for _ in range(D)]
    for i in range(1, D):
        children[parents_row[i]].append(i)
    paths = []
    stack = [[0]]
    while stack:
        p = stack.pop()
        if children[p[-1]]:
            for c in children[p[-1]]:
                stack.append(p + [c])
        else:
            paths.append(p)
    return paths


def replay_row(wl, b):
    """Decode every branch of row b linearly.

    Returns ``{(path tuple, node): (out, lse, chosen)}`` for every node on
    every root-to-leaf path.
    """
    base = LinearState(wl, b)
    res = {}
    for path in branch_paths([int(x) for x in wl.parents[b]]):
        st = base.clone()
        for node in path:
            st.append(wl.tree_u[b, node])
            res[(tuple(path), node)] = st.attend(wl.q[b, node], wl.q_idx[b, node], wl.w_idx[b, node])
    return res


def replay_commit(wl, b, accepted_last):
    """State of row b after linearly decoding its accepted path."""
    par = [int(x) for x in wl.parents[b]]
    path = [int(accepted_last)]
    while par[path[-1]] >= 0:
        path.append(par[path[-1]])
    path.reverse()
    st = LinearState(wl, b)
    for node in path:
        st.append(wl.tree_u[b, node])
    return st, path
