"""Pins of the refresh schedules (Sec. 4.3) to the plain accepted-path
refresh: writing a designated chain's CSA entries through at compression
time and skipping their copies at commit leaves exactly the committed state
that the plain commit leaves, over every slot a later round can see, for any
designated chain, any accepted node, capacity failures, and two rounds in a
row.  Slots past the committed length hold either what they held or a
written-through entry."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import tv_oracle as O


def _visible(wl, com, b):
    d = wl.dims
    L = int(com["lens"][b])
    n4, n128 = L // d["ratio_csa"], L // d["ratio_hca"]
    b4, b128 = int(wl.c4_base[b]), int(wl.c128_base[b])
    cap = d["ring_cap"]
    slots = [q & (cap - 1) for q in range(max(0, L - cap), L)]
    return (L, com["c4"][b4:b4 + n4], com["c4_idx"][b4:b4 + n4], com["c128"][b128:b128 + n128],
            com["ring"][b, slots], com["accept_nodes"][b], com["accept_len"][b], com["status"][b])


def _round(wl, accepted, primary):
    anc, depth, st = O.build_tree_mask(wl.parents)
    scr4, scr128, w4, w128, st = O.branch_compress(wl, anc, depth, st)
    plain = O.commit_accepted_path(wl, anc, depth, scr4, scr128, accepted, st)
    pools = O.write_through(wl, anc, depth, scr4, w4, primary, st)
    f2 = O.commit_accepted_path(wl, anc, depth, scr4, scr128, accepted, st, primary_last=primary, pools=pools)
    return plain, f2, pools, (anc, depth, scr4, w4, st)


def _check(wl, plain, f2, pools):
    for b in range(wl.B):
        for x, y in zip(_visible(wl, plain, b), _visible(wl, f2, b)):
            assert np.array_equal(np.asarray(x), np.asarray(y)), b
    # beyond the visible slots: the original bytes or a written-through entry
    for k, wt, orig in (("c4", pools[0], wl.c4), ("c4_idx", pools[1], wl.c4_idx)):
        for s in np.nonzero(np.any(f2[k] != plain[k], axis=-1))[0]:
            assert np.array_equal(f2[k][s], wt[s]) or np.array_equal(f2[k][s], orig[s])
    assert np.array_equal(f2["c128"], plain["c128"])
    # the write-through touches only slots past the committed entries and below the capacity
    for b in range(wl.B):
        n4, base, cap = int(wl.lens[b]) // wl.dims["ratio_csa"], int(wl.c4_base[b]), int(wl.c4_cap[b])
        changed = np.nonzero(np.any(pools[0] != wl.c4, axis=-1) | np.any(pools[1] != wl.c4_idx, axis=-1))[0]
        end = int(wl.c4_base[b + 1]) if b + 1 < wl.B else len(wl.c4)
        mine = changed[(changed >= base) & (changed < end)]
        assert np.all((mine >= base + n4) & (mine < base + cap)), (b, mine - base, n4, cap)


def _lens_with_closures(B, rng):
    return [int(4 * rng.integers(300, 600) + rng.integers(0, 4)) for _ in range(B)]


@pytest.mark.parametrize("seed", range(6))
def test_write_through_then_skip_equals_plain_refresh(seed):
    rng = np.random.default_rng(seed)
    B, D = 6, 8
    wl = synth.make_workload("C0", B=B, D=D, tree="random", lens=_lens_with_closures(B, rng), seed=900 + seed)
    anc, depth, _ = O.build_tree_mask(wl.parents)
    accepted = rng.integers(0, D, size=B).astype(np.int32)
    primary = rng.integers(-1, D + 1, size=B).astype(np.int32)  # -1 and D: no designated chain
    primary[0] = accepted[0]                                     # the accepted chain is the cached one
    # accepted node on the designated chain, below its end
    deep = np.argmax(depth[1])
    primary[1] = deep
    accepted[1] = wl.parents[1, deep] if deep > 0 else 0
    plain, f2, pools, _ = _round(wl, accepted, primary)
    _check(wl, plain, f2, pools)


def test_chain_tree_needs_no_csa_copy():
    """A single chain: every CSA entry the commit needs was written through."""
    wl = synth.make_workload("C0", D=8, chain=True, lens=2041)  # closures at depths 2 and 6
    D = wl.D
    accepted = np.array([D - 1], np.int32)
    primary = np.array([D - 1], np.int32)
    plain, f2, pools, (anc, depth, scr4, w4, st) = _round(wl, accepted, primary)
    _check(wl, plain, f2, pools)
    assert w4.sum() == 2
    # the commit itself copied no CSA entry: its pools equal the written-through ones
    assert np.array_equal(f2["c4"], pools[0]) and np.array_equal(f2["c4_idx"], pools[1])


def test_write_through_is_invisible_before_commit():
    rng = np.random.default_rng(3)
    wl = synth.make_workload("C0", B=4, D=8, tree="random", lens=_lens_with_closures(4, rng))
    anc, depth, st = O.build_tree_mask(wl.parents)
    scr4, _, w4, _, st = O.branch_compress(wl, anc, depth, st)
    primary = np.full(4, 7, np.int32)
    c4, c4i = O.write_through(wl, anc, depth, scr4, w4, primary, st)
    for b in range(4):
        n4 = int(wl.lens[b]) // wl.dims["ratio_csa"]
        base = int(wl.c4_base[b])
        assert np.array_equal(c4[base:base + n4], wl.c4[base:base + n4])
        assert np.array_equal(c4i[base:base + n4], wl.c4_idx[base:base + n4])


def test_capacity_failure_is_the_same():
    wl = synth.make_workload("C0", B=2, D=8, chain=True, lens=[2041, 2041])
    wl.c4_cap[1] = 2041 // 4 + 1  # room for one of the two entries the chain closes
    acc = np.array([7, 7], np.int32)
    plain, f2, pools, _ = _round(wl, acc, np.array([7, 7], np.int32))
    assert list(plain["status"]) == [O.ROW_OK, O.ROW_CAPACITY] == list(f2["status"])
    _check(wl, plain, f2, pools)


def test_two_rounds_leave_no_trace_of_the_first_write_through():
    rng = np.random.default_rng(8)
    B, D = 5, 8
    wl = synth.make_workload("C0", B=B, D=D, tree="random", lens=_lens_with_closures(B, rng))
    acc1 = rng.integers(0, D, size=B).astype(np.int32)
    prim1 = rng.integers(0, D, size=B).astype(np.int32)
    plain1, f21, pools1, _ = _round(wl, acc1, prim1)
    _check(wl, plain1, f21, pools1)

    def after(com):
        return dataclasses.replace(wl, lens=com["lens"].copy(), ring=com["ring"].copy(), c4=com["c4"].copy(),
                                   c4_idx=com["c4_idx"].copy(), c128=com["c128"].copy(),
                                   parents=np.ascontiguousarray(wl.parents[:, ::1]))

    w_plain, w_f2 = after(plain1), after(f21)
    acc2 = rng.integers(0, D, size=B).astype(np.int32)
    prim2 = rng.integers(0, D, size=B).astype(np.int32)
    a2, d2, s2 = O.build_tree_mask(wl.parents)
    sp4, sp128, _, _, sp = O.branch_compress(w_plain, a2, d2, s2)
    plain2 = O.commit_accepted_path(w_plain, a2, d2, sp4, sp128, acc2, sp)
    sf4, sf128, wf4, _, sf = O.branch_compress(w_f2, a2, d2, s2)
    assert np.array_equal(sf4, sp4) and np.array_equal(sf128, sp128)  # the first write-through is invisible
    pools2 = O.write_through(w_f2, a2, d2, sf4, wf4, prim2, sf)
    f22 = O.commit_accepted_path(w_f2, a2, d2, sf4, sf128, acc2, sf, primary_last=prim2, pools=pools2)
    for b in range(B):
        for x, y in zip(_visible(wl, plain2, b), _visible(wl, f22, b)):
            assert np.array_equal(np.asarray(x), np.asarray(y)), b


@pytest.mark.parametrize("bad", [-1, 8, 1 << 20])
def test_no_designated_chain_is_the_plain_refresh(bad):
    """A designated node outside [0, D) means no chain: nothing is written
    through and the commit copies every entry, exactly as the plain refresh."""
    rng = np.random.default_rng(4)
    wl = synth.make_workload("C0", B=4, D=8, tree="random", lens=_lens_with_closures(4, rng))
    acc = rng.integers(0, 8, size=4).astype(np.int32)
    plain, f2, pools, _ = _round(wl, acc, np.full(4, bad, np.int32))
    assert np.array_equal(pools[0], wl.c4) and np.array_equal(pools[1], wl.c4_idx)
    for k in ("c4", "c4_idx", "c128", "ring", "lens", "status", "accept_nodes", "accept_len"):
        assert np.array_equal(plain[k], f2[k]), k
