"""Pins of the oracle's accepted-path selection to facts outside the oracle:
hand-worked trees, the linear-chain closed form, an independent recursive
descent, a first-maximum loop for the argmax, and invariants."""
import math
import os

import numpy as np
import pytest

import synth
from oracle import tv_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_paths.txt")


def _bits(vals):
    x = np.asarray(vals, dtype=np.float64)
    fin = np.isfinite(x)
    out = np.where(np.isnan(x), 0x7FC0, np.where(x > 0, 0x7F80, 0xFF80)).astype(np.uint16)
    out[fin] = O.f64_to_bf16(x[fin])
    return out


def _one_hot_logits(targets, vocab):
    """Logits whose unique maximum (1.0 over +0.0) sits at the given token."""
    t = np.asarray(targets)
    x = np.zeros(t.shape + (vocab,), dtype=np.uint16)
    np.put_along_axis(x, t[..., None].astype(np.int64), np.uint16(0x3F80), axis=-1)
    return x


@pytest.mark.parametrize("vals,want", [
    ([1.0, 3.0, 3.0, 2.0], 1),
    ([1.0, math.nan, 5.0, math.nan], 1),
    ([-0.0, 0.0], 0),
    ([0.0, -0.0], 0),
    ([-math.inf, -math.inf], 0),
    ([-math.inf, -3.0e38], 1),
    ([math.inf, math.nan], 1),
    ([-2.0], 0),
    ([0.5, 0.50000001, 0.5], 0),  # equal after rounding to bfloat16
])
def test_argmax_hand_cases(vals, want):
    assert int(O.target_argmax(_bits(vals))) == want


def test_argmax_against_first_maximum_loop():
    rng = np.random.default_rng(5)
    pool = np.array([-math.inf, -1.5, -0.0, 0.0, 0.25, 2.0, math.inf, math.nan])
    for _ in range(400):
        n = int(rng.integers(1, 12))
        v = _bits(rng.choice(pool, size=n, p=[.1, .2, .1, .1, .2, .2, .05, .05]))
        x = O.bf16_to_f64(v)
        best = 0
        for k in range(1, n):  # first maximum; a NaN beats every number and later NaNs
            if math.isnan(x[best]):
                break
            if math.isnan(x[k]) or x[k] > x[best]:
                best = k
        assert int(O.target_argmax(v)) == best, (v, best)


def _golden():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, par, drf, tgt, acc = [f.strip() for f in line.split("|")]
        cases.append((name, [int(v) for v in par.split()], [int(v) for v in drf.split()],
                      [int(v) for v in tgt.split()], int(acc)))
    return cases


@pytest.mark.parametrize("name,par,drf,tgt,acc", _golden(), ids=[c[0] for c in _golden()])
def test_selection_golden(name, par, drf, tgt, acc):
    vocab = 128
    t, a, n = O.select_accepted_path(np.array([par]), np.array([drf]), _one_hot_logits([tgt], vocab),
                                     np.zeros(1, np.int32))
    assert list(t[0]) == tgt
    assert int(a[0]) == acc
    assert int(n[0]) == tgt[acc]


def test_chain_closed_form():
    """On a chain, greedy verification accepts the root plus the longest
    prefix of drafts that equal the target's previous next-token."""
    rng = np.random.default_rng(9)
    for D in (1, 2, 5, 8, 16):
        par = np.arange(-1, D - 1)[None, :].repeat(50, 0)
        drf = rng.integers(0, 3, size=(50, D))
        tgt = rng.integers(0, 3, size=(50, D))
        _, a, _ = O.select_accepted_path(par, drf, _one_hot_logits(tgt, 3), np.zeros(50, np.int32))
        for b in range(50):
            m = 0
            while m + 1 < D and drf[b, m + 1] == tgt[b, m]:
                m += 1
            assert a[b] == m


def _descend(par, drf, tgt):
    """Independent definition: depth-first search through matching children,
    keeping the deepest node and the smallest index among equally deep ones."""
    D = len(par)
    kids = {i: [c for c in range(1, D) if par[c] == i] for i in range(D)}
    best = [(0, 0)]  # (-depth, index) minimum

    def go(i, dep):
        best[0] = min(best[0], (-dep, i))
        for c in kids[i]:
            if drf[c] == tgt[i]:
                go(c, dep + 1)

    go(0, 0)
    return best[0][1]


@pytest.mark.parametrize("D", [3, 8, 16, 64])
def test_random_trees_against_recursive_descent(D):
    rng = np.random.default_rng(D)
    B, vocab = 200, 3  # tiny vocabulary: many matches and duplicate siblings
    par = np.full((B, D), -1)
    for i in range(1, D):
        par[:, i] = rng.integers(0, i, size=B)
    drf = rng.integers(0, vocab, size=(B, D))
    tgt = rng.integers(0, vocab, size=(B, D))
    t, a, n = O.select_accepted_path(par, drf, _one_hot_logits(tgt, vocab), np.zeros(B, np.int32))
    for b in range(B):
        assert a[b] == _descend(par[b], drf[b], tgt[b])
        # invariants: the accepted node's path matches throughout, no child extends it
        j = int(a[b])
        while j != 0:
            assert drf[b, j] == tgt[b, par[b, j]]
            j = par[b, j]
        assert not any(par[b, c] == a[b] and drf[b, c] == tgt[b, a[b]] for c in range(1, D))
        assert n[b] == tgt[b, a[b]]


def test_rows_with_errors_are_skipped():
    par = np.array([[-1, 0, 0], [-1, 0, 1], [-1, 0, 0]])
    drf = np.array([[0, 1, 2], [0, 1, 1], [0, 2, 2]])
    tgt = np.array([[2, 0, 0], [1, 1, 0], [2, 0, 0]])
    st = np.array([O.ROW_OK, O.ROW_BAD_LEN, O.ROW_OK], np.int32)
    t, a, n = O.select_accepted_path(par, drf, _one_hot_logits(tgt, 4), st)
    assert list(a) == [2, -1, 1]
    assert list(t[1]) == [-1, -1, -1] and n[1] == -1


@pytest.mark.parametrize("name,dup", [("C0", 0), ("C1", 0), ("C3", 0), ("C1", 4)])
def test_generator_plants_the_accepted_path(name, dup):
    """The selection inputs accept the workload's own accepted node when
    siblings draft distinct tokens."""
    w = synth.make_workload(name, B=8) if name == "C3" else synth.make_workload(name)
    s = synth.make_selection(w, vocab=2000, dup_rows=dup)
    _, _, st = O.build_tree_mask(w.parents)
    t, a, n = O.select_accepted_path(w.parents, s.draft_tokens, s.target_logits, st)
    for b in range(w.B):
        if b >= dup:
            assert a[b] == s.planted_last[b]
        else:  # a duplicate sibling can only add accepted nodes, never shorten the path
            _, dep, _ = O.build_tree_mask(w.parents[b:b + 1])
            assert dep[0, a[b]] >= dep[0, s.planted_last[b]]
