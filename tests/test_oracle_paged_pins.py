"""Pins of the oracle's paged-pool reading (the three physical layers of
Sec. 4.2 sharing one page table) to things other than its own addressing:
the flat layout of the same logical state, and the linear replay, which
reads the paged state with its own page arithmetic."""
import numpy as np
import pytest

import synth
from oracle import replay as R
from oracle import tv_oracle as O

CASES = [
    dict(name="C0", lens=2047),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 3967, 1023], seed=33, topk=16),
    dict(name="C0", B=2, D=8, chain=True, lens=[253, 254], seed=34, topk=16),
    dict(name="C1", B=2, D=6, lens=[509, 639], seed=36, topk=24),
    dict(name="C1", B=2, D=8, lens=[1000, 2943], seed=47, topk=64, idx_fmt=1),
]


def _pair(case, P):
    c = dict(case)
    name = c.pop("name")
    return synth.make_workload(name, **c), synth.make_workload(name, page_size=P, **c)


@pytest.mark.parametrize("P", [128, 256])
@pytest.mark.parametrize("case", CASES)
def test_paged_state_gives_the_flat_results(case, P):
    flat, pgd = _pair(case, P)
    assert pgd.dims["page_size"] == P and pgd.page_table is not None
    a, b = O.run_round(flat), O.run_round(pgd)
    for k in ("anc", "depth", "scr_c4", "scr_c128", "sel", "status_verify"):
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(a["out"], b["out"]) and np.array_equal(a["lse"], b["lse"])
    ca, cb = a["commit"], b["commit"]
    for k in ("lens", "status", "accept_nodes", "accept_len"):
        assert np.array_equal(ca[k], cb[k]), k
    d = flat.dims
    cap = d["ring_cap"]
    written4 = np.zeros(len(cb["c4"]), dtype=bool)
    for r in range(flat.B):
        L1 = int(ca["lens"][r])
        for q in range(max(0, L1 - cap), L1):  # the raw rows the state can still use
            assert np.array_equal(ca["ring"][r, q % cap], cb["ring"][O.raw_index(pgd, r, q)])
        for s in range(L1 // d["ratio_csa"]):
            i = O.pool_index(pgd, r, s, "c4")
            written4[i] = True
            assert np.array_equal(ca["c4"][flat.c4_base[r] + s], cb["c4"][i])
            assert np.array_equal(ca["c4_idx"][flat.c4_base[r] + s], cb["c4_idx"][i])
        for s in range(L1 // d["ratio_hca"]):
            assert np.array_equal(ca["c128"][flat.c128_base[r] + s], cb["c128"][O.pool_index(pgd, r, s, "c128")])
    assert np.all(cb["c4"][~written4] == synth.inputs.BF16_NAN)  # no slot outside the state was written


@pytest.mark.parametrize("case", CASES[:4])
def test_paged_tree_oracle_equals_linear_replay(case):
    _, w = _pair(case, 128)
    res = O.run_round(w)
    for b in range(w.B):
        for (path, node), (out, lse, chosen) in R.replay_row(w, b).items():
            det = res["detail"][(b, node)]
            assert list(det["sel"]) == list(chosen)
            np.testing.assert_allclose(det["out"], out, atol=1e-10, rtol=0)
            np.testing.assert_allclose(det["lse"], lse, atol=1e-10, rtol=0)


@pytest.mark.parametrize("case", CASES[:4])
def test_paged_commit_equals_linear_replay_state(case):
    _, w = _pair(case, 128)
    com = O.run_round(w)["commit"]
    P = w.dims["page_size"]
    d = w.dims
    for b in range(w.B):
        st, path = R.replay_commit(w, b, w.accepted_last[b])
        assert com["lens"][b] == st.L
        table = [int(x) for x in w.page_table[b]]
        for q in range(max(0, st.L - d["window"]), st.L):
            assert np.array_equal(com["ring"][table[q // P], q % P], st.raw[q])
        per4 = P // d["ratio_csa"]
        for s in range(st.L // d["ratio_csa"]):
            i = table[s // per4] * per4 + s % per4
            assert np.array_equal(com["c4"][i], st.csa[s][0]) and np.array_equal(com["c4_idx"][i], st.csa[s][1])


def test_paged_commit_into_an_unallocated_page_fails_the_row():
    """Row 0 sits one token before a page boundary; with the next page taken
    out of its table, an accepted path of two or more tokens has nowhere to
    go: the row fails with CAPACITY and keeps its state, row 1 commits."""
    w = synth.make_workload("C0", B=2, D=5, lens=[127, 300], seed=48, page_size=128)
    w.accepted_last[:] = 3  # depth 2: three tokens, positions 127..129
    w.page_table[0, 1] = -1
    res = O.run_round(w)
    com = res["commit"]
    assert list(com["status"]) == [O.ROW_CAPACITY, O.ROW_OK]
    assert com["lens"][0] == 127 and com["lens"][1] == 303
    assert np.array_equal(com["ring"][w.page_table[0, 0]], w.ring[w.page_table[0, 0]])
