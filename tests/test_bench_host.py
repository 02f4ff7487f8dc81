"""Host-side accounting of bench.py, checked against the oracle on the CPU:
the per-node key counts behind the attention's flops and gathered bytes, and
the selection-layout check the benchmark applies to its first step."""
import numpy as np
import pytest

import bench
import synth
from oracle import tv_oracle as O


@pytest.mark.parametrize("case", [
    dict(name="C0", lens=2047),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 3967, 1023], seed=33, topk=16),
    dict(name="C1", B=2, D=8, lens=[127, 639], seed=41, topk=512),
])
def test_key_counts_and_layout_match_oracle(case):
    c = dict(case)
    w = synth.make_workload(c.pop("name"), **c)
    ref = O.run_round(w)
    nk = bench.node_key_counts(w.dims, w.lens, ref["depth"], ref["anc"])
    for (b, i), det in ref["detail"].items():
        assert nk[b, i] == det["n_keys"], (b, i)
    bench.check_selection_layout(w.dims, w.lens, ref["depth"], ref["anc"], ref["sel"])
    d = w.dims
    assert bench.attention_flops(d, nk) == int(nk.sum()) * 2 * d["H"] * (d["d_k"] + d["d_v"])


def test_layout_check_rejects_bad_padding():
    w = synth.make_workload("C0", B=2, D=8, tree="random", lens=[381, 3967], seed=33, topk=16)
    ref = O.run_round(w)
    sel = ref["sel"].copy()
    b, i = 0, 1
    n = int((sel[b, i] >= 0).sum())
    if n < sel.shape[-1]:
        sel[b, i, n] = 0  # a padding slot that is not -1
    else:
        sel[b, i, [0, 1]] = sel[b, i, [1, 0]]  # not ascending
    with pytest.raises(AssertionError):
        bench.check_selection_layout(w.dims, w.lens, ref["depth"], ref["anc"], sel)


def _distinct_rows(w, ref):
    """Every stored row the attention reads, by identity, from the oracle's key
    sets: committed CSA entries by index, path CSA entries by the scratch slot
    (closing node) they come from, committed and path HCA entries, committed
    window rows by position, draft rows by node."""
    d = w.dims
    r4, r128, W = d["ratio_csa"], d["ratio_hca"], d["window"]
    rows = set()
    for (b, i), det in ref["detail"].items():
        L = int(w.lens[b])
        n4 = L // r4
        path = O.node_path(ref["anc"][b], ref["depth"][b], i)
        closer = {(L + int(ref["depth"][b, j]) + 1) // r4 - 1: j for j in path
                  if (L + int(ref["depth"][b, j]) + 1) % r4 == 0}
        for s in det["sel"].tolist():
            rows.add((b, "c4", s) if s < n4 else (b, "scr4", closer[s]))
        rows.update((b, "c128", s) for s in range(L // r128))
        rows.update((b, "scr128", j) for j in path if (L + int(ref["depth"][b, j]) + 1) % r128 == 0)
        p = L + int(ref["depth"][b, i])
        rows.update((b, "ring", q) for q in range(max(0, p - W + 1), L))
        rows.update((b, "tree", j) for j in path)
    return rows


@pytest.mark.parametrize("case", [
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 3967, 1023], seed=33, topk=16),
    dict(name="C1", B=2, D=8, lens=[1000, 3001], seed=40, topk=64),
    dict(name="C1", B=2, D=8, tree=[-1, 0, 0, 1, 2, 1, 2, 3], lens=[8190, 1021], seed=52, topk=64),
    # take-all: nodes 1 and 2 (siblings at depth 1) both close block 63, and every node below each selects it
    dict(name="C1", B=2, D=8, tree=[-1, 0, 0, 1, 2, 1, 2, 3], lens=[254, 510], seed=53, topk=256),
])
def test_attention_bytes_count_each_stored_row_once(case):
    """The roofline's algorithmic bytes: queries, outputs, lse and selections,
    plus every distinct stored row the oracle's key sets read, each once (a
    sibling pair closing the same block reads two scratch rows)."""
    c = dict(case)
    w = synth.make_workload(c.pop("name"), **c)
    ref = O.run_round(w)
    d = w.dims
    fixed = d["B"] * d["D"] * (d["H"] * (d["d_k"] * 2 + d["d_v"] * 2 + 4) + d["topk"] * 4)
    want = fixed + len(_distinct_rows(w, ref)) * d["d_row"] * 2
    assert bench.attention_bytes(d, w.lens, ref["sel"], ref["depth"], ref["anc"]) == want


def test_bench_refuses_more_than_one_gpu():
    """`bench.py --gpus N` with N above 1 exits with a message before it touches a GPU."""
    import json
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    p = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in json.loads(p.stdout.strip().splitlines()[-1])["error"]
