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
