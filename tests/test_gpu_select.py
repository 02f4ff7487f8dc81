"""GPU parity of greedy accepted-path selection against the oracle: target
tokens, accepted node and next token bit for bit, on small and full-size
workloads, ties and NaN logits, ragged vocabularies, skipped rows, and a
whole round whose commit follows the selected path."""
import sys

import numpy as np
import pytest
import torch

import bench
import synth
from oracle import tv_oracle as O

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _device(w, sel):
    from paper_2609_24698_amd import DeviceRound
    r = DeviceRound(w, "cuda:0")
    r.attach_selection(sel)
    return r


def _compare(w, sel, r, status):
    t, a, n = O.select_accepted_path(w.parents, sel.draft_tokens, sel.target_logits, status)
    ok = status == O.ROW_OK
    gt, ga, gn = r.host("target_tokens"), r.host("accepted_last"), r.host("next_token")
    assert np.array_equal(gt[ok], t[ok])
    assert np.array_equal(ga[ok], a[ok])
    assert np.array_equal(gn[ok], n[ok])
    # skipped rows keep what the buffers held (targets and next token -2, accepted_last the input)
    assert np.all(gt[~ok] == -2) and np.all(gn[~ok] == -2)
    assert np.array_equal(ga[~ok], w.accepted_last[~ok])
    return a


def _run(w, sel):
    r = _device(w, sel)
    r.mask()
    r.select()
    torch.cuda.synchronize()
    return r


@pytest.mark.parametrize("vocab", [1, 7, 8, 1000, 8193, 16384, 129280])
def test_small_vocabularies(vocab):
    w = synth.make_workload("C1")
    sel = synth.make_selection(w, vocab=vocab, dup_rows=3)
    _say(f"[select] C1 B={w.B} D={w.D} vocab={vocab}")
    r = _run(w, sel)
    _compare(w, sel, r, O.build_tree_mask(w.parents)[2])


def test_ties_nan_and_signed_zero():
    """Few distinct logit values (ties everywhere), NaNs in some nodes and
    -0/+0 maxima: the first maximal index wins, a NaN beats every number."""
    w = synth.make_workload("C1", D=8, B=8)
    sel = synth.make_selection(w, vocab=4096 + 24)
    rng = np.random.default_rng(3)
    vals = np.array([0xBF80, 0x8000, 0x0000, 0x3F80], dtype=np.uint16)  # -1, -0, +0, 1
    lg = vals[rng.integers(0, 4, size=sel.target_logits.shape)]
    lg[0, :, :] = 0x8000  # all -0 and +0: index 0 wins
    lg[0, :, 17] = 0x0000
    lg[1, 2, 1000] = 0x7FC1  # a NaN in the middle
    lg[1, 2, 3000] = 0xFFC0  # a later negative NaN
    lg[2, :, :] = 0xFF80  # all -inf
    sel.target_logits = np.ascontiguousarray(lg)
    r = _run(w, sel)
    _compare(w, sel, r, O.build_tree_mask(w.parents)[2])
    assert r.host("target_tokens")[1, 2] == 1000
    assert np.all(r.host("target_tokens")[0] == 0) and np.all(r.host("target_tokens")[2] == 0)


@pytest.mark.parametrize("D,chain", [(1, False), (64, True), (64, False), (16, False)])
def test_tree_sizes(D, chain):
    """Root only, a 64-deep chain that accepts far down, and wide trees with
    duplicate sibling drafts."""
    w = synth.make_workload("C0", D=D, B=6, chain=chain, tree=None if chain else "random")
    sel = synth.make_selection(w, vocab=2048, dup_rows=4)
    _say(f"[select] C0 D={D} chain={chain}")
    r = _run(w, sel)
    a = _compare(w, sel, r, O.build_tree_mask(w.parents)[2])
    if chain:
        assert np.array_equal(a, w.accepted_last)


def test_skipped_rows():
    """Rows with a bad parent array are skipped and keep their outputs."""
    w = synth.make_workload("C1")
    sel = synth.make_selection(w, vocab=1000)
    w.parents[2, 3] = 4
    w.parents[5, 0] = 0
    w.accepted_last[:] = 1
    r = _run(w, sel)
    st = O.build_tree_mask(w.parents)[2]
    assert list(np.nonzero(st)[0]) == [2, 5]
    _compare(w, sel, r, st)


def test_c3_full_size():
    """The benchmark's ragged B=64, D=8 workload with a 129,280-token vocabulary."""
    w = bench.bench_workload("C3", 20, 5)
    sel = synth.make_selection(w)
    _say(f"[select] C3 B={w.B} D={w.D} vocab={sel.vocab}")
    r = _run(w, sel)
    a = _compare(w, sel, r, O.build_tree_mask(w.parents)[2])
    assert np.array_equal(a, sel.planted_last)


def test_round_commits_the_selected_path():
    """mask -> compress -> verify -> select -> commit on the device: the commit
    follows the selected path and equals the oracle's commit of that path."""
    w = synth.make_workload("C1", B=4, lens=[1003, 2047, 1023, 3071])
    sel = synth.make_selection(w, vocab=3000, dup_rows=2)
    anc, depth, st = O.build_tree_mask(w.parents)
    _, a, _ = O.select_accepted_path(w.parents, sel.draft_tokens, sel.target_logits, st)
    w.accepted_last[:] = 0  # the device must take the selected node, not this input
    r = _device(w, sel)
    r.mask()
    r.compress()
    r.select()
    torch.cuda.synchronize()
    assert np.array_equal(r.host("accepted_last"), a)
    # commit on the oracle's scratch bytes, so both sides see identical entries
    scr4, scr128, _, _, st2 = O.branch_compress(w, anc, depth, st)
    r.t["scr_c4"].copy_(torch.from_numpy(scr4.view(np.int16)))
    r.t["scr_c128"].copy_(torch.from_numpy(scr128.view(np.int16)))
    r.commit()
    torch.cuda.synchronize()
    com = O.commit_accepted_path(w, anc, depth, scr4, scr128, a, st2)
    assert np.array_equal(r.host("len"), com["lens"])
    assert np.array_equal(r.host("accept_nodes"), com["accept_nodes"])
    assert np.array_equal(r.host("ring"), com["ring"])
    for k in ("c4", "c4_idx", "c128"):
        assert np.array_equal(r.host(k), com[k]), k
