"""The captured multi-layer round: a graph replay gives the same bits as the
same calls issued one by one, round after round (the committed state grows),
with eager work and synchronisations between replays, and with new draft
trees written into the captured buffers between replays.  Layer 0 of the
first round is also checked against the oracle."""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import tv_oracle as O

from .parity import compare_verify

pytestmark = pytest.mark.gpu

PER_LAYER = ("out", "lse", "sel", "scr_c4", "scr_c128", "ring", "c4", "c4_idx", "c128", "len")
SHARED = ("anc", "depth", "row_status", "accepted_last", "accept_nodes", "accept_len", "target_tokens",
          "next_token")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _layers(name, n, select, **over):
    from paper_2609_24698_amd import DeviceRound
    ws = [synth.make_workload(name, seed=500 + k, max_len_margin=64, **over) for k in range(n)]
    for w in ws[1:]:  # layers of one model share the sequence: same lengths, tree and accepted node
        assert np.array_equal(w.lens, ws[0].lens)
        w.parents[:] = ws[0].parents
        w.accepted_last[:] = ws[0].accepted_last
    rounds = [DeviceRound(w, "cuda:0") for w in ws]
    if select:
        rounds[0].attach_selection(synth.make_selection(ws[0], vocab=5000, dup_rows=2))
    return ws, rounds


def _same(a, b, rnd):
    for k in SHARED:
        if k in a.layers[0].t:
            assert np.array_equal(a.layers[0].host(k), b.layers[0].host(k)), (rnd, k)
    for l, (ra, rb) in enumerate(zip(a.layers, b.layers)):
        for k in PER_LAYER:
            x, y = ra.host(k), rb.host(k)
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), (rnd, l, k)


@pytest.mark.parametrize("name,n,select,over", [
    ("C1", 3, True, {}),
    ("C0", 4, False, dict(lens=2047)),
    ("C2", 2, True, dict(B=4, lens=[32767, 20000, 4099, 1023])),
])
def test_graph_equals_eager(name, n, select, over):
    from paper_2609_24698_amd import LayeredRound
    _say(f"[graph] {name} layers={n} select={select} {over}")
    ws, ra = _layers(name, n, select, **over)
    _, rb = _layers(name, n, select, **over)
    eager, graph = LayeredRound(ra), LayeredRound(rb)
    kernels = graph.capture()
    assert kernels >= 1 + 4 * n + n
    noise = torch.empty(1 << 20, device="cuda:0")
    for rnd in range(3):
        eager.eager()
        graph.replay()
        torch.cuda.synchronize()
        if rnd == 0:  # layer 0 against the oracle
            w = ws[0]
            ref = O.run_round(w)
            nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
            g4, g128 = rb[0].host("scr_c4"), rb[0].host("scr_c128")
            compare_verify(rb[0].host("out"), rb[0].host("lse"), rb[0].host("sel"), ref, nodes, w.dims,
                           own_ref=lambda b, i: O.verify_node(w, b, i, ref["anc"], ref["depth"], g4, g128),
                           rerun=lambda b, i, chosen: O.verify_node(w, b, i, ref["anc"], ref["depth"], g4, g128,
                                                                      chosen=chosen))
        _same(eager, graph, rnd)
        noise.normal_()  # eager work of the program between replays
        torch.cuda.synchronize()
    assert np.all(rb[0].host("len") > ws[0].lens)
    graph.release()


def test_new_trees_without_recapture():
    """The graph reads the tree from device memory: a different tree shape and
    accepted node written into the captured buffers are honoured at replay."""
    from paper_2609_24698_amd import LayeredRound
    ws, ra = _layers("C1", 2, False)
    _, rb = _layers("C1", 2, False)
    eager, graph = LayeredRound(ra), LayeredRound(rb)
    graph.capture()
    rng = np.random.default_rng(11)
    for rnd in range(3):
        B, D = ws[0].parents.shape
        par = np.full((B, D), -1, dtype=np.int32)
        for i in range(1, D):
            par[:, i] = rng.integers(0, i, size=B)
        acc = rng.integers(0, D, size=B).astype(np.int32)
        for lr in (eager, graph):
            lr.layers[0].t["parents"].copy_(torch.from_numpy(par))
            lr.layers[0].t["accepted_last"].copy_(torch.from_numpy(acc))
        eager.eager()
        graph.replay()
        torch.cuda.synchronize()
        _same(eager, graph, rnd)
        assert np.array_equal(graph.layers[0].host("depth"), O.build_tree_mask(par)[1])
    graph.release()


def test_capture_reports_bad_arguments():
    """A failing check in any recorded call fails the capture; nothing is kept."""
    from paper_2609_24698_amd import LayeredRound, TvError
    _, rb = _layers("C1", 2, False)
    rb[1].t["q"] = rb[1].t["q"].view(-1)[1:]  # off a 16-byte boundary: tv_verify_attention rejects it
    g = LayeredRound(rb)
    with pytest.raises((TvError, ValueError)):
        g.capture()
    assert g.graph is None
