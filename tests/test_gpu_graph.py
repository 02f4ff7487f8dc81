"""The captured multi-layer round: a graph replay gives the same bits as the
same calls issued one by one, round after round (the committed state grows),
with eager work and synchronisations between replays, and with new draft
trees written into the captured buffers between replays.  Layer 0 of the
first round is also checked against the oracle.  The one-call layer step
(tv_verify_round: mask, compression and indexer scoring sharing launches)
gives the same bits as the separate calls."""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import tv_oracle as O

from .parity import compare_verify
from .test_gpu_parity import SMALL_CASES

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
    ("C0", 33, False, dict(B=3, D=8, tree="random", lens=[2047, 1023, 3071], topk=16)),  # two commit launches
])
def test_graph_equals_eager(name, n, select, over):
    from paper_2609_24698_amd import LayeredRound
    _say(f"[graph] {name} layers={n} select={select} {over}")
    ws, ra = _layers(name, n, select, **over)
    _, rb = _layers(name, n, select, **over)
    eager, graph = LayeredRound(ra), LayeredRound(rb)
    kernels = graph.capture()
    assert kernels >= 3 * n + 1  # per layer: mask or not, compression and scoring; top-k; attention; then the commits
    noise = torch.empty(1 << 20, device="cuda:0")
    for rnd in range(3):
        eager.eager(fused=False)
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


@pytest.mark.parametrize("name,n,select,over", [
    ("C1", 3, True, {}),
    ("C2", 2, True, dict(B=4, lens=[32767, 20000, 4099, 1023])),
    ("C4", 1, False, {}),
    ("C3", 1, False, dict(B=16)),
    ("C1", 2, False, dict(idx_fmt=1)),        # FP8 indexer keys
    ("C1", 2, False, dict(page_size=256)),    # paged pool
    ("C1", 2, False, dict(D=12)),             # beyond the scoring's fast path: compression, then scoring
    ("C1", 2, True, dict(lens=[128 * (k + 8) - 1 - (k % 6) for k in range(8)])),  # an HCA block at every depth
])
def test_one_call_layer_step_equals_calls(name, n, select, over):
    """Per layer one tv_verify_round (mask with layer 0 only) against mask,
    compress and verify issued separately, round after round, on a stream
    that is not the current one."""
    from paper_2609_24698_amd import LayeredRound
    _say(f"[one-call] {name} layers={n} select={select} {over}")
    _, ra = _layers(name, n, select, **over)
    _, rb = _layers(name, n, select, **over)
    calls, fused = LayeredRound(ra), LayeredRound(rb)
    s = torch.cuda.Stream()
    for rnd in range(3):
        calls.eager(fused=False)
        with torch.cuda.stream(s):
            fused.eager(s, fused=True)
        torch.cuda.synchronize()
        _same(calls, fused, rnd)
    assert np.all(rb[0].host("row_status") == 0)


@pytest.mark.parametrize("case", SMALL_CASES, ids=lambda c: "-".join(f"{k}{v}" for k, v in c.items() if k != "name")
                         or "base")
def test_one_call_small_cases(case):
    """The one-call layer step on the small parity cases (empty and short
    rows, lengths at block boundaries, D from 1 to 64, chains, both head
    shapes, the long-block compression, FP8 keys, paged pools): verify_round
    then commit against mask, compress, verify and commit, every output and
    the cache bit for bit, two rounds in a row."""
    from paper_2609_24698_amd import DeviceRound
    c = dict(case)
    name = c.pop("name")
    c.setdefault("max_len_margin", 64)
    _say(f"[one-call small] {name} {c}")
    ra = DeviceRound(synth.make_workload(name, **c), "cuda:0")
    rb = DeviceRound(synth.make_workload(name, **c), "cuda:0")
    keys = [k for k in PER_LAYER + SHARED if k in ra.t]
    for rnd in range(2):
        ra.round_calls()
        rb.round()
        torch.cuda.synchronize()
        for k in keys:
            assert np.array_equal(ra.host(k).view(np.uint8), rb.host(k).view(np.uint8)), (rnd, k)


def test_device_round_step_equals_calls():
    """DeviceRound.round (one-call layer step, then selection and commit)
    against round_calls, with the designated-chain refresh on."""
    _, ra = _layers("C1", 1, True)
    _, rb = _layers("C1", 1, True)
    keys = PER_LAYER + SHARED
    for r in (ra[0], rb[0]):
        r.set_primary(r.host("accepted_last"))
    for rnd in range(3):
        ra[0].round_calls()
        rb[0].round()
        torch.cuda.synchronize()
        for k in keys:
            assert np.array_equal(ra[0].host(k).view(np.uint8), rb[0].host(k).view(np.uint8)), (rnd, k)


def test_commit_failure_in_a_middle_layer():
    """A row whose layer-1 pool has no slot for the accepted path's new CSA
    entry: layer 0 commits it, layer 1 fails it (TV_ROW_CAPACITY), layer 2
    skips it; the graph's one-launch commit of all layers equals the calls
    issued layer by layer, bit for bit."""
    from paper_2609_24698_amd import LayeredRound
    ws, ra = _layers("C1", 3, False, lens=8191)  # every root closes a CSA block
    _, rb = _layers("C1", 3, False, lens=8191)
    w = ws[0]
    _, depth, _ = O.build_tree_mask(w.parents)
    rows = [b for b in range(w.B)
            if any((int(w.lens[b]) + t + 1) % 4 == 0 for t in range(int(depth[b, w.accepted_last[b]]) + 1))]
    assert rows, "no row whose accepted path closes a CSA block"
    row = rows[0]
    for r in (ra[1], rb[1]):
        r.t["c4_cap"][row] = int(w.lens[row]) // 4  # room for the committed entries only
    eager, graph = LayeredRound(ra), LayeredRound(rb)
    graph.capture()
    eager.eager(fused=False)
    graph.replay()
    torch.cuda.synchronize()
    _same(eager, graph, 0)
    assert int(rb[0].host("row_status")[row]) == O.ROW_CAPACITY
    assert int(rb[0].host("len")[row]) > int(w.lens[row])    # layer 0 committed
    assert int(rb[1].host("len")[row]) == int(w.lens[row])   # layer 1 failed
    assert int(rb[2].host("len")[row]) == int(w.lens[row])   # layer 2 skipped
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
        eager.eager(fused=False)
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
