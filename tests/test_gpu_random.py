"""GPU parity on seeded random configurations: tree size and shape, ragged
lengths (some one token short of a block boundary), top-k, indexer heads,
FP8 indexer keys and the paged pool drawn together, so that combinations the
targeted tests do not name are covered too.  Each configuration runs every
stage against the oracle, then the one-call layer step against the separate
calls for two rounds."""
import sys

import numpy as np
import pytest
import torch

import synth

from .test_gpu_parity import _check_stages, _rerun

pytestmark = pytest.mark.gpu

N_CONFIGS = 40


def random_config(k: int) -> dict:
    rng = np.random.default_rng(9100 + k)
    name = str(rng.choice(["C0", "C1"]))
    B = int(rng.integers(1, 5))
    D = int(rng.choice([1, 2, 5, 8, 12, 16]))
    lens = []
    for _ in range(B):
        if rng.random() < 0.4:  # the root or a shallow node closes a block
            lens.append(int(128 * rng.integers(2, 40) - 1 - rng.integers(0, min(D, 4))))
        else:
            lens.append(int(rng.integers(0, 6000)))
    c = dict(name=name, B=B, D=D, tree="random", lens=lens, seed=9200 + k, max_len_margin=64,
             topk=int(rng.choice([16, 64, 512])), H_idx=int(rng.choice([4, 8])),
             idx_fmt=int(rng.random() < 0.3))
    if rng.random() < 0.3:
        c["page_size"] = int(rng.choice([128, 256]))
    return c


@pytest.mark.parametrize("k", range(N_CONFIGS))
def test_random_configuration(k):
    from paper_2609_24698_amd import DeviceRound
    c = random_config(k)
    name = c.pop("name")
    print(f"[random {k}] {name} {c}", flush=True)
    sys.stdout.flush()
    from oracle import tv_oracle as O
    w = synth.make_workload(name, **c)
    ref = O.run_round(w)
    _check_stages(w, ref, DeviceRound(w, "cuda:0"), rerun=_rerun(w, ref))
    ra = DeviceRound(synth.make_workload(name, **c), "cuda:0")
    rb = DeviceRound(synth.make_workload(name, **c), "cuda:0")
    keys = [key for key in ("out", "lse", "sel", "scr_c4", "scr_c128", "ring", "c4", "c4_idx", "c128", "len",
                            "anc", "depth", "row_status", "accept_nodes", "accept_len") if key in ra.t]
    for rnd in range(2):
        ra.round_calls()
        rb.round()
        torch.cuda.synchronize()
        for key in keys:
            assert np.array_equal(ra.host(key).view(np.uint8), rb.host(key).view(np.uint8)), (rnd, key)


@pytest.mark.parametrize("k", range(8))
def test_random_graph_round(k):
    """The captured multi-layer round on random configurations: every replay
    equals the same calls issued one by one, three rounds, with the
    program's own eager work between replays."""
    from paper_2609_24698_amd import LayeredRound
    from .test_gpu_graph import _layers, _same
    c = random_config(100 + k)
    name = c.pop("name")
    c.pop("seed")
    c.pop("max_len_margin")
    n = 2 + k % 2
    select = k % 3 == 0
    print(f"[random graph {k}] {name} layers={n} select={select} {c}", flush=True)
    _, ra = _layers(name, n, select, **c)
    _, rb = _layers(name, n, select, **c)
    eager, graph = LayeredRound(ra), LayeredRound(rb)
    graph.capture()
    noise = torch.empty(1 << 20, device="cuda:0")
    for rnd in range(3):
        eager.eager(fused=False)
        graph.replay()
        torch.cuda.synchronize()
        _same(eager, graph, rnd)
        noise.normal_()
        torch.cuda.synchronize()
    graph.release()
