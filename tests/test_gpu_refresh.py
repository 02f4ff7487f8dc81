"""GPU parity of the refresh schedules (Sec. 4.3): a designated chain's CSA
entries written through at compression, their commit copies skipped.

The compression's pool writes must be exactly the oracle's write-through of
the GPU's own scratch entries; the commit must then leave exactly the oracle's
state, and over every slot a later round can see, the same state as the plain
refresh.  A twin run without a designated chain checks the same over several
rounds on the device."""
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


def _visible(r, b, d):
    L = int(r.host("len")[b])
    b4, b128 = int(r.host("c4_base")[b]), int(r.host("c128_base")[b])
    n4, n128 = L // d["ratio_csa"], L // d["ratio_hca"]
    cap = d["ring_cap"]
    slots = [q & (cap - 1) for q in range(max(0, L - cap), L)]
    return dict(len=L, c4=r.host("c4")[b4:b4 + n4], c4_idx=r.host("c4_idx")[b4:b4 + n4],
                c128=r.host("c128")[b128:b128 + n128], ring=r.host("ring")[b, slots])


def _one_round(w, primary, accepted=None):
    from paper_2609_24698_amd import DeviceRound
    if accepted is not None:
        w.accepted_last[:] = accepted
    r = DeviceRound(w, "cuda:0")
    r.set_primary(primary)
    r.mask()
    r.compress()
    torch.cuda.synchronize()
    anc, depth, st = O.build_tree_mask(w.parents)
    _, _, w4, _, st = O.branch_compress(w, anc, depth, st)
    g4, g128 = r.host("scr_c4"), r.host("scr_c128")
    pools = O.write_through(w, anc, depth, g4, w4, primary, st)
    assert np.array_equal(r.host("c4"), pools[0]) and np.array_equal(r.host("c4_idx"), pools[1])
    r.commit()
    torch.cuda.synchronize()
    untouched = dict(accept_nodes=np.full((w.B, w.D), -2, np.int32), accept_len=np.full(w.B, -2, np.int32))
    f2 = O.commit_accepted_path(w, anc, depth, g4, g128, w.accepted_last, st, primary_last=primary, pools=pools,
                                **untouched)
    plain = O.commit_accepted_path(w, anc, depth, g4, g128, w.accepted_last, st, **untouched)
    for k, dev in (("c4", "c4"), ("c4_idx", "c4_idx"), ("c128", "c128"), ("ring", "ring"), ("lens", "len"),
                   ("status", "row_status"), ("accept_nodes", "accept_nodes"), ("accept_len", "accept_len")):
        assert np.array_equal(r.host(dev), f2[k]), k
    d = w.dims
    for b in range(w.B):  # the plain refresh's committed state
        L = int(plain["lens"][b])
        assert L == int(r.host("len")[b])
        n4, base = L // d["ratio_csa"], int(w.c4_base[b])
        assert np.array_equal(r.host("c4")[base:base + n4], plain["c4"][base:base + n4])
        assert np.array_equal(r.host("c4_idx")[base:base + n4], plain["c4_idx"][base:base + n4])
    assert np.array_equal(r.host("c128"), plain["c128"])
    return r, anc, depth, w4


def _lens(B, rng):
    return [int(4 * rng.integers(300, 600) + rng.integers(0, 4)) for _ in range(B)]


@pytest.mark.parametrize("seed", range(3))
def test_random_trees_and_chains(seed):
    rng = np.random.default_rng(seed)
    B, D = 8, 8
    w = synth.make_workload("C0", B=B, D=D, tree="random", lens=_lens(B, rng), seed=700 + seed)
    _, depth, _ = O.build_tree_mask(w.parents)
    primary = rng.integers(-1, D + 1, size=B).astype(np.int32)
    acc = rng.integers(0, D, size=B).astype(np.int32)
    primary[0] = acc[0]                     # the accepted path is the cached chain
    primary[1] = int(np.argmax(depth[1]))   # accepted node strictly inside the chain
    acc[1] = w.parents[1, primary[1]] if primary[1] > 0 else 0
    _say(f"[refresh] seed={seed} primary={primary.tolist()} accepted={acc.tolist()}")
    _one_round(w, primary, acc)


def test_chain_skips_every_csa_copy():
    w = synth.make_workload("C0", D=8, chain=True, lens=2041, B=3)
    w.c4_cap[2] = 2041 // 4 + 1  # one of the chain's two CSA slots fits: the row fails at commit
    _one_round(w, np.full(3, 7, np.int32), np.array([7, 4, 7], np.int32))


def test_mla_shape_full_size():
    """The benchmark's ragged B=64 workload, the chain ending at the accepted node or elsewhere."""
    w = bench.bench_workload("C3", 20, 5)
    rng = np.random.default_rng(5)
    primary = np.where(rng.random(w.B) < 0.5, w.accepted_last, rng.integers(0, w.D, size=w.B)).astype(np.int32)
    _say(f"[refresh] C3 B={w.B}")
    _one_round(w, primary)


def test_rounds_on_device_match_the_plain_refresh():
    """Four rounds on the device with and without designated chains: after
    every round the committed state seen by the next round is the same."""
    from paper_2609_24698_amd import DeviceRound
    rng = np.random.default_rng(9)
    B, D = 6, 8
    w = synth.make_workload("C1", B=B, D=D, lens=_lens(B, rng), max_len_margin=64)
    a, b_ = DeviceRound(w, "cuda:0"), DeviceRound(w, "cuda:0")
    for rnd in range(4):
        par = np.full((B, D), -1, np.int32)
        for i in range(1, D):
            par[:, i] = rng.integers(0, i, size=B)
        acc = rng.integers(0, D, size=B).astype(np.int32)
        prim = np.where(rng.random(B) < 0.5, acc, rng.integers(0, D, size=B)).astype(np.int32)
        for r in (a, b_):
            r.t["parents"].copy_(torch.from_numpy(par))
            r.t["accepted_last"].copy_(torch.from_numpy(acc))
        b_.set_primary(prim)
        for r in (a, b_):
            r.mask()
            r.compress()
            r.verify()
            r.commit()
        torch.cuda.synchronize()
        for k in ("out", "lse", "sel", "scr_c4", "scr_c128", "accept_nodes", "accept_len", "row_status"):
            assert np.array_equal(a.host(k).view(np.uint8), b_.host(k).view(np.uint8)), (rnd, k)
        for row in range(B):
            va, vb = _visible(a, row, w.dims), _visible(b_, row, w.dims)
            for k in va:
                assert np.array_equal(np.asarray(va[k]), np.asarray(vb[k])), (rnd, row, k)
