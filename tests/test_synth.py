"""The seeded generator: determinism, shapes and the structure the configurations ask for."""
import hashlib

import numpy as np

import synth


def _digest(w):
    h = hashlib.sha256()
    for k in ("lens", "parents", "accepted_last", "ring", "c4", "c4_idx", "c128", "tree_u", "q", "q_idx", "w_idx", "gate_w"):
        h.update(np.ascontiguousarray(getattr(w, k)).tobytes())
    return h.hexdigest()


def test_same_seed_same_bytes():
    assert _digest(synth.make_workload("C0")) == _digest(synth.make_workload("C0"))
    assert _digest(synth.make_workload("C0")) != _digest(synth.make_workload("C0", seed=1))


def test_chain_twin_shares_every_kv_byte():
    a = synth.make_workload("C2", B=4)
    b = synth.make_workload("C2", B=4, chain=True)
    for k in ("lens", "ring", "c4", "c4_idx", "c128", "tree_u", "q", "q_idx", "w_idx", "gate_w"):
        assert np.array_equal(getattr(a, k), getattr(b, k)), k
    assert np.array_equal(b.parents[0], np.arange(-1, 7))


def test_ragged_lengths_and_tail_offsets():
    w = synth.make_workload("C3", B=64)
    L = w.lens.astype(np.int64)
    assert L.min() >= 1024 and L.max() <= 65536
    assert np.all(L % 128 >= 1)
    for b in range(8):
        assert L[b] % 128 == 127 - (b % 4)
    assert 8000 < L.mean() < 25000
    # every parent precedes its child
    assert np.all(w.parents[:, 0] == -1)
    for i in range(1, 8):
        assert np.all((0 <= w.parents[:, i]) & (w.parents[:, i] < i))


def test_pool_layout_and_poison():
    w = synth.make_workload("C1", B=3)
    n4 = w.lens // 4
    for b in range(3):
        base, cap = w.c4_base[b], w.c4_cap[b]
        assert cap >= n4[b]
        assert np.all(w.c4[base + n4[b]:base + cap] == synth.inputs.BF16_NAN)
        assert not np.any(w.c4[base:base + n4[b]] == synth.inputs.BF16_NAN)
    assert w.c4_base[1] == w.c4_cap[0]


def test_value_distributions():
    w = synth.make_workload("C1", B=2)
    q = (w.q.astype(np.uint32) << 16).view(np.float32)
    g = (w.gate_w.astype(np.uint32) << 16).view(np.float32)
    assert abs(q.std() - 1.0) < 0.01 and abs(q.mean()) < 0.01
    assert abs(g.std() - 0.02) < 0.003
