"""A CPU model of the device top-k's radix select, checked against a sort.

The top-k and merge kernels select the k largest order-preserving score keys
with radix passes of 13-bit digits (the last pass the remaining bits), each
restricted to the keys that share the digits found so far, and stop once the
threshold bin holds exactly the keys still needed; an ordered compaction then
takes the keys above the threshold and the lowest-index keys equal to it.
Padding slots hold key 0 and are not tested key by key: while the resolved
prefix is 0 they all fall into bin 0, which starts at minus their count.

The GPU parity tests cannot put the threshold inside that bin: only -inf and
NaN scores have keys below 2**19, and float32 scoring and the float64 oracle
do not produce them alike.  This model, written from the description above,
covers it (keys concentrated in bin 0, ties, padding between real keys) and
must give exactly the k largest keys, ties to the lower index.
"""
import numpy as np
import pytest

BITS = 13


def _radix(keys, n, n_real, k, nt):
    nr = (n + nt - 1) // nt
    pool = keys[:nr * nt]
    n_pad = nr * nt - n_real
    prefix, pmask, rem, shift = 0, 0, k, 32
    while shift > 0:
        nb = min(shift, BITS)
        sft = shift - nb
        nbins = 1 << nb
        h = np.zeros(nbins, dtype=np.int64)
        if prefix == 0:
            h[0] -= n_pad
        m = (pool & pmask) == prefix
        np.add.at(h, ((pool[m] >> sft) & (nbins - 1)).astype(np.int64), 1)
        assert h.min() >= 0
        above, found = 0, None
        for b in range(nbins - 1, -1, -1):
            if above < rem <= above + h[b]:
                found = (b, above, int(h[b]))
                break
            above += int(h[b])
        b, above, c = found
        prefix |= b << sft
        pmask |= (nbins - 1) << sft
        rem -= above
        shift = sft
        if c == rem:
            break
    return prefix, pmask, rem


def _compact(keys, n, prefix, pmask, rem):
    km = keys[:n] & pmask
    taken = km > prefix
    equal = np.nonzero((km == prefix) & (keys[:n] != 0))[0][:rem]
    taken[equal] = True
    return np.nonzero(taken)[0]


def _by_sort(keys, n, k):
    real = [e for e in range(n) if keys[e] != 0]
    return np.array(sorted(sorted(real, key=lambda e: (-int(keys[e]), e))[:k]))


@pytest.mark.parametrize("kind", ["uniform", "bin0", "tiny_ties", "mixed", "all_equal"])
def test_radix_select_model_equals_sort(kind):
    rng = np.random.default_rng(["uniform", "bin0", "tiny_ties", "mixed", "all_equal"].index(kind) + 11)
    cases = 0
    for trial in range(160):
        nt = int(rng.choice([64, 128, 512]))
        kpt = int(rng.integers(1, 5))
        k = int(rng.choice([1, 3, 16, 50, 200]))
        n = int(rng.integers(1, nt * kpt + 1))
        if kind == "uniform":
            v = rng.integers(1, 2**32, size=n)
        elif kind == "bin0":  # every key below 2**19: the threshold lies in bin 0 of the first pass
            v = rng.integers(1, 1 << 19, size=n)
        elif kind == "tiny_ties":
            v = rng.integers(1, 40, size=n)
        elif kind == "mixed":
            v = np.where(rng.random(n) < 0.5, rng.integers(1, 5, size=n), rng.integers(1, 2**32, size=n))
        else:
            v = np.ones(n, dtype=np.int64)
        keys = np.zeros(nt * kpt, dtype=np.uint32)
        keys[:n] = v.astype(np.uint32)
        if trial % 2:  # merge-like: padding slots between the real keys
            keys[:n][rng.random(n) < 0.3] = 0
        n_real = int((keys[:n] != 0).sum())
        if n_real <= k:
            continue
        cases += 1
        prefix, pmask, rem = _radix(keys, n, n_real, k, nt)
        assert np.array_equal(_compact(keys, n, prefix, pmask, rem), _by_sort(keys, n, k)), (kind, trial)
    assert cases > 50
