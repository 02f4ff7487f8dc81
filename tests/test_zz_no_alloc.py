"""The verify entry point that allocates nothing (its workspace is a static
device array) against tv_verify_attention with a caller workspace: two calls
in a row, the second on a smaller input, every output bit for bit equal
(the same kernels on the same inputs, fixed reduction orders), which is
within the oracle tolerance of the existing entry point by transitivity; the
existing entry point's own oracle parity is tested elsewhere."""
import sys

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _pair(w):
    from paper_2609_24698_amd import DeviceRound
    a, b = DeviceRound(w, "cuda:0"), DeviceRound(w, "cuda:0")
    for r in (a, b):
        r.mask()
        r.compress()
    return a, b


@pytest.mark.parametrize("first,second", [
    (dict(name="C1"), dict(name="C1", B=2, D=8, lens=[3001, 1000], seed=81, topk=64)),
    (dict(name="C3", B=16, seed=82), dict(name="C0", lens=2047)),
])
def test_noalloc_equals_workspace_entry(first, second):
    for case in (first, second):
        c = dict(case)
        w = synth.make_workload(c.pop("name"), **c)
        print(f"[noalloc] {case} B={w.B} D={w.D} max_len={w.dims['max_len']}", flush=True)
        sys.stdout.flush()
        a, b = _pair(w)
        a.verify()
        b.verify_noalloc()
        torch.cuda.synchronize()
        for k in ("out", "lse", "sel", "row_status"):
            assert np.array_equal(a.host(k).view(np.uint8), b.host(k).view(np.uint8)), k
        assert np.all(b.host("row_status") == 0)
        # nullable outputs behave as in the workspace entry point
        b.t["out"].fill_(-1)
        b.verify_noalloc(with_sel=False, with_lse=False)
        torch.cuda.synchronize()
        assert np.array_equal(a.host("out"), b.host("out"))


def test_noalloc_rejects_oversized_dims():
    from paper_2609_24698_amd import binding
    import ctypes
    d = synth.config_dims("C3")
    d["max_len"] = 1 << 20  # B=64 rows of 1M tokens: far more workspace than the static array holds
    dims = binding.make_dims(d)
    assert binding.tv_verify_workspace_bytes(dims) > binding.NOALLOC_SCRATCH_BYTES
    st = binding.lib().tv_verify_attention_noalloc(ctypes.byref(dims), None, *([None] * 12), None)
    assert st in (binding.TV_ERR_INVALID_ARG, binding.TV_ERR_WORKSPACE)
