"""The C-ABI library loads, exports every declared entry point, and rejects bad
arguments on the host before touching a GPU (these calls run without one)."""
import ctypes
import os
import re

import pytest

from paper_2609_24698_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "tv.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(tv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = binding.lib()
    names = _declared()
    assert "tv_verify_attention" in names and len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(binding.EXPORTED)


def _dims(**over):
    d = dict(B=2, D=5, H=8, d_row=256, d_k=128, v_off=128, d_v=128, d_idx=64, H_idx=8, ratio_csa=4, ratio_hca=128,
             window=128, topk=64, ring_cap=256, max_len=4096, scale=0.088)
    d.update(over)
    return binding.make_dims(d)


# ring_cap must be a power of two holding the window plus a whole accepted path (window + D): with window 16 and
# D 64 a commit of 64 rows into a 32-slot ring would write two rows to one slot.
BAD = [dict(B=0), dict(D=0), dict(D=65), dict(topk=0), dict(window=0), dict(ring_cap=200), dict(ring_cap=64),
       dict(ring_cap=128), dict(window=16, D=64, ring_cap=32), dict(window=16, D=64, ring_cap=64),
       dict(ratio_csa=0), dict(max_len=-1), dict(v_off=200), dict(scale=float("inf")),
       dict(scale=0.0), dict(scale=-0.5), dict(idx_fmt=2), dict(idx_fmt=-1)]


@pytest.mark.parametrize("over", BAD, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_bad_dims_rejected_without_gpu(over):
    lib = binding.lib()
    d = _dims(**over)
    assert lib.tv_build_tree_mask(ctypes.byref(d), None, None, None, None, None) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_verify_workspace_bytes(ctypes.byref(d)) == 0


def test_unsupported_shapes():
    lib = binding.lib()
    for over in (dict(H=16), dict(d_idx=32), dict(H_idx=3), dict(B=5000)):
        d = _dims(**over)
        assert lib.tv_build_tree_mask(ctypes.byref(d), None, None, None, None, None) == binding.TV_ERR_UNSUPPORTED


# Top-k limits: topk at most 8192; a row of more than 16,896 candidates (ratio 4) is cut into segments, at most
# 64 of them and segments x topk at most 34,816 (the 1M-token row with topk 2048: 16 segments, supported).
TOPK_LIMITS = [
    (dict(topk=8192), True), (dict(topk=8193), False),
    (dict(topk=2048, max_len=1 << 20), True),
    (dict(topk=4096, max_len=4 * 16896 * 9), False),   # 9 segments x 4096 > 34,816
    (dict(topk=64, max_len=4 * 16896 * 64), True),     # 64 segments
    (dict(topk=64, max_len=4 * 16896 * 64 + 4), False),  # 65 segments
]


@pytest.mark.parametrize("over,ok", TOPK_LIMITS, ids=lambda x: ",".join(f"{k}={v}" for k, v in x.items())
                         if isinstance(x, dict) else str(x))
def test_topk_limits_checked_without_gpu(over, ok):
    lib = binding.lib()
    d = _dims(**over)
    want = binding.TV_ERR_INVALID_ARG if ok else binding.TV_ERR_UNSUPPORTED  # null pointers come after the dims
    assert lib.tv_build_tree_mask(ctypes.byref(d), None, None, None, None, None) == want


def test_null_pointers_rejected_without_gpu():
    lib = binding.lib()
    d = _dims()
    assert lib.tv_build_tree_mask(ctypes.byref(d), None, None, None, None, None) == binding.TV_ERR_INVALID_ARG
    cache = binding.TvCache()
    assert lib.tv_branch_compress(ctypes.byref(d), ctypes.byref(cache), *([None] * 9)) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_commit_accepted_path(ctypes.byref(d), ctypes.byref(cache), *([None] * 11)) == \
        binding.TV_ERR_INVALID_ARG
    assert lib.tv_verify_attention(ctypes.byref(d), ctypes.byref(cache), *([None] * 13), 0, None) == \
        binding.TV_ERR_INVALID_ARG


def test_workspace_size_grows_with_max_len():
    lib = binding.lib()
    a = lib.tv_verify_workspace_bytes(ctypes.byref(_dims(max_len=1024)))
    b = lib.tv_verify_workspace_bytes(ctypes.byref(_dims(max_len=65536)))
    assert 0 < a < b


def test_status_strings():
    assert binding.status_string(0) == "ok"
    assert "workspace" in binding.status_string(3)
    assert binding.status_string(99) == "unknown status"


def test_profile_capacity_checked_without_gpu():
    lib = binding.lib()
    assert lib.tv_profile_enable(0) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_profile_read(None, 4, None) == binding.TV_ERR_INVALID_ARG


def test_misaligned_pointers_rejected_without_gpu():
    """Row buffers move with 16-byte accesses: an address off a 16-byte boundary is an argument error,
    found on the host before any device call (the addresses are never dereferenced)."""
    lib = binding.lib()
    d = _dims()
    ok, bad = ctypes.c_void_p(1 << 20), ctypes.c_void_p((1 << 20) + 8)
    assert lib.tv_build_tree_mask(ctypes.byref(d), bad, ok, ok, ok, None) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_build_tree_mask(ctypes.byref(d), ok, ok, ok, bad, None) == binding.TV_ERR_INVALID_ARG
    cache = binding.TvCache()
    for name, _ in binding.TvCache._fields_:
        setattr(cache, name, ok.value)
    cache.c4_idx = bad.value
    assert lib.tv_branch_compress(ctypes.byref(d), ctypes.byref(cache), *([ok] * 7), None, None) == \
        binding.TV_ERR_INVALID_ARG
    for name, _ in binding.TvCache._fields_:
        setattr(cache, name, ok.value)
    # the optional designated chains must be aligned too
    assert lib.tv_branch_compress(ctypes.byref(d), ctypes.byref(cache), *([ok] * 7), bad, None) == \
        binding.TV_ERR_INVALID_ARG
    assert lib.tv_commit_accepted_path(ctypes.byref(d), ctypes.byref(cache), *([ok] * 9), bad, None) == \
        binding.TV_ERR_INVALID_ARG


def test_select_arguments_checked_without_gpu():
    lib = binding.lib()
    d = _dims()
    ok, bad = ctypes.c_void_p(1 << 20), ctypes.c_void_p((1 << 20) + 8)
    assert lib.tv_select_workspace_bytes(ctypes.byref(d), 129280) >= 8 * 2 * 5 * 16
    need = lib.tv_select_workspace_bytes(ctypes.byref(d), 1000)
    assert need >= 8 * 2 * 5 and need % 256 == 0
    assert lib.tv_select_workspace_bytes(ctypes.byref(d), 0) == 0
    assert lib.tv_select_workspace_bytes(ctypes.byref(_dims(B=0)), 1000) == 0
    args = [ok] * 5 + [1000] + [ok, ok, None, ok, ok, need]
    assert lib.tv_select_accepted_path(ctypes.byref(_dims(D=0)), *args, None) == binding.TV_ERR_INVALID_ARG
    bad_vocab = list(args)
    bad_vocab[5] = 0
    assert lib.tv_select_accepted_path(ctypes.byref(d), *bad_vocab, None) == binding.TV_ERR_INVALID_ARG
    for k in (0, 1, 2, 3, 4, 6, 7, 9):  # every required pointer
        a = list(args)
        a[k] = None
        assert lib.tv_select_accepted_path(ctypes.byref(d), *a, None) == binding.TV_ERR_INVALID_ARG, k
        a[k] = bad
        assert lib.tv_select_accepted_path(ctypes.byref(d), *a, None) == binding.TV_ERR_INVALID_ARG, k
    a = list(args)
    a[8] = bad  # optional next_token, misaligned
    assert lib.tv_select_accepted_path(ctypes.byref(d), *a, None) == binding.TV_ERR_INVALID_ARG
    small = list(args)
    small[11] = need - 1
    assert lib.tv_select_accepted_path(ctypes.byref(d), *small, None) == binding.TV_ERR_WORKSPACE
    nows = list(args)
    nows[10] = None
    assert lib.tv_select_accepted_path(ctypes.byref(d), *nows, None) == binding.TV_ERR_WORKSPACE
    odd = list(args)
    odd[10] = ctypes.c_void_p((1 << 20) + 16)
    assert lib.tv_select_accepted_path(ctypes.byref(d), *odd, None) == binding.TV_ERR_INVALID_ARG


def test_round_graph_arguments_checked_without_gpu():
    lib = binding.lib()
    d = _dims()
    rnd = binding.TvRound()
    layers = (binding.TvLayer * 2)()
    h = ctypes.c_void_p(123)
    assert lib.tv_round_graph_create(ctypes.byref(d), ctypes.byref(rnd), layers, 2, None) == binding.TV_ERR_INVALID_ARG
    for n in (0, -1, 1025):
        assert lib.tv_round_graph_create(ctypes.byref(d), ctypes.byref(rnd), layers, n, ctypes.byref(h)) == \
            binding.TV_ERR_INVALID_ARG
        assert h.value is None  # cleared on failure
        h = ctypes.c_void_p(123)
    assert lib.tv_round_graph_create(ctypes.byref(_dims(B=0)), ctypes.byref(rnd), layers, 2, ctypes.byref(h)) == \
        binding.TV_ERR_INVALID_ARG
    assert lib.tv_round_graph_create(ctypes.byref(d), None, layers, 2, ctypes.byref(h)) == binding.TV_ERR_INVALID_ARG
    rnd.draft_tokens = 1 << 20  # selection inputs without logits
    assert lib.tv_round_graph_create(ctypes.byref(d), ctypes.byref(rnd), layers, 2, ctypes.byref(h)) == \
        binding.TV_ERR_INVALID_ARG
    assert lib.tv_round_graph_launch(None, None) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_round_graph_destroy(None) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_round_graph_kernels(None) == 0


def test_verify_round_arguments_checked_without_gpu():
    lib = binding.lib()
    d = _dims()
    rnd = binding.TvRound()
    layer = binding.TvLayer()
    assert lib.tv_verify_round(ctypes.byref(d), None, ctypes.byref(layer), None) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_verify_round(ctypes.byref(d), ctypes.byref(rnd), None, None) == binding.TV_ERR_INVALID_ARG
    assert lib.tv_verify_round(ctypes.byref(_dims(B=0)), ctypes.byref(rnd), ctypes.byref(layer), None) == \
        binding.TV_ERR_INVALID_ARG
    # without parents the mask is not built, but the layer's buffers are still checked
    assert lib.tv_verify_round(ctypes.byref(d), ctypes.byref(rnd), ctypes.byref(layer), None) == \
        binding.TV_ERR_INVALID_ARG
    rnd.parents, rnd.anc, rnd.depth, rnd.row_status = 1 << 20, 1 << 21, 1 << 22, 1 << 23
    assert lib.tv_verify_round(ctypes.byref(d), ctypes.byref(rnd), ctypes.byref(layer), None) == \
        binding.TV_ERR_INVALID_ARG  # null layer buffers
