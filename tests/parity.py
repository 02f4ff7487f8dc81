"""Comparison helpers for GPU-vs-oracle parity tests.

Tolerances: ancestor masks, depths, accepted-path lists, commit layout and
integer status are bit-exact.  Attention outputs and compressed entries are
bfloat16 and must be within max-abs 2e-2 and mean-abs 2e-3 of the oracle's
float64 value rounded to bfloat16.  CSA selections must be identical except
where the oracle's scores at the selection boundary are within 1e-5 relative
of each other (near ties that float32 scoring may order differently).
"""
from __future__ import annotations

import math

import numpy as np

from oracle import tv_oracle as O

MAX_ABS = 2e-2
MEAN_ABS = 2e-3
TIE_REL = 1e-5
# lse: the paper and the contract fix no tolerance, so it follows from the
# kernels' arithmetic.  The value product takes bfloat16 probabilities and the
# normalising sum is the sum of those same probabilities; bfloat16 has 8 bits
# of precision, so each probability is off by at most 2^-8 of itself and the
# sum by at most 2^-8 of itself: |d lse| <= ln(1 + 2^-8) = 3.9e-3 (reached
# when one key dominates a peaky softmax).  1e-4 covers the float32 logits.
LSE_ABS = math.log1p(2.0 ** -8) + 1e-4


def bf16_err(gpu_bits: np.ndarray, ref_f64: np.ndarray):
    g = O.bf16_to_f64(gpu_bits)
    r = O.round_bf16(ref_f64)
    assert np.all(np.isfinite(g)), "GPU output holds NaN/inf (unwritten or corrupted)"
    e = np.abs(g - r)
    return float(e.max()) if e.size else 0.0, float(e.mean()) if e.size else 0.0


def assert_bf16_close(gpu_bits, ref_f64, what: str):
    mx, mean = bf16_err(gpu_bits, ref_f64)
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max-abs {mx:.3e} mean-abs {mean:.3e}"
    return mx, mean


# A quantised code (an FP8 E4M3 indexer key) decided from a float32 value on
# the GPU and a float64 one in the oracle may land on either side of a
# rounding midpoint the two values straddle: a code one step away is accepted
# where the oracle's unrounded value lies within this fraction of its
# magnitude (at least the E4M3 normal threshold 2**-6) of a midpoint.  The
# GPU's pooled float32 value is off by about 1e-6 of its magnitude.
E4M3_MID_REL = 1e-4


def assert_e4m3_codes(gpu_bf16_bits, ref_pooled_f64, what: str):
    """FP8 indexer channels of compressed entries (E4M3 values held in
    bfloat16): codes equal to the oracle's rounding of its pooled value,
    except one step away at a near-midpoint.  Returns the number of such
    near-midpoint channels."""
    g = O.bf16_to_f64(gpu_bf16_bits)
    assert np.all(np.isfinite(g)), f"{what}: non-finite"
    gc = O.f64_to_e4m3(g)
    assert np.array_equal(O.e4m3_to_f64(gc), g), f"{what}: not E4M3 values"
    rc = O.f64_to_e4m3(ref_pooled_f64)
    diff = gc != rc
    if not diff.any():
        return 0
    lo, hi = np.minimum(gc, rc)[diff], np.maximum(gc, rc)[diff]
    v = ref_pooled_f64[diff]
    va, vb = np.abs(O.e4m3_to_f64(lo)), np.abs(O.e4m3_to_f64(hi))
    mid = (va + vb) / 2
    step = (hi & 0x7F).astype(int) - (lo & 0x7F).astype(int)
    near = np.abs(np.abs(v) - mid) <= E4M3_MID_REL * np.maximum(np.abs(v), 2.0 ** -6)
    same_sign = (lo & 0x80) == (hi & 0x80)
    ok = same_sign & (step == 1) & near
    assert np.all(ok), f"{what}: {int((~ok).sum())} E4M3 codes differ away from a rounding midpoint"
    return int(diff.sum())


def assert_sel_layout(gpu_sel: np.ndarray, n: int, where: str):
    """The ABI's selection layout: the first n entries strictly ascending and
    non-negative, every later slot exactly -1."""
    head, tail = gpu_sel[:n], gpu_sel[n:]
    assert np.all(head >= 0) and np.all(np.diff(head) > 0), f"{where}: selection not ascending: {head[:16]}"
    assert np.all(tail == -1), f"{where}: padding is not -1: {np.unique(tail)[:8]}"


def selection_matches(gpu_sel: np.ndarray, ref_detail: dict, k: int):
    """True if identical; 'tie' if they differ only within near-ties; False otherwise."""
    ref = np.asarray(ref_detail["sel"])
    g = gpu_sel[gpu_sel >= 0]
    if len(g) == len(ref) and np.array_equal(g, ref):
        return True
    if len(g) != len(ref):
        return False
    scores = ref_detail["scores"]
    vals = sorted(scores.values(), reverse=True)
    if len(vals) <= k:
        return False
    kth = vals[k - 1]
    diff = set(g.tolist()) ^ set(ref.tolist())
    tol = TIE_REL * max(abs(kth), 1e-30)
    if all(s in scores and abs(scores[s] - kth) <= tol for s in diff):
        return "tie"
    return False


def compare_verify(gpu_out, gpu_lse, gpu_sel, ref, nodes, dims, own_ref=None, rerun=None):
    """Compare verify outputs node by node; returns stats.

    Every node's selection must have the ABI layout (ascending, -1 padded)
    and equal the oracle's, except within near ties.

    ``own_ref(b, i)`` is given when the GPU verified against its own scratch
    entries rather than the oracle's (which may differ in the last bfloat16
    bit): the oracle's node result is then recomputed on the GPU's scratch,
    and the GPU's selection must match that one under the same near-tie rule.
    ``rerun(b, i, chosen)`` returns the oracle's result for a node with a given
    selection; nodes whose selection differs within a near tie are compared
    against the oracle run on the GPU's selection (skipped without it).
    """
    k = dims["topk"]
    ties = 0
    worst = 0.0
    sums = 0.0
    count = 0
    for (b, i) in nodes:
        det = own_ref(b, i) if own_ref is not None else ref["detail"][(b, i)]
        assert_sel_layout(gpu_sel[b, i], len(det["sel"]), f"row {b} node {i}")
        m = selection_matches(gpu_sel[b, i], det, k)
        assert m is not False, f"selection mismatch at row {b} node {i}"
        if m == "tie":
            ties += 1
            if rerun is None:
                continue
            det = rerun(b, i, gpu_sel[b, i][gpu_sel[b, i] >= 0])
        mx, mean = bf16_err(gpu_out[b, i], det["out"])
        assert mx <= MAX_ABS, f"out row {b} node {i}: max-abs {mx:.3e}"
        worst = max(worst, mx)
        sums += mean
        count += 1
        if gpu_lse is not None:
            le = np.abs(gpu_lse[b, i].astype(np.float64) - det["lse"]).max()
            assert le <= LSE_ABS, f"lse row {b} node {i}: {le:.3e}"
    mean_all = sums / max(count, 1)
    assert mean_all <= MEAN_ABS, f"out mean-abs {mean_all:.3e}"
    return dict(nodes=count, ties=ties, max_abs=worst, mean_abs=mean_all)
