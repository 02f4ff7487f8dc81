"""Benchmark of one verify round per step on one MI355X.

A step is the whole hot path over one batch: tree mask, per-branch
compression and verify attention in one library call (the mask, the CSA
entries and the indexer scoring share a launch; the HCA entries share the
top-k's), then the accepted-path commit, for B rows of D-node draft trees.
Every step commits its accepted path, so the committed context grows by the
accepted length (at most D tokens per row per step) like a decoding loop
would.  Inputs are synthetic and already resident in HBM.

Cold and warm caches.  Between two verify rounds of one layer a decoder runs
every other layer of the model, so a layer's KV is no longer in the 256 MB
Infinity Cache or the L2 when its next round starts.  The headline numbers
are therefore cold: before every timed step a 1 GiB device copy (512 MiB read,
512 MiB written) evicts both caches, outside the step's HIP event pair.  Warm
numbers (steps back to back, one step's footprint fitting the Infinity Cache)
are reported next to them, labelled.

Prints one JSON line: verified tree tokens per second (B * D per step) over K
timed cold steps; the roofline of the dominant kernel (verify attention, HBM
bound: algorithmic bytes per launch over its mean cold duration, from HIP
event pairs that the library records on the launch stream around every kernel
during K further cold steps), with its bf16 MFMA fraction; and the CPU oracle
timed on a bounded sample of the same workload.  Under "next_rows" it adds the
other workloads (each its own cold/warm step time and attention roofline,
the B=32 tree against its chain twin on identical bytes, and the 8-head
reading of the ragged workload), the greedy accepted-path selection over the
same trees, the refresh schedule (each stage its own call, so the compression
is timed alone), and a round over 61 layers issued call by call against the
same round replayed as one HIP graph; none of them is part of the step.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verified tree tokens/sec at B=64,D=8,16K ctx; % of MI355X peak HBM GB/s"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
DOMINANT = "verify_attn"
KERNEL_SOURCES = {"verify_attn": ["attn_mla.hip", "attn_common.h", "tv_common.h"],
                  "target_argmax": ["select.hip", "tv_common.h"]}
FLUSH_MIB = 512  # copy source and destination, each: 1 GiB through the caches per flush

WORKLOADS = {
    "C3": "B=64 rows, committed length log-uniform in [1024, 65536] (stratified draw, mean ~15.5K; partially "
          "filled 128-token tail), D=8 random draft trees, 64 query heads over a 576-wide latent (values 512), CSA "
          "ratio 4 with top-k 512, HCA ratio 128, window 128",
    "C1": "B=8 rows, L=8192, D=6 random trees, 64 heads over a 576-wide latent, CSA top-k 512",
    "C2": "B=32 rows, L=32768, D=8 random trees, 64 heads over a 576-wide latent, CSA top-k 512",
    "C4": "B=1 row, L=1048576, D=8 random tree, 64 heads over a 576-wide latent, CSA top-k 2048",
    "C0": "B=1 row, L=2048, tree [-1,0,0,1,1], 8 heads over one 128-wide KV head, CSA top-k 64",
}
# Workloads timed under next_rows: (label, config, overrides).
NEXT_WORKLOADS = [
    ("C0", "C0", {}),
    ("C1", "C1", {}),
    ("C2", "C2", {}),
    ("C2-chain", "C2", {"chain": True}),
    ("C4", "C4", {}),
    ("C3-8head", "C3", {"shape": "mha128"}),
    ("C3-fp8keys", "C3", {"idx_fmt": 1}),
    ("C3-paged", "C3", {"page_size": 128}),
]


def kernel_source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2609_24698_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def attention_bytes(dims, lens, sel, depth, anc):
    """Algorithmic HBM bytes of one verify-attention launch.

    Queries, outputs (bf16) and lse; the selection lists; the union over the
    row's nodes of the CSA rows they select (each row once: a committed entry
    by its index, an entry closed on a path by the scratch slot of the node
    that closed it, since siblings close the same index in different slots);
    every HCA entry a node of the row sees; the committed window rows of the
    row (the root's window is the widest); the row's draft-token rows.
    """
    B, D, H = dims["B"], dims["D"], dims["H"]
    r4 = dims["ratio_csa"]
    row = dims["d_row"] * 2
    total = B * D * H * (dims["d_k"] * 2 + dims["d_v"] * 2 + 4)
    total += B * D * dims["topk"] * 4
    for b in range(B):
        L = int(lens[b])
        n4 = L // r4
        committed, closers = set(), set()
        for i in range(D):
            si = sel[b, i][sel[b, i] >= 0]
            committed.update(int(x) for x in si[si < n4])
            on_path = set(int(x) for x in si[si >= n4])
            for j in range(D):
                q = L + int(depth[b, j]) + 1
                if (int(anc[b, i]) >> j) & 1 and q % r4 == 0 and q // r4 - 1 in on_path:
                    closers.add(j)
        total += (len(committed) + len(closers)) * row
        total += (L // dims["ratio_hca"]) * row
        hca_closers = {j for j in range(D) if (L + int(depth[b, j]) + 1) % dims["ratio_hca"] == 0}
        total += len(hca_closers) * row
        total += min(L, dims["window"] - 1) * row
        total += D * row
    return total


def step_bytes(dims, lens, sel, depth, anc):
    """Algorithmic bytes of the whole step: attention plus the indexer keys and queries."""
    n4 = sum(int(L) // dims["ratio_csa"] for L in lens)
    b = attention_bytes(dims, lens, sel, depth, anc)
    b += n4 * dims["d_idx"] * 2
    b += dims["B"] * dims["D"] * dims["H_idx"] * (dims["d_idx"] * 2 + 2)
    return b


def node_key_counts(dims, lens, depth, anc):
    """Keys node (b, i) attends to: its CSA selection, every HCA entry it sees
    (committed and closed on its path), its committed window and its path."""
    B, D = depth.shape
    r4, r128, W, k = dims["ratio_csa"], dims["ratio_hca"], dims["window"], dims["topk"]
    n = np.zeros((B, D), dtype=np.int64)
    for b in range(B):
        L = int(lens[b])
        for i in range(D):
            path = [j for j in range(D) if (int(anc[b, i]) >> j) & 1]
            ncsa = sum(1 for j in path if (L + int(depth[b, j]) + 1) % r4 == 0)
            nhca = sum(1 for j in path if (L + int(depth[b, j]) + 1) % r128 == 0)
            p = L + int(depth[b, i])
            lo = max(0, p - W + 1)
            nsel = min(k, L // r4 + ncsa)
            n[b, i] = nsel + L // r128 + nhca + max(0, L - lo) + (p - max(lo, L) + 1)
    return n


def attention_flops(dims, nkeys):
    """Dense-contraction flops of one attention launch: per attended (node,
    key) pair, the logits of every head over d_k channels and the value sum
    over d_v channels."""
    return int(nkeys.sum()) * 2 * dims["H"] * (dims["d_k"] + dims["d_v"])


def gathered_bytes(dims, nkeys):
    """Key-row bytes one attention launch gathers into LDS: every workgroup
    gathers each key of its node once."""
    return int(nkeys.sum()) * dims["d_row"] * 2


def check_selection_layout(dims, lens, depth, anc, sel):
    """The first step's selections have the ABI layout: min(topk, candidates)
    ascending indices of visible entries, then -1."""
    B, D = depth.shape
    r4, k = dims["ratio_csa"], dims["topk"]
    for b in range(B):
        L = int(lens[b])
        for i in range(D):
            path = [j for j in range(D) if (int(anc[b, i]) >> j) & 1]
            cand = L // r4 + sum(1 for j in path if (L + int(depth[b, j]) + 1) % r4 == 0)
            n = min(k, cand)
            s = sel[b, i]
            assert np.all(s[:n] >= 0) and np.all(np.diff(s[:n]) > 0) and np.all(s[:n] < cand), (b, i)
            assert np.all(s[n:] == -1), (b, i)


def _first_rows(wl, n):
    """The same workload restricted to its first n rows (pools stay shared)."""
    import dataclasses

    dims = dict(wl.dims)
    dims["B"] = n
    cut = {k: getattr(wl, k)[:n] for k in ("lens", "parents", "accepted_last", "ring", "c4_base", "c4_cap",
                                           "c128_base", "c128_cap", "tree_u", "q", "q_idx", "w_idx")}
    return dataclasses.replace(wl, dims=dims, **cut)


def cpu_baseline(wl, budget_s: float):
    """The CPU oracle (all four steps) on the first rows of the same workload.

    The oracle is a single Python thread; its numpy calls are held to one BLAS
    thread, so it uses exactly one core.  One row is timed first to size the
    sample so that the timed run takes about ``budget_s`` seconds; the sample
    is then timed as a whole.
    """
    from threadpoolctl import threadpool_limits

    from oracle import tv_oracle as O

    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        O.run_round(_first_rows(wl, 1))
        t1 = time.perf_counter() - t0
        rows = int(max(1, min(wl.B, budget_s // max(t1, 1e-3))))
        sub = _first_rows(wl, rows)
        reps = 0
        t0 = time.perf_counter()
        while True:  # whole passes over the sample until the budget is spent
            O.run_round(sub)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= budget_s or rows < wl.B:
                break
    return dict(value=round(reps * rows * wl.D / dt, 2), unit="tokens/s", cores=1, kind="oracle",
                sample=f"all four steps for the first {rows} of {wl.B} rows ({rows * wl.D} tree nodes, mean "
                       f"length {float(sub.lens.mean()):.0f}) of the same workload, {reps} pass(es), float64 "
                       f"numpy oracle on one thread (BLAS held to 1 thread; host has {os.cpu_count()} CPUs), "
                       f"{dt:.1f} s")


def bench_workload(config: str, steps: int, warmup: int, seed=None, **over):
    """The workload the benchmark times: pools and the length bound leave room
    for every step's commit (at most D tokens per row per step)."""
    import synth

    grow = (6 * steps + warmup + 2) * synth.CONFIGS[config]["D"]  # six timed regions of K steps
    return synth.make_workload(config, seed=seed, max_len_margin=grow, extra_c4=grow // 4 + 8,
                               extra_c128=grow // 128 + 4, **over)


def pmc_traffic(kernel: str, config: str):
    """Calibrated HBM bytes per launch from the committed counter summary,
    or None when the kernel's sources changed since the counters were taken."""
    pmc_file = os.path.join(ROOT, "profiles", f"{kernel}_{config}_pmc.json")
    if not os.path.exists(pmc_file):
        return None
    with open(pmc_file) as f:
        pmc = json.load(f)
    if pmc.get("source_hash") != kernel_source_hash(kernel):
        return None
    return pmc.get("hbm_bytes_per_launch")


class Flush:
    """Evicts the L2s and the Infinity Cache: a device copy of FLUSH_MIB MiB
    (read) into another FLUSH_MIB MiB (written), on the current stream."""

    def __init__(self, torch):
        n = FLUSH_MIB << 18
        self.src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        self.dst = torch.empty_like(self.src)

    def __call__(self):
        self.dst.copy_(self.src)


def time_steps(r, K, torch, flush=None, binding=None):
    """K whole steps.  With ``flush``, a cache flush precedes every step,
    outside its HIP event pair; without, the steps run back to back under one
    event pair.  With ``binding``, the library also records an event pair
    around every kernel.  Returns (per-step ms list, per-kernel dict)."""
    stream = torch.cuda.current_stream()
    if binding is not None:
        binding.tv_profile_enable(8 * K + 16)
    torch.cuda.synchronize()
    if flush is not None:
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
        for e0, e1 in ev:
            flush()
            e0.record(stream)
            r.round()
            e1.record(stream)
        torch.cuda.synchronize()
        ms = [e0.elapsed_time(e1) for e0, e1 in ev]
    else:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(K):
            r.round()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = [e0.elapsed_time(e1) / K] * K
    kern = None
    if binding is not None:
        kern = binding.tv_profile_read()
        binding.tv_profile_disable()
    return ms, kern


def attention_roofline(dims, kern, a_bytes, flops, gathered):
    launches, tot = kern[DOMINANT]
    avg = tot / launches
    achieved = a_bytes / (avg / 1e3) / 1e9
    tflops = flops / (avg / 1e3) / 1e12
    return {"bound": "hbm", "kernel": DOMINANT, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "algorithmic_bytes_per_launch": int(a_bytes),
            "avg_launch_ms": round(avg, 5), "mfma_tflops": round(tflops, 1),
            "mfma_frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4), "flops_per_launch": int(flops),
            "lds_gathered_bytes_per_launch": int(gathered)}


def measure(wl, K, W, torch, binding, flush):
    """First step (its selections, depths and lengths size the algorithmic
    bytes and are checked for the ABI layout), W warm-up steps, then: K cold
    steps, K warm steps, K cold steps with per-kernel events and K warm steps
    with per-kernel events."""
    from paper_2609_24698_amd import DeviceRound

    r = DeviceRound(wl, "cuda:0", poison_outputs=False)
    r.verify_round()
    torch.cuda.synchronize()
    st = r.host("row_status")
    assert np.all(st == 0), f"rows failed: {np.unique(st)}"
    sel0, depth0, anc0, lens0 = r.host("sel"), r.host("depth"), r.host("anc"), r.host("len").copy()
    check_selection_layout(wl.dims, lens0, depth0, anc0, sel0)
    out0 = r.host("out")
    assert not np.any((out0 & 0x7F80) == 0x7F80), "non-finite attention output"
    r.commit()
    for _ in range(W):
        r.round()
    cold, _ = time_steps(r, K, torch, flush=flush)
    warm, _ = time_steps(r, K, torch)
    _, kern_cold = time_steps(r, K, torch, flush=flush, binding=binding)
    _, kern_warm = time_steps(r, K, torch, binding=binding)
    st = r.host("row_status")
    assert np.all(st == 0), f"rows left the workload: {np.unique(st)}"
    nk = node_key_counts(wl.dims, lens0, depth0, anc0)
    a_bytes = attention_bytes(wl.dims, lens0, sel0, depth0, anc0)
    m = dict(r=r, cold=cold, warm=warm, kern_cold=kern_cold, kern_warm=kern_warm, lens0=lens0, sel0=sel0,
             depth0=depth0, anc0=anc0, a_bytes=a_bytes, s_bytes=step_bytes(wl.dims, lens0, sel0, depth0, anc0),
             flops=attention_flops(wl.dims, nk), gathered=gathered_bytes(wl.dims, nk), pairs=int(nk.sum()))
    m["roof_cold"] = attention_roofline(wl.dims, kern_cold, a_bytes, m["flops"], m["gathered"])
    m["roof_warm"] = attention_roofline(wl.dims, kern_warm, a_bytes, m["flops"], m["gathered"])
    return m


def workload_line(label, wl, m, K):
    cold_ms, warm_ms = float(np.mean(m["cold"])), float(np.mean(m["warm"]))
    tok = wl.B * wl.D
    return {"workload": label, "B": wl.B, "D": wl.D, "H": wl.dims["H"], "topk": wl.dims["topk"],
            "mean_len": round(float(wl.lens.mean()), 1),
            "cold_ms_per_step": round(cold_ms, 4), "cold_median_ms": round(float(np.median(m["cold"])), 4),
            "cold_tokens_per_s": round(tok / (cold_ms / 1e3), 1),
            "warm_ms_per_step": round(warm_ms, 4), "warm_tokens_per_s": round(tok / (warm_ms / 1e3), 1),
            "step_algorithmic_bytes": int(m["s_bytes"]),
            "step_hbm_frac_cold": round(m["s_bytes"] / (cold_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
            "attended_pairs": m["pairs"],
            "kernels_ms_cold": {k: round(v[1] / v[0], 4) for k, v in m["kern_cold"].items()},
            "kernels_ms_warm": {k: round(v[1] / v[0], 4) for k, v in m["kern_warm"].items()},
            "attention_cold": m["roof_cold"], "attention_warm": m["roof_warm"]}


def time_selection(r, wl, K, binding, torch):
    """Accepted-path selection over the same trees with a vocabulary of
    synth.VOCAB tokens, timed on its own (it follows verify in a decoding
    round but is not part of the step): K calls, per-kernel HIP events."""
    import synth

    sel = synth.make_selection(wl)
    r.attach_selection(sel)
    for _ in range(3):
        r.select()
    torch.cuda.synchronize()
    got = r.host("accepted_last")
    assert np.array_equal(got, sel.planted_last), "selection did not accept the planted paths"
    stream = torch.cuda.current_stream()
    binding.tv_profile_enable(2 * K + 4)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(K):
        r.select()
    e1.record(stream)
    torch.cuda.synchronize()
    kern = binding.tv_profile_read()
    binding.tv_profile_disable()
    n, tot = kern["target_argmax"]
    avg = tot / n
    a_bytes = wl.B * wl.D * sel.vocab * 2  # every logit read once
    achieved = a_bytes / (avg / 1e3) / 1e9
    return {"vocab": sel.vocab, "calls": K, "ms_per_call": round(e0.elapsed_time(e1) / K, 4),
            "kernels_ms_per_call": {k: round(v[1] / v[0], 4) for k, v in kern.items()},
            "roofline": {"bound": "hbm", "kernel": "target_argmax", "achieved": round(achieved, 1),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                         "traffic": None, "algorithmic_bytes_per_launch": int(a_bytes),
                         "avg_launch_ms": round(avg, 5)}}


def time_refresh(r, wl, K, binding, torch):
    """The refresh schedule with every row's accepted path designated as its
    cached chain (the case where the CSA refresh is skipped entirely): K whole
    steps with per-kernel HIP events, plain then designated, each stage its
    own call so the compression is timed alone."""
    def kernels():
        binding.tv_profile_enable(8 * K + 16)
        for _ in range(K):
            r.round_calls()
        torch.cuda.synchronize()
        kern = binding.tv_profile_read()
        binding.tv_profile_disable()
        return kern

    r.round_calls()  # the separate calls' kernels are loaded before they are timed
    torch.cuda.synchronize()
    plain_kern = kernels()
    r.set_primary(wl.accepted_last)
    kern = kernels()
    r.set_primary(None)
    status = r.host("row_status")
    assert np.all(status == 0), f"rows left the workload: {np.unique(status)}"
    out = {}
    for k in ("branch_compress", "commit_path"):
        out[k] = {"plain_ms": round(plain_kern[k][1] / plain_kern[k][0], 4),
                  "designated_chain_ms": round(kern[k][1] / kern[k][0], 4)}
    return out


def time_graph(config: str, n_layers: int, K: int, W: int, torch):
    """One round over n_layers layers sharing a draft tree (mask once;
    compress and verify per layer; commit per layer), issued call by call
    from Python and as one captured graph, on the same device state: K rounds
    each, HIP events on the stream around the K rounds.  Every layer holds
    its own copy of the workload's buffers."""
    from paper_2609_24698_amd import DeviceRound, LayeredRound

    wl = bench_workload(config, K + W + 2, 0)  # the pools take both timings' commits
    lr = LayeredRound([DeviceRound(wl, "cuda:0", poison_outputs=False) for _ in range(n_layers)])
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(W):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(K):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K, (time.perf_counter() - t0) * 1e3 / K

    eager_ms, eager_wall = timed(lr.eager)
    kernels = lr.capture()
    graph_ms, graph_wall = timed(lr.replay)
    lr.release()
    status = lr.layers[0].host("row_status")
    assert np.all(status == 0), f"rows left the workload: {np.unique(status)}"
    res = {"layers": n_layers, "kernels_per_round": kernels, "eager_ms_per_round": round(eager_ms, 4),
           "graph_ms_per_round": round(graph_ms, 4), "eager_wall_ms": round(eager_wall, 4),
           "graph_wall_ms": round(graph_wall, 4), "speedup": round(eager_ms / graph_ms, 3),
           "tokens_per_s_graph": round(wl.B * wl.D / (graph_ms / 1e3), 1)}
    del lr
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="C3", choices=sorted(WORKLOADS))
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-next", action="store_true",
                    help="skip the other workloads, the selection, the refresh schedule and the graph round")
    ap.add_argument("--no-workloads", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-select", action="store_true",
                    help="skip the separately timed accepted-path selection (not part of the step)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the separately timed multi-layer round (eager calls against one graph replay)")
    ap.add_argument("--graph-layers", type=int, default=61)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain elementwise copy of this many MiB five times (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch

    from paper_2609_24698_amd import binding

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 18  # float32 elements
        src = torch.randn(n, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": 4 * n, "copy_probe_bytes_written": 4 * n, "launches": 5}))
        return
    K, W = args.steps, args.warmup
    flush = Flush(torch)
    wl = bench_workload(args.config, K, W, args.seed)
    print(f"[bench] {args.config}: B={wl.B} D={wl.D} mean L={wl.lens.mean():.0f} "
          f"input {wl.nbytes() / 1e6:.0f} MB", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    m = measure(wl, K, W, torch, binding, flush)
    r = m["r"]
    wall = time.perf_counter() - t0
    cold_ms = float(np.mean(m["cold"]))
    warm_ms = float(np.mean(m["warm"]))
    tokens = wl.B * wl.D
    value = tokens / (cold_ms / 1e3)
    roof = dict(m["roof_cold"])
    roof["traffic"] = pmc_traffic(DOMINANT, args.config)
    roof["warm"] = {k: m["roof_warm"][k] for k in ("achieved", "frac", "avg_launch_ms", "mfma_frac")}
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(cold_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "cache": "cold: a 1 GiB device copy evicts the L2s and the Infinity Cache before every timed step",
        "warm_value": round(tokens / (warm_ms / 1e3), 1),
        "warm_ms_per_step": round(warm_ms, 4),
        "config": {"workload": f"{args.config}: {WORKLOADS[args.config]}", "B": wl.B, "D": wl.D,
                   "mean_len": round(float(wl.lens.mean()), 1), "seed": wl.seed,
                   "cold_median_ms": round(float(np.median(m["cold"])), 4),
                   "step_algorithmic_bytes": int(m["s_bytes"]),
                   "step_hbm_frac": round(m["s_bytes"] / (cold_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                   "attended_pairs": m["pairs"],
                   "kernels_ms_per_step": {k: round(v[1] / v[0], 4) for k, v in m["kern_cold"].items()},
                   "kernels_ms_per_step_warm": {k: round(v[1] / v[0], 4) for k, v in m["kern_warm"].items()}},
        "roofline": roof,
    }
    print(f"[bench] {K} cold steps: {cold_ms:.4f} ms mean, warm {warm_ms:.4f} ms; per-kernel cold ms: "
          + ", ".join(f"{k} {v[1] / v[0]:.4f}" for k, v in m["kern_cold"].items()), file=sys.stderr, flush=True)
    nxt = {}
    if not args.no_next:
        if not args.no_select:
            sel = time_selection(r, wl, K, binding, torch)
            sel["roofline"]["traffic"] = pmc_traffic("target_argmax", args.config)
            nxt["select_accepted_path"] = sel
            print(f"[bench] selection: {sel['ms_per_call']:.4f} ms per call, argmax "
                  f"{sel['roofline']['achieved']:.0f} GB/s", file=sys.stderr, flush=True)
        nxt["refresh_schedule"] = time_refresh(r, wl, K, binding, torch)
    del r, m
    torch.cuda.empty_cache()
    if not args.no_next and not args.no_workloads:
        lines = {}
        for label, cfg, over in NEXT_WORKLOADS:
            w2 = bench_workload(cfg, K, W, **over)
            m2 = measure(w2, K, W, torch, binding, flush)
            lines[label] = workload_line(label, w2, m2, K)
            print(f"[bench] {label}: cold {lines[label]['cold_ms_per_step']:.4f} ms/step, attention "
                  f"{lines[label]['attention_cold']['avg_launch_ms']:.4f} ms (frac "
                  f"{lines[label]['attention_cold']['frac']:.3f}), kernels "
                  f"{lines[label]['kernels_ms_cold']}", file=sys.stderr, flush=True)
            del m2, w2
            torch.cuda.empty_cache()
        if "C2" in lines and "C2-chain" in lines:
            t, c = lines["C2"], lines["C2-chain"]
            lines["C2_tree_vs_chain"] = {
                "step_cold_ratio": round(t["cold_ms_per_step"] / c["cold_ms_per_step"], 4),
                "step_warm_ratio": round(t["warm_ms_per_step"] / c["warm_ms_per_step"], 4),
                "attention_cold_ratio": round(t["attention_cold"]["avg_launch_ms"]
                                              / c["attention_cold"]["avg_launch_ms"], 4),
                "attended_pairs_ratio": round(t["attended_pairs"] / c["attended_pairs"], 4),
                "note": "tree over chain on identical bytes: ratio of cold step time, warm step time, cold "
                        "attention time and attended (node, key) pairs"}
        nxt["workloads"] = lines
    if not args.no_next and not args.no_graph:
        graph = {"workloads": {}}
        for cfg in dict.fromkeys([args.config, "C1"]):
            graph["workloads"][cfg] = time_graph(cfg, args.graph_layers, K, W, torch)
            g = graph["workloads"][cfg]
            print(f"[bench] {cfg} round over {g['layers']} layers: eager {g['eager_ms_per_round']:.3f} ms, "
                  f"graph {g['graph_ms_per_round']:.3f} ms ({g['kernels_per_round']} kernels)", file=sys.stderr,
                  flush=True)
        nxt["graph_round"] = graph
    if nxt:
        res["next_rows"] = nxt
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    print(f"[bench] done in {time.perf_counter() - t0:.1f} s (first workload {wall:.1f} s)", file=sys.stderr,
          flush=True)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
