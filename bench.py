"""Benchmark of one verify round per step on one MI355X.

A step is the whole hot path over one batch: tree mask, per-branch
compression, verify attention and accepted-path commit, for B rows of D-node
draft trees.  Every step commits its accepted path, so the committed context
grows by the accepted length (at most D tokens per row per step) like a
decoding loop would.  Inputs are synthetic and already resident in HBM.

Prints one JSON line: verified tree tokens per second (B * D per step) over K
timed steps with nothing else on the stream; the roofline of the dominant
kernel (verify attention, HBM bound: algorithmic bytes per launch over its
mean duration, from HIP event pairs that the library records on the launch
stream around every kernel during K further timed steps); and the CPU oracle
timed on a bounded sample of the same workload.  Under "next_rows" it adds the
greedy accepted-path selection over the same trees (target argmax over a
129,280-token vocabulary at every node, then the path), timed on its own with
the roofline of its argmax kernel; the refresh schedule (compress and commit
with each row's accepted path designated as its cached chain, against the
plain refresh); and a round over 61 layers (DeepSeek-V3's
depth; the paper does not state V4-Flash's) issued call by call against the
same round replayed as one HIP graph; neither is part of the step.
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
DOMINANT = "verify_attn"
KERNEL_SOURCES = {"verify_attn": ["attn_mla.hip", "attn_common.h", "tv_common.h"],
                  "target_argmax": ["select.hip", "tv_common.h"]}

WORKLOADS = {
    "C3": "B=64 rows, committed length log-uniform in [1024, 65536] (partially filled 128-token tail), "
          "D=8 random draft trees, 64 query heads over a 576-wide latent (values 512), CSA ratio 4 with top-k 512, "
          "HCA ratio 128, window 128",
    "C1": "B=8 rows, L=8192, D=6 random trees, 64 heads over a 576-wide latent, CSA top-k 512",
    "C2": "B=32 rows, L=32768, D=8 random trees, 64 heads over a 576-wide latent, CSA top-k 512",
    "C4": "B=1 row, L=1048576, D=8 random tree, 64 heads over a 576-wide latent, CSA top-k 2048",
    "C0": "B=1 row, L=2048, tree [-1,0,0,1,1], 8 heads over one 128-wide KV head, CSA top-k 64",
}


def kernel_source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2609_24698_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def attention_bytes(dims, lens, sel, depth, anc):
    """Algorithmic HBM bytes of one verify-attention launch.

    Queries, outputs (bf16) and lse; the selection lists; the union over the
    row's nodes of the CSA rows they select (each row once); every HCA entry a
    node of the row sees; the committed window rows of the row (the root's
    window is the widest); the row's draft-token rows.
    """
    B, D, H = dims["B"], dims["D"], dims["H"]
    row = dims["d_row"] * 2
    total = B * D * H * (dims["d_k"] * 2 + dims["d_v"] * 2 + 4)
    total += B * D * dims["topk"] * 4
    for b in range(B):
        L = int(lens[b])
        s = sel[b]
        total += len(np.unique(s[s >= 0])) * row
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

    One row is timed first to size the sample so that the timed run takes
    about ``budget_s`` seconds; the sample is then timed as a whole.
    """
    from oracle import tv_oracle as O

    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = 1
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
    return dict(value=round(reps * rows * wl.D / dt, 2), unit="tokens/s", cores=int(cores), kind="oracle",
                sample=f"all four steps for the first {rows} of {wl.B} rows ({rows * wl.D} tree nodes, mean "
                       f"length {float(sub.lens.mean()):.0f}) of the same workload, {reps} pass(es), float64 "
                       f"numpy oracle, {dt:.1f} s")


def bench_workload(config: str, steps: int, warmup: int, seed=None):
    """The workload the benchmark times: pools and the length bound leave room
    for every step's commit (at most D tokens per row per step)."""
    import synth

    grow = (3 * steps + warmup + 2) * synth.CONFIGS[config]["D"]  # three timed regions of K steps
    return synth.make_workload(config, seed=seed, max_len_margin=grow, extra_c4=grow // 4 + 8,
                               extra_c128=grow // 128 + 4)


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


def time_refresh(r, wl, K, binding, torch, plain_kern):
    """The refresh schedule with every row's accepted path designated as its
    cached chain (the case where the CSA refresh is skipped entirely): K more
    whole steps with per-kernel HIP events, against the plain steps."""
    r.set_primary(wl.accepted_last)
    binding.tv_profile_enable(8 * K + 16)
    for _ in range(K):
        r.round()
    torch.cuda.synchronize()
    kern = binding.tv_profile_read()
    binding.tv_profile_disable()
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
    ap.add_argument("--no-check", action="store_true", help="skip the sampled oracle check of the first step")
    ap.add_argument("--no-select", action="store_true",
                    help="skip the separately timed accepted-path selection (not part of the step)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the separately timed multi-layer round (eager calls against one graph replay)")
    ap.add_argument("--graph-layers", type=int, default=61)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain elementwise copy of this many MiB five times (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch

    import synth
    from paper_2609_24698_amd import DeviceRound, binding

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
    wl = bench_workload(args.config, K, W, args.seed)
    dims = wl.dims
    print(f"[bench] {args.config}: B={wl.B} D={wl.D} mean L={wl.lens.mean():.0f} "
          f"input {wl.nbytes() / 1e6:.0f} MB", file=sys.stderr, flush=True)
    r = DeviceRound(wl, "cuda:0", poison_outputs=False)

    # first step, checked against the oracle on sampled nodes
    r.mask()
    r.compress()
    r.verify()
    torch.cuda.synchronize()
    sel0 = r.host("sel")
    depth0, anc0 = r.host("depth"), r.host("anc")
    lens0 = r.host("len").copy()
    if not args.no_check:
        from oracle import tv_oracle as O

        rng = np.random.default_rng(0)
        bs = sorted(set(rng.integers(0, wl.B, size=min(4, wl.B)).tolist()))
        nodes = [(b, i) for b in bs for i in range(wl.D)]
        anc, depth, st = O.build_tree_mask(wl.parents)
        scr4, scr128, w4, w128, st = O.branch_compress(wl, anc, depth, st)
        out, lse, sel, st, det = O.verify_attention(wl, anc, depth, scr4, scr128, st, nodes)
        g = O.bf16_to_f64(r.host("out"))
        worst = 0.0
        for (b, i) in nodes:
            if np.array_equal(sel0[b, i][sel0[b, i] >= 0], det[(b, i)]["sel"]):
                worst = max(worst, float(np.abs(g[b, i] - O.round_bf16(out[b, i])).max()))
        assert worst <= 2e-2, f"first-step check failed: max-abs {worst}"
        print(f"[bench] first step matches the oracle on {len(nodes)} nodes (max-abs {worst:.2e})",
              file=sys.stderr, flush=True)
    r.commit()
    for _ in range(W):
        r.round()
    torch.cuda.synchronize()

    # Timed region 1: K whole steps, nothing else on the stream (the value).
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(K):
        r.round()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    # Timed region 2: K more steps with a HIP event pair around every kernel
    # launch, recorded by the library on the launch stream (per-kernel times).
    binding.tv_profile_enable(8 * K + 16)
    ev2, ev3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev2.record(stream)
    for _ in range(K):
        r.round()
    ev3.record(stream)
    torch.cuda.synchronize()
    kern = binding.tv_profile_read()
    binding.tv_profile_disable()
    prof_ms = ev2.elapsed_time(ev3)
    status = r.host("row_status")
    assert np.all(status == 0), f"rows left the workload: {np.unique(status)}"

    ms_per_step = gpu_ms / K
    tokens = wl.B * wl.D
    value = tokens * K / (gpu_ms / 1e3)
    launches, tot = kern[DOMINANT]
    avg_ms = tot / launches
    a_bytes = attention_bytes(dims, lens0, sel0, depth0, anc0)
    achieved = a_bytes / (avg_ms / 1e3) / 1e9
    s_bytes = step_bytes(dims, lens0, sel0, depth0, anc0)

    traffic = pmc_traffic(DOMINANT, args.config)
    select = None
    if not args.no_select:
        select = time_selection(r, wl, K, binding, torch)
        select["roofline"]["traffic"] = pmc_traffic("target_argmax", args.config)

    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_profiled": round(prof_ms / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.config}: {WORKLOADS[args.config]}", "B": wl.B, "D": wl.D,
                   "mean_len": round(float(wl.lens.mean()), 1), "seed": wl.seed,
                   "step_algorithmic_bytes": int(s_bytes),
                   "step_hbm_frac": round(s_bytes / (ms_per_step / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                   "kernels_ms_per_step": {k: round(v[1] / K, 4) for k, v in kern.items()}},
        "roofline": {"bound": "hbm", "kernel": DOMINANT, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": int(a_bytes), "avg_launch_ms": round(avg_ms, 5)},
    }
    refresh = time_refresh(r, wl, K, binding, torch, kern)
    graph = None
    if not args.no_graph:
        graph = {"workloads": {}}
        for cfg in dict.fromkeys([args.config, "C1"]):
            graph["workloads"][cfg] = time_graph(cfg, args.graph_layers, K, W, torch)
    res["next_rows"] = {"refresh_schedule": refresh}
    if select is not None:
        res["next_rows"]["select_accepted_path"] = select
        print(f"[bench] selection: {select['ms_per_call']:.4f} ms per call, argmax "
              f"{select['roofline']['achieved']:.0f} GB/s", file=sys.stderr, flush=True)
    if graph is not None:
        res["next_rows"]["graph_round"] = graph
        for cfg, g in graph["workloads"].items():
            print(f"[bench] {cfg} round over {g['layers']} layers: eager {g['eager_ms_per_round']:.3f} ms, "
                  f"graph {g['graph_ms_per_round']:.3f} ms ({g['kernels_per_round']} kernels)", file=sys.stderr,
                  flush=True)
    print(f"[bench] {K} steps in {gpu_ms:.2f} ms GPU ({wall * 1e3:.2f} ms wall); per-kernel ms/step: "
          + ", ".join(f"{k} {v[1] / K:.4f}" for k, v in kern.items()), file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
