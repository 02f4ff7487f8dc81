"""GPU parity at full workload sizes, on error rows, and for the variants the
small cases do not reach.

Full sizes run in the benchmark's launch configuration (its workload, its
length bound, hence its split plan) and compare every stage on sampled nodes
the oracle computes one by one: masks, commit layout and row status over all
rows, compressed entries over all closing nodes, verify outputs on the
sampled nodes.
"""
import sys

import numpy as np
import pytest
import torch

import bench
import synth
from oracle import tv_oracle as O

from .parity import assert_bf16_close, compare_verify
from .test_gpu_parity import _check_stages

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _rerun(w, ref):
    def f(b, i, chosen):
        return O.verify_node(w, b, i, ref["anc"], ref["depth"], ref["scr_c4"], ref["scr_c128"], chosen=chosen)
    return f


def _device(w):
    from paper_2609_24698_amd import DeviceRound
    return DeviceRound(w, "cuda:0")


def _full(config, rows, chain=False):
    if chain:
        w = synth.make_workload(config, chain=True)
    else:
        w = bench.bench_workload(config, 20, 5)
    rows = sorted(set(int(b) for b in rows))
    nodes = [(b, i) for b in rows for i in range(w.D)]
    _say(f"[workload] {config} chain={chain} B={w.B} D={w.D} rows={rows} lens={[int(w.lens[b]) for b in rows]}")
    ref = O.run_round(w, nodes)
    r = _device(w)
    stats = _check_stages(w, ref, r, nodes, rerun=_rerun(w, ref))
    _say(f"  {stats}")
    return stats


def test_c2_tree_full_size():
    _full("C2", [0, 13, 31])


def test_c2_chain_twin_full_size():
    """The chain twin of the B=32 workload: identical bytes, parents [-1, 0, 1, ...]."""
    _full("C2", [0, 31], chain=True)


def test_c3_full_size():
    w = bench.bench_workload("C3", 20, 5)
    order = np.argsort(w.lens)
    # the longest and shortest rows, rows whose tree closes an HCA block, one more
    rows = [order[-1], order[-2], order[0], 0, 1, 2, 3, 40]
    _full("C3", rows)


def test_batch_above_256_rows():
    """300 ragged rows of the 8-head shape (more rows than one scoring or
    ranking workgroup has threads): sampled rows on both sides of row 256."""
    lens = np.random.default_rng(91).integers(520, 3100, size=300).tolist()
    w = synth.make_workload("C0", seed=91, B=300, lens=lens, max_len_margin=16)
    rows = [0, 255, 256, 299, int(np.argmax(w.lens))]
    rows = sorted(set(rows))
    nodes = [(b, i) for b in rows for i in range(w.D)]
    _say(f"[workload] C0 B={w.B} D={w.D} rows={rows} lens={[int(w.lens[b]) for b in rows]}")
    ref = O.run_round(w, nodes)
    stats = _check_stages(w, ref, _device(w), nodes, rerun=_rerun(w, ref))
    _say(f"  {stats}")


def test_c4_full_size():
    """One row of 1M committed tokens: 262,144 indexer candidates per node
    (the global-memory top-k path) and split attention with the combine."""
    _full("C4", [0])


@pytest.mark.parametrize("topk,zero_w", [(512, False), (2048, False), (512, True)],
                         ids=["k512", "k2048", "k512-all-ties"])
def test_segmented_topk(topk, zero_w):
    """Rows longer than one top-k segment (16,896 candidates): every segment
    keeps its own top-k and a merge selects among the survivors.  Row 0 has
    three segments, row 1 two.  With zero indexer weights on two nodes every
    score ties at 0 and the selection is the lowest logical indices across
    segment boundaries."""
    w = synth.make_workload("C1", B=2, D=8, lens=[140001, 70000], seed=75, topk=topk)
    if zero_w:
        w.w_idx[0, 3] = 0
        w.w_idx[1, 5] = 0
    nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
    ref = O.run_round(w, nodes)
    r = _device(w)
    stats = _check_stages(w, ref, r, nodes, rerun=_rerun(w, ref))
    _say(f"  segmented top-k k={topk} zero_w={zero_w}: {stats}")
    if zero_w:
        sel = r.host("sel")
        assert np.array_equal(sel[0, 3], np.arange(topk)) and np.array_equal(sel[1, 5], np.arange(topk))


@pytest.mark.parametrize("D", [8, 6, 1])
def test_hca_blocks(D):
    """Every row closes an HCA block inside its tree (committed lengths one to
    D short of a multiple of 128), at every depth of the tree across the rows,
    for a full binary-ish tree (D=8), a ragged one (D=6) and the root alone
    (D=1); the entries match the oracle."""
    lens = [128 * (k + 8) - 1 - (k % D) for k in range(12)]
    w = synth.make_workload("C1", B=len(lens), D=D, lens=lens, seed=80 + D, topk=64, tree="random")
    nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
    ref = O.run_round(w, nodes)
    stats = _check_stages(w, ref, _device(w), nodes, rerun=_rerun(w, ref))
    _say(f"  HCA blocks D={D}: {stats}")


def test_topk_crowded_threshold():
    """Committed indexer keys drawn from three distinct vectors, so each
    node's scores take three values and the top-k threshold falls inside a
    class of hundreds of exactly equal scores, which are taken lowest logical
    index first.  Row 1 is long enough for two top-k segments and the
    merge."""
    w = synth.make_workload("C1", B=2, D=8, lens=[9001, 40003], seed=79, topk=512)
    base = [w.c4_idx[int(w.c4_base[0]) + t].copy() for t in range(3)]
    for b in range(w.B):
        n4 = int(w.lens[b]) // w.dims["ratio_csa"]
        c0 = int(w.c4_base[b])
        for s_ in range(n4):
            w.c4_idx[c0 + s_] = base[s_ % 3]
    nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
    ref = O.run_round(w, nodes)
    r = _device(w)
    stats = _check_stages(w, ref, r, nodes, rerun=_rerun(w, ref))
    # Equal scores are equal in both precisions here (same query, same key),
    # so the selection is exact: score descending, then lower index.
    sel, k = r.host("sel"), w.dims["topk"]
    for (b, i) in nodes:
        sc = ref["detail"][(b, i)]["scores"]
        want = sorted(sorted(sc, key=lambda e: (-sc[e], e))[:k])
        got = sel[b, i][sel[b, i] >= 0].tolist()
        assert got == want, f"row {b} node {i}: tie order differs"
    _say(f"  crowded threshold: {stats}")


@pytest.mark.parametrize("config", ["C1", "C0"])
def test_softmax_restart(config):
    """A committed window key whose logit exceeds the first tile's maximum by
    far more than the fixed reference's slack (for many heads its first-pass
    probability overflows float32): the split must run again from the largest
    logit seen and still match the oracle.  Only key channels that are not
    value channels are scaled (the shared latent's 64 rope channels; the
    8-head shape's whole key), so the outputs keep their usual magnitude."""
    w = synth.make_workload(config, B=2, D=8, lens=[6000, 3001], seed=76, topk=256, tree="random")
    cap, d_k, v_off, d_v = w.dims["ring_cap"], w.dims["d_k"], w.dims["v_off"], w.dims["d_v"]
    key_only = np.ones(d_k, dtype=bool)  # key channels that are not value channels
    key_only[max(v_off, 0):min(v_off + d_v, d_k)] = False
    for b in range(w.B):
        L = int(w.lens[b])
        row = O.bf16_to_f64(w.ring[b, (L - 1) % cap])
        row[:d_k][key_only] *= 200.0 if config == "C1" else 100.0
        w.ring[b, (L - 1) % cap] = O.f64_to_bf16(row)
    nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
    ref = O.run_round(w, nodes)
    r = _device(w)
    stats = _check_stages(w, ref, r, nodes, rerun=_rerun(w, ref))
    _say(f"  restart case: {stats}")


def test_mla_many_units():
    """72 rows of the shared-latent shape (576 node units, more than two per
    compute unit), lengths from a few hundred to a few thousand, and in every
    third row a committed window key whose logits exceed the first tile's
    maxima by far (those units restart from the larger reference)."""
    rng = np.random.default_rng(78)
    lens = rng.integers(300, 3000, size=72).tolist()
    w = synth.make_workload("C1", B=72, D=8, lens=lens, seed=78, topk=128, tree="random")
    cap, d_k, d_v = w.dims["ring_cap"], w.dims["d_k"], w.dims["d_v"]
    for b in range(0, w.B, 3):
        L = int(w.lens[b])
        row = O.bf16_to_f64(w.ring[b, (L - 1) % cap])
        row[d_v:d_k] *= 60.0  # rope channels only: keys, not values
        w.ring[b, (L - 1) % cap] = O.f64_to_bf16(row)
    rows = [0, 1, 3, 35, 69, 70, int(np.argmax(w.lens)), int(np.argmin(w.lens))]
    nodes = [(b, i) for b in sorted(set(rows)) for i in range(w.D)]
    _say(f"[workload] C1 shape B=72 rows={sorted(set(rows))}")
    ref = O.run_round(w, nodes)
    stats = _check_stages(w, ref, _device(w), nodes, rerun=_rerun(w, ref))
    _say(f"  {stats}")


def _small(B=5, D=8, lens=(1003, 2047, 999, 1023, 1500), seed=71, **over):
    return synth.make_workload("C1", B=B, D=D, lens=list(lens), seed=seed, topk=64, **over)


def test_row_errors():
    """A bad parent array, an accepted node outside the tree, a pool too small
    for the path's new entry and a length beyond the bound each fail their own
    row only; the row keeps its cache and its outputs stay unwritten."""
    w = _small()
    assert (int(w.lens[3]) + 1) % 4 == 0  # the root of row 3 closes a CSA block
    w.parents[1, 3] = 5                   # parent after the node
    w.accepted_last[2] = w.D              # outside the tree
    w.c4_cap[3] = int(w.lens[3]) // 4     # no slot for the entry the root closes
    w.lens[4] = w.dims["max_len"] + 1     # beyond the bound
    ref = O.run_round(w)
    assert list(ref["commit"]["status"]) == [O.ROW_OK, O.ROW_BAD_PARENT, O.ROW_BAD_ACCEPT, O.ROW_CAPACITY,
                                             O.ROW_BAD_LEN]
    r = _device(w)
    _check_stages(w, ref, r, rerun=_rerun(w, ref))


def test_row_errors_one_call():
    """The same row errors through the one-call layer step (mask, CSA entries
    and scoring in one launch, HCA entries in the top-k's): every output, the
    cache and the row status equal the separate calls' bit for bit, two
    rounds in a row."""
    w = _small()
    w.parents[1, 3] = 5
    w.accepted_last[2] = w.D
    w.c4_cap[3] = int(w.lens[3]) // 4
    w.lens[4] = w.dims["max_len"] + 1
    ra, rb = _device(w), _device(w)
    keys = ("out", "lse", "sel", "scr_c4", "scr_c128", "anc", "depth", "row_status", "accept_nodes", "accept_len",
            "ring", "c4", "c4_idx", "c128", "len")
    for rnd in range(2):
        ra.round_calls()
        rb.round()
        torch.cuda.synchronize()
        for k in keys:
            assert np.array_equal(ra.host(k).view(np.uint8), rb.host(k).view(np.uint8)), (rnd, k)
    assert list(rb.host("row_status")) == [O.ROW_OK, O.ROW_BAD_PARENT, O.ROW_BAD_ACCEPT, O.ROW_CAPACITY,
                                           O.ROW_BAD_LEN]


def test_deterministic():
    """Two launches on the same inputs give the same bits (fixed reduction orders)."""
    w = _small(seed=72)
    r = _device(w)
    r.mask()
    r.compress()
    r.verify()
    torch.cuda.synchronize()
    first = {k: r.host(k).copy() for k in ("scr_c4", "scr_c128", "out", "lse", "sel")}
    r.verify()
    r.compress()
    r.verify()
    torch.cuda.synchronize()
    for k, v in first.items():
        assert np.array_equal(r.host(k).view(np.uint8), v.view(np.uint8)), k


@pytest.mark.parametrize("over", [dict(H_idx=1), dict(H_idx=64), dict(D=16), dict(D=16, H_idx=4)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_indexer_variants(over):
    """Indexer head counts and tree sizes served by the general scoring kernel."""
    D = over.pop("D", 8)
    w = _small(B=3, D=D, lens=(1003, 4095, 2046), seed=73, **over)
    ref = O.run_round(w)
    r = _device(w)
    _check_stages(w, ref, r, rerun=_rerun(w, ref))


@pytest.mark.parametrize("idx_fmt,page_size", [(0, 0), (1, 0), (1, 128)], ids=["bf16-keys", "fp8-keys",
                                                                                "fp8-keys-paged"])
def test_round_on_own_scratch(idx_fmt, page_size):
    """The whole round on the GPU's own intermediates: verify reads the GPU's
    scratch entries (which may differ from the oracle's in the last bit) and
    commit stores them."""
    w = _small(B=4, lens=(1003, 2047, 1023, 3071), seed=74, idx_fmt=idx_fmt, page_size=page_size)
    ref = O.run_round(w)
    r = _device(w)
    r.round()
    torch.cuda.synchronize()
    d = w.dims
    nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
    g4, g128 = r.host("scr_c4"), r.host("scr_c128")

    def own_ref(b, i):
        return O.verify_node(w, b, i, ref["anc"], ref["depth"], g4, g128)

    def rerun_own(b, i, chosen):
        return O.verify_node(w, b, i, ref["anc"], ref["depth"], g4, g128, chosen=chosen)

    stats = compare_verify(r.host("out"), r.host("lse"), r.host("sel"), ref, nodes, d, own_ref=own_ref,
                           rerun=rerun_own)
    _say(f"  own scratch: {stats}")
    com = ref["commit"]
    assert np.array_equal(r.host("len"), com["lens"])
    assert np.array_equal(r.host("ring"), com["ring"])
    assert np.array_equal(r.host("accept_len"), com["accept_len"])
    assert np.array_equal(r.host("accept_nodes"), com["accept_nodes"])
    # the committed pools are the oracle's commit of the GPU's own scratch, bit for bit
    own = O.commit_accepted_path(w, ref["anc"], ref["depth"], g4, g128, w.accepted_last, ref["status_verify"])
    for name in ("c4", "c4_idx", "c128"):
        assert np.array_equal(r.host(name), own[name]), name
    for name in ("c4", "c128") + (("c4_idx",) if idx_fmt == 0 else ()):
        g, o = r.host(name), com[name]
        diff = np.any(g != o, axis=-1)
        if diff.any():  # only entries the path closed, within the bfloat16 tolerance
            assert_bf16_close(g[diff], O.bf16_to_f64(o[diff]), f"committed {name} entries")


def test_c3_fp8_keys_full_size():
    """The ragged B=64 workload with FP8 (E4M3) indexer keys, in the
    benchmark's length bound: sampled rows, every closing node's entry."""
    w = bench.bench_workload("C3", 20, 5, idx_fmt=1)
    assert w.c4_idx.dtype == np.uint8
    order = np.argsort(w.lens)
    rows = sorted(set(int(b) for b in [order[-1], order[0], 0, 1, 2, 3, 21]))
    nodes = [(b, i) for b in rows for i in range(w.D)]
    _say(f"[workload] C3 FP8 keys rows={rows} lens={[int(w.lens[b]) for b in rows]}")
    ref = O.run_round(w, nodes)
    stats = _check_stages(w, ref, _device(w), nodes, rerun=_rerun(w, ref))
    _say(f"  {stats}")


def test_c3_paged_full_size():
    """The ragged B=64 workload in a paged pool of 128-token pages, in the
    benchmark's length bound: sampled rows, every row's commit."""
    w = bench.bench_workload("C3", 20, 5, page_size=128)
    assert w.page_table is not None
    order = np.argsort(w.lens)
    rows = sorted(set(int(b) for b in [order[-1], order[0], 0, 1, 2, 3, 17]))
    nodes = [(b, i) for b in rows for i in range(w.D)]
    _say(f"[workload] C3 paged rows={rows} lens={[int(w.lens[b]) for b in rows]}")
    ref = O.run_round(w, nodes)
    stats = _check_stages(w, ref, _device(w), nodes, rerun=_rerun(w, ref))
    _say(f"  {stats}")


def test_paged_row_errors():
    """Paged pool: a row whose accepted path runs into a page its table does
    not allocate fails with CAPACITY and keeps its state; a row with a bad
    parent array fails on its own; the others commit."""
    w = synth.make_workload("C1", B=3, D=5, lens=[127, 300, 1023], seed=52, topk=64, page_size=128)
    w.accepted_last[:] = 3  # depth 2: positions L .. L+2
    w.page_table[0, 1] = -1  # row 0: positions 128, 129 have no page
    w.parents[1, 2] = 4
    ref = O.run_round(w)
    assert list(ref["commit"]["status"]) == [O.ROW_CAPACITY, O.ROW_BAD_PARENT, O.ROW_OK]
    _check_stages(w, ref, _device(w), rerun=_rerun(w, ref))


def test_c3_alt_shape_full_size():
    """The alternative reading of "shapes as config 1" on the ragged B=64
    workload: 8 query heads over one 128-wide key and value head, top-k 512,
    in the benchmark's length bound."""
    w = bench.bench_workload("C3", 20, 5, shape="mha128")
    order = np.argsort(w.lens)
    rows = sorted(set(int(b) for b in [order[-1], order[0], 0, 1, 2, 33]))
    nodes = [(b, i) for b in rows for i in range(w.D)]
    _say(f"[workload] C3 alt shape H={w.dims['H']} rows={rows} lens={[int(w.lens[b]) for b in rows]}")
    ref = O.run_round(w, nodes)
    stats = _check_stages(w, ref, _device(w), nodes, rerun=_rerun(w, ref))
    _say(f"  {stats}")


def test_nullable_outputs():
    """sel and lse may be NULL (the selection then lives in the workspace) and
    next_token may be NULL: the outputs that are given equal, bit for bit,
    those of a call with every output given, and the buffers not passed stay
    untouched."""
    w = _small(seed=77)
    full, bare = _device(w), _device(w)
    for r in (full, bare):
        r.mask()
        r.compress()
    full.verify()
    bare.verify(with_sel=False, with_lse=False)
    torch.cuda.synchronize()
    assert np.array_equal(bare.host("out"), full.host("out"))
    assert np.all(bare.host("sel") == -2) and np.all(np.isnan(bare.host("lse")))
    ref = O.run_round(w)
    nodes = [(b, i) for b in range(w.B) for i in range(w.D)]
    compare_verify(full.host("out"), full.host("lse"), full.host("sel"), ref, nodes, w.dims, rerun=_rerun(w, ref))
    sel = synth.make_selection(w, vocab=5000)
    tgt, acc, nxt = O.select_accepted_path(w.parents, sel.draft_tokens, sel.target_logits, ref["status_verify"])
    for r in (full, bare):
        r.attach_selection(sel)
    full.select()
    bare.select(with_next=False)
    torch.cuda.synchronize()
    for r in (full, bare):
        assert np.array_equal(r.host("target_tokens"), tgt) and np.array_equal(r.host("accepted_last"), acc)
    assert np.array_equal(full.host("next_token"), nxt)
    assert np.all(bare.host("next_token") == -2)
