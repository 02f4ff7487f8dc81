"""GPU parity: every call of the C ABI against the CPU oracle on the same seeded inputs.

Stage by stage: the mask and depth must be bit-exact; scratch entries within
the bfloat16 tolerance; verify is run on the oracle's scratch bytes (so both
sides see identical inputs) and compared node by node; commit is run on the
same scratch and must reproduce the oracle's cache bit for bit.  A final pass
runs the whole round on the GPU's own intermediates.
"""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import tv_oracle as O

from .parity import assert_bf16_close, assert_e4m3_codes, compare_verify

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _round(case):
    from paper_2609_24698_amd import DeviceRound

    c = dict(case)
    name = c.pop("name")
    nodes = c.pop("nodes", None)
    w = synth.make_workload(name, **c)
    _say(f"[parity] {name} {c} B={w.B} D={w.D} lens[:4]={w.lens[:4].tolist()}")
    ref = O.run_round(w, nodes)
    r = DeviceRound(w, "cuda:0")
    return w, ref, r


def _rerun(w, ref):
    """The oracle's result for a node on a given selection (for nodes where
    several selections are correct)."""
    def f(b, i, chosen):
        return O.verify_node(w, b, i, ref["anc"], ref["depth"], ref["scr_c4"], ref["scr_c128"], chosen=chosen)
    return f


def _check_stages(w, ref, r, nodes=None, rerun=None):
    d = w.dims
    B, D = w.B, w.D
    # verify preprocess
    r.mask()
    torch.cuda.synchronize()
    assert np.array_equal(r.host("anc"), ref["anc"])
    assert np.array_equal(r.host("depth"), ref["depth"])
    st_mask = O.build_tree_mask(w.parents)[2]
    assert np.array_equal(r.host("row_status"), st_mask)
    # per-branch compression
    r.compress()
    torch.cuda.synchronize()
    g4, g128 = r.host("scr_c4"), r.host("scr_c128")
    w4, w128 = ref["w4"], ref["w128"]
    if w4.any():
        if d.get("idx_fmt", 0) == O.IDX_E4M3:  # latent channels bfloat16, indexer channels E4M3 codes
            d_row = d["d_row"]
            assert_bf16_close(g4[w4][:, :d_row], O.bf16_to_f64(ref["scr_c4"][w4][:, :d_row]), "scratch CSA entries")
            pooled = np.stack([ref["pooled"][(b, i, 0)][d_row:] for b, i in zip(*np.nonzero(w4))])
            near = assert_e4m3_codes(g4[w4][:, d_row:], pooled, "scratch CSA indexer keys")
            _say(f"  FP8 keys: {int(w4.sum())} entries, {near} near-midpoint codes")
        else:
            assert_bf16_close(g4[w4], O.bf16_to_f64(ref["scr_c4"][w4]), "scratch CSA entries")
    if w128.any():
        assert_bf16_close(g128[w128], O.bf16_to_f64(ref["scr_c128"][w128]), "scratch HCA entries")
    assert np.all(g4[~w4] == 0xFFFF) and np.all(g128[~w128] == 0xFFFF), "scratch slot written that closes nothing"
    # verify on the oracle's scratch bytes
    r.t["scr_c4"].copy_(torch.from_numpy(ref["scr_c4"].view(np.int16)))
    r.t["scr_c128"].copy_(torch.from_numpy(ref["scr_c128"].view(np.int16)))
    r.verify()
    torch.cuda.synchronize()
    assert np.array_equal(r.host("row_status"), ref["status_verify"])
    ok_nodes = [(b, i) for b in range(B) for i in range(D) if ref["status_verify"][b] == 0]
    if nodes is not None:
        ok_nodes = [n for n in nodes if n in ref["detail"]]
    stats = compare_verify(r.host("out"), r.host("lse"), r.host("sel"), ref, ok_nodes, d,
                           rerun=rerun if rerun is not None else _rerun(w, ref))
    _say(f"  verify {stats}")
    bad_rows = [b for b in range(B) if ref["status_verify"][b] != 0]
    for b in bad_rows:  # skipped rows keep their poisoned outputs
        assert np.all(r.host("out")[b] == 0xFFFF)
    # commit on the same scratch
    r.commit()
    torch.cuda.synchronize()
    com = ref["commit"]
    assert np.array_equal(r.host("row_status"), com["status"])
    assert np.array_equal(r.host("len"), com["lens"])
    assert np.array_equal(r.host("ring"), com["ring"])
    assert np.array_equal(r.host("c4"), com["c4"])
    assert np.array_equal(r.host("c4_idx"), com["c4_idx"])
    assert np.array_equal(r.host("c128"), com["c128"])
    okc = com["status"] == 0
    assert np.array_equal(r.host("accept_len")[okc], com["accept_len"][okc])
    assert np.array_equal(r.host("accept_nodes")[okc], com["accept_nodes"][okc])
    assert np.all(r.host("accept_len")[~okc] == -2)
    return stats


SMALL_CASES = [
    dict(name="C0"),
    dict(name="C0", lens=2045),
    dict(name="C0", lens=2046),
    dict(name="C0", lens=2047),
    dict(name="C0", lens=99),
    dict(name="C0", lens=5),
    dict(name="C0", lens=0),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 3967, 1023], seed=33, topk=16),
    dict(name="C0", B=2, D=8, chain=True, lens=[253, 4094], seed=34),
    dict(name="C0", B=2, D=1, tree=[-1], lens=[511, 512], seed=35),
    dict(name="C0", B=2, D=64, tree="random", lens=[1150, 3001], seed=36),
    dict(name="C0", B=2, D=6, tree="random", lens=[391, 2303], seed=37, scale=8.0 / np.sqrt(128)),
    dict(name="C1", B=2, D=8, lens=[1000, 3001], seed=40, topk=64),
    dict(name="C1", B=2, D=8, lens=[127, 639], seed=41, topk=512),
    dict(name="C1", B=1, D=8, chain=True, lens=[5119], seed=42, topk=128, scale=8.0 / 24.0),
    # compression blocks of 512 and 256 tokens (more rows than the compression kernel's 1024 threads cover in
    # one pass of its gate-logit loop, 128 tokens) with a larger ring
    dict(name="C0", B=2, D=8, tree="random", lens=[1535, 4090], seed=38, ratio_csa=16, ratio_hca=512, ring_cap=512),
    dict(name="C1", B=2, D=8, lens=[1791, 3327], seed=43, topk=64, ratio_hca=256, ring_cap=256),
    # FP8 (E4M3) indexer keys, both scoring kernels (8 indexer heads and D <= 8; the general one)
    dict(name="C0", lens=2047, idx_fmt=1),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 3967, 1023], seed=44, topk=16, idx_fmt=1),
    dict(name="C1", B=2, D=8, lens=[1000, 3001], seed=45, topk=64, idx_fmt=1),
    dict(name="C1", B=2, D=12, tree="random", lens=[2043, 5119], seed=46, topk=128, H_idx=4, idx_fmt=1),
    # the paged three-layer pool (raw rows, CSA and HCA entries through one page table per row)
    dict(name="C0", lens=2047, page_size=128),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 3967, 1023], seed=49, topk=16, page_size=256),
    dict(name="C1", B=2, D=8, lens=[1000, 3007], seed=50, topk=64, page_size=128),
    dict(name="C1", B=2, D=12, tree="random", lens=[2043, 5119], seed=51, topk=128, H_idx=4, idx_fmt=1,
         page_size=128),
]


@pytest.mark.parametrize("case", SMALL_CASES, ids=lambda c: "-".join(f"{k}{v}" for k, v in c.items() if k != "name")
                         or "base")
def test_stages_small(case):
    w, ref, r = _round(case)
    _check_stages(w, ref, r)


def test_c1_full():
    w, ref, r = _round(dict(name="C1"))
    _check_stages(w, ref, r)
