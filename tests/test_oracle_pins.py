"""Pins of the CPU oracle to facts that do not come from the oracle itself.

Each test checks the oracle against a definition written out by brute force,
a closed form, a library routine, a hand-derived fixture, an invariant, or the
independent linear replay.
"""
import os

import numpy as np
import pytest
import torch

import synth
from oracle import replay as R
from oracle import tv_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# bfloat16 rounding
# --------------------------------------------------------------------------
def test_bf16_roundtrip_all_finite_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = O.bf16_to_f64(bits)
    fin = np.isfinite(vals)
    back = O.f64_to_bf16(vals[fin])
    # +0 and -0 both stay themselves; every finite pattern maps back to itself
    assert np.array_equal(back, bits[fin])


def test_bf16_matches_torch_on_float32_values():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(200000) * s for s in (1e-30, 1e-3, 1.0, 1e3, 1e30)])
    x = x.astype(np.float32)  # torch rounds float32 -> bfloat16 once, to nearest even
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.f64_to_bf16(x.astype(np.float64)), ref)


def test_bf16_two_independent_roundings_agree():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(500000) * np.exp(rng.uniform(-40, 40, 500000))
    assert np.array_equal(O.f64_to_bf16(x), R._to_bf16(x))


def test_bf16_hand_cases():
    # bfloat16 spacing just above 1.0 is 2**-7.
    cases = {
        1.0 + 2 ** -8: 0x3F80,                 # exact tie, even neighbour is 1.0
        1.0 + 3 * 2 ** -8: 0x3F82,             # exact tie, even neighbour is 1 + 2**-6
        1.0 + 2 ** -8 + 2 ** -30: 0x3F81,      # just above the tie: one rounding gives 1 + 2**-7
        -(1.0 + 2 ** -8 + 2 ** -30): 0xBF81,
        2.0 ** -133: 0x0001,                   # smallest subnormal
        0.0: 0x0000,
        (2 - 2 ** -7) * 2.0 ** 127: 0x7F7F,     # largest finite bfloat16
        (2 - 2 ** -8) * 2.0 ** 127: 0x7F80,     # tie between it and 2**128: rounds to inf (even)
    }
    for x, want in cases.items():
        assert int(O.f64_to_bf16(np.array([x]))[0]) == want, x


# --------------------------------------------------------------------------
# FP8 E4M3 (indexer keys, FP8 reading)
# --------------------------------------------------------------------------
def test_e4m3_decode_matches_torch_on_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = O.e4m3_to_f64(codes)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan) and list(codes[nan]) == [0x7F, 0xFF]
    assert np.array_equal(got[~nan], ref[~nan]) and np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_e4m3_roundtrip_every_finite_code():
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], dtype=np.uint8)
    assert np.array_equal(O.f64_to_e4m3(O.e4m3_to_f64(codes)), codes)


def test_e4m3_matches_torch_within_range():
    # torch rounds float32 -> e4m3fn once, to nearest even; inside +-464 it agrees
    # with the saturating reading (beyond, torch gives NaN and the reading +-448)
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(100000) * s for s in (1e-3, 0.03, 1.0, 30.0)])
    x = np.clip(x, -464.0, 464.0).astype(np.float32)
    mids = O.e4m3_to_f64(np.arange(0, 0x7E, dtype=np.uint8))
    x = np.concatenate([x, ((mids[:-1] + mids[1:]) / 2).astype(np.float32)])  # every exact midpoint
    x = np.concatenate([x, -x])
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(O.f64_to_e4m3(x.astype(np.float64)), ref)


def test_e4m3_two_independent_roundings_agree():
    rng = np.random.default_rng(6)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-9, 7, 20000))
    mids = O.e4m3_to_f64(np.arange(0, 0x7E, dtype=np.uint8))
    x = np.concatenate([x, (mids[:-1] + mids[1:]) / 2, [1e4, -1e4, 448.0, 464.0, 465.0]])
    assert np.array_equal(O.f64_to_e4m3(x), R._to_e4m3(x))


def test_e4m3_hand_cases():
    # E4M3 spacing just above 1.0 is 2**-3; subnormals are multiples of 2**-9.
    cases = [
        (1.0, 0x38),
        (1.0 + 2 ** -4, 0x38),                   # exact tie, even neighbour is 1.0
        (1.0 + 3 * 2 ** -4, 0x3A),               # exact tie, even neighbour is 1.25
        (1.0 + 2 ** -4 + 2 ** -20, 0x39),        # just above the tie
        (-(1.0 + 2 ** -4 + 2 ** -20), 0xB9),
        (448.0, 0x7E),                            # largest finite
        (464.0, 0x7E),                            # tie between 448 and 480 (not finite): even is 448
        (1e6, 0x7E), (-1e6, 0xFE),                # saturation
        (2.0 ** -9, 0x01),                        # smallest subnormal
        (2.0 ** -10, 0x00),                       # tie between 0 and 2**-9: even is 0
        (3 * 2.0 ** -10, 0x02),                   # tie between 1 and 2 subnormal units: even is 2
        (7.5 * 2.0 ** -9, 0x08),                  # tie between the largest subnormal and 2**-6: even is 2**-6
        (0.0, 0x00), (-0.0, 0x80),
    ]
    for x, want in cases:
        assert int(O.f64_to_e4m3(np.array([x]))[0]) == want, x


def test_fp8_compressed_key_is_the_e4m3_rounding_of_the_pooled_key():
    """With FP8 indexer keys a CSA scratch entry keeps its latent channels as
    bfloat16 and its indexer channels as E4M3 values (held in bfloat16): the
    compression of a block differs from the bfloat16 reading only there."""
    w8 = synth.make_workload("C0", lens=2047, idx_fmt=1)
    w16 = synth.make_workload("C0", lens=2047)
    d_row = w8.dims["d_row"]
    assert w8.c4_idx.dtype == np.uint8
    for w in (w8, w16):
        w.c4_idx[:] = 0  # committed keys do not enter the compression; align the two workloads
    r8, r16 = O.run_round(w8), O.run_round(w16)
    assert r8["w4"].any()
    a, b = r8["scr_c4"][r8["w4"]], r16["scr_c4"][r16["w4"]]
    assert np.array_equal(a[:, :d_row], b[:, :d_row])
    ka, kb = O.bf16_to_f64(a[:, d_row:]), O.bf16_to_f64(b[:, d_row:])
    assert np.array_equal(O.round_e4m3(ka), ka)  # E4M3 values
    # both are one rounding of the same pooled value: to E4M3 (spacing 2**(E-3) for |v| in [2**E, 2**(E+1)),
    # at least 2**-9) and to bfloat16 (spacing 2**(E-7))
    E = np.floor(np.log2(np.maximum(np.abs(kb), 2.0 ** -6)))
    assert np.all(np.abs(ka - kb) <= np.maximum(2.0 ** (E - 4), 2.0 ** -10) + 2.0 ** (E - 8))
    assert np.any(ka != kb)


# --------------------------------------------------------------------------
# verification plan
# --------------------------------------------------------------------------
def _read_plans():
    out = []
    with open(os.path.join(GOLDEN, "tree_plans.txt")) as f:
        lines = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    for i in range(0, len(lines), 3):
        par = [int(x) for x in lines[i][3:]]
        anc = [int(x) for x in lines[i + 1][1:]]
        dep = [int(x) for x in lines[i + 2][1:]]
        out.append((lines[i][1], par, anc, dep))
    return out


@pytest.mark.parametrize("name,par,anc,dep", _read_plans())
def test_tree_plan_golden(name, par, anc, dep):
    a, d, st = O.build_tree_mask(np.array([par]))
    assert st[0] == O.ROW_OK
    assert [int(x) for x in a[0]] == anc
    assert [int(x) for x in d[0]] == dep


def _random_parents(rng, B, D):
    p = np.zeros((B, D), dtype=np.int32)
    p[:, 0] = -1
    for i in range(1, D):
        p[:, i] = rng.integers(0, i, size=B)
    return p


@pytest.mark.parametrize("D", [1, 2, 5, 8, 33, 64])
def test_tree_mask_brute_force_walk(D):
    rng = np.random.default_rng(D)
    par = _random_parents(rng, 16, D)
    anc, depth, st = O.build_tree_mask(par)
    assert np.all(st == 0)
    for b in range(16):
        for i in range(D):
            walk, j = 0, i
            steps = -1
            while j >= 0:
                walk |= 1 << j
                j = int(par[b, j])
                steps += 1
            assert int(anc[b, i]) == walk
            assert depth[b, i] == steps
            assert bin(int(anc[b, i])).count("1") == depth[b, i] + 1
            assert int(anc[b, i]) & 1 and (int(anc[b, i]) >> i) & 1


def test_tree_mask_chain_is_lower_triangular():
    D = 64
    anc, depth, st = O.build_tree_mask(np.arange(-1, D - 1)[None, :])
    assert [int(x) for x in anc[0]] == [(1 << (i + 1)) - 1 for i in range(D)]
    assert list(depth[0]) == list(range(D))


@pytest.mark.parametrize("bad", [[0, 0, 1], [-1, 1, 0], [-1, 0, 2], [-1, -1, 0], [-1, 0, 5], [3, 0, 1]])
def test_tree_mask_rejects_bad_parents(bad):
    par = np.array([[-1, 0, 1], bad])
    anc, depth, st = O.build_tree_mask(par)
    assert list(st) == [O.ROW_OK, O.ROW_BAD_PARENT]
    assert np.all(anc[1] == 0) and np.all(depth[1] == 0)


# --------------------------------------------------------------------------
# compression special cases
# --------------------------------------------------------------------------
def test_compress_zero_gate_is_block_mean():
    rng = np.random.default_rng(3)
    toks = rng.standard_normal((128, 640))
    np.testing.assert_allclose(O.compress_block(toks, np.zeros(640)), toks.mean(axis=0), rtol=0, atol=1e-14)


def test_compress_dominant_gate_returns_that_token():
    rng = np.random.default_rng(4)
    toks = rng.standard_normal((4, 320))
    gate = np.zeros(320)
    gate[7] = 1.0
    toks[:, 7] = [0.0, 0.0, 900.0, 0.0]  # token 2's gate logit dominates by e^900
    np.testing.assert_array_equal(O.compress_block(toks, gate), toks[2])


def test_compress_invariant_to_block_permutation():
    rng = np.random.default_rng(5)
    toks = rng.standard_normal((128, 640))
    gate = rng.standard_normal(640) * 0.02
    perm = rng.permutation(128)
    np.testing.assert_allclose(O.compress_block(toks[perm], gate), O.compress_block(toks, gate), atol=1e-13)


def test_compress_two_tokens_closed_form():
    # Two tokens: weights are the logistic of the logit difference.
    t = np.array([[1.0, 2.0, 3.0], [-1.0, 0.5, 4.0]])
    g = np.array([0.3, -0.2, 0.1])
    z0, z1 = t[0] @ g, t[1] @ g
    w0 = 1.0 / (1.0 + np.exp(z1 - z0))
    np.testing.assert_allclose(O.compress_block(t, g), w0 * t[0] + (1 - w0) * t[1], atol=1e-15)


# --------------------------------------------------------------------------
# indexer scoring and top-k
# --------------------------------------------------------------------------
def test_indexer_scores_one_hot_keys_closed_form():
    # Key s = unit vector e_s, so q_h . k_s = q_h[s] and the score is sum_h w_h max(0, q_h[s]).
    rng = np.random.default_rng(6)
    q = rng.standard_normal((8, 64))
    w = rng.standard_normal(8)
    S = O.indexer_scores(np.eye(64), q, w)
    for s in range(64):
        assert S[s] == pytest.approx(sum(w[h] * max(0.0, q[h, s]) for h in range(8)), abs=1e-12)


def test_topk_against_stable_library_sort_with_exact_ties():
    # Zero keys score exactly 0 for every node; with only 40 nonzero keys the
    # k = 64 boundary falls inside the block of ties, which the lower logical
    # index must win.  Duplicated nonzero keys add ties away from the boundary.
    rng = np.random.default_rng(7)
    w = synth.make_workload("C0", lens=2048)
    n4 = 512
    keys = w.c4_idx[:n4].copy()
    live = np.sort(rng.choice(n4, size=40, replace=False))
    dead = np.setdiff1d(np.arange(n4), live)
    keys[dead] = 0
    keys[live[20:]] = keys[live[:20]]
    w.c4_idx[:n4] = keys
    anc, depth, st = O.build_tree_mask(w.parents)
    scr4 = np.zeros((1, 5, 320), np.uint16)
    scr128 = np.zeros((1, 5, 256), np.uint16)
    for i in range(5):
        r = O.verify_node(w, 0, i, anc, depth, scr4, scr128)
        S = O.indexer_scores(O.bf16_to_f64(keys), O.bf16_to_f64(w.q_idx[0, i]), O.bf16_to_f64(w.w_idx[0, i]))
        ref = np.sort(np.argsort(-S, kind="stable")[:64])
        assert np.sum(S > 0) < 64 < np.sum(S >= 0)  # the boundary sits in the zero ties
        assert list(r["sel"]) == list(ref)


def test_topk_takes_everything_when_candidates_fit():
    w = synth.make_workload("C0", lens=99)
    res = O.run_round(w)
    for i in range(5):
        assert len(res["detail"][(0, i)]["sel"]) == 25
        assert list(res["sel"][0, i, :25]) == list(range(25))
        assert np.all(res["sel"][0, i, 25:] == -1)


def _read_counts():
    cases = []
    with open(os.path.join(GOLDEN, "key_counts.txt")) as f:
        lines = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    for i in range(0, len(lines), 6):
        L = int(lines[i][2])
        vals = {ln[0]: [int(x) for x in ln[1:]] for ln in lines[i + 1:i + 6]}
        cases.append((L, vals))
    return cases


@pytest.mark.parametrize("L,vals", _read_counts())
def test_key_counts_golden(L, vals):
    w = synth.make_workload("C0", lens=L)
    res = O.run_round(w)
    for i in range(5):
        det = res["detail"][(0, i)]
        assert len(det["scores"]) == vals["cand4"][i]
        assert len(det["sel"]) == vals["sel"][i]
        assert det["n_keys"] == vals["keys"][i]
        assert vals["keys"][i] == vals["sel"][i] + vals["hca"][i] + vals["win"][i]


# --------------------------------------------------------------------------
# attention arithmetic against a library routine
# --------------------------------------------------------------------------
@pytest.mark.parametrize("shape", ["mha128", "mla"])
def test_attention_matches_torch_sdpa(shape, monkeypatch):
    w = synth.make_workload("C0", lens=700, shape=shape, topk=32, seed=11)
    anc, depth, st = O.build_tree_mask(w.parents)
    scr4, scr128, *_ = O.branch_compress(w, anc, depth, st)
    captured = {}
    real_stack = np.stack

    def spy(arrs, *a, **k):  # capture the gathered key rows of the node
        r = real_stack(arrs, *a, **k)
        if r.ndim == 2 and r.shape[1] == w.dims["d_row"]:
            captured["R"] = r
        return r

    d = w.dims
    for i in range(5):
        monkeypatch.setattr(O.np, "stack", spy)
        r = O.verify_node(w, 0, i, anc, depth, scr4, scr128)
        monkeypatch.setattr(O.np, "stack", real_stack)
        Rw = torch.from_numpy(captured["R"])
        Q = torch.from_numpy(O.bf16_to_f64(w.q[0, i]))
        K = Rw[:, :d["d_k"]]
        V = Rw[:, d["v_off"]:d["v_off"] + d["d_v"]]
        sc = float(np.float32(d["scale"]))
        ref = torch.nn.functional.scaled_dot_product_attention(Q[None], K[None], V[None], scale=sc)[0]
        np.testing.assert_allclose(r["out"], ref.numpy(), atol=1e-12)
        lse_ref = torch.logsumexp(sc * Q @ K.T, dim=1).numpy()
        np.testing.assert_allclose(r["lse"], lse_ref, atol=1e-12)


def test_attention_zero_query_is_mean_of_values():
    w = synth.make_workload("C0", lens=300, seed=12)
    w.q[:] = 0
    res = O.run_round(w)
    for i in range(5):
        det = res["detail"][(0, i)]
        # uniform softmax: lse is log of the key count
        np.testing.assert_allclose(det["lse"], np.log(det["n_keys"]), atol=1e-12)


# --------------------------------------------------------------------------
# the whole method against the linear replay
# --------------------------------------------------------------------------
REPLAY_CASES = [
    dict(name="C0", lens=2048),
    dict(name="C0", lens=2045),
    dict(name="C0", lens=2046),
    dict(name="C0", lens=2047),
    dict(name="C0", lens=5, seed=31),
    dict(name="C0", lens=0, seed=32),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 382, 383], seed=33, topk=16),
    dict(name="C0", B=2, D=8, chain=True, lens=[253, 254], seed=34, topk=16),
    dict(name="C0", B=2, D=12, tree="random", lens=[126, 1023], seed=35, topk=8, window=16, ring_cap=128),
    dict(name="C1", B=2, D=6, lens=[509, 510], seed=36, topk=24),
    dict(name="C0", B=2, D=6, tree="random", lens=[391, 127], seed=37, topk=12, scale=8.0 / np.sqrt(128)),
    # FP8 indexer keys
    dict(name="C0", lens=2047, idx_fmt=1),
    dict(name="C0", B=3, D=8, tree="random", lens=[381, 382, 383], seed=38, topk=16, idx_fmt=1),
    dict(name="C1", B=2, D=6, lens=[509, 510], seed=39, topk=24, idx_fmt=1),
]


def _mk(case):
    c = dict(case)
    return synth.make_workload(c.pop("name"), **c)


@pytest.mark.parametrize("case", REPLAY_CASES)
def test_tree_oracle_equals_linear_replay(case):
    w = _mk(case)
    res = O.run_round(w)
    for b in range(w.B):
        rp = R.replay_row(w, b)
        for (path, node), (out, lse, chosen) in rp.items():
            det = res["detail"][(b, node)]
            assert list(det["sel"]) == list(chosen)
            np.testing.assert_allclose(det["out"], out, atol=1e-10, rtol=0)
            np.testing.assert_allclose(det["lse"], lse, atol=1e-10, rtol=0)


@pytest.mark.parametrize("case", REPLAY_CASES)
def test_commit_equals_linear_replay_state(case):
    w = _mk(case)
    res = O.run_round(w)
    com = res["commit"]
    d = w.dims
    for b in range(w.B):
        st, path = R.replay_commit(w, b, w.accepted_last[b])
        assert com["lens"][b] == st.L
        assert com["accept_len"][b] == len(path)
        assert list(com["accept_nodes"][b, :len(path)]) == path
        cap = d["ring_cap"]
        for q in range(max(0, st.L - cap), st.L):
            assert np.array_equal(com["ring"][b, q % cap], st.raw[q])
        n4, n128 = st.L // d["ratio_csa"], st.L // d["ratio_hca"]
        b4, b128 = w.c4_base[b], w.c128_base[b]
        for s in range(n4):
            assert np.array_equal(com["c4"][b4 + s], st.csa[s][0])
            assert np.array_equal(com["c4_idx"][b4 + s], st.csa[s][1])
        for s in range(n128):
            assert np.array_equal(com["c128"][b128 + s], st.hca[s])
        # nothing past the new entries was written
        assert np.all(com["c4"][b4 + n4:b4 + w.c4_cap[b]] == synth.inputs.BF16_NAN)
        idx_nan = synth.inputs.E4M3_NAN if d["idx_fmt"] == 1 else synth.inputs.BF16_NAN
        assert np.all(com["c4_idx"][b4 + n4:b4 + w.c4_cap[b]] == idx_nan)
        assert np.all(com["c128"][b128 + n128:b128 + w.c128_cap[b]] == synth.inputs.BF16_NAN)


# --------------------------------------------------------------------------
# branch isolation (Sec. 3.1, Sec. 3.2)
# --------------------------------------------------------------------------
def test_other_branches_do_not_change_a_node():
    w = synth.make_workload("C0", B=1, D=8, tree="random", lens=[1023], seed=41, topk=16)
    base = O.run_round(w)
    anc = base["anc"]
    for i in range(8):
        others = [j for j in range(8) if not (int(anc[0, i]) >> j) & 1]
        if not others:
            continue
        w2 = synth.make_workload("C0", B=1, D=8, tree="random", lens=[1023], seed=41, topk=16)
        for j in others:
            w2.tree_u[0, j] ^= np.uint16(0x0040)
            w2.q[0, j] ^= np.uint16(0x0040)
            w2.q_idx[0, j] ^= np.uint16(0x0040)
        r2 = O.run_round(w2)
        assert np.array_equal(r2["out"][0, i], base["out"][0, i])
        assert np.array_equal(r2["sel"][0, i], base["sel"][0, i])


def test_rejected_nodes_leave_no_trace_in_commit():
    w = synth.make_workload("C0", B=1, D=8, tree="random", lens=[1019], seed=42, topk=16)
    base = O.run_round(w)["commit"]
    anc, depth, _ = O.build_tree_mask(w.parents)
    acc = int(w.accepted_last[0])
    rejected = [j for j in range(8) if not (int(anc[0, acc]) >> j) & 1]
    assert rejected
    for j in rejected:
        w.tree_u[0, j] ^= np.uint16(0x0100)
    com = O.run_round(w)["commit"]
    for k in ("ring", "c4", "c4_idx", "c128", "lens", "accept_nodes", "accept_len"):
        assert np.array_equal(com[k], base[k]), k


def test_chain_tree_equals_linear_verification():
    # top-k = 1 drafting gives a chain (Sec. 5.1): node i is token i of one linear sequence.
    w = synth.make_workload("C0", B=1, D=8, chain=True, lens=[509], seed=43, topk=16)
    res = O.run_round(w)
    st = R.LinearState(w, 0)
    for i in range(8):
        st.append(w.tree_u[0, i])
        out, lse, chosen = st.attend(w.q[0, i], w.q_idx[0, i], w.w_idx[0, i])
        np.testing.assert_allclose(res["out"][0, i], out, atol=1e-10)
        assert list(res["detail"][(0, i)]["sel"]) == chosen


# --------------------------------------------------------------------------
# row status handling
# --------------------------------------------------------------------------
def test_row_errors_skip_rows():
    w = synth.make_workload("C0", B=4, D=5, lens=[300, 301, 302, 303], seed=50)
    w.parents[1, 3] = 3            # BAD_PARENT
    w.accepted_last[2] = 5         # BAD_ACCEPT (D = 5)
    w.c4_cap[3] = 300 // 4         # no room for any new CSA entry
    w.dims["max_len"] = 1000
    res = O.run_round(w)
    st = res["commit"]["status"]
    assert st[1] == O.ROW_BAD_PARENT
    assert st[2] == O.ROW_BAD_ACCEPT
    anc, depth, _ = O.build_tree_mask(w.parents)
    acc = int(w.accepted_last[3])
    closes = any((303 + int(depth[3, j]) + 1) % 4 == 0 for j in range(5) if (int(anc[3, acc]) >> j) & 1)
    assert st[3] == (O.ROW_CAPACITY if closes else O.ROW_OK)
    assert res["commit"]["lens"][1] == 301 and res["commit"]["lens"][2] == 302
    assert np.all(np.isnan(res["out"][1]))


def test_len_beyond_bound_is_flagged():
    w = synth.make_workload("C0", B=2, D=5, lens=[300, 301], seed=51)
    w.dims["max_len"] = 300
    res = O.run_round(w)
    assert list(res["status_verify"]) == [O.ROW_OK, O.ROW_BAD_LEN]


def test_given_selection_replaces_only_the_csa_rows():
    """A given selection reproduces the node exactly when it is the top-k
    itself; swapping one chosen entry for an unchosen one changes exactly one
    attended CSA row (the committed entry's row), checked against SDPA over
    the explicitly gathered keys."""
    w = synth.make_workload("C0", lens=1500, topk=32, seed=12)
    anc, depth, st = O.build_tree_mask(w.parents)
    scr4, scr128, *_ = O.branch_compress(w, anc, depth, st)
    d = w.dims
    base = O.verify_node(w, 0, 3, anc, depth, scr4, scr128)
    same = O.verify_node(w, 0, 3, anc, depth, scr4, scr128, chosen=base["sel"])
    assert np.array_equal(same["out"], base["out"]) and np.array_equal(same["sel"], base["sel"])
    unchosen = sorted(set(base["scores"]) - set(base["sel"].tolist()))
    swapped = np.sort(np.concatenate([base["sel"][1:], [unchosen[0]]]))
    alt = O.verify_node(w, 0, 3, anc, depth, scr4, scr128, chosen=swapped)
    assert np.array_equal(alt["sel"], swapped) and alt["n_keys"] == base["n_keys"]
    assert not np.allclose(alt["out"], base["out"])
    # brute force on the swapped set: committed CSA rows of the set, every HCA
    # entry, the window (committed ring rows and the root path's draft rows)
    n4 = int(w.lens[0]) // d["ratio_csa"]
    assert all(s < n4 for s in swapped)  # node 3 closes no block at this length
    rows = [O.bf16_to_f64(w.c4[w.c4_base[0] + s]) for s in swapped]
    rows += [O.bf16_to_f64(w.c128[w.c128_base[0] + s]) for s in range(int(w.lens[0]) // d["ratio_hca"])]
    path = O.node_path(anc[0], depth[0], 3)
    L, p = int(w.lens[0]), int(w.lens[0]) + int(depth[0, 3])
    for qpos in range(max(0, p - d["window"] + 1), p + 1):
        src = w.ring[0, qpos % d["ring_cap"]] if qpos < L else w.tree_u[0, path[qpos - L]]
        rows.append(O.bf16_to_f64(src[:d["d_row"]]))
    R = torch.from_numpy(np.stack(rows))
    Q = torch.from_numpy(O.bf16_to_f64(w.q[0, 3]))
    sc = float(np.float32(d["scale"]))
    ref = torch.nn.functional.scaled_dot_product_attention(
        Q[None], R[None, :, :d["d_k"]], R[None, :, d["v_off"]:d["v_off"] + d["d_v"]], scale=sc)[0]
    np.testing.assert_allclose(alt["out"], ref.numpy(), atol=1e-12)
