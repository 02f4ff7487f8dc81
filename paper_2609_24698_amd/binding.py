"""ctypes binding of ``libtv.so``: the C ABI of ``include/tv.h`` with torch tensors.

Argument marshalling only.  Every step runs in the library's HIP kernels; there
is no Python or CPU fallback, and loading fails loudly when the library has
not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libtv.so")

TV_OK, TV_ERR_INVALID_ARG, TV_ERR_UNSUPPORTED, TV_ERR_WORKSPACE, TV_ERR_LAUNCH, TV_ERR_DEVICE = range(6)
ROW_OK, ROW_BAD_PARENT, ROW_BAD_ACCEPT, ROW_CAPACITY, ROW_BAD_LEN = range(5)

EXPORTED = (
    "tv_build_tree_mask", "tv_branch_compress", "tv_verify_workspace_bytes", "tv_verify_attention",
    "tv_verify_attention_noalloc", "tv_verify_round",
    "tv_commit_accepted_path", "tv_select_workspace_bytes", "tv_select_accepted_path", "tv_round_graph_create", "tv_round_graph_kernels",
    "tv_round_graph_launch", "tv_round_graph_destroy", "tv_status_string", "tv_profile_enable", "tv_profile_disable", "tv_profile_read",
)


class TvError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where}: {status_string(code)} ({code})")
        self.code = code


class TvDims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "B", "D", "H", "d_row", "d_k", "v_off", "d_v", "d_idx", "H_idx", "ratio_csa", "ratio_hca", "window",
        "topk", "ring_cap", "max_len")] + [("scale", ctypes.c_float)] + [(n, ctypes.c_int32) for n in (
            "idx_fmt", "page_size", "page_stride")]


class TvCache(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "ring", "c4", "c4_idx", "c128", "c4_base", "c4_cap", "c128_base", "c128_cap", "len", "page_table")]


class TvLayer(ctypes.Structure):
    _fields_ = [("cache", TvCache)] + [(n, ctypes.c_void_p) for n in (
        "tree_u", "gate_w", "q", "q_idx", "w_idx", "scr_c4", "scr_c128", "out", "lse", "sel", "workspace")] + [
        ("workspace_bytes", ctypes.c_size_t)]


class TvRound(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "parents", "anc", "depth", "row_status", "accepted_last", "accept_nodes", "accept_len", "primary_last",
        "draft_tokens", "target_logits")] + [("vocab", ctypes.c_int32)] + [(n, ctypes.c_void_p) for n in (
            "target_tokens", "next_token", "select_workspace")] + [("select_workspace_bytes", ctypes.c_size_t)]


class TvKernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2609_24698_amd._build.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        dp = ctypes.POINTER(TvDims)
        cp = ctypes.POINTER(TvCache)
        L.tv_build_tree_mask.argtypes = [dp, vp, vp, vp, vp, vp]
        L.tv_branch_compress.argtypes = [dp, cp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.tv_verify_workspace_bytes.argtypes = [dp]
        L.tv_verify_workspace_bytes.restype = sz
        L.tv_verify_attention.argtypes = [dp, cp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.tv_verify_attention_noalloc.argtypes = [dp, cp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.tv_commit_accepted_path.argtypes = [dp, cp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.tv_select_workspace_bytes.argtypes = [dp, i32]
        L.tv_select_workspace_bytes.restype = sz
        L.tv_select_accepted_path.argtypes = [dp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, sz, vp]
        L.tv_verify_round.argtypes = [dp, ctypes.POINTER(TvRound), ctypes.POINTER(TvLayer), vp]
        L.tv_round_graph_create.argtypes = [dp, ctypes.POINTER(TvRound), ctypes.POINTER(TvLayer), i32,
                                            ctypes.POINTER(vp)]
        L.tv_round_graph_kernels.argtypes = [vp]
        L.tv_round_graph_kernels.restype = i32
        L.tv_round_graph_launch.argtypes = [vp, vp]
        L.tv_round_graph_destroy.argtypes = [vp]
        L.tv_status_string.argtypes = [ctypes.c_int]
        L.tv_status_string.restype = ctypes.c_char_p
        L.tv_profile_enable.argtypes = [i32]
        L.tv_profile_read.argtypes = [ctypes.POINTER(TvKernelTime), i32, ctypes.POINTER(i32)]
        for name in ("tv_build_tree_mask", "tv_branch_compress", "tv_verify_attention", "tv_verify_attention_noalloc",
                     "tv_verify_round", "tv_commit_accepted_path",
                     "tv_select_accepted_path", "tv_round_graph_create", "tv_round_graph_launch",
                     "tv_round_graph_destroy", "tv_profile_enable", "tv_profile_disable", "tv_profile_read"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().tv_status_string(int(code)).decode()


def _check(code: int, where: str) -> None:
    if code != TV_OK:
        raise TvError(code, where)


def make_dims(d: dict) -> TvDims:
    d = dict(d)
    for k in ("idx_fmt", "page_size", "page_stride"):
        d.setdefault(k, 0)
    return TvDims(**{f: (float(d[f]) if f == "scale" else int(d[f])) for f, _ in TvDims._fields_})


def _ptr(t: Optional[torch.Tensor], dtype=None) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"expected {dtype}, got {t.dtype}")
    return t.data_ptr()


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _stream(stream) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def make_cache(ring, c4, c4_idx, c128, c4_base, c4_cap, c128_base, c128_cap, lens, page_table=None) -> TvCache:
    """Cache struct over device tensors (bf16/int16 pools, int64 bases, int32 caps and lengths; an int32
    page table for a paged pool)."""
    return TvCache(_ptr(ring), _ptr(c4), _ptr(c4_idx), _ptr(c128), _ptr(c4_base, torch.int64),
                   _ptr(c4_cap, torch.int32), _ptr(c128_base, torch.int64), _ptr(c128_cap, torch.int32),
                   _ptr(lens, torch.int32), _ptr(page_table, torch.int32))


def tv_build_tree_mask(dims: TvDims, parents, anc, depth, row_status, stream=None) -> None:
    _check(lib().tv_build_tree_mask(ctypes.byref(dims), _ptr(parents, torch.int32), _ptr(anc, torch.int64),
                                    _ptr(depth, torch.int32), _ptr(row_status, torch.int32), _stream(stream)),
           "tv_build_tree_mask")


def tv_branch_compress(dims: TvDims, cache: TvCache, tree_u, anc, depth, gate_w, scr_c4, scr_c128, row_status,
                       primary_last=None, stream=None) -> None:
    _check(lib().tv_branch_compress(ctypes.byref(dims), ctypes.byref(cache), _ptr(tree_u), _ptr(anc, torch.int64),
                                    _ptr(depth, torch.int32), _ptr(gate_w), _ptr(scr_c4), _ptr(scr_c128),
                                    _ptr(row_status, torch.int32), _ptr(primary_last, torch.int32),
                                    _stream(stream)),
           "tv_branch_compress")


def tv_verify_workspace_bytes(dims: TvDims) -> int:
    return int(lib().tv_verify_workspace_bytes(ctypes.byref(dims)))


def tv_verify_attention(dims: TvDims, cache: TvCache, tree_u, anc, depth, scr_c4, scr_c128, q, q_idx, w_idx, out,
                        lse, sel, row_status, workspace, stream=None) -> None:
    _check(lib().tv_verify_attention(ctypes.byref(dims), ctypes.byref(cache), _ptr(tree_u), _ptr(anc, torch.int64),
                                     _ptr(depth, torch.int32), _ptr(scr_c4), _ptr(scr_c128), _ptr(q), _ptr(q_idx),
                                     _ptr(w_idx), _ptr(out), _ptr(lse, torch.float32), _ptr(sel, torch.int32),
                                     _ptr(row_status, torch.int32), _ptr(workspace), workspace.numel() *
                                     workspace.element_size(), _stream(stream)),
           "tv_verify_attention")


NOALLOC_SCRATCH_BYTES = 64 << 20  # TV_NOALLOC_SCRATCH_BYTES


def tv_verify_attention_noalloc(dims: TvDims, cache: TvCache, tree_u, anc, depth, scr_c4, scr_c128, q, q_idx,
                                w_idx, out, lse, sel, row_status, stream=None) -> None:
    _check(lib().tv_verify_attention_noalloc(ctypes.byref(dims), ctypes.byref(cache), _ptr(tree_u),
                                             _ptr(anc, torch.int64), _ptr(depth, torch.int32), _ptr(scr_c4),
                                             _ptr(scr_c128), _ptr(q), _ptr(q_idx), _ptr(w_idx), _ptr(out),
                                             _ptr(lse, torch.float32), _ptr(sel, torch.int32),
                                             _ptr(row_status, torch.int32), _stream(stream)),
           "tv_verify_attention_noalloc")


def tv_commit_accepted_path(dims: TvDims, cache: TvCache, tree_u, anc, depth, scr_c4, scr_c128, accepted_last,
                            accept_nodes, accept_len, row_status, primary_last=None, stream=None) -> None:
    _check(lib().tv_commit_accepted_path(ctypes.byref(dims), ctypes.byref(cache), _ptr(tree_u),
                                         _ptr(anc, torch.int64), _ptr(depth, torch.int32), _ptr(scr_c4),
                                         _ptr(scr_c128), _ptr(accepted_last, torch.int32),
                                         _ptr(accept_nodes, torch.int32), _ptr(accept_len, torch.int32),
                                         _ptr(row_status, torch.int32), _ptr(primary_last, torch.int32),
                                         _stream(stream)),
           "tv_commit_accepted_path")


def tv_select_workspace_bytes(dims: TvDims, vocab: int) -> int:
    return int(lib().tv_select_workspace_bytes(ctypes.byref(dims), int(vocab)))


def tv_select_accepted_path(dims: TvDims, parents, anc, depth, draft_tokens, target_logits, vocab: int,
                            target_tokens, accepted_last, next_token, row_status, workspace, stream=None) -> None:
    _check(lib().tv_select_accepted_path(ctypes.byref(dims), _ptr(parents, torch.int32), _ptr(anc, torch.int64),
                                         _ptr(depth, torch.int32), _ptr(draft_tokens, torch.int32),
                                         _ptr(target_logits), int(vocab), _ptr(target_tokens, torch.int32),
                                         _ptr(accepted_last, torch.int32), _ptr(next_token, torch.int32),
                                         _ptr(row_status, torch.int32), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)),
           "tv_select_accepted_path")


def tv_profile_enable(capacity: int) -> None:
    _check(lib().tv_profile_enable(int(capacity)), "tv_profile_enable")


def tv_profile_disable() -> None:
    _check(lib().tv_profile_disable(), "tv_profile_disable")


def tv_profile_read(max_entries: int = 32) -> dict:
    arr = (TvKernelTime * max_entries)()
    n = ctypes.c_int32(0)
    _check(lib().tv_profile_read(arr, max_entries, ctypes.byref(n)), "tv_profile_read")
    return {arr[k].name.decode(): (int(arr[k].launches), float(arr[k].total_ms)) for k in range(n.value)}


# ---------------------------------------------------------------------------
# Device-resident round state: uploads host arrays and owns every buffer the
# four calls read or write.
# ---------------------------------------------------------------------------
def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device)
    if a.dtype == np.uint64:
        return torch.from_numpy(a.view(np.int64)).to(device)
    return torch.from_numpy(a).to(device)


def layer_struct(cache: TvCache, t) -> TvLayer:
    """The TvLayer of one layer's buffers (``t``: DeviceRound.t)."""
    return TvLayer(cache, _ptr(t["tree_u"]), _ptr(t["gate_w"]), _ptr(t["q"]), _ptr(t["q_idx"]), _ptr(t["w_idx"]),
                   _ptr(t["scr_c4"]), _ptr(t["scr_c128"]), _ptr(t["out"]), _ptr(t["lse"]), _ptr(t["sel"]),
                   _ptr(t["workspace"]), _nbytes(t["workspace"]))


def round_struct(t, parents, vocab: int = 0) -> TvRound:
    """The TvRound of the shared tree buffers ``t`` (a DeviceRound.t), with
    the selection buffers when ``t`` holds target logits."""
    sel = "target_logits" in t
    return TvRound(_ptr(parents), _ptr(t["anc"]), _ptr(t["depth"]), _ptr(t["row_status"]),
                   _ptr(t["accepted_last"]), _ptr(t["accept_nodes"]), _ptr(t["accept_len"]),
                   _ptr(t.get("primary_last"), torch.int32),
                   _ptr(t["draft_tokens"]) if sel else None, _ptr(t["target_logits"]) if sel else None,
                   vocab if sel else 0, _ptr(t["target_tokens"]) if sel else None,
                   _ptr(t["next_token"]) if sel else None, _ptr(t["select_ws"]) if sel else None,
                   _nbytes(t["select_ws"]) if sel else 0)


class DeviceRound:
    """Device buffers of one verify round built from host arrays.

    ``src`` needs the attributes dims, lens, parents, accepted_last, ring, c4,
    c4_idx, c128, c4_base, c4_cap, c128_base, c128_cap, tree_u, q, q_idx,
    w_idx, gate_w (numpy, bfloat16 data as uint16).
    """

    def __init__(self, src, device="cuda:0", poison_outputs: bool = True):
        dev = torch.device(device)
        d = dict(src.dims)
        self.host_dims = d
        self.dims = make_dims(d)
        B, D, H = d["B"], d["D"], d["H"]
        d_u = d["d_row"] + d["d_idx"]
        T = {}
        for k in ("parents", "accepted_last", "ring", "c4", "c4_idx", "c128", "c4_base", "c4_cap", "c128_base",
                  "c128_cap", "tree_u", "q", "q_idx", "w_idx", "gate_w"):
            T[k] = _dev(getattr(src, k), dev)
        T["len"] = _dev(src.lens.astype(np.int32), dev)
        pt = getattr(src, "page_table", None)
        T["page_table"] = _dev(pt.astype(np.int32), dev) if pt is not None else None
        fill = -1 if poison_outputs else 0  # 0xFFFF bf16 is NaN: unwritten outputs show up
        T["anc"] = torch.full((B, D), fill, dtype=torch.int64, device=dev)
        T["depth"] = torch.full((B, D), fill, dtype=torch.int32, device=dev)
        T["row_status"] = torch.full((B,), fill, dtype=torch.int32, device=dev)
        T["scr_c4"] = torch.full((B, D, d_u), fill, dtype=torch.int16, device=dev)
        T["scr_c128"] = torch.full((B, D, d["d_row"]), fill, dtype=torch.int16, device=dev)
        T["out"] = torch.full((B, D, H, d["d_v"]), fill, dtype=torch.int16, device=dev)
        T["lse"] = torch.full((B, D, H), float("nan"), dtype=torch.float32, device=dev)
        T["sel"] = torch.full((B, D, d["topk"]), -2, dtype=torch.int32, device=dev)
        T["accept_nodes"] = torch.full((B, D), -2, dtype=torch.int32, device=dev)
        T["accept_len"] = torch.full((B,), -2, dtype=torch.int32, device=dev)
        ws = tv_verify_workspace_bytes(self.dims)
        if ws == 0:
            raise TvError(TV_ERR_INVALID_ARG, "tv_verify_workspace_bytes")
        T["workspace"] = torch.empty(ws, dtype=torch.uint8, device=dev)
        self.t = T
        self.cache = make_cache(T["ring"], T["c4"], T["c4_idx"], T["c128"], T["c4_base"], T["c4_cap"],
                                T["c128_base"], T["c128_cap"], T["len"], T["page_table"])

    def mask(self, stream=None):
        t = self.t
        tv_build_tree_mask(self.dims, t["parents"], t["anc"], t["depth"], t["row_status"], stream)

    def set_primary(self, primary_last):
        """Designate a chain per row (the refresh schedule of compress and
        commit); None goes back to the plain refresh."""
        if primary_last is None:
            self.t.pop("primary_last", None)
        else:
            self.t["primary_last"] = _dev(np.asarray(primary_last, dtype=np.int32), self.t["parents"].device)

    def compress(self, stream=None):
        t = self.t
        tv_branch_compress(self.dims, self.cache, t["tree_u"], t["anc"], t["depth"], t["gate_w"], t["scr_c4"],
                           t["scr_c128"], t["row_status"], t.get("primary_last"), stream)

    def verify(self, stream=None, with_sel: bool = True, with_lse: bool = True):
        t = self.t
        tv_verify_attention(self.dims, self.cache, t["tree_u"], t["anc"], t["depth"], t["scr_c4"], t["scr_c128"],
                            t["q"], t["q_idx"], t["w_idx"], t["out"], t["lse"] if with_lse else None,
                            t["sel"] if with_sel else None, t["row_status"], t["workspace"], stream)

    def verify_noalloc(self, stream=None, with_sel: bool = True, with_lse: bool = True):
        """verify() through the entry point that takes no workspace."""
        t = self.t
        tv_verify_attention_noalloc(self.dims, self.cache, t["tree_u"], t["anc"], t["depth"], t["scr_c4"],
                                    t["scr_c128"], t["q"], t["q_idx"], t["w_idx"], t["out"],
                                    t["lse"] if with_lse else None, t["sel"] if with_sel else None,
                                    t["row_status"], stream)

    def verify_round(self, stream=None, with_mask: bool = True):
        """mask + compress + verify in one library call (tv_verify_round),
        bit-identical to the three calls with fewer launches.
        ``with_mask=False`` reuses the masks already in anc/depth."""
        t = self.t
        rnd = round_struct(t, t["parents"] if with_mask else None, getattr(self, "vocab", 0))
        layer = layer_struct(self.cache, t)
        _check(lib().tv_verify_round(ctypes.byref(self.dims), ctypes.byref(rnd), ctypes.byref(layer),
                                     _stream(stream)), "tv_verify_round")

    def commit(self, stream=None):
        t = self.t
        tv_commit_accepted_path(self.dims, self.cache, t["tree_u"], t["anc"], t["depth"], t["scr_c4"],
                                t["scr_c128"], t["accepted_last"], t["accept_nodes"], t["accept_len"],
                                t["row_status"], t.get("primary_last"), stream)

    def attach_selection(self, sel, fill: int = -2):
        """Upload the draft tokens and target logits of ``sel`` (a synth
        Selection) and allocate the selection outputs and workspace."""
        t, d = self.t, self.host_dims
        dev = t["parents"].device
        self.vocab = int(sel.vocab)
        t["draft_tokens"] = _dev(sel.draft_tokens.astype(np.int32), dev)
        t["target_logits"] = _dev(sel.target_logits, dev)
        t["target_tokens"] = torch.full((d["B"], d["D"]), fill, dtype=torch.int32, device=dev)
        t["next_token"] = torch.full((d["B"],), fill, dtype=torch.int32, device=dev)
        ws = tv_select_workspace_bytes(self.dims, self.vocab)
        if ws == 0:
            raise TvError(TV_ERR_INVALID_ARG, "tv_select_workspace_bytes")
        t["select_ws"] = torch.empty(ws, dtype=torch.uint8, device=dev)

    def select(self, stream=None, with_next: bool = True):
        """Greedy selection; writes accepted_last, which commit then reads."""
        t = self.t
        tv_select_accepted_path(self.dims, t["parents"], t["anc"], t["depth"], t["draft_tokens"],
                                t["target_logits"], self.vocab, t["target_tokens"], t["accepted_last"],
                                t["next_token"] if with_next else None, t["row_status"], t["select_ws"], stream)

    def round(self, stream=None):
        """One step: mask, compression and verification in one call, then
        selection (when attached) and commit."""
        self.verify_round(stream)
        if "target_logits" in self.t:
            self.select(stream)
        self.commit(stream)

    def round_calls(self, stream=None):
        """round() issued one library call per stage, all on ``stream``."""
        self.mask(stream)
        self.compress(stream)
        self.verify(stream)
        if "target_logits" in self.t:
            self.select(stream)
        self.commit(stream)

    def host(self, name: str) -> np.ndarray:
        x = self.t[name].cpu().numpy()
        if x.dtype == np.int16:
            return x.view(np.uint16)
        if name == "anc":
            return x.view(np.uint64)
        return x


# ---------------------------------------------------------------------------
# A round over several layers: shared tree buffers, per-layer state.
# ---------------------------------------------------------------------------
class LayeredRound:
    """One verify round over several layers that share a draft tree.

    ``layers`` are DeviceRound objects (one per layer, each with its own
    cache, tokens, queries, outputs and workspace); the tree buffers (parents,
    masks, depths, row status, accepted path) and, when layer 0 has a
    selection attached, the selection buffers are layer 0's.  ``eager()``
    issues the calls one by one; ``capture()`` records the same sequence into
    a HIP graph that ``replay()`` launches.
    """

    def __init__(self, layers):
        self.layers = list(layers)
        self.dims = self.layers[0].dims
        self.graph = None

    def _shared(self):
        return self.layers[0].t

    def eager(self, stream=None, fused: bool = True):
        """The round call by call.  ``fused``: per layer one tv_verify_round
        (the mask with layer 0), as the graph records it; otherwise mask,
        compress and verify as separate calls on one stream."""
        t0 = self._shared()
        if fused:
            for k, r in enumerate(self.layers):
                rnd = round_struct(t0, t0["parents"] if k == 0 else None)
                layer = layer_struct(r.cache, r.t)
                _check(lib().tv_verify_round(ctypes.byref(self.dims), ctypes.byref(rnd), ctypes.byref(layer),
                                             _stream(stream)), "tv_verify_round")
        else:
            self._calls(stream)
        self._finish(stream)

    def _calls(self, stream):
        t0 = self._shared()
        tv_build_tree_mask(self.dims, t0["parents"], t0["anc"], t0["depth"], t0["row_status"], stream)
        for r in self.layers:
            t = r.t
            tv_branch_compress(self.dims, r.cache, t["tree_u"], t0["anc"], t0["depth"], t["gate_w"], t["scr_c4"],
                               t["scr_c128"], t0["row_status"], t0.get("primary_last"), stream)
            tv_verify_attention(self.dims, r.cache, t["tree_u"], t0["anc"], t0["depth"], t["scr_c4"], t["scr_c128"],
                                t["q"], t["q_idx"], t["w_idx"], t["out"], t["lse"], t["sel"], t0["row_status"],
                                t["workspace"], stream)

    def _finish(self, stream):
        t0 = self._shared()
        L0 = self.layers[0]
        if "target_logits" in t0:
            tv_select_accepted_path(self.dims, t0["parents"], t0["anc"], t0["depth"], t0["draft_tokens"],
                                    t0["target_logits"], L0.vocab, t0["target_tokens"], t0["accepted_last"],
                                    t0["next_token"], t0["row_status"], t0["select_ws"], stream)
        for r in self.layers:
            t = r.t
            tv_commit_accepted_path(self.dims, r.cache, t["tree_u"], t0["anc"], t0["depth"], t["scr_c4"],
                                    t["scr_c128"], t0["accepted_last"], t0["accept_nodes"], t0["accept_len"],
                                    t0["row_status"], t0.get("primary_last"), stream)

    def capture(self) -> int:
        """Record the round into a graph; returns the number of kernels in it."""
        t0 = self._shared()
        layers = (TvLayer * len(self.layers))()
        for k, r in enumerate(self.layers):
            layers[k] = layer_struct(r.cache, r.t)
        rnd = round_struct(t0, t0["parents"], getattr(self.layers[0], "vocab", 0))
        self._keep = (layers, rnd)
        h = ctypes.c_void_p()
        _check(lib().tv_round_graph_create(ctypes.byref(self.dims), ctypes.byref(rnd), layers, len(self.layers),
                                           ctypes.byref(h)), "tv_round_graph_create")
        self.release()
        self.graph = h
        return int(lib().tv_round_graph_kernels(h))

    def replay(self, stream=None):
        if self.graph is None:
            raise RuntimeError("capture() first")
        _check(lib().tv_round_graph_launch(self.graph, _stream(stream)), "tv_round_graph_launch")

    def release(self):
        if self.graph is not None:
            _check(lib().tv_round_graph_destroy(self.graph), "tv_round_graph_destroy")
            self.graph = None

    def __del__(self):
        try:
            self.release()
        except Exception:
            pass
