"""ctypes binding of the C ABI in include/ml2.h (argument marshalling only).

Every call goes straight to ``libml2.so``; all arithmetic runs in its HIP
kernels.  Device buffers are torch tensors (``tensor.data_ptr()``) or raw
integer device addresses; the stream defaults to torch's current stream.
The library must have been built (``python -m paper_2411_10764_amd.build``):
there is no fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libml2.so")

ML2_OK = 0
ML2_ERR_INVALID_ARG = 1
ML2_ERR_UNSUPPORTED = 2
ML2_ERR_OUT_OF_MEMORY = 3
ML2_ERR_HIP = 4
ML2_MAX_DEPTH = 32
ML2_MAX_TREE_NODES = 3062
ML2_MAX_FEATURES = 256
ML2_MAX_TOPK = 16384
ML2_MAX_STREAM_K = 4096

EXPORTED = (
    "ml2_load_ensemble", "ml2_free_ensemble", "ml2_ensemble_num_features",
    "ml2_ensemble_num_trees", "ml2_ensemble_depth", "ml2_score_validity",
    "ml2_score_perf", "ml2_score", "ml2_score_single_pass", "ml2_topk_workspace_bytes", "ml2_filter_topk", "ml2_filter_topk_noalloc",
    "ml2_rerank",
    "ml2_rerank_workspace_bytes",
    "ml2_explorer_create", "ml2_explorer_free", "ml2_explorer_reset", "ml2_explorer_rounds",
    "ml2_explorer_round", "ml2_stream_explorer_create", "ml2_stream_explorer_free",
    "ml2_stream_explorer_reset", "ml2_stream_explorer_rounds", "ml2_stream_explorer_begin",
    "ml2_stream_explorer_chunk", "ml2_stream_explorer_end", "ml2_last_error",
)
# include/ml2_probe.h: microbenchmarks behind the roofline figures
EXPORTED_PROBE = ("ml2_probe_visit", "ml2_probe_lds", "ml2_probe_valu", "ml2_tune_walk_plan",
                  "ml2_tune_layout")


class Ml2Error(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"ml2 status {status}: {message}")
        self.status = status


class ml2_ensemble_desc(ctypes.Structure):
    _fields_ = [
        ("num_trees", ctypes.c_int32),
        ("num_features", ctypes.c_int32),
        ("base_score", ctypes.c_float),
        ("tree_node_offset", ctypes.c_void_p),
        ("left_child", ctypes.c_void_p),
        ("right_child", ctypes.c_void_p),
        ("split_feature", ctypes.c_void_p),
        ("split_threshold", ctypes.c_void_p),
        ("leaf_value", ctypes.c_void_p),
        ("default_left", ctypes.c_void_p),
    ]


_lib = None


def lib():
    """The loaded libml2.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2411_10764_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.ml2_load_ensemble.restype = I32
        L.ml2_load_ensemble.argtypes = [P, ctypes.POINTER(P)]
        L.ml2_free_ensemble.restype = None
        L.ml2_free_ensemble.argtypes = [P]
        for f in ("ml2_ensemble_num_features", "ml2_ensemble_num_trees", "ml2_ensemble_depth"):
            getattr(L, f).restype = I32
            getattr(L, f).argtypes = [P]
        L.ml2_score_validity.restype = I32
        L.ml2_score_validity.argtypes = [P, P, I64, I64, P, P, P]
        L.ml2_score_perf.restype = I32
        L.ml2_score_perf.argtypes = [P, P, I64, I64, P, P, P]
        L.ml2_score.restype = I32
        L.ml2_score.argtypes = [P, P, P, I64, I64, P, P, P, P]
        L.ml2_score_single_pass.restype = I32
        L.ml2_score_single_pass.argtypes = [P, P, P, I64, I64]
        L.ml2_topk_workspace_bytes.restype = I32
        L.ml2_topk_workspace_bytes.argtypes = [I64, I32, ctypes.POINTER(SZ)]
        L.ml2_filter_topk.restype = I32
        L.ml2_filter_topk.argtypes = [P, P, I64, I32, P, P, P, P, SZ, P]
        L.ml2_filter_topk_noalloc.restype = I32
        L.ml2_filter_topk_noalloc.argtypes = [P, P, I64, I32, P, P, P, P]
        L.ml2_rerank.restype = I32
        L.ml2_rerank.argtypes = [P, P, I64, I64, P, I32, I32, P, P, P, P, P, SZ, P]
        L.ml2_rerank_workspace_bytes.restype = I32
        L.ml2_rerank_workspace_bytes.argtypes = [P, I32, ctypes.POINTER(SZ)]
        L.ml2_explorer_create.restype = I32
        L.ml2_explorer_create.argtypes = [P, P, P, I64, I32, I32, I32, ctypes.POINTER(P)]
        L.ml2_explorer_free.restype = None
        L.ml2_explorer_free.argtypes = [P]
        L.ml2_explorer_reset.restype = I32
        L.ml2_explorer_reset.argtypes = [P]
        L.ml2_explorer_rounds.restype = I32
        L.ml2_explorer_rounds.argtypes = [P]
        L.ml2_explorer_round.restype = I32
        L.ml2_explorer_round.argtypes = [P, P, I64, I32, P, P, P, P]
        L.ml2_stream_explorer_create.restype = I32
        L.ml2_stream_explorer_create.argtypes = [P, P, P, I64, I32, I32, I32, ctypes.POINTER(P)]
        L.ml2_stream_explorer_free.restype = None
        L.ml2_stream_explorer_free.argtypes = [P]
        L.ml2_stream_explorer_reset.restype = I32
        L.ml2_stream_explorer_reset.argtypes = [P]
        L.ml2_stream_explorer_rounds.restype = I32
        L.ml2_stream_explorer_rounds.argtypes = [P]
        L.ml2_stream_explorer_begin.restype = I32
        L.ml2_stream_explorer_begin.argtypes = [P, P]
        L.ml2_stream_explorer_chunk.restype = I32
        L.ml2_stream_explorer_chunk.argtypes = [P, P, I64, I64, I64, P]
        L.ml2_stream_explorer_end.restype = I32
        L.ml2_stream_explorer_end.argtypes = [P, P, P, P, P]
        L.ml2_last_error.restype = ctypes.c_char_p
        L.ml2_last_error.argtypes = []
        D = ctypes.POINTER(ctypes.c_double)
        L.ml2_probe_visit.restype = I32
        L.ml2_probe_visit.argtypes = [I32, I32, I32, I32, I32, I32, I32, D, D]
        L.ml2_probe_lds.restype = I32
        L.ml2_probe_lds.argtypes = [I32, I32, I32, D, D]
        L.ml2_probe_valu.restype = I32
        L.ml2_probe_valu.argtypes = [I32, I32, D, D]
        L.ml2_tune_walk_plan.restype = I32
        L.ml2_tune_walk_plan.argtypes = [I32, I32, I32, I32, I32]
        L.ml2_tune_layout.restype = I32
        L.ml2_tune_layout.argtypes = [I32]
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != ML2_OK:
        msg = lib().ml2_last_error()
        raise Ml2Error(status, msg.decode() if msg else "")


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _rows(X):
    """(pointer, n, ld) of a 2-D row-major float32 device tensor."""
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be a 2-D tensor with unit column stride")
    return X.data_ptr(), X.shape[0], X.stride(0)


class Ensemble:
    """An ensemble loaded on the current device (owns the library handle)."""

    def __init__(self, handle: int):
        self.handle = handle

    @property
    def num_features(self) -> int:
        return lib().ml2_ensemble_num_features(self.handle)

    @property
    def num_trees(self) -> int:
        return lib().ml2_ensemble_num_trees(self.handle)

    @property
    def depth(self) -> int:
        return lib().ml2_ensemble_depth(self.handle)

    def free(self) -> None:
        if self.handle:
            lib().ml2_free_ensemble(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - interpreter shutdown order
        try:
            self.free()
        except Exception:
            pass


def make_desc(ens):
    """(descriptor, keep-alive arrays) from a gen.Ensemble-like object."""
    arrays = (
        np.ascontiguousarray(ens.offsets, np.int64),
        np.ascontiguousarray(ens.left, np.int32),
        np.ascontiguousarray(ens.right, np.int32),
        np.ascontiguousarray(ens.feature, np.int32),
        np.ascontiguousarray(ens.threshold, np.float32),
        np.ascontiguousarray(ens.value, np.float32),
    )
    dl = getattr(ens, "default_left", None)
    if dl is not None:
        dl = np.ascontiguousarray(dl, np.uint8)
        arrays = arrays + (dl,)
    off, left, right, feat, thr, val = arrays[:6]
    d = ml2_ensemble_desc(int(off.shape[0] - 1), int(ens.num_features), float(ens.base_score),
                          off.ctypes.data, left.ctypes.data, right.ctypes.data,
                          feat.ctypes.data, thr.ctypes.data, val.ctypes.data,
                          None if dl is None else dl.ctypes.data)
    return d, arrays


def ml2_load_ensemble(ens) -> Ensemble:
    """Load a gen.Ensemble-like tree ensemble (or an ml2_ensemble_desc)."""
    if isinstance(ens, ml2_ensemble_desc):
        d, keep = ens, None
    else:
        d, keep = make_desc(ens)
    h = ctypes.c_void_p()
    _check(lib().ml2_load_ensemble(ctypes.byref(d), ctypes.byref(h)))
    del keep
    return Ensemble(h.value)


def ml2_free_ensemble(e: Ensemble) -> None:
    e.free()


def ml2_score_validity(v: Ensemble, X, valid_out, margin_out=None, stream=None) -> None:
    xp, n, ld = _rows(X)
    _check(lib().ml2_score_validity(v.handle, xp, n, ld, _ptr(valid_out), _ptr(margin_out),
                                    _stream(stream)))


def ml2_score_perf(p: Ensemble, X, valid, score_out, stream=None) -> None:
    xp, n, ld = _rows(X)
    _check(lib().ml2_score_perf(p.handle, xp, n, ld, _ptr(valid), _ptr(score_out),
                                _stream(stream)))


def ml2_score(v: Ensemble, p: Ensemble, X, valid_out, margin_out, score_out,
              stream=None) -> None:
    """Validity and performance in one call (one pass over the pool where
    the ensembles allow it)."""
    xp, n, ld = _rows(X)
    _check(lib().ml2_score(v.handle, p.handle, xp, n, ld, _ptr(valid_out), _ptr(margin_out),
                           _ptr(score_out), _stream(stream)))


def ml2_score_single_pass(v: Ensemble, p: Ensemble, X) -> bool:
    xp, n, ld = _rows(X)
    return bool(lib().ml2_score_single_pass(v.handle, p.handle, xp, n, ld))


def ml2_topk_workspace_bytes(n: int, k: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().ml2_topk_workspace_bytes(n, k, ctypes.byref(out)))
    return int(out.value)


def ml2_filter_topk(valid, scores, k: int, topk_idx, topk_score, num_selected, workspace,
                    workspace_bytes: int | None = None, n: int | None = None,
                    stream=None) -> None:
    if n is None:
        n = scores.shape[0]
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    _check(lib().ml2_filter_topk(_ptr(valid), _ptr(scores), n, k, _ptr(topk_idx),
                                 _ptr(topk_score), _ptr(num_selected), _ptr(workspace),
                                 workspace_bytes, _stream(stream)))


def ml2_filter_topk_noalloc(valid, scores, k: int, topk_idx, topk_score, num_selected,
                            n: int | None = None, stream=None) -> None:
    """ml2_filter_topk with the library's static workspace (allocates nothing)."""
    if n is None:
        n = scores.shape[0]
    _check(lib().ml2_filter_topk_noalloc(_ptr(valid), _ptr(scores), n, k, _ptr(topk_idx),
                                         _ptr(topk_score), _ptr(num_selected), _stream(stream)))


def ml2_rerank_workspace_bytes(a: Ensemble, m: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().ml2_rerank_workspace_bytes(a.handle, m, ctypes.byref(out)))
    return int(out.value)


def ml2_rerank(a: Ensemble, X, rows, keep: int, row_scores, out_idx, out_score, num_selected,
               workspace, workspace_bytes: int | None = None, m: int | None = None,
               stream=None) -> None:
    xp, n, ld = _rows(X)
    if m is None:
        m = rows.shape[0]
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    _check(lib().ml2_rerank(a.handle, xp, n, ld, _ptr(rows), m, keep, _ptr(row_scores),
                            _ptr(out_idx), _ptr(out_score), _ptr(num_selected), _ptr(workspace),
                            workspace_bytes, _stream(stream)))


class Explorer:
    """An ml2_explorer over one pool of n candidates (owns the handle; holds
    references to its ensembles so they outlive it)."""

    def __init__(self, v: Ensemble, p: Ensemble, a: Ensemble | None, n: int, k: int,
                 keep: int, max_rounds: int):
        h = ctypes.c_void_p()
        _check(lib().ml2_explorer_create(v.handle, p.handle, a.handle if a else None, n, k, keep,
                                         max_rounds, ctypes.byref(h)))
        self.handle = h.value
        self.models = (v, p, a)
        self.n, self.k, self.keep = n, k, keep

    @property
    def rounds(self) -> int:
        return lib().ml2_explorer_rounds(self.handle)

    def reset(self) -> None:
        _check(lib().ml2_explorer_reset(self.handle))

    def round(self, X, out_idx, out_score, num_selected, rescore: bool = True,
              stream=None) -> None:
        xp, n, ld = _rows(X)
        if n != self.n:
            raise ValueError(f"pool has {n} rows, the explorer was made for {self.n}")
        _check(lib().ml2_explorer_round(self.handle, xp, ld, 1 if rescore else 0, _ptr(out_idx),
                                        _ptr(out_score), _ptr(num_selected), _stream(stream)))

    def free(self) -> None:
        if self.handle:
            lib().ml2_explorer_free(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - interpreter shutdown order
        try:
            self.free()
        except Exception:
            pass


class StreamExplorer:
    """An ml2_stream_explorer: the explorer's rounds over a pool that arrives
    in chunks of rows (owns the handle; holds references to its ensembles)."""

    def __init__(self, v: Ensemble, p: Ensemble, a: Ensemble | None, max_chunk_rows: int,
                 k: int, keep: int, max_rounds: int):
        h = ctypes.c_void_p()
        _check(lib().ml2_stream_explorer_create(v.handle, p.handle, a.handle if a else None,
                                                max_chunk_rows, k, keep, max_rounds,
                                                ctypes.byref(h)))
        self.handle = h.value
        self.models = (v, p, a)
        self.k, self.keep = k, keep

    @property
    def rounds(self) -> int:
        return lib().ml2_stream_explorer_rounds(self.handle)

    def reset(self) -> None:
        _check(lib().ml2_stream_explorer_reset(self.handle))

    def begin(self, stream=None) -> None:
        _check(lib().ml2_stream_explorer_begin(self.handle, _stream(stream)))

    def chunk(self, X, row0: int, stream=None) -> None:
        xp, m, ld = _rows(X)
        _check(lib().ml2_stream_explorer_chunk(self.handle, xp, m, ld, row0, _stream(stream)))

    def end(self, out_idx, out_score, num_selected, stream=None) -> None:
        _check(lib().ml2_stream_explorer_end(self.handle, _ptr(out_idx), _ptr(out_score),
                                             _ptr(num_selected), _stream(stream)))

    def free(self) -> None:
        if self.handle:
            lib().ml2_stream_explorer_free(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - interpreter shutdown order
        try:
            self.free()
        except Exception:
            pass


class Pipeline:
    """Device buffers for validity -> masked performance -> top-k on one pool
    (plumbing around the three calls; every step runs in libml2.so)."""

    def __init__(self, v: Ensemble, p: Ensemble, n: int, k: int, device="cuda",
                 with_margin: bool = False):
        import torch
        self.v, self.p, self.n, self.k = v, p, n, k
        self.valid = torch.empty(n, dtype=torch.uint8, device=device)
        self.margin = torch.empty(n, dtype=torch.float32, device=device) if with_margin else None
        self.score = torch.empty(n, dtype=torch.float32, device=device)
        self.idx = torch.empty(max(k, 1), dtype=torch.int32, device=device)
        self.top = torch.empty(max(k, 1), dtype=torch.float32, device=device)
        self.num = torch.empty(1, dtype=torch.int32, device=device)
        self.ws_bytes = ml2_topk_workspace_bytes(n, k)
        # 256-byte alignment holds for torch's caching allocator blocks
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        if self.ws.data_ptr() % 256:
            raise RuntimeError("top-k workspace is not 256-byte aligned")

    def run(self, X, stream=None) -> None:
        ml2_score_validity(self.v, X, self.valid, self.margin, stream)
        ml2_score_perf(self.p, X, self.valid, self.score, stream)
        ml2_filter_topk(self.valid, self.score, self.k, self.idx, self.top, self.num, self.ws,
                        self.ws_bytes, self.n, stream)


# ---- microbenchmarks (include/ml2_probe.h) ---------------------------------

def _probe(fn, *args):
    ms, work = ctypes.c_double(), ctypes.c_double()
    _check(fn(*args, ctypes.byref(ms), ctypes.byref(work)))
    return ms.value, work.value


def ml2_probe_visit(depth: int, trees_per_lane: int, lanes_per_candidate: int, waves: int,
                    features: int, iters: int, blocks: int):
    """(ms, node visits) of the walk's inner loop over a resident chunk at
    the given shape."""
    return _probe(lib().ml2_probe_visit, depth, trees_per_lane, lanes_per_candidate, waves,
                  features, iters, blocks)


def ml2_probe_lds(mode: int, iters: int, blocks: int):
    """(ms, bytes read) of LDS reads of 4/8/16 bytes (mode % 3), consecutive
    (mode < 3) or random."""
    return _probe(lib().ml2_probe_lds, mode, iters, blocks)


def ml2_probe_valu(iters: int, blocks: int):
    """(ms, lane additions) of chains of 32-bit adds."""
    return _probe(lib().ml2_probe_valu, iters, blocks)


# ---- tuning overrides (include/ml2_probe.h) --------------------------------

def ml2_tune_walk_plan(split: int = 0, group: int = 0, waves: int = 0, nbuf: int = 0,
                       chunk: int = 0) -> None:
    """Force the walks' launch shape for every later call (zeros: the
    planner's choice); results are unchanged, only the shape differs."""
    _check(lib().ml2_tune_walk_plan(split, group, waves, nbuf, chunk))


def ml2_tune_layout(layout: int = 0) -> None:
    """Force the layout of later loads: 0 the loader's choice, 1 perfect,
    2 ragged (where the ensemble allows it)."""
    _check(lib().ml2_tune_layout(layout))
