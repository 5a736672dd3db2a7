"""CPU oracle for candidate scoring -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never calls it and
shares no code with it.

The arithmetic lives in ``ml2_oracle.c`` (plain C, one candidate and one
tree at a time, full-sort selection); this module compiles it with the host
compiler and wraps it with ctypes.  See the header of ``ml2_oracle.c`` for
what is computed and which passages of the paper it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ml2_oracle.c")
_LIB = os.path.join(_HERE, "libml2_oracle.so")


def build() -> str:
    """Compile the oracle (IEEE float32: no fast-math, no contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
           "-ffp-contract=off", "-fno-fast-math", "-fno-unsafe-math-optimizations",
           _SRC, "-o", _LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _Ens(ctypes.Structure):
    _fields_ = [
        ("num_trees", ctypes.c_int32),
        ("num_features", ctypes.c_int32),
        ("base_score", ctypes.c_float),
        ("offsets", ctypes.c_void_p),
        ("left", ctypes.c_void_p),
        ("right", ctypes.c_void_p),
        ("feature", ctypes.c_void_p),
        ("threshold", ctypes.c_void_p),
        ("value", ctypes.c_void_p),
        ("default_left", ctypes.c_void_p),
    ]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        lib.ml2o_tree_leaf.restype = ctypes.c_float
        lib.ml2o_tree_leaf.argtypes = [P, ctypes.c_int32, P]
        lib.ml2o_leaves.restype = None
        lib.ml2o_leaves.argtypes = [P, P, P]
        lib.ml2o_margin.restype = ctypes.c_float
        lib.ml2o_margin.argtypes = [P, P]
        lib.ml2o_validity.restype = None
        lib.ml2o_validity.argtypes = [P, P, ctypes.c_int64, ctypes.c_int64, P, P, ctypes.c_int32]
        lib.ml2o_perf.restype = None
        lib.ml2o_perf.argtypes = [P, P, ctypes.c_int64, ctypes.c_int64, P, P, ctypes.c_int32]
        lib.ml2o_topk.restype = ctypes.c_int64
        lib.ml2o_topk.argtypes = [P, P, ctypes.c_int64, ctypes.c_int64, P, P]
        lib.ml2o_rerank.restype = ctypes.c_int64
        lib.ml2o_rerank.argtypes = [P, P, ctypes.c_int64, ctypes.c_int64, P, ctypes.c_int64,
                                    ctypes.c_int64, P, P, P]
        _lib = lib
    return _lib


class OracleEnsemble:
    """Holds the arrays of an ensemble (gen.Ensemble-like) alive for C."""

    def __init__(self, ens):
        self.arrays = (
            np.ascontiguousarray(ens.offsets, np.int64),
            np.ascontiguousarray(ens.left, np.int32),
            np.ascontiguousarray(ens.right, np.int32),
            np.ascontiguousarray(ens.feature, np.int32),
            np.ascontiguousarray(ens.threshold, np.float32),
            np.ascontiguousarray(ens.value, np.float32),
        )
        dl = getattr(ens, "default_left", None)
        self.dl = None if dl is None else np.ascontiguousarray(dl, np.uint8)
        off, left, right, feat, thr, val = self.arrays
        self.num_trees = int(off.shape[0] - 1)
        self.num_features = int(ens.num_features)
        self.s = _Ens(self.num_trees, self.num_features, float(ens.base_score),
                      off.ctypes.data, left.ctypes.data, right.ctypes.data,
                      feat.ctypes.data, thr.ctypes.data, val.ctypes.data,
                      None if self.dl is None else self.dl.ctypes.data)

    @property
    def ptr(self):
        return ctypes.addressof(self.s)


def _as_oracle(ens) -> OracleEnsemble:
    return ens if isinstance(ens, OracleEnsemble) else OracleEnsemble(ens)


def _rows(X):
    X = np.asarray(X, dtype=np.float32)
    if X.ndim == 1:
        X = X[None, :]
    if not X.flags.c_contiguous:
        X = np.ascontiguousarray(X)
    return X


def tree_leaf(ens, t: int, x) -> np.float32:
    e = _as_oracle(ens)
    x = np.ascontiguousarray(x, np.float32)
    return np.float32(_load().ml2o_tree_leaf(e.ptr, t, x.ctypes.data))


def leaves(ens, x) -> np.ndarray:
    e = _as_oracle(ens)
    x = np.ascontiguousarray(x, np.float32)
    out = np.empty(e.num_trees, np.float32)
    _load().ml2o_leaves(e.ptr, x.ctypes.data, out.ctypes.data)
    return out


def margin(ens, x) -> np.float32:
    e = _as_oracle(ens)
    x = np.ascontiguousarray(x, np.float32)
    return np.float32(_load().ml2o_margin(e.ptr, x.ctypes.data))


def validity(ens, X, threads: int = 1):
    """(valid u8 [n], margin f32 [n]) for the rows of X."""
    e = _as_oracle(ens)
    X = _rows(X)
    n, ld = X.shape
    valid = np.zeros(n, np.uint8)
    marg = np.zeros(n, np.float32)
    _load().ml2o_validity(e.ptr, X.ctypes.data, n, ld, valid.ctypes.data, marg.ctypes.data, threads)
    return valid, marg


def perf(ens, X, valid=None, threads: int = 1) -> np.ndarray:
    """Scores f32 [n]; -inf where valid == 0 (valid None = all valid)."""
    e = _as_oracle(ens)
    X = _rows(X)
    n, ld = X.shape
    score = np.zeros(n, np.float32)
    vp = None
    if valid is not None:
        valid = np.ascontiguousarray(valid, np.uint8)
        assert valid.shape == (n,)
        vp = valid.ctypes.data
    _load().ml2o_perf(e.ptr, X.ctypes.data, n, ld, vp, score.ctypes.data, threads)
    return score


def topk(valid, score, k: int):
    """(idx i32 [k], score f32 [k], num_selected) by (score desc, index asc)."""
    score = np.ascontiguousarray(score, np.float32)
    n = score.shape[0]
    vp = None
    if valid is not None:
        valid = np.ascontiguousarray(valid, np.uint8)
        assert valid.shape == (n,)
        vp = valid.ctypes.data
    idx = np.empty(max(k, 0), np.int32)
    out = np.empty(max(k, 0), np.float32)
    sel = _load().ml2o_topk(vp, score.ctypes.data, n, k, idx.ctypes.data, out.ctypes.data)
    if sel < 0:
        raise MemoryError("oracle top-k allocation failed")
    return idx, out, int(sel)


def rerank(a_ens, X, rows, keep: int):
    """Model A's second level: (row_scores f32 [m], idx i32 [keep],
    score f32 [keep], num_selected) over the pool rows listed in `rows`
    (entries outside [0, n) are skipped), by (score desc, row asc)."""
    e = _as_oracle(a_ens)
    X = np.ascontiguousarray(X, np.float32)
    n, ld = (X.shape[0], X.shape[1]) if X.ndim == 2 else (0, 1)
    assert n == 0 or ld >= e.num_features
    rows = np.ascontiguousarray(rows, np.int32)
    m = rows.shape[0]
    row_scores = np.empty(max(m, 1), np.float32)
    idx = np.empty(max(keep, 1), np.int32)
    out = np.empty(max(keep, 1), np.float32)
    sel = _load().ml2o_rerank(e.ptr, X.ctypes.data if n else None, n, ld, rows.ctypes.data, m,
                              keep, row_scores.ctypes.data, idx.ctypes.data, out.ctypes.data)
    if sel < 0:
        raise MemoryError("oracle re-rank allocation failed")
    return row_scores[:m], idx[:keep], out[:keep], int(sel)


def explore(v_ens, p_ens, a_ens, X, k: int, keep: int, rounds: int, threads: int = 1):
    """The explorer's rounds over a fixed pool with fixed models (Section 2):
    each round holds the k best accepted rows not proposed before (by P),
    model A (or P's order when a_ens is None) keeps `keep` of them, and those
    are proposed.  Returns [(idx i32 [keep], score f32 [keep], num)] per
    round; -1/-inf pad a round once the pool runs dry."""
    valid, _ = validity(v_ens, X, threads)
    score = perf(p_ens, X, valid, threads)
    proposed = np.zeros(valid.shape[0], bool)
    out = []
    for _ in range(rounds):
        mask = (valid != 0) & ~proposed
        held, held_score, n_held = topk(mask.astype(np.uint8), score, k)
        if a_ens is not None:
            _, idx, top, num = rerank(a_ens, X, held, keep)
        else:
            idx, top = held[:keep].copy(), held_score[:keep].copy()
            num = min(n_held, keep)
        proposed[idx[idx >= 0]] = True
        out.append((idx, top, num))
    return out


def explore_stream(v_ens, p_ens, a_ens, chunks, k: int, keep: int, rounds: int,
                   threads: int = 1):
    """The explorer's rounds over a pool that arrives in row chunks
    (Section 2: the explorer applies V and P to the candidate configurations
    until (alpha+1)N are held and model A keeps N; a configuration proposed
    once is not proposed again).  ``chunks`` is the list of (row0, X_chunk)
    the pool arrives in, the same every round: row ``row0 + i`` of the pool
    is ``X_chunk[i]``; a row that arrives in several chunks is one
    configuration.  By definition a round works on the set of distinct rows,
    so this runs ``explore`` over those rows in row order (ties by position
    are then ties by row) and reports pool rows.  Returns [(idx i32 [keep],
    score f32 [keep], num)] per round; -1/-inf pad a round once the pool runs
    dry."""
    rows = {}
    F = None
    for row0, Xc in chunks:
        Xc = np.asarray(Xc, np.float32)
        F = Xc.shape[1] if Xc.ndim == 2 else F
        for i in range(Xc.shape[0]):
            rows.setdefault(int(row0) + i, Xc[i])
    ids = np.array(sorted(rows), np.int64)
    if ids.size == 0:
        return [(np.full(keep, -1, np.int32), np.full(keep, -np.inf, np.float32), 0)
                for _ in range(rounds)]
    X = np.stack([rows[int(i)] for i in ids]).astype(np.float32)
    out = []
    for idx, top, num in explore(v_ens, p_ens, a_ens, X, k, keep, rounds, threads):
        pool = np.where(idx >= 0, ids[np.maximum(idx, 0)], -1).astype(np.int32)
        out.append((pool, top, num))
    return out


def pipeline(v_ens, p_ens, X, k: int, threads: int = 1):
    """Validity -> masked performance -> top-k, as the explorer applies them."""
    valid, marg = validity(v_ens, X, threads)
    score = perf(p_ens, X, valid, threads)
    idx, top, sel = topk(valid, score, k)
    return dict(valid=valid, margin=marg, score=score, idx=idx, top=top, num=sel)
