"""Seeded synthetic workloads for candidate scoring (input generation only).

The paper tunes the convolution layers of ResNet18 on an extended VTA and
scores candidate configurations with XGBoost models (Section 3 "Experimental
Setup"; Appendix A.3 "Experimental HyperParameter", Table 3).  Its profiled
configuration spaces and trained models are not public, so every workload
here is synthetic, scaled up from the paper's shapes:

* visible features (tile width, tile height, virtual threads; Appendix A.4,
  Table 5) become integer knob columns log2(tile) uniform on {0..8};
* hidden compiler features (derived sizes and branch flags; Appendix A.4,
  Table 5) become lognormal(0,1) columns;
* models V and P (Section 2, "ML Model P", "ML Model V") become perfect
  binary trees of a fixed depth with split features uniform over the
  columns, thresholds drawn from the split column's own distribution and
  leaves N(0, 0.5) (validity) or N(0, 0.1) (performance).

This module holds no tree walking, no summation and no selection: it only
produces inputs, through the C generator in ``ml2gen.c`` (counter-based,
so results do not depend on the thread count).  Both the GPU path and the
CPU oracle take their inputs from here.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ml2gen.c")
_LIB = os.path.join(_HERE, "libml2gen.so")

STREAM_FEATURES = 0
STREAM_VALIDITY = 1
STREAM_PERF = 2
STREAM_SECOND_LEVEL = 3


def build() -> str:
    """Compile the generator with the host C compiler (always rebuilds)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
           "-ffp-contract=off", "-fno-fast-math", _SRC, "-o", _LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.ml2gen_hash.restype = ctypes.c_uint64
        lib.ml2gen_hash.argtypes = [ctypes.c_uint64] * 3
        lib.ml2gen_features.restype = None
        lib.ml2gen_features.argtypes = [
            ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
            ctypes.c_double]
        lib.ml2gen_ragged_trees.restype = ctypes.c_int64
        lib.ml2gen_ragged_trees.argtypes = [
            ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_double] + [ctypes.c_void_p] * 7
        lib.ml2gen_perfect_trees.restype = None
        lib.ml2gen_perfect_trees.argtypes = [
            ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_void_p]
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def hash64(seed: int, stream: int, ctr: int) -> int:
    return int(_load().ml2gen_hash(seed, stream, ctr))


@dataclasses.dataclass(frozen=True)
class Ensemble:
    """A tree ensemble in the general child-pointer form.

    Tree t owns nodes ``offsets[t] .. offsets[t+1]-1``; node ids in
    ``left``/``right`` are tree-local (0 = root); a leaf has -1 on both.
    Internal nodes go LEFT iff ``x[feature] < threshold``.
    """
    num_features: int
    base_score: float
    offsets: np.ndarray       # int64 [T+1]
    left: np.ndarray          # int32 [nodes]
    right: np.ndarray         # int32 [nodes]
    feature: np.ndarray       # int32 [nodes]
    threshold: np.ndarray     # float32 [nodes]
    value: np.ndarray         # float32 [nodes] (leaves only)
    # uint8 [nodes] or None: a missing (NaN) feature value goes left at an
    # internal node with a nonzero entry, right otherwise (None: always right)
    default_left: np.ndarray | None = None

    @property
    def num_trees(self) -> int:
        return int(self.offsets.shape[0] - 1)

    def with_base(self, base: float) -> "Ensemble":
        return dataclasses.replace(self, base_score=float(np.float32(base)))


def perfect_ensemble(seed: int, stream: int, trees: int, depth: int, F: int, K: int,
                     leaf_sigma: float, base_score: float = 0.0) -> Ensemble:
    """`trees` perfect trees of `depth` split levels (see ml2gen.c)."""
    nodes = (2 << depth) - 1
    total = trees * nodes
    off = np.empty(trees + 1, np.int64)
    left = np.empty(total, np.int32)
    right = np.empty(total, np.int32)
    feat = np.empty(total, np.int32)
    thr = np.empty(total, np.float32)
    val = np.empty(total, np.float32)
    _load().ml2gen_perfect_trees(
        seed, stream, trees, depth, F, K, float(leaf_sigma),
        off.ctypes.data, left.ctypes.data, right.ctypes.data, feat.ctypes.data,
        thr.ctypes.data, val.ctypes.data)
    return Ensemble(F, float(np.float32(base_score)), off, left, right, feat, thr, val)


def ragged_ensemble(seed: int, stream: int, trees: int, max_depth: int, F: int, K: int,
                    leaf_sigma: float, base_score: float = 0.0, p_split: float = 0.9,
                    decay: float = 0.9, p_left: float = 0.5,
                    max_nodes: int = 2047) -> Ensemble:
    """`trees` ragged trees of at most `max_depth` split levels with default
    directions for missing values (see ml2gen.c)."""
    cap = trees * max_nodes
    off = np.empty(trees + 1, np.int64)
    left = np.empty(cap, np.int32)
    right = np.empty(cap, np.int32)
    feat = np.empty(cap, np.int32)
    thr = np.empty(cap, np.float32)
    val = np.empty(cap, np.float32)
    dl = np.empty(cap, np.uint8)
    total = _load().ml2gen_ragged_trees(
        seed, stream, trees, max_depth, max_nodes, float(p_split), float(decay),
        float(p_left), F, K, float(leaf_sigma), off.ctypes.data, left.ctypes.data,
        right.ctypes.data, feat.ctypes.data, thr.ctypes.data, val.ctypes.data, dl.ctypes.data)
    if total < 0:
        raise MemoryError("ragged tree generation failed")
    return Ensemble(F, float(np.float32(base_score)), off, left[:total].copy(),
                    right[:total].copy(), feat[:total].copy(), thr[:total].copy(),
                    val[:total].copy(), dl[:total].copy())


def features(seed: int, n: int, F: int, K: int, *, rows=None, row0: int = 0,
             ld: int | None = None, out: np.ndarray | None = None,
             threads: int | None = None, missing: float = 0.0) -> np.ndarray:
    """Rows of the seeded N x F candidate matrix as float32 [m, ld].

    With ``rows`` (int64 indices) the output holds those global rows in that
    order; otherwise rows ``row0 .. row0+n-1``.  With ``missing`` > 0 each
    hidden value is NaN (missing) with that probability.
    """
    ld = F if ld is None else ld
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        m = rows.shape[0]
    else:
        m = n
    if out is None:
        out = np.zeros((m, ld), np.float32)
    assert out.dtype == np.float32 and out.flags.c_contiguous and out.shape == (m, ld)
    _load().ml2gen_features(
        seed, rows.ctypes.data if rows is not None else None, row0, m, F, K, ld,
        out.ctypes.data, threads or default_threads(), float(missing))
    return out


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic scoring workload: pool size, feature split, ensembles, k."""
    name: str
    n: int
    F: int
    K: int                       # knob (visible) columns; the rest are hidden
    v_trees: int
    v_depth: int
    p_trees: int
    p_depth: int
    k: int
    seed: int
    base_v: float = 0.0          # validity margin bias (float32 value)
    calib_quantile: float | None = None  # invalid fraction base_v was fixed for
    # Second level (model A) and the paper's feature split: with
    # visible_only, V and P split on the K knob columns only (their
    # num_features is K) and A, over all F columns, re-ranks the k held
    # configurations and keeps `keep`.
    a_trees: int = 0
    a_depth: int = 0
    keep: int = 0
    visible_only: bool = False
    # Paper-shaped models (Table 3): P and A as ragged trees of at most
    # p_depth / a_depth levels with default directions, grown with
    # ragged_ensemble's defaults; hidden values missing with this probability.
    ragged: bool = False
    ragged_max_nodes: int = 255
    missing: float = 0.0

    def _vp_features(self) -> int:
        return self.K if self.visible_only else self.F

    def validity(self) -> Ensemble:
        return perfect_ensemble(self.seed, STREAM_VALIDITY, self.v_trees, self.v_depth,
                                self._vp_features(), self.K, 0.5, self.base_v)

    def perf(self) -> Ensemble:
        if self.ragged:
            return ragged_ensemble(self.seed, STREAM_PERF, self.p_trees, self.p_depth,
                                   self._vp_features(), self.K, 0.1,
                                   max_nodes=self.ragged_max_nodes)
        return perfect_ensemble(self.seed, STREAM_PERF, self.p_trees, self.p_depth,
                                self._vp_features(), self.K, 0.1, 0.0)

    def second_level(self) -> Ensemble:
        assert self.a_trees > 0, f"workload {self.name} has no second-level model"
        if self.ragged:
            return ragged_ensemble(self.seed, STREAM_SECOND_LEVEL, self.a_trees, self.a_depth,
                                   self.F, self.K, 0.1, max_nodes=self.ragged_max_nodes)
        return perfect_ensemble(self.seed, STREAM_SECOND_LEVEL, self.a_trees, self.a_depth,
                                self.F, self.K, 0.1, 0.0)

    def features(self, rows=None, **kw) -> np.ndarray:
        kw.setdefault("missing", self.missing)
        return features(self.seed, self.n, self.F, self.K, rows=rows, **kw)


# Margin biases of the calibrated workloads.  Each is -(float32) of the
# p-quantile of the zero-bias validity margins of the first 65536 candidates,
# computed by oracle/calibrate_base.py (p = 0.4 for "medium", p = 0.9 for
# "skewed"); tests/test_workloads.py recomputes them.
_BASE_V_MEDIUM = 1.4281009435653687     # float32 0x3fb6cc03
_BASE_V_SKEWED = -8.522647857666016      # float32 0xc1085cc4

WORKLOADS = {
    "tiny": Workload("tiny", 4096, 32, 16, 50, 5, 50, 5, 32, 1),
    "medium": Workload("medium", 262144, 64, 32, 200, 6, 200, 6, 128, 2,
                       _BASE_V_MEDIUM, 0.4),
    "large": Workload("large", 4194304, 96, 48, 500, 8, 500, 8, 512, 3),
    "roofline": Workload("roofline", 16777216, 128, 64, 300, 6, 1000, 8, 1024, 4),
    "skewed": Workload("skewed", 8388608, 64, 32, 200, 6, 800, 10, 256, 5,
                       _BASE_V_SKEWED, 0.9),
    # The explorer as the paper runs it (Section 2): V and P on the visible
    # (knob) columns, A (300 rounds as in Table 3, depth 12 = the deepest
    # perfect layout; Table 3's 14 needs the ragged layout) on visible +
    # hidden columns; k = (alpha+1)N = 1024 held, N = 512 kept (alpha = 1).
    "explorer": Workload("explorer", 16777216, 128, 64, 300, 6, 1000, 8, 1024, 6,
                         a_trees=300, a_depth=12, keep=512, visible_only=True),
    # The models as Table 3 sizes them: V 300 rounds of depth 5; P and A 300
    # rounds of depth up to 14 (ragged, default directions for missing
    # values; trees of about 100 nodes, as trained on a few hundred profiled
    # configurations); 5 % of the hidden values missing; (alpha+1)N = 20
    # held and N = 10 kept (Section 3).
    "paper": Workload("paper", 16777216, 128, 64, 300, 5, 300, 14, 20, 7,
                      a_trees=300, a_depth=14, keep=10, visible_only=True, ragged=True,
                      missing=0.05),
    # Diagnostic, not a benchmark configuration: the 16M x 128 pool with
    # small ensembles (V and P 40 trees of depth 5, about 300 node visits
    # per candidate), where reading the pool from HBM, not walking trees,
    # bounds the step.
    "hbm": Workload("hbm", 16777216, 128, 64, 40, 5, 40, 5, 1024, 8),
}
CALIBRATION_ROWS = 65536
