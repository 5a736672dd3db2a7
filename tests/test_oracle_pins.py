"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with itself: the expected values
come from hand computation (golden files), closed forms, brute force over
the whole knob grid with an independent path-predicate evaluator, exact
summation bounds, and an independent sort.
"""
import json
import math
import os

import numpy as np
import pytest

import gen
import oracle
from tests.treeutil import (ensemble_from_trees, path_predicate_leaves,
                            random_ragged_ensemble)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _f(v):
    return np.float32(float(v)) if not isinstance(v, str) else np.float32(float(v))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def _tree(node):
    if isinstance(node, list):
        f, t, l, r = node
        return (int(f), float(t), _tree(l), _tree(r))
    return float(node)


# ---- the split rule (go left iff x < t) --------------------------------------

def _stump(t):
    return ensemble_from_trees([(0, t, 1.0, 2.0)], 1)


@pytest.mark.parametrize("x,t,expect", [
    (3.0, 3.0, 2.0),                                    # tie goes right
    (float(np.nextafter(np.float32(3), np.float32(-np.inf))), 3.0, 1.0),
    (1e30, float("inf"), 1.0),                          # finite < +inf
    (float("inf"), float("inf"), 2.0),                  # inf < inf is false
    (float("nan"), 3.0, 2.0),                           # NaN goes right
    (float("nan"), float("inf"), 2.0),
    (-0.0, 0.0, 2.0),                                   # -0 == +0: not less
    (0.0, -0.0, 2.0),
    (-1e-45, 0.0, 1.0),                                 # negative subnormal < 0
    (2.0 ** -141, 2.0 ** -140, 1.0),                    # subnormals not flushed
    (2.0 ** -140, 2.0 ** -140, 2.0),
    (-float("inf"), -float("inf"), 2.0),
    (-float("inf"), -3.0, 1.0),
])
def test_split_rule(x, t, expect):
    e = _stump(t)
    got = oracle.tree_leaf(e, 0, np.array([x], np.float32))
    assert got == np.float32(expect)


# ---- hand-computed pipeline ---------------------------------------------------

def _golden_pipeline():
    g = _load("hand_pipeline.json")
    F = g["num_features"]
    V = ensemble_from_trees([_tree(t) for t in g["validity"]["trees"]], F, g["validity"]["base"])
    P = ensemble_from_trees([_tree(t) for t in g["perf"]["trees"]], F, g["perf"]["base"])
    X = np.array([[float(v) for v in row] for row in g["candidates"]], np.float32)
    return g, V, P, X


def test_golden_leaves_margins_mask():
    g, V, P, X = _golden_pipeline()
    exp = g["expected"]
    for i, x in enumerate(X):
        assert np.array_equal(oracle.leaves(V, x), np.array(exp["validity_leaves"][i], np.float32))
    valid, margin = oracle.validity(V, X)
    assert np.array_equal(margin, np.array(exp["margin"], np.float32))
    assert np.array_equal(valid, np.array(exp["valid"], np.uint8))
    score = oracle.perf(P, X, valid)
    assert np.array_equal(score, np.array([float(s) for s in exp["score"]], np.float32))


@pytest.mark.parametrize("k", ["2", "5", "0"])
def test_golden_topk(k):
    g, V, P, X = _golden_pipeline()
    r = oracle.pipeline(V, P, X, int(k))
    e = g["expected"]["topk"][k]
    assert r["num"] == e["num"]
    assert np.array_equal(r["idx"], np.array(e["idx"], np.int32))
    assert np.array_equal(r["top"], np.array([float(s) for s in e["score"]], np.float32))


# ---- fold order, strict decision ---------------------------------------------

@pytest.mark.parametrize("case", _load("order_witness.json")["cases"])
def test_order_witness(case):
    trees = [float(v) for v in case["leaves"]]
    V = ensemble_from_trees(trees, 1, case["base"])
    valid, margin = oracle.validity(V, np.zeros((1, 1), np.float32))
    assert margin[0] == np.float32(case["margin"])
    assert valid[0] == case["valid"]


def test_strict_margin_beats_sigmoid_reading():
    # sigmoid(1e-8) rounds to exactly 0.5 in float32, so a "sigmoid > 0.5" test
    # would reject this candidate; the hinge decision (margin > 0) accepts it.
    m = np.float32(1e-8)
    sig = np.float32(1) / (np.float32(1) + np.exp(-m, dtype=np.float32))
    assert sig == np.float32(0.5)
    V = ensemble_from_trees([1e-8], 1)
    valid, _ = oracle.validity(V, np.zeros((1, 1), np.float32))
    assert valid[0] == 1


def test_base_score_added_first():
    # base 2^24, leaves 1, 1: ((2^24 + 1) + 1) = 2^24 in float32 (each +1 is
    # lost to rounding), whereas base + (1 + 1) would be 2^24 + 2.
    V = ensemble_from_trees([1.0, 1.0], 1, 16777216.0)
    _, m = oracle.validity(V, np.zeros((1, 1), np.float32))
    assert m[0] == np.float32(16777216.0)


def test_permuting_constant_trees_changes_only_fold_order():
    rng = np.random.default_rng(7)
    leaves = (rng.integers(-2 ** 20, 2 ** 20, size=64) * 2.0 ** -10).tolist()  # dyadic, exact
    a = ensemble_from_trees(leaves, 1, 0.5)
    b = ensemble_from_trees(list(reversed(leaves)), 1, 0.5)
    x = np.zeros((1, 1), np.float32)
    exact = math.fsum(leaves) + 0.5
    assert float(oracle.margin(a, x[0])) == exact
    assert float(oracle.margin(b, x[0])) == exact


# ---- brute force over the whole knob grid --------------------------------------

def _knob_grid(F):
    axes = np.meshgrid(*[np.arange(9, dtype=np.float32)] * F, indexing="ij")
    return np.stack([a.ravel() for a in axes], axis=1)


@pytest.mark.parametrize("F,depth,trees,seed", [(3, 4, 40, 11), (4, 5, 30, 12), (4, 3, 60, 13)])
def test_brute_force_knob_grid_perfect(F, depth, trees, seed):
    """Every point of {0..8}^F (729 or 6561 candidates, as the paper
    enumerates whole configuration spaces), perfect generator trees."""
    X = _knob_grid(F)
    ens = gen.perfect_ensemble(seed, 1, trees, depth, F, F, 0.5)
    want = path_predicate_leaves(ens, X)
    got = np.stack([oracle.leaves(ens, x) for x in X])
    assert np.array_equal(got, want)


def test_brute_force_knob_grid_ragged():
    rng = np.random.default_rng(5)
    F = 4
    ens = random_ragged_ensemble(
        rng, 50, 7, F, lambda r, f: float(r.integers(0, 9)),
        lambda r: float(r.normal(0, 0.5)), p_split=0.75)
    X = _knob_grid(F)
    want = path_predicate_leaves(ens, X)
    got = np.stack([oracle.leaves(ens, x) for x in X])
    assert np.array_equal(got, want)


# ---- fold accuracy against the exact sum --------------------------------------

def test_fold_within_summation_bound():
    """|fl(sum) - sum| <= gamma_{T} * sum|partial terms| (Higham, recursive
    summation); a dropped or doubled leaf would break it by orders of magnitude."""
    w = gen.WORKLOADS["medium"]
    X = w.features(rows=np.arange(200, dtype=np.int64))
    V = w.validity()
    ov = oracle.OracleEnsemble(V)
    u = 2.0 ** -24
    T = V.num_trees
    gamma = T * u / (1 - T * u)
    for x in X:
        lv = oracle.leaves(ov, x)
        terms = [float(V.base_score)] + [float(v) for v in lv]
        exact = math.fsum(terms)
        got = float(oracle.margin(ov, x))
        assert abs(got - exact) <= gamma * sum(abs(t) for t in terms) + 1e-30


def test_dyadic_fold_is_exact():
    rng = np.random.default_rng(3)
    F = 6
    ens = random_ragged_ensemble(
        rng, 80, 6, F, lambda r, f: float(r.integers(0, 9)),
        lambda r: float(r.integers(-4096, 4096)) * 2.0 ** -8, base=0.375)
    X = rng.integers(0, 9, size=(300, F)).astype(np.float32)
    leaves = path_predicate_leaves(ens, X)
    _, m = oracle.validity(ens, X)
    for i in range(X.shape[0]):
        assert float(m[i]) == math.fsum([0.375] + leaves[i].astype(np.float64).tolist())


# ---- masked performance --------------------------------------------------------

def test_perf_masks_invalid_to_minus_inf():
    rng = np.random.default_rng(1)
    F = 3
    P = random_ragged_ensemble(rng, 10, 4, F, lambda r, f: float(r.integers(0, 9)),
                               lambda r: float(r.integers(-64, 64)) * 2.0 ** -6)
    X = rng.integers(0, 9, size=(50, F)).astype(np.float32)
    valid = (rng.random(50) < 0.5).astype(np.uint8)
    s = oracle.perf(P, X, valid)
    full = oracle.perf(P, X, None)
    leaves = path_predicate_leaves(P, X)
    for i in range(50):
        exact = math.fsum(leaves[i].astype(np.float64).tolist())
        assert float(full[i]) == exact
        assert s[i] == (full[i] if valid[i] else -np.inf)


# ---- selection ----------------------------------------------------------------

def _sorted_reference(valid, score, k):
    inc = [i for i in range(len(score))
           if (valid is None or valid[i]) and not np.isnan(score[i])]
    inc.sort(key=lambda i: (-float(score[i]), i))
    return inc[:k]


@pytest.mark.parametrize("seed", range(5))
def test_topk_against_independent_sort(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 3000))
    # coarse scores to force many ties, plus -0.0 / +0.0 and NaN
    score = (rng.integers(-20, 20, size=n) * 0.25).astype(np.float32)
    score[rng.random(n) < 0.05] = -0.0
    score[rng.random(n) < 0.02] = np.nan
    valid = (rng.random(n) < 0.6).astype(np.uint8)
    for k in (0, 1, 7, 100, n + 5):
        idx, top, num = oracle.topk(valid, score, k)
        ref = _sorted_reference(valid, score, k)
        assert num == len(ref)
        assert idx[:num].tolist() == ref
        assert np.array_equal(top[:num], score[ref], equal_nan=False)
        assert np.all(idx[num:] == -1) and np.all(top[num:] == -np.inf)


def test_topk_constant_trees_select_lowest_indices():
    V = ensemble_from_trees([0.5], 2)
    P = ensemble_from_trees([0.25, 0.125], 2)
    X = np.zeros((1000, 2), np.float32)
    r = oracle.pipeline(V, P, X, 17)
    assert r["num"] == 17
    assert r["idx"].tolist() == list(range(17))
    assert np.all(r["top"] == np.float32(0.375))


def test_topk_signed_zero_ties_by_index():
    score = np.array([0.0, -0.0, 0.0, -0.0], np.float32)
    idx, top, num = oracle.topk(None, score, 4)
    assert idx.tolist() == [0, 1, 2, 3]
    assert np.signbit(top).tolist() == [False, True, False, True]


def test_topk_empty_pool():
    idx, top, num = oracle.topk(None, np.zeros(0, np.float32), 3)
    assert num == 0 and idx.tolist() == [-1, -1, -1]
