"""Pins of the oracle on deep ragged trees with per-node default directions
for missing values (XGBoost's rule: a NaN feature takes the node's default
branch; Table 3's models are 300 rounds of depth up to 14): brute force
against the independent path-predicate evaluator, hand-checked stumps, and
the shape of the generator's trees."""
import numpy as np
import pytest

import gen
import oracle
from tests.treeutil import ensemble_from_trees, fold_left_f32, path_predicate_leaves


def _with_default_left(ens, dl):
    import dataclasses
    return dataclasses.replace(ens, default_left=np.asarray(dl, np.uint8))


def test_stump_default_direction():
    # one split on feature 0 at 1.0: left leaf 10, right leaf 20
    base = ensemble_from_trees([(0, 1.0, 10.0, 20.0)], num_features=1)
    x = np.array([[0.0], [1.0], [np.nan], [np.inf], [-np.inf]], np.float32)
    right = _with_default_left(base, [0, 0, 0])
    left = _with_default_left(base, [1, 0, 0])
    assert list(oracle.validity(right, x)[1]) == [10, 20, 20, 20, 10]
    assert list(oracle.validity(left, x)[1]) == [10, 20, 10, 20, 10]
    assert list(oracle.validity(base, x)[1]) == [10, 20, 20, 20, 10]  # no array: right


def _depth(ens, t):
    base = int(ens.offsets[t])
    best, stack = 0, [(0, 0)]
    while stack:
        node, d = stack.pop()
        l = int(ens.left[base + node])
        if l < 0:
            best = max(best, d)
        else:
            stack += [(l, d + 1), (int(ens.right[base + node]), d + 1)]
    return best


def test_generator_shape():
    e = gen.ragged_ensemble(3, 2, 60, 14, 10, 5, 0.1, max_nodes=300)
    sizes = np.diff(e.offsets)
    assert sizes.max() <= 300 and sizes.min() >= 3
    depths = [_depth(e, t) for t in range(60)]
    assert max(depths) == 14 and min(depths) >= 1
    for t in range(60):  # breadth-first ids: children adjacent, after the parent
        base = int(e.offsets[t])
        for i in range(int(sizes[t])):
            l, r = int(e.left[base + i]), int(e.right[base + i])
            if l >= 0:
                assert r == l + 1 and l > i
    internal = e.left >= 0
    assert 0.3 < e.default_left[internal].mean() < 0.7
    assert not e.default_left[~internal].any()


@pytest.mark.parametrize("seed", range(4))
def test_ragged_brute_force(seed):
    F, K = 8, 4
    e = gen.ragged_ensemble(seed, 1, 12, 14, F, K, 0.5, base_score=0.25, max_nodes=200)
    X = gen.features(seed, 300, F, K, missing=0.3)
    assert np.isnan(X[:, K:]).mean() > 0.2 and not np.isnan(X[:, :K]).any()
    leaves = path_predicate_leaves(e, X)
    want = np.array([fold_left_f32(e.base_score, leaves[i]) for i in range(X.shape[0])],
                    np.float32)
    _, got = oracle.validity(e, X)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_missing_values_are_seeded_and_hidden_only():
    a = gen.features(5, 100, 12, 6, missing=0.5)
    b = gen.features(5, 100, 12, 6, missing=0.5, threads=1)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    c = gen.features(5, 100, 12, 6)
    present = ~np.isnan(a)
    assert np.array_equal(a[present], c[present])  # the same values where present
    assert 0.35 < np.isnan(a[:, 6:]).mean() < 0.65
