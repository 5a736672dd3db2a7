"""Pins of the oracle's second level (model A re-rank, Section 2 "Hidden
Feature Extractor & ML Model A"): brute force against an independent
evaluator (every leaf's path predicate) and Python's sort, plus the
definitional special cases (skipped entries, duplicates, padding, ties,
signed zero)."""
import numpy as np
import pytest

import oracle
from tests.treeutil import (ensemble_from_trees, fold_left_f32, path_predicate_leaves,
                            random_ragged_ensemble)


def _brute(ens, X, rows, keep):
    """Expected (row_scores, idx, score, num) written out from the definition."""
    n = X.shape[0]
    leaves = path_predicate_leaves(ens, X) if n else np.zeros((0, ens.num_trees), np.float32)
    scores = []
    entries = []
    for r in rows:
        if 0 <= r < n:
            s = fold_left_f32(ens.base_score, leaves[r])
            scores.append(s)
            entries.append((float(s), int(r)))
        else:
            scores.append(np.float32(-np.inf))
    entries.sort(key=lambda e: (-e[0], e[1]))
    sel = entries[:keep]
    idx = [r for _, r in sel] + [-1] * (keep - len(sel))
    top = [s for s, _ in sel] + [-np.inf] * (keep - len(sel))
    return (np.array(scores, np.float32), np.array(idx, np.int32), np.array(top, np.float32),
            len(sel))


def _thr(rng, f):
    return float(rng.integers(0, 5))


@pytest.mark.parametrize("seed", range(6))
def test_rerank_brute_force(seed):
    rng = np.random.default_rng(seed)
    F = 6
    A = random_ragged_ensemble(rng, 7, 4, F, _thr, lambda r: float(np.float32(r.normal(0, 1))),
                               p_split=0.7, base=float(np.float32(rng.normal())))
    n = 40
    X = rng.integers(0, 5, size=(n, F)).astype(np.float32)
    m = int(rng.integers(0, 30))
    rows = rng.integers(-3, n + 3, size=m).astype(np.int32)  # some out of range, repeats
    keep = int(rng.integers(0, 25))
    got = oracle.rerank(A, X, rows, keep)
    want = _brute(A, X, rows, keep)
    assert np.array_equal(got[0].view(np.uint32), want[0].view(np.uint32))
    assert np.array_equal(got[1], want[1])
    assert np.array_equal(got[2].view(np.uint32), want[2].view(np.uint32))
    assert got[3] == want[3]


def test_rerank_ties_go_to_lower_row_and_duplicates_count_twice():
    # one tree with a single leaf: every row scores the same
    A = ensemble_from_trees([0.25], num_features=2, base=1.0)
    X = np.zeros((10, 2), np.float32)
    rows = np.array([7, 3, -1, 9, 3, 12, 0], np.int32)
    row_scores, idx, top, num = oracle.rerank(A, X, rows, 4)
    assert list(idx) == [0, 3, 3, 7] and num == 4
    assert np.all(top == np.float32(1.25))
    assert row_scores[2] == -np.inf and row_scores[5] == -np.inf


def test_rerank_padding_and_empty():
    A = ensemble_from_trees([0.5], num_features=1)
    X = np.zeros((3, 1), np.float32)
    _, idx, top, num = oracle.rerank(A, X, np.array([2, 1], np.int32), 5)
    assert list(idx) == [1, 2, -1, -1, -1] and num == 2
    assert np.all(np.isneginf(top[2:]))
    rs, idx, top, num = oracle.rerank(A, X, np.zeros(0, np.int32), 3)
    assert num == 0 and list(idx) == [-1, -1, -1] and rs.shape == (0,)
    rs, idx, top, num = oracle.rerank(A, X, np.array([0, 1], np.int32), 0)
    assert num == 0 and idx.shape == (0,)
    rs, idx, top, num = oracle.rerank(A, np.zeros((0, 1), np.float32), np.array([0, 1], np.int32), 2)
    assert num == 0 and np.all(np.isneginf(rs)) and list(idx) == [-1, -1]


def test_rerank_signed_zero():
    # base -0.0 plus a -0.0 leaf folds to -0.0 (rows 0 and 2), base -0.0 plus a
    # +0.0 leaf to +0.0 (row 1).  -0.0 and +0.0 are equal in the order, so the
    # three tie and go by row; each kept entry reports its own score, sign of
    # zero included (the selection returns the scores it ranked, as the
    # top-k does).
    A = ensemble_from_trees([(0, 0.5, -0.0, 0.0)], num_features=1, base=-0.0)
    X = np.array([[0.0], [1.0], [0.0]], np.float32)  # rows 0, 2 -> -0.0; row 1 -> +0.0
    row_scores, idx, top, num = oracle.rerank(A, X, np.array([2, 1, 0], np.int32), 3)
    assert np.signbit(row_scores[0]) and not np.signbit(row_scores[1])
    assert list(idx) == [0, 1, 2] and num == 3
    assert list(np.signbit(top)) == [True, False, True]
    assert np.all(top == 0.0)


def test_rerank_order_is_score_then_row():
    # scores decided by feature 0; several rows share a score
    A = ensemble_from_trees([(0, 1.5, 1.0, (0, 2.5, 3.0, 2.0))], num_features=1)
    X = np.array([[0], [2], [3], [1], [2], [0]], np.float32)  # scores 1, 3, 2, 1, 3, 1
    _, idx, top, num = oracle.rerank(A, X, np.arange(6, dtype=np.int32), 6)
    assert list(idx) == [1, 4, 2, 0, 3, 5]
    assert list(top) == [3, 3, 2, 1, 1, 1]
