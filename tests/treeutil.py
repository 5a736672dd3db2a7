"""Test helpers: hand-built ensembles, random ragged trees and an independent
path-predicate evaluator.

The evaluator never walks a tree.  For every leaf it collects the conditions
on its root path (``x[f] < t`` for a left turn, ``not (x[f] < t)`` for a
right turn) and marks the candidates that satisfy all of them; a well-formed
tree partitions the input space, so exactly one leaf per tree must hold.
"""
from __future__ import annotations

import numpy as np

import gen


def ensemble_from_trees(trees, num_features, base=0.0):
    """Build a gen.Ensemble from nested tuples.

    A tree is either a float (a leaf) or ``(feature, threshold, left, right)``.
    Nodes are numbered in pre-order, so the layout is not breadth-first: this
    exercises general child pointers.
    """
    off = [0]
    left, right, feat, thr, val = [], [], [], [], []

    def emit(node):
        i = len(left) - off[-1]
        left.append(-1); right.append(-1); feat.append(-1); thr.append(0.0); val.append(0.0)
        g = len(left) - 1
        if isinstance(node, tuple):
            f, t, l, r = node
            feat[g] = f
            thr[g] = t
            li = emit(l)
            ri = emit(r)
            left[g] = li
            right[g] = ri
        else:
            val[g] = node
        return i

    for tr in trees:
        emit(tr)
        off.append(len(left))
    return gen.Ensemble(
        num_features, float(np.float32(base)),
        np.asarray(off, np.int64), np.asarray(left, np.int32), np.asarray(right, np.int32),
        np.asarray(feat, np.int32), np.asarray(thr, np.float32), np.asarray(val, np.float32))


def random_ragged_ensemble(rng, n_trees, max_depth, num_features, threshold_sampler,
                           leaf_sampler, p_split=0.7, base=0.0):
    """Random general trees: each node splits with probability p_split until
    max_depth; children are emitted in a shuffled order (ids are not BFS)."""
    trees = []

    def grow(d):
        if d < max_depth and rng.random() < p_split:
            f = int(rng.integers(num_features))
            return (f, float(threshold_sampler(rng, f)), grow(d + 1), grow(d + 1))
        return float(leaf_sampler(rng))

    for _ in range(n_trees):
        trees.append(grow(0))
    return ensemble_from_trees(trees, num_features, base)


def leaf_paths(ens, t):
    """[(conditions, value)] for tree t; a condition is (feature, thr,
    default_left, went_left)."""
    base = int(ens.offsets[t])
    dl_arr = getattr(ens, "default_left", None)
    out = []
    stack = [(0, [])]
    while stack:
        node, conds = stack.pop()
        g = base + node
        l, r = int(ens.left[g]), int(ens.right[g])
        if l < 0 and r < 0:
            out.append((conds, np.float32(ens.value[g])))
            continue
        f, th = int(ens.feature[g]), np.float32(ens.threshold[g])
        dl = bool(dl_arr[g]) if dl_arr is not None else False
        stack.append((l, conds + [(f, th, dl, True)]))
        stack.append((r, conds + [(f, th, dl, False)]))
    return out


def path_predicate_leaves(ens, X):
    """float32 [n, T]: the leaf each tree assigns to each row of X, found by
    checking every leaf's path conditions.  Asserts the partition property."""
    X = np.asarray(X, np.float32)
    n = X.shape[0]
    out = np.zeros((n, ens.num_trees), np.float32)
    for t in range(ens.num_trees):
        hits = np.zeros(n, np.int64)
        for conds, value in leaf_paths(ens, t):
            m = np.ones(n, bool)
            for f, th, dl, went_left in conds:
                # left: a present value below the threshold, or a missing
                # value at a node whose default is left
                x = X[:, f]
                left = (x < th) | (np.isnan(x) & dl)
                m &= left if went_left else ~left
            hits += m
            out[m, t] = value
        assert np.all(hits == 1), f"tree {t}: leaves do not partition the inputs"
    return out


def fold_left_f32(base, leaves):
    """Reference left fold used only to state expected values in tests."""
    m = np.float32(base)
    for v in leaves:
        m = np.float32(m + np.float32(v))
    return m
