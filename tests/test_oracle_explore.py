"""Pins of the oracle's explorer rounds (Section 2: each iteration proposes
N configurations; V and P fill (alpha+1)N held ones, model A keeps N; a
configuration is proposed once): brute force from an independent evaluator
(leaf path predicates) and Python's sort, and the loop's invariants."""
import numpy as np
import pytest

import oracle
from tests.treeutil import fold_left_f32, path_predicate_leaves, random_ragged_ensemble


def _thr(rng, f):
    return float(rng.integers(0, 6))


def _ens(rng, trees, sigma, base=0.0):
    return random_ragged_ensemble(rng, trees, 4, 5, _thr,
                                  lambda r: float(np.float32(r.normal(0, sigma))), p_split=0.8,
                                  base=base)


def _margins(ens, X):
    leaves = path_predicate_leaves(ens, X)
    return np.array([fold_left_f32(ens.base_score, leaves[i]) for i in range(X.shape[0])],
                    np.float32)


def _brute(V, P, A, X, k, keep, rounds):
    valid = _margins(V, X) > 0
    ps = _margins(P, X)
    as_ = _margins(A, X) if A is not None else None
    proposed = set()
    out = []
    for _ in range(rounds):
        cand = [i for i in range(X.shape[0]) if valid[i] and i not in proposed]
        held = sorted(cand, key=lambda i: (-float(ps[i]), i))[:k]
        by = as_ if A is not None else ps
        kept = sorted(held, key=lambda i: (-float(by[i]), i))[:keep]
        proposed.update(kept)
        sc = [float(by[i]) for i in kept]
        out.append((kept + [-1] * (keep - len(kept)), sc + [-np.inf] * (keep - len(kept))))
    return out


@pytest.mark.parametrize("seed,with_a", [(0, True), (1, True), (2, False), (3, True)])
def test_explore_brute_force(seed, with_a):
    rng = np.random.default_rng(seed)
    V = _ens(rng, 5, 1.0, base=0.3)
    P = _ens(rng, 6, 1.0)
    A = _ens(rng, 7, 1.0) if with_a else None
    X = rng.integers(0, 6, size=(50, 5)).astype(np.float32)
    k, keep, rounds = 7, 3, 12  # enough rounds to run the pool dry
    got = oracle.explore(V, P, A, X, k, keep, rounds)
    want = _brute(V, P, A, X, k, keep, rounds)
    for r, ((idx, top, num), (widx, wtop)) in enumerate(zip(got, want)):
        assert list(idx) == widx, f"round {r}"
        assert np.array_equal(top.view(np.uint32), np.array(wtop, np.float32).view(np.uint32))
        assert num == sum(i >= 0 for i in widx)


def test_explore_invariants():
    rng = np.random.default_rng(9)
    V, P, A = _ens(rng, 4, 1.0, base=1.0), _ens(rng, 5, 1.0), _ens(rng, 6, 1.0)
    X = rng.integers(0, 6, size=(80, 5)).astype(np.float32)
    out = oracle.explore(V, P, A, X, 6, 4, 30)
    valid, _ = oracle.validity(V, X)
    seen = [i for idx, _, _ in out for i in idx if i >= 0]
    assert len(seen) == len(set(seen)), "a row was proposed twice"
    assert all(valid[i] for i in seen), "a rejected row was proposed"
    assert len(seen) == int(valid.sum()), "the loop stops before the accepted rows run out"
    nums = [num for _, _, num in out]
    assert nums == sorted(nums, reverse=True)


def _brute_stream(V, P, A, chunks, k, keep, rounds):
    """Expected rounds over a chunked pool, from the definition: every
    distinct row (the first copy of a row arriving twice), its leaves by path
    predicates, Python's sort."""
    rows = {}
    for row0, Xc in chunks:
        for i in range(Xc.shape[0]):
            rows.setdefault(row0 + i, Xc[i])
    ids = sorted(rows)
    X = np.array([rows[i] for i in ids], np.float32)
    valid = dict(zip(ids, _margins(V, X) > 0))
    ps = dict(zip(ids, _margins(P, X)))
    by = dict(zip(ids, _margins(A, X))) if A is not None else ps
    proposed = set()
    out = []
    for _ in range(rounds):
        cand = [i for i in ids if valid[i] and i not in proposed]
        held = sorted(cand, key=lambda i: (-float(ps[i]), i))[:k]
        kept = sorted(held, key=lambda i: (-float(by[i]), i))[:keep]
        proposed.update(kept)
        sc = [float(by[i]) for i in kept]
        out.append((kept + [-1] * (keep - len(kept)), sc + [-np.inf] * (keep - len(kept))))
    return out


@pytest.mark.parametrize("seed,with_a", [(4, True), (5, False), (6, True)])
def test_explore_stream_brute_force(seed, with_a):
    """Chunks with gaps between them, a chunk overlapping another (its shared
    rows arrive twice with the same features), an empty chunk, and rows far
    apart in the id space."""
    rng = np.random.default_rng(seed)
    V = _ens(rng, 5, 1.0, base=0.3)
    P = _ens(rng, 6, 1.0)
    A = _ens(rng, 7, 1.0) if with_a else None
    pool = rng.integers(0, 6, size=(120, 5)).astype(np.float32)
    spans = [(0, 30), (45, 70), (60, 95), (95, 95), (100, 120)]  # ids 1000 + [a, b)
    chunks = [(1000 + a, pool[a:b]) for a, b in spans]
    k, keep, rounds = 6, 3, 30
    got = oracle.explore_stream(V, P, A, chunks, k, keep, rounds)
    want = _brute_stream(V, P, A, chunks, k, keep, rounds)
    for r, ((idx, top, num), (widx, wtop)) in enumerate(zip(got, want)):
        assert list(idx) == widx, f"round {r}"
        assert np.array_equal(top.view(np.uint32), np.array(wtop, np.float32).view(np.uint32))
        assert num == sum(i >= 0 for i in widx)
    proposed = [i for idx, _, _ in got for i in idx if i >= 0]
    assert len(proposed) == len(set(proposed)), "a row was proposed twice"
    assert all(1000 <= i < 1030 or 1045 <= i < 1095 or 1100 <= i < 1120 for i in proposed)


def test_explore_stream_of_contiguous_chunks_is_the_pool():
    # chunks that tile the pool give the pool's rounds, rows and scores
    rng = np.random.default_rng(8)
    V, P, A = _ens(rng, 4, 1.0, base=0.5), _ens(rng, 5, 1.0), _ens(rng, 6, 1.0)
    X = rng.integers(0, 6, size=(64, 5)).astype(np.float32)
    chunks = [(0, X[:10]), (10, X[10:11]), (11, X[11:40]), (40, X[40:])]
    got = oracle.explore_stream(V, P, A, chunks, 5, 2, 20)
    want = _brute(V, P, A, X, 5, 2, 20)
    for (idx, top, _), (widx, wtop) in zip(got, want):
        assert list(idx) == widx
        assert np.array_equal(top.view(np.uint32), np.array(wtop, np.float32).view(np.uint32))
