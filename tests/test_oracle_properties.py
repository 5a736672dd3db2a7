"""Property tests of the oracle on random small inputs (hypothesis)."""
import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from tests.treeutil import path_predicate_leaves, random_ragged_ensemble

floats32 = st.floats(width=32, allow_nan=True, allow_infinity=True)


@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 2 ** 31), F=st.integers(1, 6), depth=st.integers(0, 7),
       n=st.integers(1, 40))
def test_walker_matches_path_predicates(seed, F, depth, n):
    rng = np.random.default_rng(seed)
    ens = random_ragged_ensemble(
        rng, 12, depth, F,
        lambda r, f: float(np.float32(r.normal(0, 2))) if r.random() < 0.8 else float(r.integers(-2, 3)),
        lambda r: float(np.float32(r.normal(0, 1))))
    X = rng.normal(0, 2, size=(n, F)).astype(np.float32)
    X[rng.random((n, F)) < 0.1] = np.nan
    ties = rng.random((n, F)) < 0.2          # values equal to integer thresholds
    X[ties] = rng.integers(-2, 3, size=int(ties.sum()))
    want = path_predicate_leaves(ens, X)
    got = np.stack([oracle.leaves(ens, x) for x in X])
    assert np.array_equal(got, want, equal_nan=True)


@settings(max_examples=80, deadline=None)
@given(scores=st.lists(st.floats(width=32, allow_nan=True, allow_infinity=True), max_size=300),
       mask_seed=st.integers(0, 2 ** 31), k=st.integers(0, 400))
def test_topk_invariants(scores, mask_seed, k):
    score = np.array(scores, np.float32)
    n = score.shape[0]
    valid = (np.random.default_rng(mask_seed).random(n) < 0.7).astype(np.uint8)
    idx, top, num = oracle.topk(valid, score, k)
    included = [i for i in range(n) if valid[i] and not np.isnan(score[i])]
    assert num == min(k, len(included))
    sel = idx[:num].tolist()
    assert len(set(sel)) == num and all(valid[i] and not np.isnan(score[i]) for i in sel)
    assert np.array_equal(top[:num], score[sel])
    for a, b in zip(sel, sel[1:]):
        assert score[a] > score[b] or (score[a] == score[b] and a < b)
    if num:
        last = sel[-1]
        chosen = set(sel)
        for j in included:
            if j not in chosen:
                assert score[j] < score[last] or (score[j] == score[last] and j > last)
    assert np.all(idx[num:] == -1) and np.all(top[num:] == -np.inf)
