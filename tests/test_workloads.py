"""The seeded input generator: determinism, shapes, distributions, and the
calibrated validity biases."""
import numpy as np
import pytest

import gen


def test_thread_count_independent():
    w = gen.WORKLOADS["medium"]
    a = gen.features(w.seed, 3000, w.F, w.K, threads=1)
    b = gen.features(w.seed, 3000, w.F, w.K, threads=7)
    assert np.array_equal(a, b)


def test_row_selection_matches_contiguous_rows():
    w = gen.WORKLOADS["large"]
    rows = np.array([0, 5, 4095, 123456, w.n - 1], np.int64)
    sel = w.features(rows=rows)
    for j, r in enumerate(rows):
        one = gen.features(w.seed, 1, w.F, w.K, row0=int(r))
        assert np.array_equal(sel[j], one[0])


def test_padded_stride_leaves_tail_columns():
    w = gen.WORKLOADS["tiny"]
    X = gen.features(w.seed, 10, w.F, w.K, ld=w.F + 3)
    assert X.shape == (10, w.F + 3)
    assert np.all(X[:, w.F:] == 0)
    assert np.array_equal(X[:, :w.F], gen.features(w.seed, 10, w.F, w.K))


def test_feature_distributions():
    w = gen.WORKLOADS["medium"]
    X = gen.features(w.seed, 20000, w.F, w.K)
    knobs = X[:, :w.K]
    assert np.all(knobs == np.round(knobs)) and knobs.min() == 0 and knobs.max() == 8
    counts = np.bincount(knobs.astype(np.int64).ravel(), minlength=9) / knobs.size
    assert np.all(np.abs(counts - 1 / 9) < 0.005)
    z = np.log(X[:, w.K:].astype(np.float64))
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01


def test_perfect_tree_shape():
    e = gen.perfect_ensemble(9, 2, 5, 4, 10, 4, 0.1)
    nodes = 31
    assert e.offsets.tolist() == [i * nodes for i in range(6)]
    for t in range(5):
        b = t * nodes
        for i in range(nodes):
            if i < 15:
                assert e.left[b + i] == 2 * i + 1 and e.right[b + i] == 2 * i + 2
                f = e.feature[b + i]
                assert 0 <= f < 10
                if f < 4:
                    assert e.threshold[b + i] in np.arange(9, dtype=np.float32)
                else:
                    assert e.threshold[b + i] > 0
            else:
                assert e.left[b + i] == -1 and e.right[b + i] == -1


def test_leaf_scales():
    v = gen.perfect_ensemble(3, 1, 200, 6, 64, 32, 0.5)
    p = gen.perfect_ensemble(3, 2, 200, 6, 64, 32, 0.1)
    lv = v.value[v.left < 0].astype(np.float64)
    lp = p.value[p.left < 0].astype(np.float64)
    assert abs(lv.std() - 0.5) < 0.02 and abs(lp.std() - 0.1) < 0.004


def test_streams_differ():
    a = gen.perfect_ensemble(4, 1, 3, 3, 8, 4, 0.5)
    b = gen.perfect_ensemble(4, 2, 3, 3, 8, 4, 0.5)
    assert not np.array_equal(a.value, b.value)


@pytest.mark.parametrize("name", ["medium", "skewed"])
def test_calibrated_bias_reproduces(name):
    from oracle.calibrate_base import calibrated_base
    w = gen.WORKLOADS[name]
    assert calibrated_base(w) == w.base_v
