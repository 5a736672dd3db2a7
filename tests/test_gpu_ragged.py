"""GPU parity of the ragged layout (Table 3's deep models: 300 rounds up to
depth 14, with XGBoost's per-node default directions for missing values)
through the C ABI against the CPU oracle, bit for bit.  Inputs are seeded and
synthetic; missing values are NaN in the hidden columns."""
import json
import os
import sys

import numpy as np
import pytest

import gen
import oracle
from tests.test_gpu_parity import check_pipeline
from tests.test_gpu_rerank import check_rerank

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2411_10764_amd import ml2  # noqa: E402
from paper_2411_10764_amd.xgboost_json import load_xgboost_json  # noqa: E402

DEV = "cuda:0"
THREADS = gen.default_threads()
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _note(msg):
    print(f"[gpu-ragged] {msg}", flush=True)
    sys.stdout.flush()


def _paper_models(seed, F, K, trees=300, depth=14, max_nodes=400):
    V = gen.perfect_ensemble(seed, 1, trees, 5, K, K, 0.5)
    P = gen.ragged_ensemble(seed, 2, trees, depth, K, K, 0.1, max_nodes=max_nodes)
    A = gen.ragged_ensemble(seed, 3, trees, depth, F, K, 0.1, max_nodes=max_nodes)
    return V, P, A


def test_depth_reported():
    V, P, A = _paper_models(61, 32, 16, trees=40)
    for e in (V, P, A):
        h = ml2.ml2_load_ensemble(e)
        want = max(int(max(_depth(e, t) for t in range(e.num_trees))), 1)
        assert h.depth == want
        h.free()


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


def test_paper_shaped_pipeline_with_missing_values():
    n, F, K = 6000, 32, 16
    V, _, A = _paper_models(62, F, K)
    # P on all columns here so that the missing values reach a ragged model
    P = gen.ragged_ensemble(62, 2, 300, 14, F, K, 0.1, max_nodes=400)
    X = gen.features(62, n, F, K, missing=0.1)
    _note(f"paper-shaped pipeline n={n} F={F}")
    check_pipeline(V, P, X, 64)
    rows = np.arange(0, n, 7, dtype=np.int32)
    check_rerank(A, X, rows, 100)


@pytest.mark.parametrize("split,waves,nbuf,group", [
    (1, 4, 1, 0), (1, 8, 1, 0), (2, 8, 1, 0), (1, 4, 2, 0), (2, 4, 1, 0), (1, 2, 1, 0),
    (1, 8, 1, 1), (1, 8, 1, 2), (1, 4, 2, 4), (2, 8, 1, 1), (2, 8, 1, 2)])
def test_ragged_plans(tune, split, waves, nbuf, group):
    """Launch shapes of the ragged walks; group 0 leaves the trees per lane
    to the planner."""
    for key, val in (("SPLIT", split), ("WAVES", waves), ("NBUF", nbuf), ("GROUP", group)):
        if val:
            tune(**{key.lower(): val})
    n, F, K = 3000, 40, 20
    V = gen.ragged_ensemble(63, 1, 60, 9, F, K, 0.5, base_score=0.2, max_nodes=300)
    P = gen.ragged_ensemble(63, 2, 90, 14, F, K, 0.1, max_nodes=300)
    X = gen.features(63, n, F, K, missing=0.2)
    _note(f"ragged plan S={split} W={waves} nbuf={nbuf} G={group}")
    check_pipeline(V, P, X, 50)


@pytest.mark.parametrize("split,group", [(0, 0), (1, 2), (1, 4), (2, 0), (2, 1)])
def test_ragged_shallow_trees(tune, split, group):
    """Shallow trees (one to three splits; walks that end after a step or
    two, lanes that run through a slot's trees in a few steps, single-leaf
    padding trees after P's 37), V a slot of exactly four trees; the default
    plan, groups of two and four trees per lane, and two lanes per
    candidate."""
    for key, val in (("SPLIT", split), ("GROUP", group)):
        if val:
            tune(**{key.lower(): val})
    n, F, K = 2500, 24, 12
    V = gen.ragged_ensemble(66, 1, 4, 3, F, K, 0.5, base_score=0.1, p_split=0.3)
    P = gen.ragged_ensemble(66, 2, 37, 6, F, K, 0.1, p_split=0.3, decay=0.5)
    X = gen.features(66, n, F, K, missing=0.1)
    _note(f"shallow ragged S={split} G={group}: P trees of "
          f"{int(np.diff(P.offsets).max())} nodes at most")
    check_pipeline(V, P, X, 30)


@pytest.mark.parametrize("split", [1, 2])
def test_ragged_widest_rows(tune, split):
    """256 features: the node word's feature byte offset reaches 255 x 256
    (one lane per candidate) and its half (two lanes per candidate)."""
    tune(split=split)
    n, F, K = 1500, 256, 128
    V = gen.ragged_ensemble(67, 1, 20, 9, F, K, 0.5, base_score=0.1, max_nodes=200)
    P = gen.ragged_ensemble(67, 2, 30, 12, F, K, 0.1, max_nodes=300)
    feats = np.concatenate([V.feature[V.left >= 0], P.feature[P.left >= 0]])
    assert feats.max() >= 250, "the trees should split on the last features"
    X = gen.features(67, n, F, K, missing=0.1)
    _note(f"ragged F=256 S={split}: largest split feature {int(feats.max())}")
    check_pipeline(V, P, X, 25)


@pytest.mark.parametrize("seed", range(12))
def test_ragged_random_shapes(tune, seed):
    """Seeded random ragged ensembles, feature counts, pool sizes (ragged
    tails), missing fractions and launch shapes (lanes per candidate, trees
    per lane), each against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    F = int(rng.integers(1, 201))
    K = int(rng.integers(0, F + 1))
    n = int(rng.integers(1, 5000))
    split = int(rng.choice([0, 1, 2]))
    group = int(rng.choice([0, 1, 2, 4])) if split != 2 else int(rng.choice([0, 1, 2]))
    for key, val in (("SPLIT", split), ("GROUP", group)):
        if val:
            tune(**{key.lower(): val})
    V = gen.ragged_ensemble(2000 + seed, 1, int(rng.integers(1, 60)), int(rng.integers(1, 16)),
                            F, K, 0.5, base_score=float(rng.normal(0, 0.5)),
                            p_split=float(rng.uniform(0.5, 1.0)), max_nodes=int(rng.integers(3, 600)))
    P = gen.ragged_ensemble(2000 + seed, 2, int(rng.integers(1, 120)), int(rng.integers(1, 16)),
                            F, K, 0.1, p_split=float(rng.uniform(0.5, 1.0)),
                            max_nodes=int(rng.integers(3, 600)))
    X = gen.features(2000 + seed, n, F, K, missing=float(rng.choice([0.0, 0.05, 0.3])))
    k = int(rng.integers(0, 200))
    _note(f"random ragged seed={seed} F={F} K={K} n={n} S={split} G={group} "
          f"V={V.num_trees} P={P.num_trees} k={k}")
    check_pipeline(V, P, X, k)


def test_forced_ragged_layout_on_perfect_trees(tune):
    """Perfect trees packed into ragged slots give the same results."""
    tune(layout=2)
    w = gen.WORKLOADS["tiny"]
    check_pipeline(w.validity(), w.perf(), w.features(), w.k)


@pytest.mark.parametrize("max_nodes,depth", [(ml2.ML2_MAX_TREE_NODES, 32), (2041, 13),
                                             (7, 3)])
def test_ragged_tree_sizes(max_nodes, depth):
    n, F, K = 2000, 24, 12
    V = gen.ragged_ensemble(64, 1, 9, depth, F, K, 0.5, p_split=0.97, decay=0.99,
                            max_nodes=max_nodes)
    P = gen.ragged_ensemble(64, 2, 13, depth, F, K, 0.1, p_split=0.97, decay=0.99,
                            max_nodes=max_nodes)
    X = gen.features(64, n, F, K, missing=0.05)
    _note(f"ragged sizes max_nodes={max_nodes} depth<={depth} "
          f"largest tree {int(np.diff(P.offsets).max())} nodes")
    check_pipeline(V, P, X, 40)


def test_xgboost_fixture_on_gpu():
    with open(os.path.join(GOLDEN, "xgboost_small.json")) as fh:
        model = json.load(fh)
    with open(os.path.join(GOLDEN, "xgboost_small_expected.json")) as fh:
        exp = json.load(fh)
    X = np.array([[np.nan if v == "nan" else v for v in row] for row in exp["inputs"]],
                 np.float32)
    e = ml2.ml2_load_ensemble(load_xgboost_json(model))
    Xd = torch.from_numpy(X).to(DEV)
    valid = torch.empty(X.shape[0], dtype=torch.uint8, device=DEV)
    margin = torch.empty(X.shape[0], dtype=torch.float32, device=DEV)
    ml2.ml2_score_validity(e, Xd, valid, margin)
    torch.cuda.synchronize()
    assert margin.cpu().numpy().tolist() == exp["margins"]
    e.free()


def test_explorer_with_ragged_models():
    n, F, K, k, keep = 4000, 32, 16, 20, 10
    V, P, A = _paper_models(65, F, K, trees=100)
    X = gen.features(65, n, F, K, missing=0.1)
    from tests.test_gpu_explorer import compare, run_rounds
    pattern = [1, 0, 0, 1, 0, 0]
    got = run_rounds(V, P, A, X, k, keep, pattern)
    compare(got, oracle.explore(V, P, A, X, k, keep, len(pattern), THREADS))
