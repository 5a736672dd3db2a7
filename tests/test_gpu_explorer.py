"""GPU parity of the explorer's rounds (ml2_explorer_*) through the C ABI
against the oracle's rounds: every round's proposed rows, their scores and
counts must be bit-identical, whether the round rescores the pool or reuses
the stored scores.  Inputs are seeded and synthetic."""
import sys

import numpy as np
import pytest

import gen
import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2411_10764_amd import ml2  # noqa: E402

DEV = "cuda:0"
THREADS = gen.default_threads()


def _note(msg):
    print(f"[gpu-explorer] {msg}", flush=True)
    sys.stdout.flush()


def run_rounds(V, P, A, X, k, keep, rescore_pattern, max_rounds=None):
    n = X.shape[0]
    Xd = torch.from_numpy(np.ascontiguousarray(X)).to(DEV)
    v, p = ml2.ml2_load_ensemble(V), ml2.ml2_load_ensemble(P)
    a = ml2.ml2_load_ensemble(A) if A is not None else None
    ex = ml2.Explorer(v, p, a, n, k, keep, max_rounds or len(rescore_pattern))
    idx = torch.empty(keep, dtype=torch.int32, device=DEV)
    top = torch.empty(keep, dtype=torch.float32, device=DEV)
    num = torch.empty(1, dtype=torch.int32, device=DEV)
    out = []
    for rescore in rescore_pattern:
        ex.round(Xd, idx, top, num, rescore=bool(rescore))
        torch.cuda.synchronize()
        out.append((idx.cpu().numpy().copy(), top.cpu().numpy().copy(), int(num.item())))
    assert ex.rounds == len(rescore_pattern)
    ex.free()
    return out


def compare(got, want):
    assert len(got) == len(want)
    for r, (g, w) in enumerate(zip(got, want)):
        assert np.array_equal(g[0], w[0]), f"round {r}: proposed rows differ"
        assert np.array_equal(g[1].view(np.uint32), w[1].view(np.uint32)), f"round {r}: scores"
        assert g[2] == w[2], f"round {r}: count"


def _models(seed, F, K, depth=6):
    V = gen.perfect_ensemble(seed, 1, 40, 5, K, K, 0.5)
    P = gen.perfect_ensemble(seed, 2, 50, depth, K, K, 0.1)
    A = gen.perfect_ensemble(seed, 3, 60, depth + 1, F, K, 0.1)
    return V, P, A


PATTERN = [1, 0, 0, 1, 0, 1, 0, 0, 0, 1, 0, 0]


def test_explorer_matches_oracle():
    n, F, K, k, keep = 4096, 32, 16, 20, 10
    V, P, A = _models(51, F, K)
    X = gen.features(51, n, F, K)
    _note(f"explorer n={n} k={k} keep={keep} rounds={len(PATTERN)}")
    got = run_rounds(V, P, A, X, k, keep, PATTERN)
    compare(got, oracle.explore(V, P, A, X, k, keep, len(PATTERN), THREADS))


def test_explorer_without_second_level():
    n, F, K, k, keep = 3000, 24, 12, 16, 6
    V, P, _ = _models(52, F, K)
    X = gen.features(52, n, F, K)
    got = run_rounds(V, P, None, X, k, keep, PATTERN)
    compare(got, oracle.explore(V, P, None, X, k, keep, len(PATTERN), THREADS))


@pytest.mark.parametrize("rescore", [0, 1])
def test_explorer_runs_dry(rescore):
    """Fewer accepted rows than rounds * keep: the last rounds are padded."""
    n, F, K, k, keep, rounds = 200, 16, 8, 12, 8, 20
    V, P, A = _models(53, F, K, depth=5)
    X = gen.features(53, n, F, K)
    pattern = [1] + [rescore] * (rounds - 1)
    got = run_rounds(V, P, A, X, k, keep, pattern)
    want = oracle.explore(V, P, A, X, k, keep, rounds, THREADS)
    assert want[-1][2] == 0, "the pool should run dry in this case"
    compare(got, want)


def test_explorer_reset_and_round_limit():
    n, F, K, k, keep = 1000, 16, 8, 10, 5
    V, P, A = _models(54, F, K, depth=5)
    X = gen.features(54, n, F, K)
    Xd = torch.from_numpy(X).to(DEV)
    v, p, a = (ml2.ml2_load_ensemble(e) for e in (V, P, A))
    ex = ml2.Explorer(v, p, a, n, k, keep, 2)
    idx = torch.empty(keep, dtype=torch.int32, device=DEV)
    top = torch.empty(keep, dtype=torch.float32, device=DEV)
    num = torch.empty(1, dtype=torch.int32, device=DEV)
    ex.round(Xd, idx, top, num)
    first = idx.cpu().numpy().copy()
    ex.round(Xd, idx, top, num, rescore=False)
    with pytest.raises(ml2.Ml2Error) as ei:
        ex.round(Xd, idx, top, num)
    assert ei.value.status == ml2.ML2_ERR_INVALID_ARG
    ex.reset()
    assert ex.rounds == 0
    ex.round(Xd, idx, top, num, rescore=False)  # no stored scores yet: it scores
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), first)
    bad = torch.zeros((n, K - 1), dtype=torch.float32, device=DEV)
    with pytest.raises(ml2.Ml2Error):
        ex.round(bad, idx, top, num)  # ld < the ensembles' feature count
    ex.free()
    for e in (v, p, a):
        e.free()


def test_explorer_create_errors():
    L = ml2.lib()
    V, P, A = _models(55, 16, 8, depth=4)
    v, p = ml2.ml2_load_ensemble(V), ml2.ml2_load_ensemble(P)
    h = __import__("ctypes").c_void_p()
    ref = __import__("ctypes").byref(h)
    assert L.ml2_explorer_create(v.handle, p.handle, None, 100, 5, 6, 3, ref) == \
        ml2.ML2_ERR_INVALID_ARG  # keep > k
    assert L.ml2_explorer_create(v.handle, p.handle, None, 0, 5, 2, 3, ref) == \
        ml2.ML2_ERR_INVALID_ARG  # empty pool
    assert L.ml2_explorer_create(v.handle, p.handle, None, 100, 5, 2, 0, ref) == \
        ml2.ML2_ERR_INVALID_ARG  # no rounds
    assert L.ml2_explorer_create(v.handle, p.handle, None, 100, ml2.ML2_MAX_TOPK + 1, 2, 3,
                                 ref) == ml2.ML2_ERR_UNSUPPORTED
    assert L.ml2_explorer_create(v.handle, None, None, 100, 5, 2, 3, ref) == \
        ml2.ML2_ERR_INVALID_ARG
    v.free()
    p.free()
