"""GPU parity of the explorer over a streamed pool (ml2_stream_explorer_*)
through the C ABI against the oracle's rounds over the distinct rows the
chunks carry: every round's proposed rows, their scores and counts must be
bit-identical.  The chunks come out of order, leave gaps, overlap (a row
arrives twice in a round) and pass through one device staging buffer that
is overwritten between chunks.  Inputs are seeded and synthetic."""
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
    print(f"[gpu-stream] {msg}", flush=True)
    sys.stdout.flush()


def run_stream(V, P, A, chunks, k, keep, rounds, max_rows=None):
    """Rounds over `chunks` [(row0, X_chunk)], each chunk copied into one
    staging buffer on the stream right before its call."""
    v, p = ml2.ml2_load_ensemble(V), ml2.ml2_load_ensemble(P)
    a = ml2.ml2_load_ensemble(A) if A is not None else None
    F = chunks[0][1].shape[1]
    max_rows = max_rows or max(1, max(c.shape[0] for _, c in chunks))
    ex = ml2.StreamExplorer(v, p, a, max_rows, k, keep, rounds)
    stage = torch.empty((max_rows, F), dtype=torch.float32, device=DEV)
    host = [(row0, torch.from_numpy(np.ascontiguousarray(c)).pin_memory()) for row0, c in chunks]
    idx = torch.empty(keep, dtype=torch.int32, device=DEV)
    top = torch.empty(keep, dtype=torch.float32, device=DEV)
    num = torch.empty(1, dtype=torch.int32, device=DEV)
    out = []
    for _ in range(rounds):
        ex.begin()
        for row0, hc in host:
            m = hc.shape[0]
            if m:
                stage[:m].copy_(hc, non_blocking=True)
            ex.chunk(stage[:m], row0)
        ex.end(idx, top, num)
        torch.cuda.synchronize()
        out.append((idx.cpu().numpy().copy(), top.cpu().numpy().copy(), int(num.item())))
    assert ex.rounds == rounds
    ex.free()
    return out


def compare(got, want):
    assert len(got) == len(want)
    for r, (g, w) in enumerate(zip(got, want)):
        assert np.array_equal(g[0], w[0]), f"round {r}: proposed rows differ"
        assert np.array_equal(g[1].view(np.uint32), w[1].view(np.uint32)), f"round {r}: scores"
        assert g[2] == w[2], f"round {r}: count"


def _models(seed, F, K):
    V = gen.perfect_ensemble(seed, 1, 40, 5, K, K, 0.5)
    P = gen.perfect_ensemble(seed, 2, 50, 6, K, K, 0.1)
    A = gen.perfect_ensemble(seed, 3, 60, 7, F, K, 0.1)
    return V, P, A


def _chunks(X, spans, base):
    """Chunks of X over [a, b) spans, pool rows base + a .."""
    return [(base + a, X[a:b]) for a, b in spans]


# out of order, gaps, an overlap (rows 300..359 arrive twice), an empty chunk,
# single-row chunks, a chunk smaller than k
SPANS = [(400, 700), (0, 10), (10, 11), (11, 360), (300, 400), (700, 700), (750, 1000),
         (1000, 1007)]


@pytest.mark.parametrize("with_a", [True, False])
def test_stream_matches_oracle(with_a):
    F, K, k, keep, rounds = 32, 16, 20, 10, 45
    V, P, A = _models(71, F, K)
    A = A if with_a else None
    X = gen.features(71, 1007, F, K)
    chunks = _chunks(X, SPANS, 123456)
    _note(f"stream with_a={with_a}: {len(chunks)} chunks, k={k} keep={keep} rounds={rounds}")
    got = run_stream(V, P, A, chunks, k, keep, rounds)
    want = oracle.explore_stream(V, P, A, chunks, k, keep, rounds, THREADS)
    compare(got, want)
    assert got[-1][2] == 0, "the pool should run dry within the rounds"


def test_stream_large_chunks_paper_k():
    """(alpha+1)N = 20 held and N = 10 kept over a 2^20-row pool in seven
    uneven chunks (two overlapping) of 128-feature rows, V and P on the 64
    knob columns, A on all 128."""
    F, K, n = 128, 64, 1 << 20
    V = gen.perfect_ensemble(72, 1, 300, 6, K, K, 0.5)
    P = gen.perfect_ensemble(72, 2, 300, 8, K, K, 0.1)
    A = gen.perfect_ensemble(72, 3, 300, 12, F, K, 0.1)
    X = gen.features(72, n, F, K)
    cuts = [0, 100000, 250000, 250001, 600000, 900000, n]
    spans = [(a, b) for a, b in zip(cuts, cuts[1:])] + [(550000, 650000)]
    chunks = _chunks(X, spans[::-1], 7)
    _note(f"stream large: {n} rows in {len(chunks)} chunks")
    got = run_stream(V, P, A, chunks, 20, 10, 4)
    compare(got, oracle.explore_stream(V, P, A, chunks, 20, 10, 4, THREADS))


def test_stream_ragged_models_missing_values():
    F, K = 40, 20
    V = gen.ragged_ensemble(73, 1, 60, 7, K, K, 0.5, base_score=0.3, max_nodes=200)
    P = gen.ragged_ensemble(73, 2, 80, 14, K, K, 0.1, max_nodes=300)
    A = gen.ragged_ensemble(73, 3, 90, 14, F, K, 0.1, max_nodes=300)
    X = gen.features(73, 3000, F, K, missing=0.1)
    chunks = _chunks(X, [(0, 1000), (2000, 3000), (900, 2100)], 0)
    got = run_stream(V, P, A, chunks, 64, 32, 12)
    compare(got, oracle.explore_stream(V, P, A, chunks, 64, 32, 12, THREADS))


def test_stream_largest_k():
    F, K = 16, 8
    V, P, A = _models(74, F, K)
    X = gen.features(74, 20000, F, K)
    chunks = _chunks(X, [(0, 9000), (9000, 20000)], 50)
    k = ml2.ML2_MAX_STREAM_K
    got = run_stream(V, P, A, chunks, k, 1000, 3)
    compare(got, oracle.explore_stream(V, P, A, chunks, k, 1000, 3, THREADS))


def test_stream_round_with_no_chunk():
    F, K = 16, 8
    V, P, A = _models(75, F, K)
    v, p, a = (ml2.ml2_load_ensemble(e) for e in (V, P, A))
    ex = ml2.StreamExplorer(v, p, a, 100, 8, 4, 2)
    idx = torch.full((4,), 5, dtype=torch.int32, device=DEV)
    top = torch.zeros(4, dtype=torch.float32, device=DEV)
    num = torch.full((1,), 9, dtype=torch.int32, device=DEV)
    ex.begin()
    ex.end(idx, top, num)
    torch.cuda.synchronize()
    assert int(num.item()) == 0 and idx.tolist() == [-1] * 4
    assert torch.all(torch.isneginf(top))
    ex.reset()
    assert ex.rounds == 0
    ex.free()


def test_stream_argument_errors():
    F, K = 16, 8
    V, P, A = _models(76, F, K)
    v, p, a = (ml2.ml2_load_ensemble(e) for e in (V, P, A))
    with pytest.raises(ml2.Ml2Error) as ei:
        ml2.StreamExplorer(v, p, a, 100, ml2.ML2_MAX_STREAM_K + 1, 4, 2)
    assert ei.value.status == ml2.ML2_ERR_UNSUPPORTED
    for args in ((0, 8, 4, 2), (100, 8, 9, 2), (100, 8, 4, 0)):
        with pytest.raises(ml2.Ml2Error) as ei:
            ml2.StreamExplorer(v, p, a, *args)
        assert ei.value.status == ml2.ML2_ERR_INVALID_ARG
    ex = ml2.StreamExplorer(v, p, a, 100, 8, 4, 1)
    X = torch.zeros((101, F), dtype=torch.float32, device=DEV)
    narrow = torch.zeros((10, F - 1), dtype=torch.float32, device=DEV)
    idx = torch.empty(4, dtype=torch.int32, device=DEV)
    top = torch.empty(4, dtype=torch.float32, device=DEV)
    num = torch.empty(1, dtype=torch.int32, device=DEV)
    bad = [lambda: ex.chunk(X[:10], 0),                  # no round open
           lambda: ex.end(idx, top, num)]                # no round open
    for call in bad:
        with pytest.raises(ml2.Ml2Error) as ei:
            call()
        assert ei.value.status == ml2.ML2_ERR_INVALID_ARG
    ex.begin()
    with pytest.raises(ml2.Ml2Error):
        ex.begin()                                       # already open
    for call in (lambda: ex.chunk(X, 0),                 # more rows than max_chunk_rows
                 lambda: ex.chunk(X[:10], -1),           # negative row0
                 lambda: ex.chunk(X[:10], (1 << 31) - 5),  # rows beyond 2^31 - 1
                 lambda: ex.chunk(narrow, 0)):           # row stride below A's features
        with pytest.raises(ml2.Ml2Error) as ei:
            call()
        assert ei.value.status == ml2.ML2_ERR_INVALID_ARG
    ex.chunk(X[:10], 0)
    ex.end(idx, top, num)
    with pytest.raises(ml2.Ml2Error):
        ex.begin()                                       # every round used
    torch.cuda.synchronize()
    ex.free()
