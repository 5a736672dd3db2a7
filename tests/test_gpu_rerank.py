"""GPU parity of the second level (model A re-rank, Section 2 "Hidden Feature
Extractor & ML Model A") through the C ABI against the CPU oracle: the row
scores, the kept rows and their scores must be bit-identical.  Inputs are
seeded and synthetic."""
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
    print(f"[gpu-rerank] {msg}", flush=True)
    sys.stdout.flush()


def _to_dev(X, ld=None):
    n, F = X.shape
    ld = F if ld is None else ld
    buf = torch.full((n * ld + 4,), float("nan"), dtype=torch.float32, device=DEV)
    view = buf[:n * ld].view(n, ld)
    if n:
        view[:, :F] = torch.from_numpy(np.ascontiguousarray(X)).to(DEV)
    return view


def rerank_gpu(A, Xd, rows, keep, a=None):
    m = rows.shape[0]
    own = a is None
    a = ml2.ml2_load_ensemble(A) if own else a
    if isinstance(rows, torch.Tensor):
        rows_d = rows.to(device=DEV, dtype=torch.int32)
    elif m:
        rows_d = torch.from_numpy(np.ascontiguousarray(rows, np.int32)).to(DEV)
    else:
        rows_d = torch.empty(1, dtype=torch.int32, device=DEV)
    rs = torch.full((max(m, 1),), 7.0, dtype=torch.float32, device=DEV)
    idx = torch.full((max(keep, 1),), -7, dtype=torch.int32, device=DEV)
    top = torch.empty(max(keep, 1), dtype=torch.float32, device=DEV)
    num = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    wsb = ml2.ml2_rerank_workspace_bytes(a, m)
    ws = torch.full((wsb // 4,), float("nan"), dtype=torch.float32, device=DEV)
    ml2.ml2_rerank(a, Xd, rows_d, keep, rs, idx, top, num, ws, wsb, m=m)
    torch.cuda.synchronize()
    out = (rs.cpu().numpy()[:m], idx.cpu().numpy()[:keep], top.cpu().numpy()[:keep],
           int(num.item()))
    if own:
        a.free()
    return out


def check_rerank(A, X, rows, keep, ld=None):
    Xd = _to_dev(X, ld)
    got = rerank_gpu(A, Xd, rows, keep)
    want = oracle.rerank(A, X, rows, keep)
    assert np.array_equal(got[0].view(np.uint32), want[0].view(np.uint32)), "row scores differ"
    assert np.array_equal(got[1], want[1]), "kept rows differ"
    assert np.array_equal(got[2].view(np.uint32), want[2].view(np.uint32)), "kept scores differ"
    assert got[3] == want[3]
    return got


def test_explorer_chain_tiny():
    """V and P on the visible columns -> top-(alpha+1)N -> A on all columns
    keeps N, every step on the GPU, against the oracle chain."""
    n, F, K, k, keep = 4096, 32, 16, 64, 32
    V = gen.perfect_ensemble(41, 1, 50, 5, K, K, 0.5)
    P = gen.perfect_ensemble(41, 2, 60, 6, K, K, 0.1)
    A = gen.perfect_ensemble(41, 3, 70, 7, F, K, 0.1)
    X = gen.features(41, n, F, K)
    _note(f"chain n={n} F={F} K={K} k={k} keep={keep}")
    Xd = _to_dev(X)
    v, p, a = (ml2.ml2_load_ensemble(e) for e in (V, P, A))
    pipe = ml2.Pipeline(v, p, n, k, device=DEV)
    pipe.run(Xd)
    got = rerank_gpu(A, Xd, pipe.idx, keep, a=a)
    want_chain = oracle.pipeline(V, P, X, k, THREADS)
    assert np.array_equal(pipe.idx.cpu().numpy(), want_chain["idx"])
    want = oracle.rerank(A, X, want_chain["idx"], keep)
    assert np.array_equal(got[0].view(np.uint32), want[0].view(np.uint32))
    assert np.array_equal(got[1], want[1])
    assert np.array_equal(got[2].view(np.uint32), want[2].view(np.uint32))
    assert got[3] == want[3] == keep
    for e in (v, p, a):
        e.free()


@pytest.mark.parametrize("case", ["skips", "duplicates", "pad", "keep0", "m0", "out_of_range"])
def test_rerank_edge_rows(case):
    rng = np.random.default_rng(7)
    n, F, K = 1000, 24, 12
    A = gen.perfect_ensemble(43, 3, 33, 6, F, K, 0.1)
    X = gen.features(43, n, F, K)
    rows, keep = {
        "skips": (np.array([5, -1, 17, -1, 999, 0], np.int32), 4),
        "duplicates": (np.array([3, 3, 3, 10, 10, 500], np.int32), 6),
        "pad": (rng.integers(0, n, 9).astype(np.int32), 20),
        "keep0": (rng.integers(0, n, 9).astype(np.int32), 0),
        "m0": (np.zeros(0, np.int32), 5),
        "out_of_range": (np.array([n, n + 5, -3, 2 ** 31 - 1, 1], np.int32), 3),
    }[case]
    _note(f"edge {case} m={rows.shape[0]} keep={keep}")
    check_rerank(A, X, rows, keep)


def test_rerank_empty_pool():
    A = gen.perfect_ensemble(44, 3, 10, 4, 8, 4, 0.1)
    Xd = torch.empty((0, 8), dtype=torch.float32, device=DEV)
    rs, idx, top, num = rerank_gpu(A, Xd, np.array([0, 1, -1], np.int32), 2)
    assert num == 0 and idx.tolist() == [-1, -1] and np.all(np.isneginf(top))
    assert np.all(np.isneginf(rs))


def test_rerank_max_list():
    """m = keep = ML2_MAX_TOPK (the largest single-workgroup sort)."""
    rng = np.random.default_rng(9)
    n, F, K = 20000, 16, 8
    A = gen.perfect_ensemble(45, 3, 20, 5, F, K, 0.1)
    X = gen.features(45, n, F, K)
    m = ml2.ML2_MAX_TOPK
    rows = rng.integers(-50, n, m).astype(np.int32)
    _note(f"max list m={m}")
    check_rerank(A, X, rows, m)


@pytest.mark.parametrize("m", [1, 20, 64, 65, 129, 200, 700, 5000])
def test_rerank_list_sizes(m):
    """List sizes that change the leaf walk's waves per workgroup (1..4), its
    row tiles and its tree-chunk size."""
    rng = np.random.default_rng(11 + m)
    n, F, K = 6000, 40, 20
    A = gen.perfect_ensemble(46, 3, 90, 7, F, K, 0.1)
    X = gen.features(46, n, F, K)
    rows = rng.integers(-2, n, m).astype(np.int32)
    _note(f"list m={m}")
    check_rerank(A, X, rows, min(m, 50))


@pytest.mark.parametrize("depth,F,ld", [(12, 128, 128), (12, 256, 256), (10, 64, 67), (8, 128, 130),
                                         (3, 5, 5), (1, 1, 1)])
def test_rerank_shapes(depth, F, ld):
    """The explorer's A shape (depth 12 over 128 columns), a ragged row stride,
    and a narrow pool."""
    rng = np.random.default_rng(depth)
    n = 2500
    A = gen.perfect_ensemble(47, 3, 24, depth, F, F // 2, 0.1)
    X = gen.features(47, n, F, F // 2)
    rows = rng.integers(0, n, 1024).astype(np.int32)
    _note(f"shape depth={depth} F={F} ld={ld}")
    check_rerank(A, X, rows, 512, ld=ld)


def test_rerank_argument_errors():
    L = ml2.lib()
    A = gen.perfect_ensemble(48, 3, 4, 3, 8, 4, 0.1)
    a = ml2.ml2_load_ensemble(A)
    X = torch.zeros((10, 8), dtype=torch.float32, device=DEV)
    buf = torch.zeros(64, dtype=torch.int32, device=DEV)
    P = buf.data_ptr()
    xp = X.data_ptr()
    s = torch.cuda.current_stream().cuda_stream
    wsb = ml2.ml2_rerank_workspace_bytes(a, 5)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=DEV)
    ok = dict(n=10, ld=8, rows=P, m=5, keep=3, rs=P, idx=P, sc=P, num=P, ws=ws.data_ptr(),
              wsb=wsb)

    def call(**kw):
        c = dict(ok, **kw)
        return L.ml2_rerank(a.handle, xp, c["n"], c["ld"], c["rows"], c["m"], c["keep"], c["rs"],
                            c["idx"], c["sc"], c["num"], c["ws"], c["wsb"], s)

    assert call(m=-1) == ml2.ML2_ERR_INVALID_ARG
    assert call(keep=-1) == ml2.ML2_ERR_INVALID_ARG
    assert call(ld=7) == ml2.ML2_ERR_INVALID_ARG
    assert call(num=None) == ml2.ML2_ERR_INVALID_ARG
    assert call(rows=None) == ml2.ML2_ERR_INVALID_ARG
    assert call(rs=None) == ml2.ML2_ERR_INVALID_ARG
    assert call(idx=None) == ml2.ML2_ERR_INVALID_ARG
    assert call(ws=None) == ml2.ML2_ERR_INVALID_ARG
    assert call(wsb=wsb - 1) == ml2.ML2_ERR_INVALID_ARG
    assert call(m=ml2.ML2_MAX_TOPK + 1) == ml2.ML2_ERR_UNSUPPORTED
    assert call(keep=ml2.ML2_MAX_TOPK + 1) == ml2.ML2_ERR_UNSUPPORTED
    assert L.ml2_rerank(None, xp, 10, 8, P, 5, 3, P, P, P, P, P, 1 << 20, s) == \
        ml2.ML2_ERR_INVALID_ARG
    with pytest.raises(ml2.Ml2Error) as ei:
        ml2.ml2_rerank_workspace_bytes(a, -1)
    assert ei.value.status == ml2.ML2_ERR_INVALID_ARG
    with pytest.raises(ml2.Ml2Error) as ei:
        ml2.ml2_rerank_workspace_bytes(a, ml2.ML2_MAX_TOPK + 1)
    assert ei.value.status == ml2.ML2_ERR_UNSUPPORTED
    assert ml2.ml2_rerank_workspace_bytes(a, 1000) >= 16 * 1000 * 4
    torch.cuda.synchronize()
    a.free()
