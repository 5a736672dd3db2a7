"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Masks, top-k indices and scores must be bit-identical to the oracle (the
fold order is fixed, so scores are expected at 0 ulp; the accepted bar for
scores is |gpu - oracle| <= 1e-5 * max(|oracle|, 1), and anything above
0 ulp is reported).  Inputs are seeded and synthetic.
"""
import math
import sys

import numpy as np
import pytest

import gen
import oracle
from tests.treeutil import ensemble_from_trees, random_ragged_ensemble

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2411_10764_amd import ml2  # noqa: E402

DEV = "cuda:0"
THREADS = gen.default_threads()


def _note(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


def _to_dev(X, ld=None, offset=0):
    """Device copy of X with row stride ld (>= F) and the first row `offset`
    floats into the allocation (offset 1 breaks 16-byte alignment)."""
    n, F = X.shape
    ld = F if ld is None else ld
    buf = torch.full((offset + n * ld + 4,), float("nan"), dtype=torch.float32, device=DEV)
    view = buf[offset:offset + n * ld].view(n, ld) if n else buf[offset:offset].view(0, ld)
    if n:
        view[:, :F] = torch.from_numpy(np.ascontiguousarray(X)).to(DEV)
    return view


def run_gpu(V, P, X, k, ld=None, offset=0, perf_mask=True):
    n = X.shape[0]
    Xd = _to_dev(X, ld, offset)
    v = ml2.ml2_load_ensemble(V)
    p = ml2.ml2_load_ensemble(P)
    valid = torch.empty(max(n, 1), dtype=torch.uint8, device=DEV)
    margin = torch.empty(max(n, 1), dtype=torch.float32, device=DEV)
    score = torch.empty(max(n, 1), dtype=torch.float32, device=DEV)
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=DEV)
    top = torch.empty(max(k, 1), dtype=torch.float32, device=DEV)
    num = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    wsb = ml2.ml2_topk_workspace_bytes(n, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    ml2.ml2_score_validity(v, Xd, valid, margin)
    ml2.ml2_score_perf(p, Xd, valid if perf_mask else None, score)
    ml2.ml2_filter_topk(valid if perf_mask else None, score, k, idx, top, num, ws, wsb, n)
    torch.cuda.synchronize()
    out = dict(valid=valid.cpu().numpy()[:n], margin=margin.cpu().numpy()[:n],
               score=score.cpu().numpy()[:n], idx=idx.cpu().numpy()[:k],
               top=top.cpu().numpy()[:k], num=int(num.item()))
    v.free()
    p.free()
    return out


def assert_scores(got, want, what):
    same = (got.view(np.uint32) == want.view(np.uint32)) | (np.isnan(got) & np.isnan(want))
    if not np.all(same):
        bad = np.flatnonzero(~same)
        tol = 1e-5 * np.maximum(np.abs(want[bad].astype(np.float64)), 1.0)
        err = np.abs(got[bad].astype(np.float64) - want[bad].astype(np.float64))
        _note(f"{what}: {bad.size} entries differ from the oracle above 0 ulp "
              f"(max abs err {err.max():.3g})")
        assert np.all(err <= tol), f"{what}: {int((err > tol).sum())} entries beyond 1e-5 rel"


def check_pipeline(V, P, X, k, **kw):
    got = run_gpu(V, P, X, k, **kw)
    perf_mask = kw.get("perf_mask", True)
    valid, margin = oracle.validity(V, X, THREADS)
    score = oracle.perf(P, X, valid if perf_mask else None, THREADS)
    idx, top, num = oracle.topk(valid if perf_mask else None, score, k)
    assert np.array_equal(got["valid"], valid), "validity mask differs"
    assert_scores(got["margin"], margin, "margin")
    assert_scores(got["score"], score, "score")
    assert got["num"] == num
    assert np.array_equal(got["idx"], idx), "top-k indices differ"
    assert np.array_equal(got["top"].view(np.uint32), top.view(np.uint32)), "top-k scores differ"
    return got


# ---- the workloads ---------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny", "medium"])
def test_workload_exact(name):
    w = gen.WORKLOADS[name]
    _note(f"{name}: n={w.n} F={w.F} V={w.v_trees}x{w.v_depth} P={w.p_trees}x{w.p_depth} k={w.k}")
    X = w.features()
    got = check_pipeline(w.validity(), w.perf(), X, w.k)
    _note(f"{name}: invalid fraction {1 - got['valid'].mean():.4f}, top-k exact")


def test_golden_hand_pipeline():
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_pipeline.json")))

    def tree(node):
        return (int(node[0]), float(node[1]), tree(node[2]), tree(node[3])) \
            if isinstance(node, list) else float(node)

    V = ensemble_from_trees([tree(t) for t in g["validity"]["trees"]], 3, g["validity"]["base"])
    P = ensemble_from_trees([tree(t) for t in g["perf"]["trees"]], 3, g["perf"]["base"])
    X = np.array([[float(v) for v in r] for r in g["candidates"]], np.float32)
    for k in ("2", "5", "0"):
        got = run_gpu(V, P, X, int(k))
        e = g["expected"]
        assert np.array_equal(got["margin"], np.array(e["margin"], np.float32))
        assert np.array_equal(got["valid"], np.array(e["valid"], np.uint8))
        assert np.array_equal(got["score"], np.array([float(s) for s in e["score"]], np.float32))
        assert got["num"] == e["topk"][k]["num"]
        assert got["idx"].tolist() == e["topk"][k]["idx"]


def test_order_witness():
    import json
    import os
    cases = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                        "order_witness.json")))["cases"]
    for c in cases:
        V = ensemble_from_trees([float(v) for v in c["leaves"]], 1, c["base"])
        got = run_gpu(V, V, np.zeros((70, 1), np.float32), 3)
        assert np.all(got["margin"] == np.float32(c["margin"]))
        assert np.all(got["valid"] == c["valid"])


# ---- ragged trees, special values, shapes ------------------------------------------

def _special_features(rng, n, F, K):
    X = np.empty((n, F), np.float32)
    X[:, :K] = rng.integers(0, 9, size=(n, K))
    X[:, K:] = np.exp(rng.normal(0, 1, size=(n, F - K)))
    r = rng.random((n, F))
    X[r < 0.03] = np.nan
    X[(r >= 0.03) & (r < 0.05)] = -0.0
    X[(r >= 0.05) & (r < 0.06)] = np.float32(2.0 ** -140)        # subnormal
    X[(r >= 0.06) & (r < 0.07)] = np.inf
    X[(r >= 0.07) & (r < 0.08)] = -np.inf
    return X


def _thr_sampler(K):
    def f(r, feat):
        u = r.random()
        if u < 0.05:
            return float(2.0 ** -140)
        if u < 0.08:
            return 0.0
        if u < 0.10:
            return float("inf")
        return float(r.integers(0, 9)) if feat < K else float(np.float32(np.exp(r.normal())))
    return f


@pytest.mark.parametrize("seed,n,F,depth,trees", [
    (1, 1, 5, 3, 3), (2, 63, 7, 5, 17), (3, 64, 16, 6, 9), (4, 65, 33, 7, 30),
    (5, 257, 64, 9, 12), (6, 5000, 40, 4, 41), (7, 3000, 96, 10, 6), (8, 700, 128, 8, 25),
])
def test_ragged_trees_and_special_values(seed, n, F, depth, trees):
    rng = np.random.default_rng(seed)
    K = F // 2
    V = random_ragged_ensemble(rng, trees, depth, F, _thr_sampler(K),
                               lambda r: float(np.float32(r.normal(0, 0.5))), p_split=0.8,
                               base=float(np.float32(rng.normal(0, 0.3))))
    P = random_ragged_ensemble(rng, trees + 3, depth, F, _thr_sampler(K),
                               lambda r: float(np.float32(r.normal(0, 0.1))), p_split=0.8)
    X = _special_features(rng, n, F, K)
    _note(f"ragged seed={seed} n={n} F={F} depth<={depth}")
    check_pipeline(V, P, X, min(n, 37))


@pytest.mark.parametrize("ld,offset", [(None, 0), (70, 0), (64, 1), (67, 3)])
def test_strides_and_alignment(ld, offset):
    w = gen.WORKLOADS["tiny"]
    X = w.features()[:1000]
    _note(f"stride ld={ld} offset={offset}")
    check_pipeline(w.validity(), w.perf(), X, 50, ld=ld, offset=offset)


@pytest.mark.parametrize("depth,F,trees", [(1, 1, 5), (1, 256, 40), (11, 8, 3), (12, 256, 2),
                                           (6, 256, 33)])
def test_depth_and_width_limits(depth, F, trees):
    V = gen.perfect_ensemble(21, 1, trees, depth, F, F // 2, 0.5)
    P = gen.perfect_ensemble(21, 2, trees, depth, F, F // 2, 0.1)
    X = gen.features(21, 1500, F, F // 2)
    _note(f"limits depth={depth} F={F} trees={trees}")
    check_pipeline(V, P, X, 100)


@pytest.mark.parametrize("split,group,waves,nbuf,chunk,depth", [
    (1, 4, 4, 1, 0, 7), (1, 8, 8, 1, 0, 7), (1, 8, 4, 2, 0, 7), (1, 8, 4, 1, 16, 7),
    (2, 8, 8, 1, 0, 7), (2, 4, 8, 1, 16, 7), (2, 4, 4, 1, 0, 7), (2, 8, 8, 1, 32, 7),
    (2, 4, 8, 1, 16, 6), (2, 2, 8, 1, 0, 8), (2, 1, 8, 1, 0, 9), (2, 1, 8, 1, 0, 10),
    (1, 4, 6, 1, 0, 10), (1, 2, 8, 1, 0, 10), (1, 4, 8, 1, 0, 10), (1, 2, 6, 1, 0, 11),
])
def test_walk_plans(tune, split, group, waves, nbuf, chunk, depth):
    """Every launch shape of the walks (lanes per candidate, trees per lane,
    waves, staging mode, chunk size), forced through the tuning overrides."""
    for key, val in (("SPLIT", split), ("GROUP", group), ("WAVES", waves), ("NBUF", nbuf),
                     ("CHUNK", chunk)):
        tune(**{key.lower(): val})
    F, K = 40, 20
    V = gen.perfect_ensemble(31, 1, 70, depth, F, K, 0.5)
    P = gen.perfect_ensemble(31, 2, 90, depth, F, K, 0.1)
    X = gen.features(31, 3001, F, K)
    _note(f"plan S={split} G={group} W={waves} nbuf={nbuf} chunk={chunk} depth={depth}")
    check_pipeline(V, P, X, 64)


@pytest.mark.parametrize("seed", range(12))
def test_perfect_random_shapes(tune, seed):
    """Seeded random perfect ensembles (depth 1..12), feature counts, row
    strides and alignment, pool sizes and launch plans (overrides that do not
    fit are ignored by the planner), each against the oracle."""
    rng = np.random.default_rng(3000 + seed)
    depth = int(rng.integers(1, 13))
    F = int(rng.integers(1, 257))
    K = int(rng.integers(0, F + 1))
    n = int(rng.integers(1, 4000))
    ld = F + int(rng.choice([0, 0, 1, 3, 4]))
    offset = int(rng.choice([0, 0, 1]))
    for key, choices in (("SPLIT", [0, 1, 2]), ("GROUP", [0, 1, 2, 4, 8]), ("WAVES", [0, 4, 8]),
                         ("NBUF", [0, 1, 2]), ("CHUNK", [0, 0, 16, 32])):
        val = int(rng.choice(choices))
        if val:
            tune(**{key.lower(): val})
    tv = int(rng.integers(1, 80)) if depth <= 9 else int(rng.integers(1, 12))
    tp = int(rng.integers(1, 80)) if depth <= 9 else int(rng.integers(1, 12))
    V = gen.perfect_ensemble(4000 + seed, 1, tv, depth, F, K, 0.5, float(rng.normal(0, 0.3)))
    P = gen.perfect_ensemble(4000 + seed, 2, tp, depth, F, K, 0.1)
    X = gen.features(4000 + seed, n, F, K)
    k = int(rng.integers(0, 300))
    _note(f"random perfect seed={seed} depth={depth} F={F} ld={ld} offset={offset} n={n} "
          f"V={tv} P={tp} k={k}")
    check_pipeline(V, P, X, k, ld=ld, offset=offset)


@pytest.mark.parametrize("F,ld,trees", [(40, 40, 30), (128, 128, 48), (128, 131, 20),
                                         (132, 132, 16), (6, 6, 1)])
def test_resident_ensemble(tune, F, ld, trees):
    """Ensembles that fit one chunk (never restaged) with two lanes per
    candidate: rows prefetched whole into the staging registers where they
    are aligned and at most 128 wide, loaded directly otherwise."""
    tune(split=2)
    K = max(F // 2, 1)
    V = gen.perfect_ensemble(33, 1, trees, 5, F, K, 0.5)
    P = gen.perfect_ensemble(33, 2, trees, 4, F, K, 0.1)
    X = gen.features(33, 5003, F, K)
    _note(f"resident F={F} ld={ld} trees={trees}")
    check_pipeline(V, P, X, 40, ld=ld)


@pytest.mark.parametrize("F", [72, 96, 124, 128])
def test_row_widths_two_lanes(tune, F):
    """Two lanes per candidate with the ensemble streamed in several chunks:
    row widths whose last line-batch is partial (the validity walk's halves
    share each line, the perf walk's halves take alternate lines)."""
    tune(split=2)
    K = F // 2
    V = gen.perfect_ensemble(34, 1, 160, 6, F, K, 0.5)
    P = gen.perfect_ensemble(34, 2, 120, 7, F, K, 0.1)
    X = gen.features(34, 7001, F, K)
    _note(f"row width F={F} (two lanes per candidate, streamed)")
    check_pipeline(V, P, X, 64)


def test_perf_without_mask():
    w = gen.WORKLOADS["tiny"]
    check_pipeline(w.validity(), w.perf(), w.features(), 64, perf_mask=False)


def test_empty_pool():
    w = gen.WORKLOADS["tiny"]
    got = run_gpu(w.validity(), w.perf(), np.zeros((0, w.F), np.float32), 5)
    assert got["num"] == 0 and got["idx"].tolist() == [-1] * 5
    assert np.all(got["top"] == -np.inf)


# ---- selection edge cases ----------------------------------------------------------

def _topk_gpu(valid, score, k):
    n = score.shape[0]
    s = torch.from_numpy(score).to(DEV) if n else torch.empty(1, device=DEV)
    v = torch.from_numpy(valid).to(DEV) if valid is not None and n else None
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=DEV)
    top = torch.empty(max(k, 1), dtype=torch.float32, device=DEV)
    num = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    wsb = ml2.ml2_topk_workspace_bytes(n, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    ml2.ml2_filter_topk(v, s, k, idx, top, num, ws, wsb, n)
    torch.cuda.synchronize()
    return idx.cpu().numpy()[:k], top.cpu().numpy()[:k], int(num.item())


def _check_topk(valid, score, k):
    gi, gt, gn = _topk_gpu(valid, score, k)
    oi, ot, on = oracle.topk(valid, score, k)
    assert gn == on
    assert np.array_equal(gi, oi)
    assert np.array_equal(gt.view(np.uint32), ot.view(np.uint32))


@pytest.mark.parametrize("case", ["constant", "dups", "signed_zero", "nan", "few_valid",
                                  "k_zero", "k_max", "no_mask", "all_invalid", "extremes"])
def test_topk_edge_cases(case):
    rng = np.random.default_rng(sum(map(ord, case)))
    n, k = 100000, 300
    score = rng.normal(0, 1, n).astype(np.float32)
    valid = (rng.random(n) < 0.5).astype(np.uint8)
    if case == "constant":
        score[:] = 0.75
    elif case == "dups":
        score = (rng.integers(0, 5, n) * 0.5).astype(np.float32)
    elif case == "signed_zero":
        score[:] = 0.0
        score[rng.random(n) < 0.5] = -0.0
    elif case == "nan":
        score[rng.random(n) < 0.3] = np.nan
    elif case == "few_valid":
        valid[:] = 0
        valid[rng.choice(n, 17, replace=False)] = 1
    elif case == "k_zero":
        k = 0
    elif case == "k_max":
        k = ml2.ML2_MAX_TOPK
    elif case == "no_mask":
        valid = None
    elif case == "all_invalid":
        valid[:] = 0
    elif case == "extremes":
        score[rng.random(n) < 0.2] = -np.inf
        score[rng.random(n) < 0.2] = np.inf
        score[rng.random(n) < 0.1] = np.float32(1e-45)
    _check_topk(valid, score, k)


@pytest.mark.parametrize("n", [1, 2, 255, 256, 257, 4096, 1 << 20])
def test_topk_sizes(n):
    rng = np.random.default_rng(n)
    score = rng.normal(0, 1, n).astype(np.float32)
    valid = (rng.random(n) < 0.7).astype(np.uint8)
    for k in (1, 33, 1024):
        _check_topk(valid, score, k)


def test_repeatable_across_streams():
    w = gen.WORKLOADS["medium"]
    X = torch.from_numpy(w.features()).to(DEV)
    v, p = ml2.ml2_load_ensemble(w.validity()), ml2.ml2_load_ensemble(w.perf())
    outs = []
    for s in (torch.cuda.Stream(), torch.cuda.current_stream()):
        with torch.cuda.stream(s):
            pipe = ml2.Pipeline(v, p, w.n, w.k, device=DEV, with_margin=True)
            pipe.run(X)
        s.synchronize()
        outs.append([t.cpu().numpy().copy() for t in (pipe.valid, pipe.margin, pipe.score,
                                                      pipe.idx, pipe.top, pipe.num)])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


# ---- full-size workloads: every row against the oracle ------------------------------

def _second_level_check(w, X, Xd, idx, num):
    """Model A over the GPU's held rows, on the GPU and in the oracle."""
    A = w.second_level()
    a = ml2.ml2_load_ensemble(A)
    m = w.k
    rows = torch.from_numpy(idx.astype(np.int32)).to(DEV)
    row_scores = torch.empty(m, dtype=torch.float32, device=DEV)
    out_idx = torch.empty(w.keep, dtype=torch.int32, device=DEV)
    out_top = torch.empty(w.keep, dtype=torch.float32, device=DEV)
    out_num = torch.empty(1, dtype=torch.int32, device=DEV)
    wsb = ml2.ml2_rerank_workspace_bytes(a, m)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    ml2.ml2_rerank(a, Xd, rows, w.keep, row_scores, out_idx, out_top, out_num, ws, wsb, m=m)
    torch.cuda.synchronize()
    o_rs, o_idx, o_top, o_num = oracle.rerank(A, X, idx.astype(np.int32), w.keep)
    assert_scores(row_scores.cpu().numpy(), o_rs, "model A scores of the held rows")
    assert int(out_num.item()) == o_num
    assert np.array_equal(out_idx.cpu().numpy(), o_idx), "model A's kept rows differ"
    assert np.array_equal(out_top.cpu().numpy().view(np.uint32), o_top.view(np.uint32))
    a.free()


@pytest.mark.slow
@pytest.mark.parametrize("name", ["large", "roofline", "skewed", "hbm", "paper", "explorer"])
def test_full_size_whole_pool(name):
    """Every row of the full-size pool against the oracle: mask bytes,
    margins and scores bit for bit, and the top-k (indices, scores, count)
    equal to the oracle's selection over the oracle's own scores."""
    import time
    w = gen.WORKLOADS[name]
    _note(f"{name}: generating {w.n} x {w.F} features on the host")
    X = w.features()
    V, P = w.validity(), w.perf()
    Xd = torch.from_numpy(X).to(DEV)
    v, p = ml2.ml2_load_ensemble(V), ml2.ml2_load_ensemble(P)
    pipe = ml2.Pipeline(v, p, w.n, w.k, device=DEV, with_margin=True)
    _note(f"{name}: running the GPU pipeline")
    pipe.run(Xd)
    torch.cuda.synchronize()
    valid = pipe.valid.cpu().numpy()
    margin = pipe.margin.cpu().numpy()
    score = pipe.score.cpu().numpy()
    idx = pipe.idx.cpu().numpy()[: w.k]
    top = pipe.top.cpu().numpy()[: w.k]
    num = int(pipe.num.item())
    v.free()
    p.free()
    _note(f"{name}: oracle on all {w.n} rows ({THREADS} threads)")
    t0 = time.perf_counter()
    ov, om = oracle.validity(V, X, THREADS)
    os_ = oracle.perf(P, X, ov, THREADS)
    oidx, otop, onum = oracle.topk(ov, os_, w.k)
    _note(f"{name}: oracle took {time.perf_counter() - t0:.1f} s")
    assert np.array_equal(valid, ov), f"validity mask differs on {int((valid != ov).sum())} rows"
    assert_scores(margin, om, "margin")
    assert_scores(score, os_, "score")
    assert num == onum
    assert np.array_equal(idx, oidx), "top-k indices differ"
    assert np.array_equal(top.view(np.uint32), otop.view(np.uint32)), "top-k scores differ"
    if w.a_trees:
        _second_level_check(w, X, Xd, idx, num)
    del Xd
    _note(f"{name}: invalid fraction {1 - int(ov.sum()) / w.n:.4f}; every row and the "
          f"top-{w.k} identical to the oracle")


# ---- one GPU's share and the merge of shards ---------------------------------------

@pytest.mark.slow
def test_shard_merge_matches_whole():
    """One GPU's share of the 16M-candidate pool with eight GPUs (2^21 rows x
    128, the same ensembles), split into eight uneven contiguous pseudo-shards.
    Each shard runs the whole path on its rows; the union of the shards'
    top-k lists, selected again with ml2_filter_topk, must equal the top-k of
    the undivided share bit for bit (indices and scores), because each
    candidate's scores do not depend on the shard and the key order (score
    descending, index ascending) is the same in every shard."""
    w = gen.WORKLOADS["roofline"]
    n, G, k = 1 << 21, 8, w.k
    _note(f"shard merge: {n} x {w.F} rows, {G} pseudo-shards, k = {k}")
    X = gen.features(w.seed, n, w.F, w.K)
    Xd = torch.from_numpy(X).to(DEV)
    v, p = ml2.ml2_load_ensemble(w.validity()), ml2.ml2_load_ensemble(w.perf())
    whole = ml2.Pipeline(v, p, n, k, device=DEV)
    whole.run(Xd)
    rng = np.random.default_rng(11)
    cuts = np.sort(rng.choice(np.arange(1, n), G - 1, replace=False))
    bounds = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    cat_score = torch.full((G * k,), -math.inf, dtype=torch.float32, device=DEV)
    cat_valid = torch.zeros(G * k, dtype=torch.uint8, device=DEV)
    cat_idx = torch.full((G * k,), -1, dtype=torch.int64, device=DEV)
    for g in range(G):
        r0, r1 = int(bounds[g]), int(bounds[g + 1])
        part = ml2.Pipeline(v, p, r1 - r0, k, device=DEV)
        part.run(Xd[r0:r1])
        m = part.num[0]
        sl = slice(g * k, (g + 1) * k)
        used = torch.arange(k, device=DEV) < m
        cat_score[sl] = torch.where(used, part.top[:k], cat_score[sl])
        cat_valid[sl] = used.to(torch.uint8)
        cat_idx[sl] = torch.where(used, part.idx[:k].to(torch.int64) + r0, cat_idx[sl])
    merged = ml2.Pipeline(v, p, G * k, k, device=DEV)
    ml2.ml2_filter_topk(cat_valid, cat_score, k, merged.idx, merged.top, merged.num,
                        merged.ws, merged.ws_bytes, G * k)
    torch.cuda.synchronize()
    num = int(whole.num.item())
    assert int(merged.num.item()) == num == k
    got_idx = cat_idx[merged.idx[:num].to(torch.int64)].cpu().numpy()
    assert np.array_equal(got_idx, whole.idx[:num].cpu().numpy().astype(np.int64))
    assert np.array_equal(merged.top[:num].cpu().numpy().view(np.uint32),
                          whole.top[:num].cpu().numpy().view(np.uint32))
    ov, _ = oracle.validity(w.validity(), X, THREADS)
    os_ = oracle.perf(w.perf(), X, ov, THREADS)
    oidx, otop, onum = oracle.topk(ov, os_, k)
    assert onum == num
    assert np.array_equal(got_idx, oidx.astype(np.int64)), "merged top-k differs from the oracle's"
    assert np.array_equal(merged.top[:num].cpu().numpy().view(np.uint32), otop.view(np.uint32))
    _note(f"shard merge: shards {np.diff(bounds).tolist()}; merged top-{k} identical to the "
          "undivided share's and to the oracle's")
    v.free()
    p.free()
