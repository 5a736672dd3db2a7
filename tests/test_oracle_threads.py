"""Pins of the oracle's multi-threaded range split.

The oracle scores a pool on several threads by cutting it into contiguous
row ranges (row i belongs to the range lo = n*t/threads); each row's margin
is still the serial left fold of that row, so the outputs must not depend
on the thread count.  Pinned two ways: (1) every thread count gives the
bytes of one thread, on pool sizes that the thread counts do not divide,
and those bytes equal the path-predicate evaluator's leaves folded in tree
order (independent of the walker); (2) a ThreadSanitizer build of the
oracle scores a pool on several thread counts without a reported race.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import gen
import oracle
from tests.treeutil import fold_left_f32, path_predicate_leaves, random_ragged_ensemble

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _expected(ens, X, mask=None):
    leaves = path_predicate_leaves(ens, X)
    out = np.array([fold_left_f32(ens.base_score, leaves[i]) for i in range(X.shape[0])],
                   np.float32)
    if mask is not None:
        out[mask == 0] = -np.inf
    return out


@pytest.mark.parametrize("n", [1, 5, 97, 1013])
def test_thread_count_does_not_change_outputs(n):
    rng = np.random.default_rng(n)
    F = 7
    V = random_ragged_ensemble(rng, 11, 5, F, lambda r, f: float(r.integers(0, 9)),
                               lambda r: float(np.float32(r.normal(0, 0.5))), p_split=0.8,
                               base=0.125)
    P = gen.perfect_ensemble(seed=n, stream=gen.STREAM_PERF, trees=13, depth=4, F=F, K=4,
                             leaf_sigma=0.1)
    X = gen.features(seed=n, n=n, F=F, K=4, missing=0.0)
    X[rng.random(X.shape) < 0.05] = np.nan  # missing values go right (no default_left)
    want_m = _expected(V, X)
    want_v = (want_m > 0).astype(np.uint8)
    want_s = _expected(P, X, want_v)
    for threads in (1, 2, 3, 7, 16, 64, 256):
        valid, marg = oracle.validity(V, X, threads)
        score = oracle.perf(P, X, valid, threads)
        assert np.array_equal(valid, want_v), f"mask on {threads} threads"
        assert np.array_equal(marg.view(np.uint32), want_m.view(np.uint32)), \
            f"margins on {threads} threads"
        assert np.array_equal(score.view(np.uint32), want_s.view(np.uint32)), \
            f"scores on {threads} threads"


def test_thread_ranges_cover_every_row_once():
    # Rows untouched by every range keep a sentinel; rows scored twice cannot
    # be seen in the output, so the margins are compared with the serial ones
    # on a pool whose size is prime and smaller than some thread counts.
    ens = gen.perfect_ensemble(seed=3, stream=gen.STREAM_VALIDITY, trees=5, depth=3, F=4, K=4,
                               leaf_sigma=0.5)
    for n in (2, 3, 13, 31):
        X = gen.features(seed=n, n=n, F=4, K=4)
        for threads in (1, 4, 13, 32):
            score = oracle.perf(ens, X, None, threads)
            assert np.array_equal(score.view(np.uint32), _expected(ens, X).view(np.uint32))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_thread_sanitizer_finds_no_race(tmp_path):
    exe = str(tmp_path / "oracle_tsan")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fsanitize=thread", "-pthread",
           "-ffp-contract=off", "-fno-fast-math",
           os.path.join(ROOT, "oracle", "ml2_oracle.c"),
           os.path.join(HERE, "oracle_threads_driver.c"), "-o", exe, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitizer" in (r.stderr or "").lower():
        pytest.skip(f"ThreadSanitizer unavailable: {r.stderr[-300:]}")
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=66")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    assert "ThreadSanitizer" not in run.stderr, run.stderr[-2000:]
    assert run.returncode == 0, run.stderr[-2000:]
    assert "threads ok" in run.stdout
