"""The allocation-free selection (ml2_filter_topk_noalloc) against
ml2_filter_topk with a caller workspace and against the oracle: two calls in
a row on one device, the second with a smaller pool and k, so the second
call runs on the scratch the first one left behind."""
import sys

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2411_10764_amd import ml2  # noqa: E402

DEV = "cuda:0"


def _inputs(seed, n):
    rng = np.random.default_rng(seed)
    score = rng.normal(0, 3, n).astype(np.float32)
    score[rng.random(n) < 0.05] = np.float32(1.25)   # ties broken by index
    score[rng.random(n) < 0.01] = -0.0
    score[rng.random(n) < 0.01] = np.nan
    valid = (rng.random(n) < 0.6).astype(np.uint8)
    return valid, score


def _with_workspace(vd, sd, n, k):
    idx = torch.full((max(k, 1),), -7, dtype=torch.int32, device=DEV)
    top = torch.full((max(k, 1),), 7.0, dtype=torch.float32, device=DEV)
    num = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    wsb = ml2.ml2_topk_workspace_bytes(n, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    ml2.ml2_filter_topk(vd, sd, k, idx, top, num, ws, wsb, n)
    torch.cuda.synchronize()
    return idx.cpu().numpy()[:k], top.cpu().numpy()[:k], int(num.item())


def _noalloc(vd, sd, n, k):
    idx = torch.full((max(k, 1),), -7, dtype=torch.int32, device=DEV)
    top = torch.full((max(k, 1),), 7.0, dtype=torch.float32, device=DEV)
    num = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    ml2.ml2_filter_topk_noalloc(vd, sd, k, idx, top, num, n)
    torch.cuda.synchronize()
    return idx.cpu().numpy()[:k], top.cpu().numpy()[:k], int(num.item())


@pytest.mark.parametrize("first,second", [((1 << 20, 1024), (5000, 100)),
                                          ((300000, ml2.ML2_MAX_TOPK), (777, 7))])
def test_noalloc_matches_workspace_call(first, second):
    for call, (n, k) in enumerate((first, second)):
        print(f"[no-alloc] call {call}: n={n} k={k}", flush=True)
        sys.stdout.flush()
        valid, score = _inputs(100 * call + k, n)
        vd = torch.from_numpy(valid).to(DEV)
        sd = torch.from_numpy(score).to(DEV)
        got = _noalloc(vd, sd, n, k)
        ref = _with_workspace(vd, sd, n, k)
        o_idx, o_top, o_num = oracle.topk(valid, score, k)
        assert got[2] == ref[2] == o_num
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[0], o_idx)
        assert np.array_equal(got[1].view(np.uint32), ref[1].view(np.uint32))
        assert np.array_equal(got[1].view(np.uint32), o_top.view(np.uint32))


def test_noalloc_empty_and_k_zero():
    vd = torch.ones(10, dtype=torch.uint8, device=DEV)
    sd = torch.arange(10, dtype=torch.float32, device=DEV)
    idx, top, num = _noalloc(vd, sd, 0, 4)
    assert num == 0 and list(idx) == [-1] * 4 and np.all(np.isneginf(top))
    idx, top, num = _noalloc(vd, sd, 10, 0)
    assert num == 0
    idx, top, num = _noalloc(vd, sd, 10, 3)
    assert num == 3 and list(idx) == [9, 8, 7]
