"""The C-ABI library without a GPU: it loads, exports every symbol the
header declares, and rejects bad arguments synchronously (before any HIP
call) with the documented status codes."""
import ctypes
import os
import re

import numpy as np
import pytest

import gen
from paper_2411_10764_amd import ml2
from tests.treeutil import ensemble_from_trees

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "ml2.h")
PROBE_HEADER = os.path.join(os.path.dirname(HEADER), "ml2_probe.h")


def _header_functions(path=HEADER):
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ml2_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = ml2.lib()
    declared = _header_functions()
    assert declared, "no declarations parsed"
    for name in declared:
        assert hasattr(L, name), f"{name} not exported"
    assert sorted(ml2.EXPORTED) == declared


def test_exports_every_probe_symbol():
    L = ml2.lib()
    declared = _header_functions(PROBE_HEADER)
    assert declared == sorted(ml2.EXPORTED_PROBE)
    for name in declared:
        assert hasattr(L, name), f"{name} not exported"


@pytest.mark.parametrize("call", [
    lambda L, ms, w: L.ml2_probe_visit(7, 4, 2, 8, 128, 10, 4, ms, w),    # depth 6, 8 or 10
    lambda L, ms, w: L.ml2_probe_visit(8, 3, 1, 8, 64, 10, 4, ms, w),     # shape not built
    lambda L, ms, w: L.ml2_probe_visit(8, 4, 4, 8, 64, 10, 4, ms, w),     # shape not built
    lambda L, ms, w: L.ml2_probe_visit(8, 8, 2, 8, 128, 10, 4, ms, w),    # beyond the LDS
    lambda L, ms, w: L.ml2_probe_visit(8, 4, 2, 9, 128, 10, 4, ms, w),    # 1 to 8 waves
    lambda L, ms, w: L.ml2_probe_visit(8, 4, 2, 0, 128, 10, 4, ms, w),    # 1 to 8 waves
    lambda L, ms, w: L.ml2_probe_visit(8, 4, 2, 8, 128, 0, 4, ms, w),     # iters >= 1
    lambda L, ms, w: L.ml2_probe_visit(8, 4, 2, 8, 128, 10, 0, ms, w),    # blocks >= 1
    lambda L, ms, w: L.ml2_probe_visit(8, 4, 2, 8, 128, 10, 4, None, w),  # NULL output
    lambda L, ms, w: L.ml2_probe_lds(6, 10, 4, ms, w),        # mode 0..5
    lambda L, ms, w: L.ml2_probe_lds(0, 1 << 21, 4, ms, w),   # iters <= 2^20
    lambda L, ms, w: L.ml2_probe_lds(0, 10, 65537, ms, w),    # blocks <= 65536
    lambda L, ms, w: L.ml2_probe_valu(10, 4, ms, None),       # NULL output
])
def test_probe_argument_errors(call):
    """Probe arguments are checked before any HIP call."""
    L = ml2.lib()
    ms, w = ctypes.c_double(-1.0), ctypes.c_double(-1.0)
    assert call(L, ctypes.byref(ms), ctypes.byref(w)) == ml2.ML2_ERR_INVALID_ARG
    assert ms.value == -1.0 and w.value == -1.0


@pytest.mark.parametrize("args", [(-1, 0, 0, 0, 0), (3, 0, 0, 0, 0), (0, 17, 0, 0, 0),
                                  (0, 0, 9, 0, 0), (0, 0, 0, 3, 0), (0, 0, 0, 0, -4)])
def test_tune_walk_plan_argument_errors(args):
    """The launch-plan override rejects out-of-range fields and leaves the
    current override unchanged (no GPU needed: it only records the fields)."""
    L = ml2.lib()
    assert L.ml2_tune_walk_plan(*args) == ml2.ML2_ERR_INVALID_ARG
    assert "ml2_tune_walk_plan" in L.ml2_last_error().decode()
    assert L.ml2_tune_walk_plan(2, 4, 8, 1, 16) == ml2.ML2_OK
    assert L.ml2_tune_walk_plan(0, 0, 0, 0, 0) == ml2.ML2_OK


def test_tune_layout_argument_errors():
    L = ml2.lib()
    for bad in (-1, 3):
        assert L.ml2_tune_layout(bad) == ml2.ML2_ERR_INVALID_ARG
    for good in (1, 2, 0):
        assert L.ml2_tune_layout(good) == ml2.ML2_OK


def test_header_constants_match_binding():
    text = open(HEADER).read()
    for name in ("ML2_MAX_DEPTH", "ML2_MAX_TREE_NODES", "ML2_MAX_FEATURES", "ML2_MAX_TOPK",
                 "ML2_MAX_STREAM_K"):
        m = re.search(rf"#define {name} (\d+)", text)
        assert m and int(m.group(1)) == getattr(ml2, name)
    for name, val in (("ML2_OK", 0), ("ML2_ERR_INVALID_ARG", 1), ("ML2_ERR_UNSUPPORTED", 2),
                      ("ML2_ERR_OUT_OF_MEMORY", 3), ("ML2_ERR_HIP", 4)):
        assert re.search(rf"{name} = {val}\b", text)
        assert getattr(ml2, name) == val


def _load_status(ens):
    d, keep = ml2.make_desc(ens)
    h = ctypes.c_void_p(12345)
    st = ml2.lib().ml2_load_ensemble(ctypes.byref(d), ctypes.byref(h))
    return st, h.value, ml2.lib().ml2_last_error().decode()


def _base_ens():
    return ensemble_from_trees([(0, 1.0, 0.5, (1, 2.0, -0.5, 0.25)), 0.125], 2)


def _mutate(ens, **kw):
    import dataclasses
    arrays = {k: getattr(ens, k).copy() for k in
              ("offsets", "left", "right", "feature", "threshold", "value")}
    for k, fn in kw.items():
        if k in arrays:
            fn(arrays[k])
    base = kw.get("base_score", ens.base_score)
    nf = kw.get("num_features", ens.num_features)
    return dataclasses.replace(ens, num_features=nf, base_score=base, **arrays)


@pytest.mark.parametrize("case,status,needle", [
    ("feature_out_of_range", ml2.ML2_ERR_INVALID_ARG, "split feature"),
    ("negative_feature", ml2.ML2_ERR_INVALID_ARG, "split feature"),
    ("nan_threshold", ml2.ML2_ERR_INVALID_ARG, "NaN"),
    ("inf_leaf", ml2.ML2_ERR_INVALID_ARG, "not finite"),
    ("cycle", ml2.ML2_ERR_INVALID_ARG, "reached twice"),
    ("half_leaf", ml2.ML2_ERR_INVALID_ARG, "out of range"),
    ("orphan", ml2.ML2_ERR_INVALID_ARG, "unreachable"),
    ("bad_offsets", ml2.ML2_ERR_INVALID_ARG, "empty"),
    ("nan_base", ml2.ML2_ERR_INVALID_ARG, "base_score"),
    ("overflow", ml2.ML2_ERR_INVALID_ARG, "overflow"),
    ("too_many_features", ml2.ML2_ERR_UNSUPPORTED, "num_features"),
])
def test_load_rejects(case, status, needle):
    e = _base_ens()
    if case == "feature_out_of_range":
        e = _mutate(e, feature=lambda a: a.__setitem__(0, 2))
    elif case == "negative_feature":
        e = _mutate(e, feature=lambda a: a.__setitem__(0, -3))
    elif case == "nan_threshold":
        e = _mutate(e, threshold=lambda a: a.__setitem__(0, np.nan))
    elif case == "inf_leaf":
        e = _mutate(e, value=lambda a: a.__setitem__(1, np.inf))
    elif case == "cycle":
        e = _mutate(e, left=lambda a: a.__setitem__(2, 0), right=lambda a: a.__setitem__(2, 3))
    elif case == "half_leaf":
        e = _mutate(e, right=lambda a: a.__setitem__(2, -1))
    elif case == "orphan":
        e = ensemble_from_trees([(0, 1.0, 0.5, 0.25)], 2)
        e = _mutate(e, offsets=lambda a: a.__setitem__(1, 4),
                    left=lambda a: None)
        import dataclasses
        e = dataclasses.replace(e, left=np.append(e.left, -1), right=np.append(e.right, -1),
                                feature=np.append(e.feature, -1),
                                threshold=np.append(e.threshold, 0),
                                value=np.append(e.value, 1.0).astype(np.float32))
    elif case == "bad_offsets":
        e = _mutate(e, offsets=lambda a: a.__setitem__(2, a[1]))
    elif case == "nan_base":
        e = _mutate(e, base_score=float("nan"))
    elif case == "overflow":
        e = _mutate(e, value=lambda a: a.__setitem__(1, 3e38))
    elif case == "too_many_features":
        e = _mutate(e, num_features=ml2.ML2_MAX_FEATURES + 1)
    st, h, msg = _load_status(e)
    assert st == status, msg
    assert h is None
    assert needle in msg


def _caterpillar(depth):
    """A tree whose right spine has `depth` splits (2 * depth + 1 nodes)."""
    from tests.treeutil import ensemble_from_trees
    tree = 1.0
    for _ in range(depth):
        tree = (0, 0.5, -1.0, tree)
    return ensemble_from_trees([tree], num_features=4)


def test_load_rejects_depth_beyond_limit():
    e = _caterpillar(ml2.ML2_MAX_DEPTH + 1)
    st, h, msg = _load_status(e)
    assert st == ml2.ML2_ERR_UNSUPPORTED and "depth" in msg and h is None


def test_load_rejects_deep_tree_beyond_node_limit():
    # deeper than the perfect layout and larger than a ragged chunk holds
    e = gen.ragged_ensemble(1, 1, 1, 20, 4, 4, 0.5, p_split=1.0, decay=1.0,
                            max_nodes=ml2.ML2_MAX_TREE_NODES + 2)
    assert np.diff(e.offsets)[0] > ml2.ML2_MAX_TREE_NODES
    st, h, msg = _load_status(e)
    assert st == ml2.ML2_ERR_UNSUPPORTED and "nodes" in msg and h is None


def test_load_null_arguments():
    L = ml2.lib()
    h = ctypes.c_void_p()
    assert L.ml2_load_ensemble(None, ctypes.byref(h)) == ml2.ML2_ERR_INVALID_ARG
    d, keep = ml2.make_desc(_base_ens())
    assert L.ml2_load_ensemble(ctypes.byref(d), None) == ml2.ML2_ERR_INVALID_ARG
    d.split_threshold = None
    assert L.ml2_load_ensemble(ctypes.byref(d), ctypes.byref(h)) == ml2.ML2_ERR_INVALID_ARG
    d2, keep2 = ml2.make_desc(_base_ens())
    d2.num_trees = 0
    assert L.ml2_load_ensemble(ctypes.byref(d2), ctypes.byref(h)) == ml2.ML2_ERR_INVALID_ARG


def test_score_one_call_rejects_null_ensembles():
    L = ml2.lib()
    P = 1 << 20  # never dereferenced
    assert L.ml2_score(None, None, P, 10, 8, P, None, P, None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_score_single_pass(None, None, P, 10, 8) == 0


def test_score_calls_reject_null_ensemble():
    L = ml2.lib()
    assert L.ml2_score_validity(None, 4096, 10, 4, 8192, None, None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_score_perf(None, 4096, 10, 4, None, 8192, None) == ml2.ML2_ERR_INVALID_ARG
    assert b"NULL" in L.ml2_last_error()


def test_topk_workspace_bytes():
    assert ml2.ml2_topk_workspace_bytes(0, 0) > 0
    b1 = ml2.ml2_topk_workspace_bytes(1 << 24, 1024)
    assert b1 % 256 == 0 and b1 >= 1024 * 8
    with pytest.raises(ml2.Ml2Error) as ei:
        ml2.ml2_topk_workspace_bytes(10, ml2.ML2_MAX_TOPK + 1)
    assert ei.value.status == ml2.ML2_ERR_UNSUPPORTED
    with pytest.raises(ml2.Ml2Error) as ei:
        ml2.ml2_topk_workspace_bytes(-1, 3)
    assert ei.value.status == ml2.ML2_ERR_INVALID_ARG
    with pytest.raises(ml2.Ml2Error):
        ml2.ml2_topk_workspace_bytes(10, -1)


def test_filter_topk_argument_errors():
    L = ml2.lib()
    P = 1 << 20  # never dereferenced: every case fails validation first
    ws = ml2.ml2_topk_workspace_bytes(100, 8)
    cases = [
        dict(n=-1, k=8), dict(n=100, k=-1), dict(n=100, k=8, num=None),
        dict(n=100, k=8, ws=None), dict(n=100, k=8, scores=None), dict(n=100, k=8, idx=None),
        dict(n=100, k=8, ws_bytes=ws - 1), dict(n=100, k=8, ws_ptr=P + 8),
    ]
    for c in cases:
        st = L.ml2_filter_topk(None, c.get("scores", P), c["n"], c["k"], c.get("idx", P), P,
                               c.get("num", P),
                               c.get("ws_ptr", c.get("ws", P)) if "ws" not in c or c["ws"] else None,
                               c.get("ws_bytes", ws), None)
        assert st == ml2.ML2_ERR_INVALID_ARG, c
    st = L.ml2_filter_topk(None, P, 100, ml2.ML2_MAX_TOPK + 1, P, P, P, P, 1 << 30, None)
    assert st == ml2.ML2_ERR_UNSUPPORTED


def test_filter_topk_noalloc_argument_errors():
    """The allocation-free selection validates like ml2_filter_topk (no
    workspace argument) before touching the device."""
    L = ml2.lib()
    P = 1 << 20  # never dereferenced: every case fails validation first
    for n, k, scores, idx, num in ((-1, 8, P, P, P), (100, -1, P, P, P), (100, 8, P, P, None),
                                   (100, 8, None, P, P), (100, 8, P, None, P),
                                   (1 << 31, 8, P, P, P)):
        st = L.ml2_filter_topk_noalloc(None, scores, n, k, idx, P, num, None)
        assert st == ml2.ML2_ERR_INVALID_ARG, (n, k)
    st = L.ml2_filter_topk_noalloc(None, P, 100, ml2.ML2_MAX_TOPK + 1, P, P, P, None)
    assert st == ml2.ML2_ERR_UNSUPPORTED
    assert "static" in L.ml2_last_error().decode()


def test_rerank_null_ensemble():
    L = ml2.lib()
    P = 1 << 20  # never dereferenced: the NULL ensemble fails validation first
    assert L.ml2_rerank(None, P, 10, 4, P, 5, 3, P, P, P, P, P, 1 << 20, None) == \
        ml2.ML2_ERR_INVALID_ARG
    assert b"NULL" in L.ml2_last_error()
    import ctypes
    b = ctypes.c_size_t()
    assert L.ml2_rerank_workspace_bytes(None, 5, ctypes.byref(b)) == ml2.ML2_ERR_INVALID_ARG


def test_explorer_null_handles():
    import ctypes
    L = ml2.lib()
    h = ctypes.c_void_p()
    assert L.ml2_explorer_create(None, None, None, 10, 4, 2, 3, ctypes.byref(h)) == \
        ml2.ML2_ERR_INVALID_ARG
    assert h.value is None
    assert L.ml2_explorer_create(None, None, None, 10, 4, 2, 3, None) == ml2.ML2_ERR_INVALID_ARG
    P = 1 << 20  # never dereferenced
    assert L.ml2_explorer_round(None, P, 8, 1, P, P, P, None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_explorer_reset(None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_explorer_rounds(None) == -1
    L.ml2_explorer_free(None)


def test_stream_explorer_null_handles():
    import ctypes
    L = ml2.lib()
    h = ctypes.c_void_p()
    assert L.ml2_stream_explorer_create(None, None, None, 100, 4, 2, 3, ctypes.byref(h)) == \
        ml2.ML2_ERR_INVALID_ARG
    assert h.value is None
    assert L.ml2_stream_explorer_create(None, None, None, 100, 4, 2, 3, None) == \
        ml2.ML2_ERR_INVALID_ARG
    P = 1 << 20  # never dereferenced
    assert L.ml2_stream_explorer_begin(None, None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_stream_explorer_chunk(None, P, 10, 8, 0, None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_stream_explorer_end(None, P, P, P, None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_stream_explorer_reset(None) == ml2.ML2_ERR_INVALID_ARG
    assert L.ml2_stream_explorer_rounds(None) == -1
    L.ml2_stream_explorer_free(None)
