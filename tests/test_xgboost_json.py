"""The XGBoost JSON loader against a hand-built model in the format's
published schema (tests/golden/xgboost_small.json, hand-computed margins in
xgboost_small_expected.json), and its refusals.  Compatibility with files
written by XGBoost itself is unpinned here: XGBoost is not installed."""
import copy
import json
import os

import numpy as np
import pytest

import oracle
from paper_2411_10764_amd.xgboost_json import load_xgboost_json

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fixture():
    with open(os.path.join(GOLDEN, "xgboost_small.json")) as fh:
        model = json.load(fh)
    with open(os.path.join(GOLDEN, "xgboost_small_expected.json")) as fh:
        exp = json.load(fh)
    X = np.array([[np.nan if v == "nan" else v for v in row] for row in exp["inputs"]],
                 np.float32)
    return model, exp, X


def test_loader_structure():
    model, _, _ = _fixture()
    e = load_xgboost_json(model)
    assert e.num_trees == 2 and e.num_features == 3 and e.base_score == 0.5
    assert list(np.diff(e.offsets)) == [5, 5]  # the pruned node is dropped
    # breadth-first: children adjacent
    for t in range(2):
        b = int(e.offsets[t])
        for i in range(5):
            if e.left[b + i] >= 0:
                assert e.right[b + i] == e.left[b + i] + 1
    assert list(e.default_left[:5]) == [1, 0, 0, 0, 0]


def test_loader_margins_and_leaves():
    model, exp, X = _fixture()
    e = load_xgboost_json(json.dumps(model))
    leaves = np.array([oracle.leaves(e, x) for x in X])
    assert np.array_equal(leaves, np.array(exp["leaves"], np.float32))
    _, margins = oracle.validity(e, X)
    assert list(margins) == exp["margins"]


def test_loader_logistic_intercept():
    model, exp, X = _fixture()
    m = copy.deepcopy(model)
    m["learner"]["objective"]["name"] = "binary:logistic"
    e = load_xgboost_json(m)
    assert e.base_score == 0.0  # logit(0.5)
    _, margins = oracle.validity(e, X)
    assert list(margins) == [v - 0.5 for v in exp["margins"]] == exp["logistic_margins"]


def test_loader_path(tmp_path):
    model, exp, X = _fixture()
    p = tmp_path / "m.json"
    p.write_text(json.dumps(model))
    _, margins = oracle.validity(load_xgboost_json(str(p)), X)
    assert list(margins) == exp["margins"]


@pytest.mark.parametrize("edit", ["dart", "multiclass", "categorical", "objective", "one_child"])
def test_loader_refusals(edit):
    model, _, _ = _fixture()
    m = copy.deepcopy(model)
    lr = m["learner"]
    if edit == "dart":
        lr["gradient_booster"]["name"] = "dart"
    elif edit == "multiclass":
        lr["learner_model_param"]["num_class"] = "3"
    elif edit == "categorical":
        lr["gradient_booster"]["model"]["trees"][1]["split_type"][2] = 1
    elif edit == "objective":
        lr["objective"]["name"] = "rank:pairwise"
    else:
        lr["gradient_booster"]["model"]["trees"][0]["right_children"][1] = -1
    with pytest.raises(ValueError):
        load_xgboost_json(m)
