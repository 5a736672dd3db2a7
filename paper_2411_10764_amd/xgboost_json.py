"""Tree ensembles from XGBoost's JSON model format.

ML2Tuner's models V, P and A are XGBoost (v2.1.1) gbtree ensembles (Section 3
"Experimental Setup", Table 3).  ``load_xgboost_json`` turns a model saved
with ``Booster.save_model("model.json")`` into the arrays of the C ABI's
``ml2_ensemble_desc`` (host-side parsing only; ``ml2.ml2_load_ensemble``
accepts the result).

What is read, per the format's published schema:
  learner.learner_model_param: num_feature, num_class, num_target, base_score
  learner.objective.name
  learner.gradient_booster: name "gbtree"; model.trees[*]: left_children,
      right_children, split_indices, split_conditions (the threshold of a
      split, the value of a leaf), default_left, split_type (optional)
Each tree is renumbered breadth-first from its root, so nodes left unreachable
by pruning are dropped and the two children of a node are adjacent.

Not supported (ValueError): other boosters (dart, gblinear), several outputs
(num_class > 1, num_target > 1, a tree_info entry other than 0), categorical
splits, and objectives whose margin-space intercept is not known here.
"""
from __future__ import annotations

import dataclasses
import json
import math
import os
from collections import deque

import numpy as np

# Objectives whose margin-space intercept is base_score itself, and those
# whose prediction is sigmoid(margin) (intercept logit(base_score)).
_IDENTITY_OBJECTIVES = {
    "reg:squarederror", "reg:squaredlogerror", "reg:pseudohubererror", "reg:absoluteerror",
    "reg:quantileerror", "binary:hinge", "binary:logitraw",
}
_LOGIT_OBJECTIVES = {"binary:logistic", "reg:logistic"}


@dataclasses.dataclass(frozen=True)
class TreeEnsemble:
    """A tree ensemble in the general child-pointer form of ml2_ensemble_desc."""
    num_features: int
    base_score: float
    offsets: np.ndarray       # int64 [T+1]
    left: np.ndarray          # int32 [nodes], tree-local ids, -1 for a leaf
    right: np.ndarray         # int32 [nodes]
    feature: np.ndarray       # int32 [nodes]
    threshold: np.ndarray     # float32 [nodes]
    value: np.ndarray         # float32 [nodes] (leaves)
    default_left: np.ndarray  # uint8 [nodes]
    objective: str = ""

    @property
    def num_trees(self) -> int:
        return int(self.offsets.shape[0] - 1)


def _intercept(objective: str, base_score: float) -> float:
    if objective in _IDENTITY_OBJECTIVES:
        return base_score
    if objective in _LOGIT_OBJECTIVES:
        if not 0.0 < base_score < 1.0:
            raise ValueError(f"base_score {base_score} is not a probability")
        return math.log(base_score / (1.0 - base_score))
    raise ValueError(f"objective {objective!r}: margin-space intercept unknown")


def _base_score(text) -> float:
    if isinstance(text, (int, float)):
        return float(text)
    s = str(text).strip()
    if s.startswith("["):  # newer writers store a vector
        vals = json.loads(s)
        if len(vals) != 1:
            raise ValueError("several base scores (multi-output model)")
        return float(vals[0])
    return float(s)


def load_xgboost_json(src) -> TreeEnsemble:
    """Parse a model: a path, a JSON string or an already-decoded dict."""
    if isinstance(src, dict):
        model = src
    elif isinstance(src, (str, os.PathLike)) and os.path.exists(src):
        with open(src) as fh:
            model = json.load(fh)
    else:
        model = json.loads(src)
    learner = model["learner"]
    lmp = learner["learner_model_param"]
    num_features = int(lmp["num_feature"])
    if int(lmp.get("num_class", "0")) > 1 or int(lmp.get("num_target", "1")) > 1:
        raise ValueError("models with several outputs are not supported")
    objective = learner.get("objective", {}).get("name", "")
    base = _intercept(objective, _base_score(lmp["base_score"]))
    booster = learner["gradient_booster"]
    if booster.get("name", "gbtree") != "gbtree":
        raise ValueError(f"booster {booster.get('name')!r} is not supported (gbtree only)")
    body = booster["model"]
    trees = body["trees"]
    if any(int(i) != 0 for i in body.get("tree_info", [])):
        raise ValueError("trees of several outputs are not supported")

    offsets = [0]
    cols = {k: [] for k in ("left", "right", "feature", "threshold", "value", "default_left")}
    for ti, tree in enumerate(trees):
        lc = tree["left_children"]
        rc = tree["right_children"]
        si = tree["split_indices"]
        sc = tree["split_conditions"]
        dl = tree.get("default_left", [0] * len(lc))
        st = tree.get("split_type", [0] * len(lc))
        order = {0: 0}
        queue = deque([0])
        nodes = []
        while queue:  # breadth-first renumbering of the reachable nodes
            old = queue.popleft()
            nodes.append(old)
            l, r = int(lc[old]), int(rc[old])
            if l == -1:
                continue
            if r == -1:
                raise ValueError(f"tree {ti} node {old}: one child only")
            if int(st[old]) != 0:
                raise ValueError(f"tree {ti} node {old}: categorical split")
            for c in (l, r):
                if c in order:
                    raise ValueError(f"tree {ti}: node {c} reached twice")
                order[c] = len(order)
                queue.append(c)
        for old in nodes:
            l, r = int(lc[old]), int(rc[old])
            leaf = l == -1
            cols["left"].append(-1 if leaf else order[l])
            cols["right"].append(-1 if leaf else order[r])
            cols["feature"].append(-1 if leaf else int(si[old]))
            cols["threshold"].append(0.0 if leaf else float(sc[old]))
            cols["value"].append(float(sc[old]) if leaf else 0.0)
            cols["default_left"].append(0 if leaf else int(bool(dl[old])))
        offsets.append(offsets[-1] + len(nodes))
    return TreeEnsemble(
        num_features, float(np.float32(base)), np.asarray(offsets, np.int64),
        np.asarray(cols["left"], np.int32), np.asarray(cols["right"], np.int32),
        np.asarray(cols["feature"], np.int32), np.asarray(cols["threshold"], np.float32),
        np.asarray(cols["value"], np.float32), np.asarray(cols["default_left"], np.uint8),
        objective)
