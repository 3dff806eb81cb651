"""Node lists from a trained booster's JSON text dump.

A gradient-boosting library such as XGBoost (the model of Section 3.1) can
write each tree as one JSON object: a split node carries "nodeid", "split"
(feature name), "split_condition", "yes" and "no" (the children's node ids;
"yes" is taken when x < split_condition) and "children"; a leaf carries
"nodeid" and "leaf".  This module turns a list of such objects (or their JSON
text) into the node lists that at_ensemble_import and at_trees_pad take.
Features are never missing here, so a dump's "missing" branch is ignored.
"""
from __future__ import annotations

import json

import numpy as np


def _feature_index(name) -> int:
    if isinstance(name, (int, np.integer)):
        return int(name)
    s = str(name)
    if s.startswith("f") and s[1:].isdigit():
        return int(s[1:])
    if s.isdigit():
        return int(s)
    raise ValueError(f"split feature {name!r} is neither 'f<k>' nor an integer")


def trees_from_xgboost_dump(dumps) -> dict:
    """dumps: list of per-tree JSON strings or already-parsed dicts.  Returns
    dict(offsets, left, right, feature, threshold, value): nodes renumbered in
    preorder (root first, then the "yes" subtree, then the "no" subtree)."""
    offs, L, R, Fe, Th, V = [0], [], [], [], [], []
    for t, d in enumerate(dumps):
        root = json.loads(d) if isinstance(d, (str, bytes)) else d
        order = []            # preorder list of node dicts
        index = {}            # nodeid -> preorder position

        def visit(node):
            nid = int(node["nodeid"])
            if nid in index:
                raise ValueError(f"tree {t}: node id {nid} appears twice")
            index[nid] = len(order)
            order.append(node)
            if "leaf" in node:
                return
            kids = {int(c["nodeid"]): c for c in node.get("children", [])}
            for side in ("yes", "no"):
                cid = int(node[side])
                if cid not in kids:
                    raise ValueError(f"tree {t}: node {nid} names child {cid} that is not among its children")
                visit(kids[cid])

        visit(root)
        for node in order:
            if "leaf" in node:
                L.append(-1)
                R.append(-1)
                Fe.append(0)
                Th.append(0.0)
                V.append(float(node["leaf"]))
            else:
                L.append(index[int(node["yes"])])
                R.append(index[int(node["no"])])
                Fe.append(_feature_index(node["split"]))
                Th.append(float(node["split_condition"]))
                V.append(0.0)
        offs.append(offs[-1] + len(order))
    return {"offsets": np.asarray(offs, np.int32), "left": np.asarray(L, np.int32),
            "right": np.asarray(R, np.int32), "feature": np.asarray(Fe, np.int32),
            "threshold": np.asarray(Th, np.float32), "value": np.asarray(V, np.float32)}
