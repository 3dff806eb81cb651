"""Oracle pins: trees of any shape in node-list form (Section 3.1).

The oracle walks node lists directly.  It is pinned by a hand-worked
ensemble, by the full-tree oracle (itself pinned in test_oracle_model.py) on
full trees written as node lists, and by brute force: every input of a small
grid satisfies the split conditions of exactly one root-to-leaf path, and
the oracle returns that leaf.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))


def golden():
    with open(os.path.join(HERE, "golden", "trained_trees_worked_example.json")) as f:
        return json.load(f)


def test_hand_worked_example():
    g = golden()
    s = oracle.predict_nodes(g["trees"], np.asarray(g["rows"], np.int32))
    assert s.tolist() == g["scores"]


def heap_to_nodes(fid, thr, leaf, rng):
    """Full heap trees as node lists, each tree's non-root nodes shuffled."""
    T, n_int = fid.shape
    m = 2 * n_int + 1
    offs, L, R, Fe, Th, V = [0], [], [], [], [], []
    for t in range(T):
        pos = np.concatenate([[0], 1 + rng.permutation(m - 1)])   # heap node h is stored at pos[h]
        l, r = np.full(m, -1), np.full(m, -1)
        fe, th, v = np.zeros(m, int), np.zeros(m), np.zeros(m)
        for h in range(m):
            p = pos[h]
            if h < n_int:
                l[p], r[p] = pos[2 * h + 1], pos[2 * h + 2]
                fe[p], th[p] = fid[t, h], thr[t, h]
            else:
                v[p] = leaf[t, h - n_int]
        offs.append(offs[-1] + m)
        L.append(l), R.append(r), Fe.append(fe), Th.append(th), V.append(v)
    cat = np.concatenate
    return {"offsets": np.array(offs), "left": cat(L), "right": cat(R), "feature": cat(Fe),
            "threshold": cat(Th).astype(np.float32), "value": cat(V).astype(np.float32)}


@pytest.mark.parametrize("depth,T,F", [(1, 7, 5), (3, 40, 12), (6, 25, 110)])
def test_full_trees_equal_the_full_tree_oracle(depth, T, F):
    fid, thr, leaf = W.make_ensemble(T, depth, F, seed=depth)
    rng = np.random.default_rng(100 + depth)
    trees = heap_to_nodes(fid, thr, leaf, rng)
    x = rng.integers(0, 36, size=(300, F)).astype(np.int32)
    a = oracle.predict_nodes(trees, x)
    b = oracle.predict(fid, thr, leaf, x)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def paths(trees, t):
    """Every root-to-leaf path of tree t: (list of (feature, threshold, went_left), value)."""
    o = trees["offsets"][t]
    out = []

    def go(i, conds):
        j = o + i
        if trees["left"][j] < 0:
            out.append((conds, trees["value"][j]))
            return
        f, th = int(trees["feature"][j]), float(trees["threshold"][j])
        go(int(trees["left"][j]), conds + [(f, th, True)])
        go(int(trees["right"][j]), conds + [(f, th, False)])

    go(0, [])
    return out


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_brute_force_leaf_is_the_unique_satisfied_path(seed):
    F, vals = 3, 6
    trees = W.make_node_trees(12, 5, F, seed=seed, p_leaf=0.2)
    # thresholds inside the grid, halves and integers
    rng = np.random.default_rng(seed)
    trees["threshold"] = (rng.integers(0, 2 * vals + 1, size=len(trees["left"])) / 2.0).astype(np.float32)
    grid = np.stack(np.meshgrid(*[np.arange(vals)] * F, indexing="ij"), -1).reshape(-1, F).astype(np.int32)
    for t in range(len(trees["offsets"]) - 1):
        one = {k: v for k, v in trees.items()}
        lo, hi = trees["offsets"][t], trees["offsets"][t + 1]
        for k in ("left", "right", "feature", "threshold", "value"):
            one[k] = trees[k][lo:hi]
        one["offsets"] = np.array([0, hi - lo])
        got = oracle.predict_nodes(one, grid)
        ps = paths(trees, t)
        for x, g in zip(grid, got):
            sat = [v for conds, v in ps if all((x[f] < th) == left for f, th, left in conds)]
            assert len(sat) == 1
            assert np.float32(sat[0]) == g


def test_fold_order_is_tree_order():
    # single-leaf trees 1e8, 1, -1e8: ((0 + 1e8) + 1) - 1e8 = 0 in fp32
    trees = {"offsets": [0, 1, 2, 3], "left": [-1] * 3, "right": [-1] * 3, "feature": [0] * 3,
             "threshold": [0.0] * 3, "value": [1e8, 1.0, -1e8]}
    assert oracle.predict_nodes(trees, np.zeros((1, 1), np.int32))[0] == 0.0


def test_extreme_thresholds():
    # a negative threshold never holds for x >= 0; one above 255 always does
    trees = {"offsets": [0, 3, 6], "left": [1, -1, -1, 1, -1, -1], "right": [2, -1, -1, 2, -1, -1],
             "feature": [0, 0, 0, 1, 0, 0], "threshold": [-0.5, 0, 0, 1e6, 0, 0],
             "value": [0, 1.0, 2.0, 0, 4.0, 8.0]}
    x = np.array([[0, 0], [31, 254]], np.int32)
    assert oracle.predict_nodes(trees, x).tolist() == [6.0, 6.0]


@pytest.mark.parametrize("bad", ["child_range", "cycle", "feature_range", "empty_tree"])
def test_rejects_malformed_lists(bad):
    trees = {"offsets": [0, 3], "left": [1, -1, -1], "right": [2, -1, -1], "feature": [0, 0, 0],
             "threshold": [1.0, 0, 0], "value": [0, 1.0, 2.0]}
    if bad == "child_range":
        trees["right"] = [3, -1, -1]
    elif bad == "cycle":
        trees["left"] = [1, 0, -1]
        trees["right"] = [2, 0, -1]
    elif bad == "feature_range":
        trees["feature"] = [2, 0, 0]
    else:
        trees["offsets"] = [0, 0, 3]
    with pytest.raises(ValueError):
        oracle.predict_nodes(trees, np.array([[0, 0], [5, 5]], np.int32))
