"""CPU checks of the C-ABI library: it loads, exports every declared entry
point, validates arguments before touching the device, and its host-side
threshold helper agrees bit for bit with the oracle's."""
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "autotensor.h")


@pytest.fixture(scope="module")
def P():
    from paper_1805_08166_amd import build as B
    if B.stale():
        B.build()
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(at_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(P):
    names = declared_functions()
    assert len(names) >= 17
    for n in names:
        assert hasattr(P.lib(), n), n
    assert sorted(P.EXPORTED) == names


def test_thresholds_match_oracle_bitwise(P):
    for seed, chain0, n, base, steps in [(2000, 0, 64, 0, 500), (2003, 100, 17, 250, 33), (7, 5, 3, 0, 1),
                                         (2 ** 40 + 5, 2 ** 31, 4, 2 ** 31, 9)]:
        got = P.at_sa_thresholds(seed, chain0, n, base, steps)
        want = oracle.thresholds(seed, chain0, n, base, steps)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def expect_status(P, fn, status):
    with pytest.raises(P.ATError) as ei:
        fn()
    assert ei.value.status == status, str(ei.value)


def test_argument_errors_before_device_use(P):
    INVALID, UNSUPPORTED = -1, -2
    expect_status(P, lambda: P.at_space_create(0, (0, 4, 4)), INVALID)
    expect_status(P, lambda: P.at_space_create(0, (4, 4)), INVALID)
    expect_status(P, lambda: P.at_space_create(7, (4, 4, 4)), INVALID)
    expect_status(P, lambda: P.at_space_create(1, (2, 4, 8, 8, 4, 3, 3, 1, 1)), INVALID)
    expect_status(P, lambda: P.at_space_create(1, (1, 4, 2, 2, 4, 5, 5, 0, 1)), INVALID)
    expect_status(P, lambda: P.at_space_create(0, (70000, 4, 4)), UNSUPPORTED)
    # 2^31 iterations or more
    expect_status(P, lambda: P.at_space_create(0, (2048, 2048, 1024)), UNSUPPORTED)
    expect_status(P, lambda: P.at_sa_thresholds(1, 0, 4, 0, 0), INVALID)
    fid = np.zeros((2, 3), np.uint8)
    thr = np.zeros((2, 3), np.uint8)
    leaf = np.zeros((2, 4), np.float32)
    expect_status(P, lambda: P.at_ensemble_create(fid + 9, thr, leaf, 8), INVALID)   # fid >= F
    expect_status(P, lambda: P.at_ensemble_create(fid, thr, leaf, 300), UNSUPPORTED)
    deep = np.zeros((1, (1 << 13) - 1), np.uint8)
    expect_status(P, lambda: P.at_ensemble_create(deep, deep, np.zeros((1, 1 << 13), np.float32), 8), UNSUPPORTED)
    assert "depth" in P.lib().at_last_error().decode()
    assert P.lib().at_sa_set_profiling(None, 1) == INVALID
    assert P.lib().at_sa_kernel_times(None, None, None, None, None) == INVALID
    assert P.lib().at_chains_set_path(None, 1) == INVALID
    assert P.lib().at_chains_last_plan(None, None) == INVALID
    assert P.lib().at_select_batch(None, None, 0, 4, 2, 1.0, 1, 0, None, None) == INVALID


def bitlen(x):
    return int(x).bit_length()


def test_quotient_bitlen_identity():
    # The feature kernels compute bitlen(a // b) as k + (a >> k >= b) with
    # k = bitlen(a) - bitlen(b), for a >= b >= 1.
    def fast(a, b):
        k = bitlen(a) - bitlen(b)
        return k + (1 if (a >> k) >= b else 0)
    for a in range(1, 600):
        for b in range(1, a + 1):
            assert fast(a, b) == bitlen(a // b)
    rng = np.random.default_rng(0)
    for _ in range(20000):
        a = int(rng.integers(1, 2 ** 31))
        b = int(rng.integers(1, a + 1))
        assert fast(a, b) == bitlen(a // b)


# --------------------------------------------------------------------------
# trained trees of any shape: the library's host-side padding to full trees
# --------------------------------------------------------------------------
def heap_walk(fid, thr, leaf, x):
    """Scores of full heap trees (node h: x[fid] < thr -> 2h+1, else 2h+2),
    an fp32 left fold in tree order."""
    T, n_int = fid.shape
    depth = (n_int + 1).bit_length() - 1
    out = np.zeros(len(x), np.float32)
    for i, row in enumerate(x):
        s = np.float32(0)
        for t in range(T):
            h = 0
            for _ in range(depth):
                h = 2 * h + 1 if row[fid[t, h]] < thr[t, h] else 2 * h + 2
            s = np.float32(s + leaf[t, h - n_int])
        out[i] = s
    return out


def tree_levels(trees):
    deepest = 0
    for t in range(len(trees["offsets"]) - 1):
        o = trees["offsets"][t]
        stack = [(0, 0)]
        while stack:
            i, lev = stack.pop()
            if trees["left"][o + i] < 0:
                deepest = max(deepest, lev)
            else:
                stack += [(trees["left"][o + i], lev + 1), (trees["right"][o + i], lev + 1)]
    return deepest


@pytest.mark.parametrize("max_depth,T,F,extra", [(3, 30, 7, 0), (6, 40, 110, 0), (5, 25, 176, 2), (1, 9, 4, 0)])
def test_padded_trees_reach_the_oracle_scores(P, max_depth, T, F, extra):
    import workloads as W
    trees = W.make_node_trees(T, max_depth, F, seed=50 + max_depth)
    d = P.at_trees_depth(trees)
    assert d == tree_levels(trees)
    fid, thr, leaf = P.at_trees_pad(trees, F, max(1, d) + extra)
    rng = np.random.default_rng(max_depth)
    x = rng.integers(0, 40, size=(200, F)).astype(np.int32)
    x[:4] = [0, 254, 33, 1][:4] if F == 1 else np.array([0, 254, 33, 1])[:, None]
    want = oracle.predict_nodes(trees, x)
    assert np.array_equal(heap_walk(fid, thr, leaf, x).view(np.uint32), want.view(np.uint32))


def test_padding_of_the_worked_example(P):
    import json
    with open(os.path.join(ROOT, "tests", "golden", "trained_trees_worked_example.json")) as f:
        g = json.load(f)
    assert P.at_trees_depth(g["trees"]) == 3
    fid, thr, leaf = P.at_trees_pad(g["trees"], g["n_features"], 3)
    # tree A (one leaf) is eight copies of 0.5 under always-left splits
    assert (leaf[0] == 0.5).all() and (thr[0] == 255).all()
    # tree B's stump: threshold 3.5 becomes 4; each side copied below
    assert fid[1, 0] == 2 and thr[1, 0] == 4
    assert leaf[1].tolist() == [-0.25] * 4 + [0.125] * 4
    assert heap_walk(fid, thr, leaf, np.asarray(g["rows"])).tolist() == g["scores"]


def test_xgboost_dump_parses_to_the_worked_example(P):
    import json
    from paper_1805_08166_amd.xgboost_dump import trees_from_xgboost_dump
    with open(os.path.join(ROOT, "tests", "golden", "trained_trees_worked_example.json")) as f:
        g = json.load(f)
    trees = trees_from_xgboost_dump(g["xgboost_dump"])
    assert trees["offsets"].tolist() == [0, 1, 4, 11]
    assert P.at_trees_depth(trees) == 3
    fid, thr, leaf = P.at_trees_pad(trees, g["n_features"], 3)
    assert heap_walk(fid, thr, leaf, np.asarray(g["rows"])).tolist() == g["scores"]
    with pytest.raises(ValueError):
        trees_from_xgboost_dump(['{"nodeid": 0, "split": "f1", "split_condition": 1, "yes": 1, "no": 2, '
                                 '"children": [{"nodeid": 1, "leaf": 0.5}]}'])


def test_tree_list_errors(P):
    INVALID, UNSUPPORTED = -1, -2
    ok = {"offsets": [0, 3], "left": [1, -1, -1], "right": [2, -1, -1], "feature": [1, 0, 0],
          "threshold": [1.5, 0, 0], "value": [0, 1.0, 2.0]}

    def bad(**kw):
        t = dict(ok)
        t.update(kw)
        return t

    assert P.at_trees_depth(ok) == 1
    expect_status(P, lambda: P.at_trees_depth(bad(right=[3, -1, -1])), INVALID)       # child out of range
    expect_status(P, lambda: P.at_trees_depth(bad(right=[1, -1, -1])), INVALID)       # node reached twice
    expect_status(P, lambda: P.at_trees_depth(bad(left=[1, 0, -1], right=[2, 2, -1])), INVALID)  # cycle
    expect_status(P, lambda: P.at_trees_depth(bad(offsets=[0, 0, 3])), INVALID)      # empty tree
    expect_status(P, lambda: P.at_trees_pad(bad(feature=[2, 0, 0]), 2, 1), INVALID)   # feature out of range
    expect_status(P, lambda: P.at_trees_pad(bad(threshold=[float("nan"), 0, 0]), 2, 1), INVALID)
    expect_status(P, lambda: P.at_trees_pad(ok, 2, 13), UNSUPPORTED)
    deep = {"offsets": [0, 5], "left": [1, 3, -1, -1, -1], "right": [2, 4, -1, -1, -1], "feature": [0] * 5,
            "threshold": [1.0] * 5, "value": [0.0] * 5}
    expect_status(P, lambda: P.at_trees_pad(deep, 2, 1), INVALID)                      # leaf below depth
    # a left spine of 13 splits, each with a leaf on its right: deeper than
    # any supported ensemble
    left = [i + 1 if i < 13 else -1 for i in range(14)] + [-1] * 13
    right = [14 + i if i < 13 else -1 for i in range(14)] + [-1] * 13
    chain = {"offsets": [0, 27], "left": left, "right": right, "feature": [0] * 27, "threshold": [1.0] * 27,
             "value": [0.0] * 27}
    assert P.at_trees_depth(chain) == 13
    expect_status(P, lambda: P.at_ensemble_import(chain, 2), UNSUPPORTED)
