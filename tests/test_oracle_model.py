"""Oracle pins: tree-ensemble prediction (Section 3.1), Philox and thresholds."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))


def single_tree(depth, fid, thr, leaf):
    n_int = (1 << depth) - 1
    return (np.full((1, n_int), fid, np.uint8) if np.isscalar(fid) else np.asarray(fid, np.uint8).reshape(1, n_int),
            np.full((1, n_int), thr, np.uint8) if np.isscalar(thr) else np.asarray(thr, np.uint8).reshape(1, n_int),
            np.asarray(leaf, np.float32).reshape(1, 1 << depth))


def test_stump_closed_form():
    # depth 1: score = leaf[0] if x[f] < t else leaf[1]
    fid, thr, leaf = single_tree(1, 3, 10, [-0.5, 0.25])
    x = np.zeros((40, 8), np.int32)
    x[:, 3] = np.arange(40)
    s = oracle.predict(fid, thr, leaf, x)
    assert (s == np.where(np.arange(40) < 10, np.float32(-0.5), np.float32(0.25))).all()


@pytest.mark.parametrize("depth", [1, 3, 6, 8, 10])
def test_path_bits_tree(depth):
    # node at level l tests feature l against threshold 1, and every leaf holds
    # its own index: the leaf reached spells x_0 .. x_{d-1} in binary (MSB
    # first), since "x >= thr" takes the right child.
    n_int = (1 << depth) - 1
    level_of = np.floor(np.log2(np.arange(n_int) + 1)).astype(np.int64)
    fid, thr, leaf = single_tree(depth, level_of, 1, np.arange(1 << depth, dtype=np.float32))
    rng = np.random.default_rng(depth)
    bits = rng.integers(0, 2, size=(64, depth)).astype(np.int32)
    x = np.zeros((64, 16), np.int32)
    x[:, :depth] = bits
    want = (bits * (1 << np.arange(depth - 1, -1, -1))).sum(1)
    s, leaves = oracle.predict(fid, thr, leaf, x, want_leaves=True)
    assert (leaves[:, 0] == want).all()
    assert (s == want.astype(np.float32)).all()


def test_threshold_direction_and_extremes():
    fid, thr, leaf = single_tree(4, 0, 0, np.arange(16))
    x = np.zeros((3, 4), np.int32)
    assert (oracle.predict(fid, thr, leaf, x) == 15).all()   # x >= 0 always: rightmost leaf
    fid, thr, leaf = single_tree(4, 0, 33, np.arange(16))
    x[:] = 32
    assert (oracle.predict(fid, thr, leaf, x) == 0).all()    # 32 < 33: leftmost leaf


def test_fold_order_is_tree_order():
    # ((0 + 1e8) + -1e8) + 1 = 1, whereas 1e8 + (-1e8 + 1) rounds to 0 in fp32
    T = 3
    fid = np.zeros((T, 1), np.uint8)
    thr = np.full((T, 1), 33, np.uint8)
    leaf = np.array([[1e8, 0], [-1e8, 0], [1.0, 0]], np.float32)
    s = oracle.predict(fid, thr, leaf, np.zeros((1, 2), np.int32))
    assert s[0] == np.float32(1.0)
    # reversed order lands elsewhere
    s2 = oracle.predict(fid, thr, leaf[::-1].copy(), np.zeros((1, 2), np.int32))
    assert s2[0] == np.float32(0.0)


def test_generated_ensemble_sum_within_rounding_bound():
    fid, thr, leaf = workloads.make_ensemble(300, 8, 176, 99)
    sp = oracle.Space(workloads.CONV2D, workloads.conv_shape("C2"))
    x = sp.features(workloads.make_configs(50, sp.n_configs, 1))
    s, leaves = oracle.predict(fid, thr, leaf, x, want_leaves=True)
    vals = leaf.astype(np.float64)[np.arange(300)[None, :], leaves.astype(np.int64)]
    exact = vals.sum(1)
    bound = 300 * np.finfo(np.float32).eps * np.abs(vals).sum(1)
    assert (np.abs(s.astype(np.float64) - exact) <= bound).all()
    # leaf index really is the path: check each tree's node decisions
    n_int = 255
    for r in range(5):
        for t in range(0, 300, 37):
            n = 0
            for _ in range(8):
                n = 2 * n + (1 if x[r, fid[t, n]] >= thr[t, n] else 0) + 1
            assert n - n_int == leaves[r, t]


def test_predict_rejects_bad_feature_ids():
    fid, thr, leaf = single_tree(2, 9, 1, np.zeros(4))
    with pytest.raises(ValueError):
        oracle.predict(fid, thr, leaf, np.zeros((1, 4), np.int32))


def rocrand_blocks(queries):
    exe = os.path.join("/tmp", f"rocrand_philox_blocks_{os.getpid()}")
    src = os.path.join(HERE, "golden", "rocrand_philox_blocks.cpp")
    subprocess.run(["hipcc", "-O1", "-o", exe, src], check=True, capture_output=True, cwd="/tmp")
    inp = "\n".join(" ".join(str(int(v)) for v in q) for q in queries) + "\n"
    out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
    os.unlink(exe)
    return np.array([[int(v) for v in line.split()] for line in out.strip().splitlines()], dtype=np.uint64)


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc (rocRAND headers) not available")
def test_philox_matches_rocrand():
    rng = np.random.default_rng(42)
    queries = [(0, 0, 0, 0, 0), (7, 0, 0, 0, 0), (2003, 5, 999, 0, 0), (2000, 63, 499, 0, 0)]
    for _ in range(60):
        seed = int(rng.integers(0, 2**63))
        c = rng.integers(0, 2**32, size=4, dtype=np.uint64)
        c[1] %= 2**29   # rocRAND's offset is counter*4 in 64 bits
        queries.append((seed, *[int(v) for v in c]))
    ref = rocrand_blocks(queries)
    for q, r in zip(queries, ref):
        got = oracle.philox(q[0], q[1:])
        assert list(got.astype(np.uint64)) == list(r), q


def test_thresholds_shape_and_schedule():
    thr = oracle.thresholds(2000, 0, 16, 0, 200)
    assert thr.dtype == np.float32 and thr.shape == (16, 200)
    assert (thr <= 0).all()
    # last step: T = 0, threshold is -0.0 (ties and improvements accepted)
    assert (thr[:, -1] == 0).all() and np.signbit(thr[:, -1]).all()
    # T_s*ln(u) / T_s = ln(u): u = exp(thr/T_s) must be uniform on (0,1)
    T = 1.0 - np.arange(199) / 199.0
    u = np.exp(thr[:, :199].astype(np.float64) / T[None, :]).ravel()
    assert 0 < u.min() and u.max() < 1
    hist = np.histogram(u, bins=10, range=(0, 1))[0]
    expected = len(u) / 10
    chi2 = ((hist - expected) ** 2 / expected).sum()
    assert chi2 < 30   # 9 dof; p ~ 4e-4
    one = oracle.thresholds(2000, 0, 4, 0, 1)
    assert (one == 0).all() and np.signbit(one).all()


def test_thresholds_use_the_step_blocks_third_word():
    # T_0 = 1: thr[c][0] = fp32(ln(u)), u = (r2 + 0.5) / 2^32 of block (chain, step)
    seed, c0, base = 77, 10, 300
    thr = oracle.thresholds(seed, c0, 3, base, 5)
    for c in range(3):
        r = oracle.philox(seed, [c0 + c, base, 0, 0])
        assert thr[c, 0] == np.float32(np.log((float(r[2]) + 0.5) / 2**32))
        r4 = oracle.philox(seed, [c0 + c, base + 4, 0, 0])
        assert thr[c, 4] == np.float32(0.0 * np.log((float(r4[2]) + 0.5) / 2**32))
    # chain0 / step_base select rows and blocks: a wider table's row for the
    # same global chain at T = 1 holds the same value
    big = oracle.thresholds(seed, c0 - 2, 6, base, 9)
    assert (big[2:5, 0] == thr[:, 0]).all()


# --------------------------------------------------------------------------
# Eq. 4: global + local model
# --------------------------------------------------------------------------
def single_tree_model(leaves):
    """Depth-1 stumps on feature 0 with threshold 0: every row (x >= 0)
    reaches leaf 1, so the prediction is the fold of leaves[t][1]."""
    T = len(leaves)
    fid = np.zeros((T, 1), np.uint8)
    thr = np.zeros((T, 1), np.uint8)
    leaf = np.zeros((T, 2), np.float32)
    leaf[:, 1] = leaves
    return fid, thr, leaf


def test_global_local_is_a_sum_of_two_folds():
    """Each model folds its own trees and the two results are added once:
    global (1e8, 1) folds to 1e8 (1e8 + 1 rounds back), local (-1e8, 1) to
    -1e8, so the sum is 0; one fold over the concatenated trees would give 1."""
    x = np.zeros((3, 4), np.int32)
    g = single_tree_model([1e8, 1.0])
    l = single_tree_model([-1e8, 1.0])
    got = oracle.predict_global_local(g, x, l, x)
    assert (got == 0.0).all()
    both = single_tree_model([1e8, 1.0, -1e8, 1.0])
    assert (oracle.predict(*both, x) == 1.0).all()


def test_global_local_special_cases():
    rng = np.random.default_rng(5)
    fid, thr, leaf = workloads.make_ensemble(40, 5, 20, 17)
    feats = rng.integers(0, 33, (300, 20)).astype(np.int32)
    g = oracle.predict(fid, thr, leaf, feats)
    zero = (fid, thr, np.zeros_like(leaf))
    assert np.array_equal(oracle.predict_global_local((fid, thr, leaf), feats, zero, feats), g + np.float32(0.0))
    neg = (fid, thr, -leaf)
    assert (oracle.predict_global_local((fid, thr, leaf), feats, neg, feats) == 0.0).all()
    # different feature sets for the two models
    fid2, thr2, leaf2 = workloads.make_ensemble(25, 3, 7, 18)
    f2 = rng.integers(0, 33, (300, 7)).astype(np.int32)
    want = (g.astype(np.float64) + oracle.predict(fid2, thr2, leaf2, f2)).astype(np.float32)
    assert np.array_equal(oracle.predict_global_local((fid, thr, leaf), feats, (fid2, thr2, leaf2), f2), want)
