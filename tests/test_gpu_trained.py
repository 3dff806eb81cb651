"""GPU parity for trained trees of any shape (Section 3.1): ensembles
imported from node lists (padded to full trees on the host) score rows and
drive annealing runs bit for bit as the oracle does on the lists themselves.
Feature rows given to the oracle come from the oracle or the seeded
generators."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
PATHS = {"trees": 1, "local": 2}


def say(msg):
    print(f"[gpu-trained] {msg}", flush=True)


@pytest.fixture(scope="module")
def P():
    import torch
    torch.cuda.set_device(0)
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def bits(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


def gpu_scores(P, ens, x):
    import torch
    d = torch.from_numpy(np.ascontiguousarray(x, np.int32)).to(DEV)
    s = torch.empty(len(x), dtype=torch.float32, device=DEV)
    lv = torch.empty((len(x), ens.n_trees), dtype=torch.int16, device=DEV)
    P.at_gbt_predict(ens, d, s, lv)
    torch.cuda.synchronize()
    return s.cpu().numpy(), lv.cpu().numpy().view(np.uint16)


def rows(F, n, seed, space=None):
    """Loop-feature rows of random configurations (oracle) followed by
    random small integers, up to n rows."""
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 40, size=(n, F)).astype(np.int32)
    if space is not None:
        m = min(n // 2, 1500)
        x[:m] = space.features(W.make_configs(m, space.n_configs, seed))
    return x


@pytest.mark.parametrize("max_depth,T,F,n", [(6, 300, 110, 4096 + 37), (8, 500, 176, 3000), (10, 200, 176, 1500),
                                             (3, 1000, 192, 2048 + 5), (1, 64, 176, 700), (12, 8, 176, 300)])
def test_imported_trees_score_as_the_oracle(P, max_depth, T, F, n):
    say(f"import depth<={max_depth} T={T} F={F} n={n}")
    trees = W.make_node_trees(T, max_depth, F, seed=70 + max_depth)
    ens = P.at_ensemble_import(trees, F)
    sp = None
    if F == 176:
        sp = oracle.Space(W.CONV2D, W.conv_shape("C2"))
    elif F == 110:
        sp = oracle.Space(W.GEMM, (512, 512, 512))
    x = rows(F, n, 80 + max_depth, sp)
    got, _ = gpu_scores(P, ens, x)
    want = oracle.predict_nodes(trees, x)
    assert np.array_equal(bits(got), bits(want))


def heap_as_nodes(fid, thr, leaf):
    """Full heap trees written as node lists in heap order."""
    T, n_int = fid.shape
    m = 2 * n_int + 1
    h = np.arange(m)
    inner = h < n_int
    left = np.where(inner, 2 * h + 1, -1)
    right = np.where(inner, 2 * h + 2, -1)
    offs = np.arange(T + 1) * m
    feat = np.zeros((T, m), np.int32)
    th = np.zeros((T, m), np.float32)
    val = np.zeros((T, m), np.float32)
    feat[:, :n_int], th[:, :n_int], val[:, n_int:] = fid, thr, leaf
    return {"offsets": offs, "left": np.tile(left, T), "right": np.tile(right, T), "feature": feat.ravel(),
            "threshold": th.ravel(), "value": val.ravel()}


def test_full_trees_import_as_created(P):
    say("full trees: import equals create (scores and leaf indices)")
    F = 176
    fid, thr, leaf = W.make_ensemble(120, 8, F, seed=91)
    a = P.at_ensemble_create(fid, thr, leaf, F)
    b = P.at_ensemble_import(heap_as_nodes(fid, thr, leaf), F)
    x = rows(F, 2000, 92)
    sa, la = gpu_scores(P, a, x)
    sb, lb = gpu_scores(P, b, x)
    assert np.array_equal(bits(sa), bits(sb)) and np.array_equal(la, lb)


def pad_in_test(trees, depth):
    """The test's own padding of node lists to full heap trees, independent
    of the library's: a leaf above the last level repeats under splits that
    always go left (x[0] < 255), thresholds rounded up to integers."""
    T = len(trees["offsets"]) - 1
    n_int = (1 << depth) - 1
    fid = np.zeros((T, n_int), np.uint8)
    thr = np.zeros((T, n_int), np.uint8)
    leaf = np.zeros((T, 1 << depth), np.float32)
    for t in range(T):
        o = trees["offsets"][t]
        todo = [(0, 0, 0)]       # heap node, list node, level
        while todo:
            h, i, lev = todo.pop()
            j = o + i
            if lev == depth:
                leaf[t, h - n_int] = trees["value"][j]
                continue
            if trees["left"][j] >= 0:
                fid[t, h] = trees["feature"][j]
                thr[t, h] = int(np.clip(np.ceil(np.float64(trees["threshold"][j])), 0, 255))
                todo += [(2 * h + 1, trees["left"][j], lev + 1), (2 * h + 2, trees["right"][j], lev + 1)]
            else:
                fid[t, h], thr[t, h] = 0, 255
                todo += [(2 * h + 1, i, lev + 1), (2 * h + 2, i, lev + 1)]
    return fid, thr, leaf


@pytest.mark.parametrize("path", sorted(PATHS))
def test_annealing_with_imported_trees(P, path):
    import torch
    say(f"annealing with imported trees, path {path}")
    shape = W.conv_shape("C2")
    sp, osp = P.at_space_create(W.CONV2D, shape), oracle.Space(W.CONV2D, shape)
    F = osp.n_features
    trees = W.make_node_trees(150, 8, F, seed=93, p_leaf=0.15)
    depth = max(1, oracle_depth(trees))
    ens_t = pad_in_test(trees, depth)
    x = rows(F, 600, 94, osp)
    # the test's padding reaches the oracle's node-list scores
    assert np.array_equal(bits(oracle.predict(*ens_t, x)), bits(oracle.predict_nodes(trees, x)))
    ens = P.at_ensemble_import(trees, F)
    n, k, steps, seed = 128, 8, 60, 2101
    ch = P.at_chains_create(sp, 0, n, k, seed)
    P.at_chains_set_path(ch, PATHS[path])
    d_thr = torch.from_numpy(P.at_sa_thresholds(seed, 0, n, 0, steps)).to(DEV)
    best = torch.zeros((n, k, 4), dtype=torch.int32, device=DEV)
    P.at_sa_run(sp, ens, ch, steps, d_thr, best)
    torch.cuda.synchronize()
    assert P.at_chains_last_path(ch) == PATHS[path]
    got = P.entries(best)
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    och.run(ens_t, steps, oracle.thresholds(seed, 0, n, 0, steps))
    assert np.array_equal(got["flag"], och.top["valid"])
    assert np.array_equal(got["cfg"], och.top["cfg"])
    assert np.array_equal(bits(got["score"]), bits(och.top["score"]))


def oracle_depth(trees):
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
