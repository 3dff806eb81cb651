"""GPU parity: the HIP path against the CPU oracle, bit for bit.

Features are int32 and compared exactly; scores are fp32 left folds in tree
order and compared bitwise (tolerance 0 ulp); annealing trajectories (proposed
configuration, its score, accept flag per step), final states and best lists
are compared exactly.  Every call goes through the C ABI.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(f"[gpu-parity] {msg}", flush=True)


@pytest.fixture(scope="module")
def P():
    import torch
    torch.cuda.set_device(0)
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def u64_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(DEV)


def gpu_features(P, sp, cfgs):
    import torch
    d = u64_dev(cfgs)
    out = torch.empty((len(cfgs), sp.n_features), dtype=torch.int32, device=DEV)
    P.at_extract_features(sp, d, out)
    torch.cuda.synchronize()
    return out


def gpu_predict(P, ens, feats_dev, leaves=False):
    import torch
    n = feats_dev.shape[0]
    s = torch.empty(n, dtype=torch.float32, device=DEV)
    lv = torch.empty((n, ens.n_trees), dtype=torch.int16, device=DEV) if leaves else None
    P.at_gbt_predict(ens, feats_dev, s, lv)
    torch.cuda.synchronize()
    return s.cpu().numpy(), (lv.cpu().numpy().view(np.uint16) if leaves else None)


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


# --------------------------------------------------------------------------
# features
# --------------------------------------------------------------------------
TINY = [(W.GEMM, (4, 4, 4)), (W.GEMM, (2, 6, 3)), (W.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1)),
        (W.CONV2D, (1, 2, 6, 6, 2, 3, 3, 1, 2)), (W.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2)),
        (W.CONV2D, (1, 1, 8, 8, 2, 7, 7, 3, 2)), (W.CONV2D, (1, 3, 5, 5, 4, 2, 2, 0, 3))]


@pytest.mark.parametrize("tmpl,shape", TINY)
def test_features_every_config_of_small_spaces(P, tmpl, shape):
    say(f"features exhaustive {shape}")
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    assert sp.n_configs == osp.n_configs and list(sp.knob_sizes) == list(osp.knob_sizes)
    cfgs = np.arange(osp.n_configs, dtype=np.uint64)
    got = gpu_features(P, sp, cfgs).cpu().numpy()
    assert np.array_equal(got, osp.features(cfgs))


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C5", "C10", "C12"])
def test_features_table1_shapes_sampled(P, name):
    say(f"features {name}")
    shape = W.conv_shape(name)
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    cfgs = W.make_configs(20011, osp.n_configs, 11)   # ragged: not a multiple of 256
    assert np.array_equal(gpu_features(P, sp, cfgs).cpu().numpy(), osp.features(cfgs))


def test_features_batched_scoring_workload_full_size(P):
    # 1,048,576 random configurations of the C2 conv space: every row compared
    wl = W.WORKLOADS["conv_c2_score1m"]
    tmpl, shape = wl["spaces"][0]
    say("features 1M C2")
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    cfgs = W.make_configs(wl["n_cfgs"], osp.n_configs, wl["cfg_seed"])
    got = gpu_features(P, sp, cfgs).cpu().numpy()
    assert np.array_equal(got, osp.features(cfgs))


def test_features_gemm_512_sampled(P):
    sp = P.at_space_create(W.GEMM, W.GEMM_512)
    osp = oracle.Space(W.GEMM, W.GEMM_512)
    cfgs = W.make_configs(50000, osp.n_configs, 3)
    assert np.array_equal(gpu_features(P, sp, cfgs).cpu().numpy(), osp.features(cfgs))


def test_features_out_of_range_rows_and_unaligned_output(P):
    import torch
    shape = W.conv_shape("C2")
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    cfgs = W.make_configs(1000, osp.n_configs, 5)
    bad = [3, 500, 999]
    cfgs[bad] = [osp.n_configs, osp.n_configs + 12345, np.uint64(2 ** 63)]
    P.at_space_errors(sp)
    # output view 4 bytes past a 16-byte boundary: scalar store path
    buf = torch.empty(1000 * 176 + 1, dtype=torch.int32, device=DEV)
    out = buf[1:].view(1000, 176)
    P.at_extract_features(sp, u64_dev(cfgs), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert P.at_space_errors(sp) == 3
    assert (got[bad] == -1).all()
    good = np.setdiff1d(np.arange(1000), bad)
    assert np.array_equal(got[good], osp.features(cfgs[good]))
    # n == 0 is a no-op
    empty = torch.empty((0, 176), dtype=torch.int32, device=DEV)
    P.at_extract_features(sp, u64_dev(np.zeros(0, np.uint64)), empty)
    with pytest.raises(P.ATError):
        P.at_extract_features(P.at_spaceset_create([sp, sp], [0, 1, 2]), u64_dev(cfgs), out)


# --------------------------------------------------------------------------
# ensemble scoring
# --------------------------------------------------------------------------
@pytest.mark.parametrize("depth,trees,F", [(1, 5, 13), (3, 37, 110), (5, 9, 176), (6, 100, 110), (8, 37, 176),
                                           (10, 11, 176), (11, 3, 64), (12, 2, 176), (1, 700, 176), (2, 1029, 176),
                                           (6, 101, 176), (7, 33, 176), (8, 1, 176), (9, 6, 176), (11, 5, 176)])
def test_predict_matches_oracle_with_leaf_indices(P, depth, trees, F):
    import torch
    say(f"predict depth {depth} trees {trees} F {F}")
    fid, thr, leaf = W.make_ensemble(trees, depth, F, 1000 + depth)
    ens = P.at_ensemble_create(fid, thr, leaf, F)
    rng = np.random.default_rng(depth)
    n = 777
    x = rng.integers(0, 34, size=(n, F)).astype(np.int32)
    s, lv = gpu_predict(P, ens, torch.from_numpy(x).to(DEV), leaves=True)
    ws, wl = oracle.predict(fid, thr, leaf, x, want_leaves=True)
    assert np.array_equal(lv, wl)
    assert np.array_equal(bits(s), bits(ws))


@pytest.mark.parametrize("depth,trees,F,thr_hi", [(1, 530, 176, 64), (2, 259, 192, 64), (5, 70, 176, 64),
                                                   (7, 19, 192, 64), (8, 15, 176, 64), (8, 13, 192, 64),
                                                   (8, 11, 176, 256), (6, 9, 192, 256)])
def test_predict_wide_thresholds_and_clamped_features(P, depth, trees, F, thr_hi):
    # thresholds up to 63 or 255 and features up to 300 (clamped to 255 on
    # the device, where x >= thr keeps its value); tree counts leave a
    # partial last chunk of the scoring kernel's tree stream
    import torch
    say(f"predict depth {depth} trees {trees} F {F} thresholds < {thr_hi}")
    rng = np.random.default_rng(7 * depth + trees)
    n_int = (1 << depth) - 1
    fid = rng.integers(0, F, size=(trees, n_int)).astype(np.uint8)
    thr = rng.integers(0, thr_hi, size=(trees, n_int)).astype(np.uint8)
    leaf = (rng.standard_normal((trees, 1 << depth)) * 0.05).astype(np.float32)
    ens = P.at_ensemble_create(fid, thr, leaf, F)
    n = 1037
    x = rng.integers(0, 301, size=(n, F)).astype(np.int32)
    xd = torch.from_numpy(x).to(DEV)
    s, _ = gpu_predict(P, ens, xd)
    s_l, lv = gpu_predict(P, ens, xd, leaves=True)
    ws, wl = oracle.predict(fid, thr, leaf, x, want_leaves=True)
    assert np.array_equal(bits(s), bits(ws))
    assert np.array_equal(bits(s_l), bits(ws)) and np.array_equal(lv, wl)


def test_predict_fold_order(P):
    import torch
    fid = np.zeros((3, 1), np.uint8)
    thr = np.full((3, 1), 33, np.uint8)
    leaf = np.array([[1e8, 0], [-1e8, 0], [1.0, 0]], np.float32)
    ens = P.at_ensemble_create(fid, thr, leaf, 2)
    s, _ = gpu_predict(P, ens, torch.zeros((5, 2), dtype=torch.int32, device=DEV))
    assert (s == 1.0).all()


def test_predict_batched_scoring_workload_full_size(P):
    wl = W.WORKLOADS["conv_c2_score1m"]
    tmpl, shape = wl["spaces"][0]
    say("predict 1M x 1000 trees")
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    cfgs = W.make_configs(wl["n_cfgs"], osp.n_configs, wl["cfg_seed"])
    feats = gpu_features(P, sp, cfgs)
    s, _ = gpu_predict(P, ens, feats)
    idx = np.random.default_rng(0).choice(len(cfgs), size=20000, replace=False)
    idx = np.concatenate([idx, [0, len(cfgs) - 1]])
    want = oracle.predict(fid, thr, leaf, osp.features(cfgs[idx]))
    assert np.array_equal(bits(s[idx]), bits(want))


# --------------------------------------------------------------------------
# annealing
# --------------------------------------------------------------------------
PATHS = {"trees": 1, "local": 2}


@pytest.fixture(params=sorted(PATHS))
def path(request):
    return request.param


def mk_chains(P, sp, chain0, n, k, seed, path):
    ch = P.at_chains_create(sp, chain0, n, k, seed)
    P.at_chains_set_path(ch, PATHS[path])
    ch.path_name = path
    return ch


def gpu_sa(P, sp, ens, chains, steps, thr, traced=True):
    import torch
    d_thr = torch.from_numpy(np.ascontiguousarray(thr, np.float32)).to(DEV)
    best = torch.zeros((chains.n_chains, chains.topk, 4), dtype=torch.int32, device=DEV)
    if traced:
        tr = torch.zeros((chains.n_chains, steps, 4), dtype=torch.int32, device=DEV)
        P.at_sa_run_traced(sp, ens, chains, steps, d_thr, best, tr)
    else:
        tr = None
        P.at_sa_run(sp, ens, chains, steps, d_thr, best)
    torch.cuda.synchronize()
    want = getattr(chains, "path_name", None)
    if want is not None and chains.n_chains > 0:
        assert P.at_chains_last_path(chains) == PATHS[want], "the run took the other path"
    return P.entries(best), (P.entries(tr) if traced else None)


def export(P, chains):
    import torch
    cfg = torch.zeros(chains.n_chains, dtype=torch.int64, device=DEV)
    sc = torch.zeros(chains.n_chains, dtype=torch.float32, device=DEV)
    P.at_chains_export(chains, cfg, sc)
    torch.cuda.synchronize()
    return cfg.cpu().numpy().view(np.uint64), sc.cpu().numpy()


def assert_same_run(best, tr, och, otr, rows=None, cur=None):
    rows = slice(None) if rows is None else rows
    if tr is not None:
        assert np.array_equal(tr["cfg"][rows], otr["cfg"]), "proposed configurations differ"
        assert np.array_equal(bits(tr["score"][rows]), bits(otr["score"])), "scores differ"
        assert np.array_equal(tr["flag"][rows], otr["valid"]), "accept decisions differ"
    assert np.array_equal(best["flag"][rows], och.top["valid"])
    assert np.array_equal(best["cfg"][rows], och.top["cfg"])
    assert np.array_equal(bits(best["score"][rows]), bits(och.top["score"]))
    if cur is not None:
        cfg, sc = cur
        assert np.array_equal(cfg[rows], och.cur_cfgs())
        assert np.array_equal(bits(sc[rows]), bits(och.score))


def sa_case(P, name, n_gpu, n_oracle, steps=None, oracle_rows=None):
    wl = W.WORKLOADS[name]
    steps = wl["steps"] if steps is None else steps
    spaces = [P.at_space_create(t, s) for t, s in wl["spaces"]]
    ospaces = [oracle.Space(t, s) for t, s in wl["spaces"]]
    F = ospaces[0].n_features
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], F, wl["ens_seed"])
    ens = P.at_ensemble_create(fid, thr, leaf, F)
    seed, k = wl["sa_seed"], wl["topk"]
    return spaces, ospaces, (fid, thr, leaf), ens, seed, k, steps


def test_sa_gemm_workload_full(P, path):
    say("sa gemm512 64x500 full")
    spaces, ospaces, ens_t, ens, seed, k, steps = sa_case(P, "gemm512_sa", 64, 64)
    n = 64
    ch = mk_chains(P, spaces[0], 0, n, k, seed, path)
    thr_g = P.at_sa_thresholds(seed, 0, n, 0, steps)
    best, tr = gpu_sa(P, spaces[0], ens, ch, steps, thr_g)
    cur = export(P, ch)
    och = oracle.Chains(ospaces, [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run(ens_t, steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=cur)


def test_sa_conv_c2_workload_full_gpu_sliced_oracle(P, path):
    say("sa conv C2 1024x500, oracle on 2 slices")
    spaces, ospaces, ens_t, ens, seed, k, steps = sa_case(P, "conv_c2_sa", 1024, 0)
    n = 1024
    ch = mk_chains(P, spaces[0], 0, n, k, seed, path)
    best, tr = gpu_sa(P, spaces[0], ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    cur = export(P, ch)
    for lo, hi in [(0, 96), (1000, 1024)]:
        och = oracle.Chains(ospaces, [0, hi - lo], seed=seed, chain0=lo, topk=k)
        otr = och.run(ens_t, steps, oracle.thresholds(seed, lo, hi - lo, 0, steps), trace=True)
        assert_same_run(best, tr, och, otr, rows=slice(lo, hi), cur=cur)


def test_sa_conv_c12_deep_ensemble_short(P, path):
    say("sa conv C12 2000 trees depth 10, 300 chains x 12 steps")
    spaces, ospaces, ens_t, ens, seed, k, _ = sa_case(P, "conv_c12_sa", 300, 300)
    n, steps = 300, 12
    ch = mk_chains(P, spaces[0], 0, n, k, seed, path)
    best, tr = gpu_sa(P, spaces[0], ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    och = oracle.Chains(ospaces, [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run(ens_t, steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_sa_twelve_workload_set_short(P, path):
    say("sa 12-workload set, 40 chains each x 60 steps")
    wl = W.WORKLOADS["resnet18_12conv_sa"]
    spaces = [P.at_space_create(t, s) for t, s in wl["spaces"]]
    ospaces = [oracle.Space(t, s) for t, s in wl["spaces"]]
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    off = W.chain_offsets(12, 40)
    sset = P.at_spaceset_create(spaces, off)
    n, steps, seed, k = int(off[-1]), 60, wl["sa_seed"], wl["topk"]
    ch = mk_chains(P, sset, 0, n, k, seed, path)
    best, tr = gpu_sa(P, sset, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    och = oracle.Chains(ospaces, off, seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_sa_ragged_set_offsets(P, path):
    shapes = [(1, 2, 4, 4, 2, 3, 3, 1, 1), (1, 2, 6, 6, 2, 1, 1, 0, 2), (1, 1, 8, 8, 2, 7, 7, 3, 2)]
    spaces = [P.at_space_create(W.CONV2D, s) for s in shapes]
    ospaces = [oracle.Space(W.CONV2D, s) for s in shapes]
    off = np.array([0, 5, 300, 301], np.int64)
    fid, thr, leaf = W.make_ensemble(30, 6, 176, 8)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    sset = P.at_spaceset_create(spaces, off)
    n, steps, seed, k = 301, 50, 21, 4
    ch = mk_chains(P, sset, 7, n, k, seed, path)
    best, tr = gpu_sa(P, sset, ens, ch, steps, P.at_sa_thresholds(seed, 7, n, 0, steps))
    och = oracle.Chains(ospaces, off, seed=seed, chain0=7, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 7, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_sa_split_tables_past_the_lds_image(P, path):
    # GEMM (720, 720, 64): 2807 split choices, more than an LDS space image
    # holds, so the tree path's chain kernel reads the space from global
    # memory; a set pairs it with a space whose image fits (blocks of 16
    # chains take either)
    big, small = (720, 720, 64), (64, 32, 128)
    fid, thr, leaf = W.make_ensemble(40, 6, 110, 17)
    ens = P.at_ensemble_create(fid, thr, leaf, 110)
    sp = P.at_space_create(W.GEMM, big)
    osp = oracle.Space(W.GEMM, big)
    assert sum(int(x) for x in osp.knob_sizes[:3]) > 1024
    n, steps, seed, k = 100, 30, 23, 5
    ch = mk_chains(P, sp, 0, n, k, seed, path)
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))
    if path != "trees":
        return
    off = np.array([0, 48, 96], np.int64)
    sset = P.at_spaceset_create([sp, P.at_space_create(W.GEMM, small)], off)
    ch = mk_chains(P, sset, 0, 96, k, seed, path)
    best, tr = gpu_sa(P, sset, ens, ch, steps, P.at_sa_thresholds(seed, 0, 96, 0, steps))
    och = oracle.Chains([osp, oracle.Space(W.GEMM, small)], off, seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, 96, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_sa_ragged_set_tail_mode(P):
    # workgroups of two chains straddle the space boundaries (chains 4-5 and
    # 300), so the chain-local tail mode reads each chain's own space tables
    shapes = [(1, 2, 4, 4, 2, 3, 3, 1, 1), (1, 2, 6, 6, 2, 1, 1, 0, 2), (1, 1, 8, 8, 2, 7, 7, 3, 2)]
    say("sa ragged set, chain-local tail mode")
    spaces = [P.at_space_create(W.CONV2D, s) for s in shapes]
    ospaces = [oracle.Space(W.CONV2D, s) for s in shapes]
    off = np.array([0, 5, 300, 301], np.int64)
    fid, thr, leaf = W.make_ensemble(300, 8, 176, 8)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    sset = P.at_spaceset_create(spaces, off)
    n, steps, seed, k = 301, 20, 21, 4
    ch = mk_chains(P, sset, 7, n, k, seed, "local")
    best, tr = gpu_sa(P, sset, ens, ch, steps, P.at_sa_thresholds(seed, 7, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    assert plan["gather"] == 2 and plan["chains_per_wg"] == 2
    och = oracle.Chains(ospaces, off, seed=seed, chain0=7, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 7, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def small_setup(P, n=70, topk=6, trees=25, depth=6, shape=(1, 2, 6, 6, 4, 3, 3, 1, 1)):
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    fid, thr, leaf = W.make_ensemble(trees, depth, 176, 99)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    return sp, osp, (fid, thr, leaf), ens


@pytest.mark.parametrize("depth,trees", [(1, 21), (2, 35), (3, 19), (11, 6), (12, 5)])
def test_sa_tree_path_depths(P, depth, trees):
    # the tree kernel's LDS copy at block sizes from 8 bytes (depth 1) to
    # 16 KB (depth 12), with a partial last tree group
    say(f"sa tree path depth {depth}, {trees} trees")
    sp, osp, ens_t, ens = small_setup(P, trees=trees, depth=depth)
    n, steps, seed, k = 150, 15, 17, 4
    ch = mk_chains(P, sp, 0, n, k, seed, "trees")
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run(ens_t, steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_sa_persistence_split_equals_full(P, path):
    sp, osp, ens_t, ens = small_setup(P)
    n, steps, seed, k = 70, 80, 5, 6
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    a = mk_chains(P, sp, 0, n, k, seed, path)
    best_a, tr_a = gpu_sa(P, sp, ens, a, steps, thr)
    b = mk_chains(P, sp, 0, n, k, seed, path)
    _, tr_b1 = gpu_sa(P, sp, ens, b, 30, thr[:, :30].copy())
    assert P.at_chains_step(b) == 30
    best_b, tr_b2 = gpu_sa(P, sp, ens, b, 50, thr[:, 30:].copy())
    assert np.array_equal(np.concatenate([tr_b1, tr_b2], axis=1), tr_a)
    assert np.array_equal(best_a, best_b)
    assert P.at_chains_step(a) == P.at_chains_step(b) == 80


def test_sa_chain_independence_and_determinism(P, path):
    sp, osp, ens_t, ens = small_setup(P)
    n, steps, seed, k = 300, 40, 9, 5
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    full = mk_chains(P, sp, 0, n, k, seed, path)
    best_f, tr_f = gpu_sa(P, sp, ens, full, steps, thr)
    again = mk_chains(P, sp, 0, n, k, seed, path)
    best_g, tr_g = gpu_sa(P, sp, ens, again, steps, thr)
    assert np.array_equal(tr_f, tr_g) and np.array_equal(best_f, best_g)
    part = mk_chains(P, sp, 250, 40, k, seed, path)
    best_p, tr_p = gpu_sa(P, sp, ens, part, steps, thr[250:290].copy())
    assert np.array_equal(tr_p, tr_f[250:290]) and np.array_equal(best_p, best_f[250:290])


def test_sa_profiled_run_is_identical_and_counts_launches(P):
    sp, osp, ens_t, ens = small_setup(P)
    n, steps, seed, k = 130, 25, 21, 4
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    plain = mk_chains(P, sp, 0, n, k, seed, "trees")
    best_a, tr_a = gpu_sa(P, sp, ens, plain, steps, thr)
    assert P.at_sa_kernel_times(plain)["tree_launches"] == 0
    prof = mk_chains(P, sp, 0, n, k, seed, "trees")
    P.at_sa_set_profiling(prof, True)
    best_b, tr_b = gpu_sa(P, sp, ens, prof, steps, thr)
    assert np.array_equal(tr_a, tr_b) and np.array_equal(best_a, best_b)
    t = P.at_sa_kernel_times(prof)
    # first run: initial draw + one tree pass, then steps x (chain + trees), then the final chain pass
    assert t["tree_launches"] == steps + 1 and t["chain_launches"] == steps + 2
    assert t["tree_ms"] > 0 and t["chain_ms"] > 0
    best_c, tr_c = gpu_sa(P, sp, ens, prof, 10, P.at_sa_thresholds(seed, 0, n, steps, 10))
    t = P.at_sa_kernel_times(prof)
    assert t["tree_launches"] == 10 and t["chain_launches"] == 11


@pytest.mark.parametrize("kind", ["zero_steps", "plus_inf", "minus_inf", "zero_temp", "topk1", "topk64", "one_by_one"])
def test_sa_edge_cases(P, path, kind):
    shape = (1, 2, 6, 6, 2, 1, 1, 0, 2) if kind == "one_by_one" else (1, 2, 6, 6, 4, 3, 3, 1, 1)
    sp, osp, ens_t, ens = small_setup(P, shape=shape)
    n, steps, seed = 65, 30, 13
    k = {"topk1": 1, "topk64": 64}.get(kind, 4)
    if kind == "zero_steps":
        steps = 0
    if kind == "plus_inf":
        thr_g = np.full((n, steps), np.inf, np.float32)
    elif kind == "minus_inf":
        thr_g = np.full((n, steps), -np.inf, np.float32)
    elif kind == "zero_temp":
        thr_g = np.full((n, steps), -0.0, np.float32)
    else:
        thr_g = P.at_sa_thresholds(seed, 0, n, 0, max(steps, 1))[:, :steps].copy()
    thr_o = thr_g.copy() if kind in ("plus_inf", "minus_inf", "zero_temp") else \
        oracle.thresholds(seed, 0, n, 0, max(steps, 1))[:, :steps].copy()
    ch = mk_chains(P, sp, 0, n, k, seed, path)
    best, tr = gpu_sa(P, sp, ens, ch, steps, thr_g, traced=steps > 0)
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run(ens_t, steps, thr_o, trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))
    if kind == "zero_steps":
        assert (best["flag"][:, 0] == 1).all() and (best["flag"][:, 1:] == 0).all()


def test_sa_rejects_mismatched_ensemble(P):
    import torch
    sp = P.at_space_create(W.GEMM, (4, 4, 4))
    fid, thr, leaf = W.make_ensemble(3, 2, 176, 1)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    ch = P.at_chains_create(sp, 0, 4, 2, 1)
    best = torch.zeros((4, 2, 4), dtype=torch.int32, device=DEV)
    thr_d = torch.zeros((4, 3), dtype=torch.float32, device=DEV)
    with pytest.raises(P.ATError) as ei:
        P.at_sa_run(sp, ens, ch, 3, thr_d, best)
    assert ei.value.status == -6


def test_sa_local_profiled_run_is_one_launch(P):
    sp, osp, ens_t, ens = small_setup(P)
    n, steps, seed, k = 130, 25, 21, 4
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    plain = mk_chains(P, sp, 0, n, k, seed, "local")
    best_a, tr_a = gpu_sa(P, sp, ens, plain, steps, thr)
    prof = mk_chains(P, sp, 0, n, k, seed, "local")
    P.at_sa_set_profiling(prof, True)
    best_b, tr_b = gpu_sa(P, sp, ens, prof, steps, thr)
    assert np.array_equal(tr_a, tr_b) and np.array_equal(best_a, best_b)
    t = P.at_sa_kernel_times(prof)
    assert t["tree_launches"] == 1 and t["chain_launches"] == 0 and t["tree_ms"] > 0


def test_sa_paths_agree_and_interleave(P):
    """The two paths give the same trajectories; a run on one path continues
    chains the other has advanced."""
    sp, osp, ens_t, ens = small_setup(P, trees=90, depth=7)
    n, steps, seed, k = 200, 60, 31, 8
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    ref = mk_chains(P, sp, 0, n, k, seed, "trees")
    best_r, tr_r = gpu_sa(P, sp, ens, ref, steps, thr)
    mix = mk_chains(P, sp, 0, n, k, seed, "local")
    _, tr_1 = gpu_sa(P, sp, ens, mix, 20, thr[:, :20].copy())
    P.at_chains_set_path(mix, PATHS["trees"])
    mix.path_name = "trees"
    _, tr_2 = gpu_sa(P, sp, ens, mix, 25, thr[:, 20:45].copy())
    P.at_chains_set_path(mix, PATHS["local"])
    mix.path_name = "local"
    best_m, tr_3 = gpu_sa(P, sp, ens, mix, 15, thr[:, 45:].copy())
    assert np.array_equal(np.concatenate([tr_1, tr_2, tr_3], axis=1), tr_r)
    assert np.array_equal(best_m, best_r)
    assert np.array_equal(export(P, mix)[0], export(P, ref)[0])


# chain-local plans: resident ensemble, streamed whole trees, streamed node
# blocks with leaves from global memory, resident tree tops with the last
# level from global memory; each checked against the oracle
LOCAL_PLANS = {
    "resident": dict(n=48, trees=40, depth=6, steps=30),
    # sixteen chains per workgroup: one resident chunk without helper waves
    "resident_wide": dict(n=4096, trees=40, depth=6, steps=10),
    "streamed": dict(n=8192, trees=1000, depth=8, steps=4),
    "gathered": dict(n=64, trees=400, depth=9, steps=20),
    "tail": dict(n=300, trees=300, depth=8, steps=25),
    "tail_depth2": dict(n=1024, trees=2000, depth=2, steps=15),
    # sixteen chains per workgroup: the tail walk without helper waves
    "tail_wide": dict(n=4096, trees=300, depth=8, steps=10),
    # four chains per workgroup, the last workgroup holding one
    "tail_ragged": dict(n=1021, trees=300, depth=8, steps=12),
    # at least 384 trees: the evaluating waves also make the next candidates
    "tail_ragged_long": dict(n=1021, trees=400, depth=8, steps=12),
}


@pytest.mark.parametrize("mode", sorted(LOCAL_PLANS))
def test_sa_local_plans_match_oracle(P, mode):
    cfg = LOCAL_PLANS[mode]
    say(f"sa local plan {mode}: {cfg}")
    shape = (1, 16, 14, 14, 32, 3, 3, 1, 1)
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    fid, thr, leaf = W.make_ensemble(cfg["trees"], cfg["depth"], 176, 404)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, steps, seed, k = cfg["n"], cfg["steps"], 55, 8
    ch = mk_chains(P, sp, 0, n, k, seed, "local")
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    assert (plan["chunks"] == 0) == (mode.startswith("resident") or mode.startswith("tail"))
    assert plan["gather"] == (2 if mode.startswith("tail") else {"gathered": 1}.get(mode, 0))
    if mode.startswith("tail") or mode.startswith("resident"):
        assert (plan["chains_per_wg"] > 4) == mode.endswith("_wide")
    # the first 160 chains, or the last 160 when the last workgroup is short
    r0 = n - 160 if mode.startswith("tail_ragged") else 0
    m = min(n - r0, 160)
    och = oracle.Chains([osp], [0, m], seed=seed, chain0=r0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, r0, m, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, rows=slice(r0, r0 + m), cur=export(P, ch))
