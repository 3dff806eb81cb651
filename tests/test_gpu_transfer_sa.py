"""GPU parity of annealing with the transfer model's energy (Section 4,
Eq. 4: global model over the context relation features plus local model
over the loop-context features) against the oracle, bit for bit: proposed
configurations, scores, accept decisions, best lists and final states.
Every call goes through the C ABI (at_sa_run_global_local)."""
import numpy as np
import pytest

import oracle
import workloads as W
from test_gpu_parity import DEV, P, assert_same_run, bits, export, say  # noqa: F401

pytestmark = pytest.mark.gpu
REL = 192


def gl_run(P, sp, glob, loc, chains, steps, thr, traced=True):
    import torch
    d_thr = torch.from_numpy(np.ascontiguousarray(thr, np.float32)).to(DEV)
    best = torch.zeros((chains.n_chains, chains.topk, 4), dtype=torch.int32, device=DEV)
    tr = torch.zeros((chains.n_chains, steps, 4), dtype=torch.int32, device=DEV) if traced else None
    P.at_sa_run_global_local(sp, glob, loc, chains, steps, d_thr, best, tr)
    torch.cuda.synchronize()
    assert P.at_chains_last_path(chains) == P.AT_SA_PATH_TREES
    return P.entries(best), (P.entries(tr) if traced else None)


def setup(P, tmpl, shape, g_trees, g_depth, l_trees, l_depth, seed=31):
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    g = W.make_ensemble(g_trees, g_depth, REL, seed)
    l = W.make_ensemble(l_trees, l_depth, sp.n_features, seed + 1)
    return sp, osp, g, l, P.at_ensemble_create(*g, REL), P.at_ensemble_create(*l, sp.n_features)


CASES = {
    # conv, the two models of different depth and tree count
    "conv": (W.CONV2D, (1, 16, 14, 14, 32, 3, 3, 1, 1), 90, 7, 60, 8),
    # stride 2 with a 1x1 window (unmutable window knobs)
    "conv_1x1_s2": (W.CONV2D, (1, 16, 14, 14, 32, 1, 1, 0, 2), 40, 6, 45, 6),
    # GEMM: 110 loop features for the local model
    "gemm": (W.GEMM, (64, 32, 128), 70, 6, 33, 5),
    # deep global model, shallow local one
    "deep_global": (W.CONV2D, (1, 8, 7, 7, 16, 3, 3, 1, 1), 20, 10, 25, 3),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_global_local_annealing_matches_oracle(P, case):
    tmpl, shape, gt, gd, lt, ld = CASES[case]
    say(f"eq4 annealing {case}")
    sp, osp, g, l, eg, el = setup(P, tmpl, shape, gt, gd, lt, ld)
    n, steps, seed, k = 200, 30, 41, 6
    ch = P.at_chains_create(sp, 0, n, k, seed)
    best, tr = gl_run(P, sp, eg, el, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run(l, steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True, global_model=g)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_global_local_fold_order(P):
    # constant stumps (1e8, 1) + (-1e8, 1): each model folded on its own,
    # then added, gives exactly 0 for every candidate (one fold would give 1)
    sp = P.at_space_create(W.CONV2D, (1, 2, 6, 6, 4, 3, 3, 1, 1))

    def stumps(vals, F):
        T = len(vals)
        return (np.zeros((T, 1), np.uint8), np.zeros((T, 1), np.uint8),
                np.repeat(np.asarray(vals, np.float32)[:, None], 2, axis=1))
    g, l = stumps([1e8, 1.0], REL), stumps([-1e8, 1.0], 176)
    n, steps = 70, 12
    ch = P.at_chains_create(sp, 0, n, 3, 5)
    best, tr = gl_run(P, sp, P.at_ensemble_create(*g, REL), P.at_ensemble_create(*l, 176), ch, steps,
                      P.at_sa_thresholds(5, 0, n, 0, steps))
    assert (tr["score"] == 0.0).all()
    assert (best["score"][best["flag"] == 1] == 0.0).all()


def test_zero_global_model_equals_plain_run(P):
    import torch
    sp, osp, g, l, eg, el = setup(P, W.CONV2D, (1, 16, 14, 14, 32, 3, 3, 1, 1), 50, 6, 70, 7)
    zero = P.at_ensemble_create(g[0], g[1], np.zeros_like(g[2]), REL)
    n, steps, seed, k = 130, 25, 3, 5
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    a = P.at_chains_create(sp, 0, n, k, seed)
    best_a, tr_a = gl_run(P, sp, zero, el, a, steps, thr)
    b = P.at_chains_create(sp, 0, n, k, seed)
    P.at_chains_set_path(b, P.AT_SA_PATH_TREES)
    best_b = torch.zeros((n, k, 4), dtype=torch.int32, device=DEV)
    tr_b = torch.zeros((n, steps, 4), dtype=torch.int32, device=DEV)
    P.at_sa_run_traced(sp, el, b, steps, torch.from_numpy(thr).to(DEV), best_b, tr_b)
    torch.cuda.synchronize()
    assert np.array_equal(tr_a, P.entries(tr_b)) and np.array_equal(best_a, P.entries(best_b))


def test_global_local_split_run_equals_full_run(P):
    sp, osp, g, l, eg, el = setup(P, W.CONV2D, (1, 16, 14, 14, 32, 3, 3, 1, 1), 40, 6, 40, 6)
    n, steps, seed, k = 100, 40, 9, 4
    thr = P.at_sa_thresholds(seed, 0, n, 0, steps)
    a = P.at_chains_create(sp, 0, n, k, seed)
    best_a, tr_a = gl_run(P, sp, eg, el, a, steps, thr)
    b = P.at_chains_create(sp, 0, n, k, seed)
    _, tr_1 = gl_run(P, sp, eg, el, b, 15, thr[:, :15].copy())
    best_b, tr_2 = gl_run(P, sp, eg, el, b, 25, thr[:, 15:].copy(), traced=False)
    assert np.array_equal(tr_1, tr_a[:, :15]) and np.array_equal(best_a, best_b)
    assert np.array_equal(export(P, a)[0], export(P, b)[0])


def test_twelve_workload_set_transfer_sliced_oracle(P):
    # the twelve ResNet-18 conv2d workloads with a 1000-tree global model on
    # the relation features and the 1000-tree local model on the loop
    # features: 512 chains per workload, oracle slices at every boundary
    wl = W.WORKLOADS["resnet18_12conv_sa"]
    spaces = [P.at_space_create(t, s) for t, s in wl["spaces"]]
    off = W.chain_offsets(12, 512)
    sset = P.at_spaceset_create(spaces, off)
    l = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    g = W.make_ensemble(wl["trees"], wl["depth"], REL, wl["ens_seed"] + 50)
    n, steps, seed, k = int(off[-1]), 40, wl["sa_seed"], wl["topk"]
    ch = P.at_chains_create(sset, 0, n, k, seed)
    best, tr = gl_run(P, sset, P.at_ensemble_create(*g, REL), P.at_ensemble_create(*l, 176), ch, steps,
                      P.at_sa_thresholds(seed, 0, n, 0, steps))
    cur = export(P, ch)
    for w in range(12):
        lo = int(off[w]) + (0 if w % 2 else 508)
        lo = min(lo, n - 4)
        osp = [oracle.Space(*wl["spaces"][int(np.searchsorted(off, lo, side="right") - 1)])]
        och = oracle.Chains(osp, [0, 4], seed=seed, chain0=lo, topk=k)
        otr = och.run(l, steps, oracle.thresholds(seed, lo, 4, 0, steps), trace=True, global_model=g)
        assert_same_run(best, tr, och, otr, rows=slice(lo, lo + 4), cur=cur)


def test_global_local_argument_errors(P):
    import torch
    sp, osp, g, l, eg, el = setup(P, W.CONV2D, (1, 2, 6, 6, 4, 3, 3, 1, 1), 5, 3, 5, 3)
    n, steps = 8, 4
    thr = torch.zeros((n, steps), dtype=torch.float32, device=DEV)
    best = torch.zeros((n, 2, 4), dtype=torch.int32, device=DEV)
    ch = P.at_chains_create(sp, 0, n, 2, 1)
    with pytest.raises(P.ATError) as ei:      # global model over the loop features
        P.at_sa_run_global_local(sp, el, el, ch, steps, thr, best)
    assert ei.value.status == -6
    with pytest.raises(P.ATError) as ei:      # local model over the relation features
        P.at_sa_run_global_local(sp, eg, eg, ch, steps, thr, best)
    assert ei.value.status == -6
    P.at_chains_set_path(ch, P.AT_SA_PATH_LOCAL)
    with pytest.raises(P.ATError) as ei:
        P.at_sa_run_global_local(sp, eg, el, ch, steps, thr, best)
    assert ei.value.status == -2
