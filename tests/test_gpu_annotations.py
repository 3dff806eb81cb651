"""GPU parity of the annotated templates (vectorize and vthread knobs) and of
the one-hot annotation rows (Appendix A.2 loop-context table) against the
oracle, bit for bit: feature rows (loop-context, full, one-hot, relation),
annealing trajectories on both paths, Eq. 4 annealing and batch selection on
annotated spaces.  Every call goes through the C ABI."""
import numpy as np
import pytest

import oracle
import workloads as W
from test_gpu_parity import DEV, P, assert_same_run, export, gpu_sa, mk_chains, path, say, u64_dev  # noqa: F401

pytestmark = pytest.mark.gpu
GEMM_VT, CONV_VT = 2, 3
TINY_VT = [(GEMM_VT, (4, 4, 4)), (GEMM_VT, (2, 6, 3)), (CONV_VT, (1, 2, 4, 4, 2, 3, 3, 1, 1)),
           (CONV_VT, (1, 2, 6, 6, 2, 1, 1, 0, 2)), (CONV_VT, (1, 1, 8, 8, 2, 7, 7, 3, 2))]


def rows(P, fn, sp, cfgs, width, offset=0):
    import torch
    d = u64_dev(cfgs)
    buf = torch.full((len(cfgs) * width + offset,), 7, dtype=torch.int32, device=DEV)
    out = buf[offset:].view(len(cfgs), width)
    fn(sp, d, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("tmpl,shape", TINY_VT)
def test_features_every_config_of_small_annotated_spaces(P, tmpl, shape):
    say(f"annotated features exhaustive {tmpl} {shape}")
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    assert sp.n_configs == osp.n_configs and list(sp.knob_sizes) == list(osp.knob_sizes)
    assert sp.n_knobs == (7 if tmpl == GEMM_VT else 10)
    cfgs = np.arange(osp.n_configs, dtype=np.uint64)
    assert np.array_equal(rows(P, P.at_extract_features, sp, cfgs, sp.n_features), osp.features(cfgs))
    assert np.array_equal(rows(P, P.at_extract_features_full, sp, cfgs, 13 * sp.n_loops), osp.features_full(cfgs))
    assert np.array_equal(rows(P, P.at_extract_features_onehot, sp, cfgs, 24 * sp.n_loops), osp.features_onehot(cfgs))
    assert np.array_equal(rows(P, P.at_extract_relation_features, sp, cfgs, 192), osp.relation_features(cfgs))


@pytest.mark.parametrize("tmpl,shape", [(W.GEMM, (4, 4, 4)), (W.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1)),
                                        (W.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2))])
def test_onehot_rows_every_config_of_small_base_spaces(P, tmpl, shape):
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    cfgs = np.arange(osp.n_configs, dtype=np.uint64)
    assert np.array_equal(rows(P, P.at_extract_features_onehot, sp, cfgs, 24 * sp.n_loops), osp.features_onehot(cfgs))


@pytest.mark.parametrize("tmpl,name", [(CONV_VT, "C1"), (CONV_VT, "C2"), (CONV_VT, "C5"), (CONV_VT, "C12"),
                                       (W.CONV2D, "C7"), (GEMM_VT, None)])
def test_onehot_rows_sampled_shapes_unaligned_and_out_of_range(P, tmpl, name):
    shape = W.GEMM_512 if name is None else W.conv_shape(name)
    say(f"one-hot rows {tmpl} {shape}")
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    cfgs = W.make_configs(3001, osp.n_configs, seed=11)
    cfgs[[5, 700, 3000]] = [osp.n_configs, osp.n_configs + 9, 2 ** 40]
    P.at_space_errors(sp)
    want = osp.features_onehot(np.where(cfgs < osp.n_configs, cfgs, 0))
    want[[5, 700, 3000]] = -1
    for off in (0, 1):          # 16-byte aligned and unaligned outputs
        got = rows(P, P.at_extract_features_onehot, sp, cfgs, 24 * sp.n_loops, offset=off)
        assert np.array_equal(got, want)
    assert P.at_space_errors(sp) == 6
    f = rows(P, P.at_extract_features, sp, cfgs[:3000], sp.n_features)
    w = osp.features(np.where(cfgs[:3000] < osp.n_configs, cfgs[:3000], 0))
    w[[5, 700]] = -1
    assert np.array_equal(f, w)


def test_onehot_rows_one_million_sampled(P):
    import torch
    shape = W.conv_shape("C2")
    sp = P.at_space_create(CONV_VT, shape)
    osp = oracle.Space(CONV_VT, shape)
    n = 1 << 20
    cfgs = W.make_configs(n, osp.n_configs, seed=3002)
    d = u64_dev(cfgs)
    out = torch.empty((n, 384), dtype=torch.int32, device=DEV)
    P.at_extract_features_onehot(sp, d, out)
    torch.cuda.synchronize()
    idx = np.concatenate([np.random.default_rng(1).choice(n, 5000, replace=False), [0, n - 1]])
    assert np.array_equal(out[torch.from_numpy(idx).to(DEV)].cpu().numpy(), osp.features_onehot(cfgs[idx]))
    hot = out.view(n, 16, 24)[:, :, 1:13]
    assert bool((hot.sum(dim=2) == 1).all())


@pytest.mark.parametrize("tmpl,shape,trees,depth", [(CONV_VT, (1, 16, 14, 14, 32, 3, 3, 1, 1), 60, 7),
                                                    (GEMM_VT, (64, 32, 128), 40, 6),
                                                    (CONV_VT, (1, 8, 14, 14, 16, 1, 1, 0, 2), 300, 8)])
def test_annealing_on_annotated_spaces_matches_oracle(P, path, tmpl, shape, trees, depth):
    say(f"annealing annotated {tmpl} {shape} on {path}")
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    fid, thr, leaf = W.make_ensemble(trees, depth, sp.n_features, 88)
    ens = P.at_ensemble_create(fid, thr, leaf, sp.n_features)
    n, steps, seed, k = 260, 30, 19, 6
    ch = mk_chains(P, sp, 0, n, k, seed, path)
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_annealing_annotated_c2_workload_sliced(P):
    # the C2 search on the annotated template: 1024 chains x 100 steps on the
    # default path (chain-local), oracle slices
    wl = W.WORKLOADS["conv_c2_sa"]
    shape = wl["spaces"][0][1]
    sp = P.at_space_create(CONV_VT, shape)
    osp = oracle.Space(CONV_VT, shape)
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, steps, seed, k = 1024, 100, wl["sa_seed"], wl["topk"]
    ch = P.at_chains_create(sp, 0, n, k, seed)
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    cur = export(P, ch)
    for lo, hi in [(0, 40), (990, 1024)]:
        och = oracle.Chains([osp], [0, hi - lo], seed=seed, chain0=lo, topk=k)
        otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, lo, hi - lo, 0, steps), trace=True)
        assert_same_run(best, tr, och, otr, rows=slice(lo, hi), cur=cur)


def test_eq4_annealing_on_an_annotated_space(P):
    import torch
    shape = (1, 16, 14, 14, 32, 3, 3, 1, 1)
    sp = P.at_space_create(CONV_VT, shape)
    osp = oracle.Space(CONV_VT, shape)
    g = W.make_ensemble(50, 6, 192, 5)
    l = W.make_ensemble(50, 7, 176, 6)
    n, steps, seed, k = 150, 25, 8, 5
    ch = P.at_chains_create(sp, 0, n, k, seed)
    thr = torch.from_numpy(P.at_sa_thresholds(seed, 0, n, 0, steps)).to(DEV)
    best = torch.zeros((n, k, 4), dtype=torch.int32, device=DEV)
    trace = torch.zeros((n, steps, 4), dtype=torch.int32, device=DEV)
    P.at_sa_run_global_local(sp, P.at_ensemble_create(*g, 192), P.at_ensemble_create(*l, 176), ch, steps, thr, best,
                             trace)
    torch.cuda.synchronize()
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run(l, steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True, global_model=g)
    assert_same_run(P.entries(best), P.entries(trace), och, otr, cur=export(P, ch))


def test_select_on_an_annotated_space(P):
    import torch
    shape = W.conv_shape("C12")
    sp = P.at_space_create(CONV_VT, shape)
    osp = oracle.Space(CONV_VT, shape)
    cand = W.make_candidates(2048, 16, osp.n_configs, 9)
    d = torch.from_numpy(np.ascontiguousarray(cand).view(np.int32).reshape(2048, 16, 4).copy()).to(DEV)
    out = torch.zeros((64, 4), dtype=torch.int32, device=DEV)
    P.at_select_batch(sp, d, 128, 61, 1.0, 3, 4, out)
    torch.cuda.synchronize()
    got = P.entries(out)
    want = oracle.select_batch(osp, cand.view(oracle.TOP_DTYPE), 128, 61, 1.0, 3, 4)
    assert np.array_equal(got["cfg"], want["cfg"]) and np.array_equal(got["flag"], want["valid"])


def test_annotated_space_set_and_template_mismatch(P):
    a = P.at_space_create(CONV_VT, (1, 2, 4, 4, 2, 3, 3, 1, 1))
    b = P.at_space_create(W.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1))
    with pytest.raises(P.ATError) as ei:
        P.at_spaceset_create([a, b], [0, 4, 8])
    assert ei.value.status == -6
    ch = P.at_chains_create(a, 0, 4, 2, 1)
    fid, thr, leaf = W.make_ensemble(3, 2, 176, 1)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    import torch
    with pytest.raises(P.ATError) as ei:
        P.at_sa_run(b, ens, ch, 2, torch.zeros((4, 2), dtype=torch.float32, device=DEV),
                    torch.zeros((4, 2, 4), dtype=torch.int32, device=DEV))
    assert ei.value.status == -1
