"""GPU parity of the transfer-learning scoring pieces (Section 4): ensembles
on the context relation features, and the global + local model of Eq. 4,
bit for bit against the oracle.  Feature rows given to the oracle come from
the oracle."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(f"[gpu-transfer] {msg}", flush=True)


@pytest.fixture(scope="module")
def P():
    import torch
    torch.cuda.set_device(0)
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def dev(a, dtype=None):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def bits(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


@pytest.mark.parametrize("depth,trees", [(8, 1000), (6, 37), (10, 130)])
def test_predict_on_relation_features(P, depth, trees):
    import torch
    osp = oracle.Space(W.CONV2D, W.conv_shape("C6"))
    cfgs = W.make_configs(2 * 256 + 41, osp.n_configs, 60 + depth)
    rel = osp.relation_features(cfgs)
    fid, thr, leaf = W.make_ensemble(trees, depth, 192, 70 + depth)
    ens = P.at_ensemble_create(fid, thr, leaf, 192)
    s = torch.empty(len(cfgs), dtype=torch.float32, device=DEV)
    P.at_gbt_predict(ens, dev(rel), s)
    torch.cuda.synchronize()
    assert np.array_equal(bits(s.cpu().numpy()), bits(oracle.predict(fid, thr, leaf, rel)))


@pytest.mark.parametrize("local_tmpl", ["conv", "gemm"])
def test_global_local_matches_oracle(P, local_tmpl):
    import torch
    say(f"global (relation features) + local ({local_tmpl} loop features)")
    if local_tmpl == "conv":
        osp = oracle.Space(W.CONV2D, W.conv_shape("C2"))
    else:
        osp = oracle.Space(W.GEMM, (512, 512, 512))
    n = 3 * 256 + 19
    cfgs = W.make_configs(n, osp.n_configs, 81)
    rel, loop = osp.relation_features(cfgs), osp.features(cfgs)
    g = W.make_ensemble(1000, 8, 192, 90)
    l = W.make_ensemble(500, 8, osp.n_features, 91)
    eg = P.at_ensemble_create(*g, 192)
    el = P.at_ensemble_create(*l, osp.n_features)
    s = torch.empty(n, dtype=torch.float32, device=DEV)
    P.at_gbt_predict_global_local(eg, dev(rel), el, dev(loop), s)
    torch.cuda.synchronize()
    want = oracle.predict_global_local(g, rel, l, loop)
    assert np.array_equal(bits(s.cpu().numpy()), bits(want))


def test_global_local_fold_order(P):
    """(1e8, 1) + (-1e8, 1): the sum of two folds is 0, one fold over the
    concatenated trees would be 1."""
    import torch
    T = 2
    fid = np.zeros((T, 1), np.uint8)
    thr = np.zeros((T, 1), np.uint8)
    lg = np.zeros((T, 2), np.float32)
    ll = np.zeros((T, 2), np.float32)
    lg[:, 1] = [1e8, 1.0]
    ll[:, 1] = [-1e8, 1.0]
    eg = P.at_ensemble_create(fid, thr, lg, 4)
    el = P.at_ensemble_create(fid, thr, ll, 4)
    x = np.zeros((300, 4), np.int32)
    s = torch.empty(300, dtype=torch.float32, device=DEV)
    P.at_gbt_predict_global_local(eg, dev(x), el, dev(x), s)
    torch.cuda.synchronize()
    assert (s.cpu().numpy() == 0.0).all()


def test_global_local_full_size_sampled(P):
    """1,048,576 conv2d C2 configurations: loop and relation features on the
    GPU, then the two-model score; sampled rows recomputed by the oracle from
    the configuration index."""
    import torch
    say("global + local, 1M configurations")
    shape = W.conv_shape("C2")
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    n = 1 << 20
    cfgs = W.make_configs(n, osp.n_configs, 3002)
    d = torch.from_numpy(cfgs.view(np.int64)).to(DEV)
    loop = torch.empty((n, 176), dtype=torch.int32, device=DEV)
    rel = torch.empty((n, 192), dtype=torch.int32, device=DEV)
    P.at_extract_features(sp, d, loop)
    P.at_extract_relation_features(sp, d, rel)
    g = W.make_ensemble(1000, 8, 192, 92)
    l = W.make_ensemble(500, 8, 176, 93)
    eg = P.at_ensemble_create(*g, 192)
    el = P.at_ensemble_create(*l, 176)
    s = torch.empty(n, dtype=torch.float32, device=DEV)
    P.at_gbt_predict_global_local(eg, rel, el, loop, s)
    torch.cuda.synchronize()
    rows = np.concatenate([np.random.default_rng(4).choice(n, 2000, replace=False), [0, n - 1]])
    want = oracle.predict_global_local(g, osp.relation_features(cfgs[rows]), l, osp.features(cfgs[rows]))
    assert np.array_equal(bits(s.cpu().numpy()[rows]), bits(want))
