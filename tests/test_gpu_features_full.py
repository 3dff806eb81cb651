"""GPU parity of the full Appendix A.2 feature rows (13 per loop, with
top-down and bottom-up) against the oracle, bit for bit, and scoring of such
rows.  Configurations and expected rows come from the seeded generators and
the oracle."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(f"[gpu-full] {msg}", flush=True)


@pytest.fixture(scope="module")
def P():
    import torch
    torch.cuda.set_device(0)
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def u64_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(DEV)


def gpu_full(P, sp, cfgs, offset=0):
    """Rows written at an element offset into a larger buffer (offset 1
    leaves them 4-byte aligned only)."""
    import torch
    F = 13 * sp.n_loops
    buf = torch.full((len(cfgs) * F + offset,), -7, dtype=torch.int32, device=DEV)
    out = buf[offset:].view(len(cfgs), F)
    P.at_extract_features_full(sp, u64_dev(cfgs), out)
    torch.cuda.synchronize()
    return out.cpu().numpy(), buf[:offset].cpu().numpy()


SMALL = [(W.GEMM, (4, 4, 4)), (W.GEMM, (2, 6, 3)), (W.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1)),
         (W.CONV2D, (1, 2, 6, 6, 2, 3, 3, 1, 2)), (W.CONV2D, (1, 3, 5, 5, 4, 2, 2, 0, 3))]


@pytest.mark.parametrize("tmpl,shape", SMALL)
def test_every_config_of_small_spaces(P, tmpl, shape):
    say(f"full rows, every config of {shape}")
    sp, osp = P.at_space_create(tmpl, shape), oracle.Space(tmpl, shape)
    cfgs = np.arange(osp.n_configs, dtype=np.uint64)
    got, _ = gpu_full(P, sp, cfgs)
    assert np.array_equal(got, osp.features_full(cfgs))


@pytest.mark.parametrize("tmpl,shape,n", [(W.CONV2D, W.conv_shape("C2"), 70000 + 13), (W.CONV2D, W.conv_shape("C12"), 3001),
                                          (W.CONV2D, W.conv_shape("C1"), 2000), (W.GEMM, (512, 512, 512), 5000 + 7)])
def test_full_shapes_sampled(P, tmpl, shape, n):
    say(f"full rows, {shape} n={n}")
    sp, osp = P.at_space_create(tmpl, shape), oracle.Space(tmpl, shape)
    cfgs = W.make_configs(n, osp.n_configs, seed=n)
    got, _ = gpu_full(P, sp, cfgs)
    idx = np.r_[0:600, n - 300:n]
    assert np.array_equal(got[idx], osp.features_full(cfgs[idx]))
    # the loop-context columns agree with at_extract_features everywhere
    import torch
    plain = torch.empty((n, sp.n_features), dtype=torch.int32, device=DEV)
    P.at_extract_features(sp, u64_dev(cfgs), plain)
    torch.cuda.synchronize()
    pl = plain.cpu().numpy().reshape(n, -1, 11)
    g = got.reshape(n, -1, 13)
    assert np.array_equal(g[:, :, :2], pl[:, :, :2]) and np.array_equal(g[:, :, 4:], pl[:, :, 2:])


def test_unaligned_output_and_out_of_range_rows(P):
    say("full rows, unaligned output, out-of-range rows")
    shape = W.conv_shape("C6")
    sp, osp = P.at_space_create(W.CONV2D, shape), oracle.Space(W.CONV2D, shape)
    cfgs = W.make_configs(1000, osp.n_configs, seed=3)
    bad = [5, 999]
    cfgs[bad] = osp.n_configs + np.array([0, 12345], dtype=np.uint64)
    P.at_space_errors(sp)
    got, pre = gpu_full(P, sp, cfgs, offset=1)
    assert (pre == -7).all()
    assert (got[bad] == -1).all()
    good = np.setdiff1d(np.arange(1000), bad)
    assert np.array_equal(got[good], osp.features_full(cfgs[good]))
    assert P.at_space_errors(sp) == 2


def test_scoring_full_rows(P):
    import torch
    say("ensemble on full rows (208 features)")
    shape = W.conv_shape("C2")
    sp, osp = P.at_space_create(W.CONV2D, shape), oracle.Space(W.CONV2D, shape)
    F = osp.n_features_full
    cfgs = W.make_configs(2048 + 45, osp.n_configs, seed=11)
    rows = osp.features_full(cfgs)
    fid, thr, leaf = W.make_ensemble(300, 8, F, seed=12)
    ens = P.at_ensemble_create(fid, thr, leaf, F)
    d = torch.from_numpy(rows).to(DEV)
    s = torch.empty(len(cfgs), dtype=torch.float32, device=DEV)
    P.at_gbt_predict(ens, d, s)
    torch.cuda.synchronize()
    want = oracle.predict(fid, thr, leaf, rows)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), want.view(np.uint32))
