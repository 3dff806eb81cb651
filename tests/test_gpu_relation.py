"""GPU parity of the context relation features (Section 4, Appendix A.2):
at_extract_relation_features against the oracle, element for element."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def P():
    import torch
    torch.cuda.set_device(0)
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def gpu_relation(P, sp, cfgs):
    import torch
    d = torch.from_numpy(np.ascontiguousarray(cfgs, np.uint64).view(np.int64)).to(DEV)
    out = torch.empty((len(cfgs), 192), dtype=torch.int32, device=DEV)
    P.at_extract_relation_features(sp, d, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("tmpl,shape", [(W.GEMM, (4, 4, 4)), (W.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1)),
                                        (W.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2))])
def test_every_config_of_small_spaces(P, tmpl, shape):
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    cfgs = np.arange(osp.n_configs, dtype=np.uint64)
    assert np.array_equal(gpu_relation(P, sp, cfgs), osp.relation_features(cfgs))


@pytest.mark.parametrize("name", sorted(W.TABLE1))
def test_table1_shapes_sampled(P, name):
    shape = W.conv_shape(name)
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    cfgs = W.make_configs(1000 + 37, osp.n_configs, 50)   # several workgroups and a ragged tail
    assert np.array_equal(gpu_relation(P, sp, cfgs), osp.relation_features(cfgs))


def test_gemm_512_and_out_of_range(P):
    sp = P.at_space_create(W.GEMM, (512, 512, 512))
    osp = oracle.Space(W.GEMM, (512, 512, 512))
    cfgs = W.make_configs(700, osp.n_configs, 51)
    got = gpu_relation(P, sp, cfgs)
    assert np.array_equal(got, osp.relation_features(cfgs))
    P.at_space_errors(sp)
    bad = cfgs.copy()
    bad[[3, 600]] = osp.n_configs + np.array([0, 5], np.uint64)
    got = gpu_relation(P, sp, bad)
    assert (got[[3, 600]] == -1).all() and P.at_space_errors(sp) == 2
    keep = np.setdiff1d(np.arange(700), [3, 600])
    assert np.array_equal(got[keep], osp.relation_features(cfgs[keep]))


def test_one_million_configs_sampled(P):
    """The batched-scoring workload's size (1,048,576 conv2d C2
    configurations), checked on a sample of rows the oracle computes."""
    shape = W.conv_shape("C2")
    sp = P.at_space_create(W.CONV2D, shape)
    osp = oracle.Space(W.CONV2D, shape)
    cfgs = W.make_configs(1 << 20, osp.n_configs, 3002)
    got = gpu_relation(P, sp, cfgs)
    rows = np.random.default_rng(9).choice(len(cfgs), 3000, replace=False)
    rows = np.concatenate([rows, [0, len(cfgs) - 1]])
    assert np.array_equal(got[rows], osp.relation_features(cfgs[rows]))
