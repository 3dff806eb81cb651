"""Oracle pins: loop-context features (Appendix A.2) against brute-force enumeration."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads
from nest_bruteforce import conv_nest, gemm_nest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "appendix_worked_examples.json")
UNROLL = (0, 512, 1500)


def gemm_bruteforce(sp, cfg, outer=None):
    v = sp.decode(cfg)
    M, N, K = sp.shape
    nest = gemm_nest(M, N, K, sp.split(0, v[0]), sp.split(1, v[1]), sp.split(2, v[2]),
                     UNROLL[v[3]], v[4])
    return nest


def conv_bruteforce(sp, cfg):
    v = sp.decode(cfg)
    return conv_nest(sp.shape, *(sp.split(j, v[j]) for j in range(6)), UNROLL[v[6]], v[7])


def compare_quantities(sp, cfg, nest):
    q = sp.loop_quantities(cfg)
    for p, (ext, ann, bu, bufs) in enumerate(nest.quantities()):
        row = [ext, ann, bu] + [x for b in bufs for x in b]
        assert list(q[p]) == row, (cfg, p, list(q[p]), row)


def test_gemm_every_config_of_a_small_space():
    sp = oracle.Space(workloads.GEMM, (4, 4, 4))
    for cfg in range(sp.n_configs):
        compare_quantities(sp, cfg, gemm_bruteforce(sp, cfg))


@pytest.mark.parametrize("shape", [(2, 6, 3), (8, 2, 4)])
def test_gemm_rectangular(shape):
    sp = oracle.Space(workloads.GEMM, shape)
    rng = np.random.default_rng(5)
    for cfg in rng.integers(0, sp.n_configs, size=150):
        compare_quantities(sp, int(cfg), gemm_bruteforce(sp, int(cfg)))


CONV_SHAPES = [
    (1, 2, 4, 4, 2, 3, 3, 1, 1),   # 3x3, stride 1: overlapping windows
    (1, 2, 6, 6, 2, 3, 3, 1, 2),   # 3x3, stride 2: windows overlap by one
    (1, 2, 6, 6, 2, 1, 1, 0, 2),   # 1x1, stride 2: window smaller than stride (gaps)
    (1, 1, 8, 8, 2, 7, 7, 3, 2),   # 7x7, stride 2, pad 3 (the C1 pattern)
    (1, 3, 5, 5, 4, 2, 2, 0, 3),   # 2x2 window, stride 3 (gaps), no padding
]


@pytest.mark.parametrize("shape", CONV_SHAPES)
def test_conv_random_configs(shape):
    sp = oracle.Space(workloads.CONV2D, shape)
    rng = np.random.default_rng(11)
    for cfg in rng.integers(0, sp.n_configs, size=60):
        compare_quantities(sp, int(cfg), conv_bruteforce(sp, int(cfg)))


def test_touch_counts_are_translation_invariant():
    # with unclipped (padded) coordinates the distinct-address count of a
    # sub-nest does not depend on where the outer loops stand
    sp = oracle.Space(workloads.CONV2D, (1, 2, 6, 6, 2, 3, 3, 1, 2))
    rng = np.random.default_rng(3)
    for cfg in rng.integers(0, sp.n_configs, size=20):
        nest = conv_bruteforce(sp, int(cfg))
        base = nest.quantities()
        outer = [int(rng.integers(0, nest.loop_extent(p))) for p in range(16)]
        moved = nest.quantities(outer)
        assert base == moved


def test_worked_examples():
    g = json.load(open(GOLDEN))
    ex = g["gemm_2x2x2"]
    sp = oracle.Space(workloads.GEMM, ex["shape"])
    want = np.array(ex["rows"])
    assert (sp.features([ex["cfg"]]).reshape(10, 11) == want).all()
    assert (gemm_bruteforce(sp, ex["cfg"]).feature_rows() == want).all()
    ex = g["conv_c2k2_h4_3x3"]
    sp = oracle.Space(workloads.CONV2D, ex["shape"])
    want = np.array(ex["rows"])
    assert (sp.features([ex["cfg"]]).reshape(16, 11) == want).all()
    assert (conv_bruteforce(sp, ex["cfg"]).feature_rows() == want).all()
    ex = g["gemm_512_unroll"]
    sp = oracle.Space(workloads.GEMM, ex["shape"])
    assert list(sp.features([ex["cfg"]]).reshape(10, 11)[:, 1]) == ex["annotations"]


def test_closed_form_spot_values_at_full_size():
    # the outermost loop's sub-nest is the whole iteration space
    sp = oracle.Space(workloads.GEMM, workloads.GEMM_512)
    rng = np.random.default_rng(0)
    for cfg in rng.integers(0, sp.n_configs, size=20):
        q = sp.loop_quantities(int(cfg))
        assert q[0, 2] == 512 ** 3
        # whole arrays are touched at the outermost loop
        assert list(q[0, 3::3]) == [512 * 512] * 3
        # the innermost loop: one level, bottom-up equals its own length
        assert q[-1, 2] == q[-1, 0]
    sp = oracle.Space(workloads.CONV2D, workloads.conv_shape("C12"))
    for cfg in rng.integers(0, sp.n_configs, size=20):
        q = sp.loop_quantities(int(cfg))
        assert q[0, 2] == 512 * 7 * 7 * 512 * 3 * 3
        assert q[0, 3] == 512 * 9 * 9      # padded input: data_pad [512][9][9]
        assert q[0, 6] == 512 * 512 * 9    # kernel
        assert q[0, 9] == 512 * 7 * 7      # output


def test_feature_value_ranges_at_full_size():
    for name in ["gemm512_sa", "conv_c2_sa", "conv_c12_sa", "resnet18_12conv_sa"]:
        for tmpl, shape in workloads.WORKLOADS[name]["spaces"]:
            sp = oracle.Space(tmpl, shape)
            cfgs = workloads.make_configs(200, sp.n_configs, 7)
            f = sp.features(cfgs)
            assert f.min() >= 0 and f.max() <= 31
            ann = f.reshape(len(cfgs), -1, 11)[:, :, 1]
            assert set(np.unique(ann)) <= set(range(9))
