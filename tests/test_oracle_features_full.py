"""Oracle pins: feature rows with the top-down and bottom-up columns of
Appendix A.2 (13 per loop), against a hand-worked example, the brute-force
nests of nest_bruteforce.py and the closed-form iteration count."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads
from test_oracle_features import conv_bruteforce, gemm_bruteforce

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "appendix_worked_examples.json")


def bitlen(x):
    return int(x).bit_length()


def full_rows_from_nest(nest):
    """13 columns per loop from the brute-force nest: the 11 loop-context
    columns with bitlen(top-down) and bitlen(bottom-up) after the annotation;
    top-down is the product of the lengths of the loops outside."""
    rows, td = [], 1
    base = nest.feature_rows()
    for p, (ext, ann, bu, bufs) in enumerate(nest.quantities()):
        r = list(base[p])
        rows.append(r[:2] + [bitlen(td), bitlen(bu)] + r[2:])
        td *= ext
    return np.array(rows)


def test_hand_worked_gemm_2x2x2():
    # tile_i = (1,1,1,2), tile_j = (1,1,2,1), tile_k = (2,1): loop lengths
    # i1 j1 i2 j2 k1 i3 j3 k2 i4 j4 = 1 1 1 1 2 1 2 1 2 1; top-down (product
    # outside) 1 1 1 1 1 2 2 4 4 8, bottom-up (product at or inside)
    # 8 8 8 8 8 4 4 2 2 1
    g = json.load(open(GOLDEN))["gemm_2x2x2"]
    sp = oracle.Space(workloads.GEMM, g["shape"])
    full = sp.features_full([g["cfg"]]).reshape(10, 13)
    assert list(full[:, 2]) == [1, 1, 1, 1, 1, 2, 2, 3, 3, 4]
    assert list(full[:, 3]) == [4, 4, 4, 4, 4, 3, 3, 2, 2, 1]
    want = np.array(g["rows"])
    assert (full[:, :2] == want[:, :2]).all() and (full[:, 4:] == want[:, 2:]).all()


def test_every_config_of_a_small_gemm_space():
    sp = oracle.Space(workloads.GEMM, (4, 4, 4))
    cfgs = np.arange(sp.n_configs, dtype=np.uint64)
    full = sp.features_full(cfgs)
    for c in range(0, sp.n_configs, 7):
        assert (full[c].reshape(10, 13) == full_rows_from_nest(gemm_bruteforce(sp, c))).all(), c


@pytest.mark.parametrize("shape", [(1, 2, 6, 6, 2, 3, 3, 1, 2), (1, 3, 5, 5, 4, 2, 2, 0, 3), (1, 2, 4, 4, 2, 3, 3, 1, 1)])
def test_random_conv_configs(shape):
    sp = oracle.Space(workloads.CONV2D, shape)
    cfgs = workloads.make_configs(40, sp.n_configs, seed=sum(shape))
    full = sp.features_full(cfgs)
    for row, c in zip(full, cfgs):
        assert (row.reshape(16, 13) == full_rows_from_nest(conv_bruteforce(sp, int(c)))).all(), int(c)


@pytest.mark.parametrize("kind,shape", [(workloads.GEMM, (512, 512, 512)), (workloads.CONV2D, workloads.conv_shape("C2")),
                                        (workloads.CONV2D, workloads.conv_shape("C12")),
                                        (workloads.CONV2D, workloads.conv_shape("C1"))])
def test_top_down_times_bottom_up_is_the_iteration_count(kind, shape):
    sp = oracle.Space(kind, shape)
    if kind == workloads.GEMM:
        total = shape[0] * shape[1] * shape[2]
    else:
        n, c, h, w, k, kh, kw, pad, s = shape
        oh, ow = (h + 2 * pad - kh) // s + 1, (w + 2 * pad - kw) // s + 1
        total = k * oh * ow * c * kh * kw
    cfgs = workloads.make_configs(30, sp.n_configs, seed=5)
    full = sp.features_full(cfgs)
    plain = sp.features(cfgs)
    L = sp.n_loops
    for row, prow, c in zip(full, plain, cfgs):
        q = sp.loop_quantities(int(c))
        ext, bu = q[:, 0], q[:, 2]
        td = np.concatenate([[1], np.cumprod(ext)[:-1]])
        assert (td * bu == total).all()
        r = row.reshape(L, 13)
        assert [bitlen(x) for x in td] == list(r[:, 2])
        assert [bitlen(x) for x in bu] == list(r[:, 3])
        pr = prow.reshape(L, 11)
        assert (r[:, :2] == pr[:, :2]).all() and (r[:, 4:] == pr[:, 2:]).all()


def test_out_of_range_config_is_rejected():
    sp = oracle.Space(workloads.GEMM, (4, 4, 4))
    with pytest.raises(ValueError):
        sp.features_full([sp.n_configs])


@pytest.mark.parametrize("name", ["C1", "C2", "C4", "C7", "C10", "C12", "gemm"])
def test_touch_counts_never_shrink_outwards(name):
    # a sub-nest touches every element its inner sub-nests touch, so each
    # buffer's touch count is non-decreasing from the innermost loop out
    # (the relation features' thresholds therefore admit innermost runs of
    # loops)
    if name == "gemm":
        sp = oracle.Space(workloads.GEMM, (512, 512, 512))
    else:
        sp = oracle.Space(workloads.CONV2D, workloads.conv_shape(name))
    for c in workloads.make_configs(200, sp.n_configs, seed=17):
        q = sp.loop_quantities(int(c))
        for col in (3, 6, 9):
            assert (np.diff(q[:, col]) <= 0).all(), (name, int(c), col)
