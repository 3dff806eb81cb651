"""Oracle pins: context relation features (Section 4, Appendix A.2).

R_t = max over the loops touching fewer than 2^t elements of a buffer of
bitlen(reuse ratio), resp. bitlen(top-down product), for t = 1..32."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W
from nest_bruteforce import bitlen
from test_oracle_features import conv_bruteforce, gemm_bruteforce

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "relation_worked_example.json")
T = 32


def from_bruteforce(nest):
    """The relation rows from literally enumerated loop quantities."""
    q = nest.quantities()
    exts = [ext for ext, _, _, _ in q]
    top = [int(np.prod(exts[:k])) for k in range(len(exts))]
    n_buf = len(q[0][3])
    out = np.zeros((2, n_buf, T), np.int64)
    for b in range(n_buf):
        for t in range(1, T + 1):
            ks = [k for k in range(len(q)) if q[k][3][b][0] < 2 ** t]
            out[0, b, t - 1] = max([bitlen(q[k][3][b][1]) for k in ks], default=0)
            out[1, b, t - 1] = max([bitlen(top[k]) for k in ks], default=0)
    return out


def test_golden_appendix_configuration():
    g = json.load(open(GOLDEN))
    sp = oracle.Space(W.GEMM, g["space"]["shape"])
    rows = sp.features([g["cfg"]])[0].reshape(10, 11)
    for i, b in enumerate("ABC"):
        assert list(rows[:, 2 + 3 * i]) == g["bitlen_touch"][b]
        assert list(rows[:, 3 + 3 * i]) == g["bitlen_reuse"][b]
    r = sp.relation_features([g["cfg"]])[0].reshape(2, 3, T)
    n = g["first_thresholds"]
    for i, b in enumerate("ABC"):
        assert list(r[0, i, :n]) == g["reuse_relation"][b]
        assert list(r[1, i, :n]) == g["top_down_relation"][b]
    assert (r[:, :, n:] == r[:, :, n - 1:n]).all()


@pytest.mark.parametrize("shape", [(4, 4, 4), (2, 6, 3)])
def test_gemm_against_bruteforce(shape):
    sp = oracle.Space(W.GEMM, shape)
    rng = np.random.default_rng(sum(shape))
    cfgs = rng.choice(int(sp.n_configs), size=min(120, int(sp.n_configs)), replace=False)
    got = sp.relation_features(cfgs.astype(np.uint64)).reshape(len(cfgs), 2, 3, T)
    for i, cfg in enumerate(cfgs):
        assert (got[i] == from_bruteforce(gemm_bruteforce(sp, int(cfg)))).all(), int(cfg)


@pytest.mark.parametrize("shape", [(1, 2, 4, 4, 2, 3, 3, 1, 1), (1, 2, 6, 6, 2, 3, 3, 1, 2),
                                   (1, 2, 6, 6, 2, 1, 1, 0, 2)])
def test_conv_against_bruteforce(shape):
    sp = oracle.Space(W.CONV2D, shape)
    rng = np.random.default_rng(7)
    cfgs = rng.choice(int(sp.n_configs), size=25, replace=False)
    got = sp.relation_features(cfgs.astype(np.uint64)).reshape(len(cfgs), 2, 3, T)
    for i, cfg in enumerate(cfgs):
        assert (got[i] == from_bruteforce(conv_bruteforce(sp, int(cfg)))).all(), int(cfg)


def test_structure_at_full_size():
    """Non-decreasing in t; at t = 32 every loop qualifies (touch counts are
    below 2^31), so the values are the maxima over the whole nest; the
    top-down relation, once any loop qualifies, is the innermost loop's."""
    sp = oracle.Space(W.CONV2D, W.conv_shape("C2"))
    cfgs = W.make_configs(200, sp.n_configs, 12)
    r = sp.relation_features(cfgs).reshape(len(cfgs), 2, 3, T)
    assert (np.diff(r, axis=-1) >= 0).all()
    f = sp.features(cfgs).reshape(len(cfgs), 16, 11)
    for b in range(3):
        assert (r[:, 0, b, -1] == f[:, :, 3 + 3 * b].max(axis=1)).all()
    for i, cfg in enumerate(cfgs):
        q = sp.loop_quantities(int(cfg))
        inner_top = int(np.prod(q[:-1, 0]))
        for b in range(3):
            touched = q[:, 3 + 3 * b]
            assert (np.diff(touched) <= 0).all()       # qualifying loops form an inner suffix
            some = touched[-1] < 2 ** np.arange(1, T + 1)
            assert (r[i, 1, b][some] == bitlen(inner_top)).all() and (r[i, 1, b][~some] == 0).all()
