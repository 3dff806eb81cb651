"""Oracle pins: schedule spaces (Section 2 multi-level tiling) and knob decoding."""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads
from nest_bruteforce import ordered_splits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "appendix_worked_examples.json")


def prime_exponents(n):
    out, p = [], 2
    while p * p <= n:
        e = 0
        while n % p == 0:
            n //= p
            e += 1
        if e:
            out.append(e)
        p += 1
    if n > 1:
        out.append(1)
    return out


def n_ordered_splits(n, k):
    """Closed form: prod over prime powers p^e of C(e+k-1, k-1)."""
    return math.prod(math.comb(e + k - 1, k - 1) for e in prime_exponents(n))


@pytest.mark.parametrize("n,k", [(1, 4), (2, 4), (12, 4), (56, 4), (64, 4), (512, 4), (512, 2), (3, 2),
                                 (7, 4), (28, 4), (112, 4), (64, 2), (14, 4)])
def test_split_count_closed_form(n, k):
    sp = oracle.Space(workloads.GEMM, (n, n, n)) if k == 4 else oracle.Space(workloads.GEMM, (1, 1, n))
    knob = 0 if k == 4 else 2
    assert sp.knob_sizes[knob] == n_ordered_splits(n, k)


@pytest.mark.parametrize("n", [1, 4, 12, 18, 32])
def test_split_order_is_lexicographic(n):
    sp = oracle.Space(workloads.GEMM, (n, n, n))
    got = [sp.split(0, i) for i in range(sp.knob_sizes[0])]
    assert got == ordered_splits(n, 4)
    got2 = [sp.split(2, i) for i in range(sp.knob_sizes[2])]
    assert got2 == ordered_splits(n, 2)


def test_space_sizes_of_the_workloads():
    # knob sizes follow from the closed-form split counts of each axis extent
    for name, wl in workloads.WORKLOADS.items():
        for tmpl, shape in wl["spaces"]:
            sp = oracle.Space(tmpl, shape)
            if tmpl == workloads.GEMM:
                M, N, K = shape
                want = [n_ordered_splits(M, 4), n_ordered_splits(N, 4), n_ordered_splits(K, 2), 3, 2]
            else:
                _, C, H, W, K, KH, KW, P, S = shape
                OH, OW = (H + 2 * P - KH) // S + 1, (W + 2 * P - KW) // S + 1
                want = [n_ordered_splits(K, 4), n_ordered_splits(OH, 4), n_ordered_splits(OW, 4),
                        n_ordered_splits(C, 2), n_ordered_splits(KH, 2), n_ordered_splits(KW, 2), 3, 2]
            assert list(sp.knob_sizes) == want, name
            assert sp.n_configs == math.prod(want)
            assert sp.n_features == (110 if tmpl == workloads.GEMM else 176)


def test_space_sizes_known_values():
    assert oracle.Space(workloads.GEMM, workloads.GEMM_512).n_configs == 2_904_000
    assert oracle.Space(workloads.CONV2D, workloads.conv_shape("C2")).n_configs == 90_316_800
    assert oracle.Space(workloads.CONV2D, workloads.conv_shape("C12")).n_configs == 844_800


def test_decode_is_mixed_radix_knob0_most_significant():
    sp = oracle.Space(workloads.GEMM, (4, 4, 4))
    sizes = sp.knob_sizes
    prev = None
    for cfg in range(sp.n_configs):
        v = sp.decode(cfg)
        # numeric order of indices == lexicographic order of knob vectors
        if prev is not None:
            assert tuple(prev) < tuple(v)
        prev = v
        assert all(0 <= v[j] < sizes[j] for j in range(len(sizes)))
        assert sp.encode(v) == cfg
    assert sp.n_configs == 10 * 10 * 3 * 3 * 2  # splits of 4: 10 (4-level), 3 (2-level)


def test_decode_round_trip_conv_tiny():
    sp = oracle.Space(workloads.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1))
    for cfg in range(0, sp.n_configs, 7):
        assert sp.encode(sp.decode(cfg)) == cfg


def test_worked_example_indices():
    g = json.load(open(GOLDEN))
    ex = g["gemm_2x2x2"]
    sp = oracle.Space(workloads.GEMM, ex["shape"])
    assert sp.n_configs == ex["n_configs"]
    v = sp.decode(ex["cfg"])
    assert [sp.split(0, v[0]), sp.split(1, v[1]), sp.split(2, v[2])] == \
        [tuple(ex["tiles"]["i"]), tuple(ex["tiles"]["j"]), tuple(ex["tiles"]["k"])]
    ex = g["conv_c2k2_h4_3x3"]
    sp = oracle.Space(workloads.CONV2D, ex["shape"])
    assert sp.n_configs == ex["n_configs"]
    assert list(sp.decode(ex["cfg"])) == ex["knobs"]
    ex = g["gemm_512_unroll"]
    sp = oracle.Space(workloads.GEMM, ex["shape"])
    v = sp.decode(ex["cfg"])
    assert [sp.split(0, v[0]), sp.split(1, v[1]), sp.split(2, v[2])] == \
        [tuple(ex["tiles"]["i"]), tuple(ex["tiles"]["j"]), tuple(ex["tiles"]["k"])]
    assert v[3] == ex["auto_unroll_index"] and v[4] == ex["unroll_explicit"]


def test_invalid_shapes_rejected():
    with pytest.raises(ValueError):
        oracle.Space(workloads.GEMM, (0, 4, 4))
    with pytest.raises(ValueError):
        oracle.Space(workloads.CONV2D, (2, 4, 4, 4, 4, 3, 3, 1, 1))  # batch must be 1
    with pytest.raises(ValueError):
        oracle.Space(workloads.CONV2D, (1, 4, 2, 2, 4, 5, 5, 0, 1))  # window larger than input
    sp = oracle.Space(workloads.GEMM, (4, 4, 4))
    with pytest.raises(ValueError):
        sp.decode(sp.n_configs)
