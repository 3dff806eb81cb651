"""CPU checks of the C-ABI library: it loads, exports every declared entry
point, validates arguments before touching the device, and its host-side
threshold helper agrees bit for bit with the oracle's."""
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "autotensor.h")


@pytest.fixture(scope="module")
def P():
    from paper_1805_08166_amd import build as B
    if B.stale():
        B.build()
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(at_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(P):
    names = declared_functions()
    assert len(names) >= 17
    for n in names:
        assert hasattr(P.lib(), n), n
    assert sorted(P.EXPORTED) == names


def test_thresholds_match_oracle_bitwise(P):
    for seed, chain0, n, base, steps in [(2000, 0, 64, 0, 500), (2003, 100, 17, 250, 33), (7, 5, 3, 0, 1),
                                         (2 ** 40 + 5, 2 ** 31, 4, 2 ** 31, 9)]:
        got = P.at_sa_thresholds(seed, chain0, n, base, steps)
        want = oracle.thresholds(seed, chain0, n, base, steps)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def expect_status(P, fn, status):
    with pytest.raises(P.ATError) as ei:
        fn()
    assert ei.value.status == status, str(ei.value)


def test_argument_errors_before_device_use(P):
    INVALID, UNSUPPORTED = -1, -2
    expect_status(P, lambda: P.at_space_create(0, (0, 4, 4)), INVALID)
    expect_status(P, lambda: P.at_space_create(0, (4, 4)), INVALID)
    expect_status(P, lambda: P.at_space_create(7, (4, 4, 4)), INVALID)
    expect_status(P, lambda: P.at_space_create(1, (2, 4, 8, 8, 4, 3, 3, 1, 1)), INVALID)
    expect_status(P, lambda: P.at_space_create(1, (1, 4, 2, 2, 4, 5, 5, 0, 1)), INVALID)
    expect_status(P, lambda: P.at_space_create(0, (70000, 4, 4)), UNSUPPORTED)
    # 2^31 iterations or more
    expect_status(P, lambda: P.at_space_create(0, (2048, 2048, 1024)), UNSUPPORTED)
    expect_status(P, lambda: P.at_sa_thresholds(1, 0, 4, 0, 0), INVALID)
    fid = np.zeros((2, 3), np.uint8)
    thr = np.zeros((2, 3), np.uint8)
    leaf = np.zeros((2, 4), np.float32)
    expect_status(P, lambda: P.at_ensemble_create(fid + 9, thr, leaf, 8), INVALID)   # fid >= F
    expect_status(P, lambda: P.at_ensemble_create(fid, thr, leaf, 300), UNSUPPORTED)
    deep = np.zeros((1, (1 << 13) - 1), np.uint8)
    expect_status(P, lambda: P.at_ensemble_create(deep, deep, np.zeros((1, 1 << 13), np.float32), 8), UNSUPPORTED)
    assert "depth" in P.lib().at_last_error().decode()
    assert P.lib().at_sa_set_profiling(None, 1) == INVALID
    assert P.lib().at_sa_kernel_times(None, None, None, None, None) == INVALID
    assert P.lib().at_chains_set_path(None, 1) == INVALID
    assert P.lib().at_chains_last_plan(None, None) == INVALID
    assert P.lib().at_select_batch(None, None, 0, 4, 2, 1.0, 1, 0, None, None) == INVALID


def bitlen(x):
    return int(x).bit_length()


def test_quotient_bitlen_identity():
    # The feature kernels compute bitlen(a // b) as k + (a >> k >= b) with
    # k = bitlen(a) - bitlen(b), for a >= b >= 1.
    def fast(a, b):
        k = bitlen(a) - bitlen(b)
        return k + (1 if (a >> k) >= b else 0)
    for a in range(1, 600):
        for b in range(1, a + 1):
            assert fast(a, b) == bitlen(a // b)
    rng = np.random.default_rng(0)
    for _ in range(20000):
        a = int(rng.integers(1, 2 ** 31))
        b = int(rng.integers(1, a + 1))
        assert fast(a, b) == bitlen(a // b)
