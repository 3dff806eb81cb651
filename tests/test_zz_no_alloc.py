"""The batch selection entry point that allocates nothing
(at_select_batch_noalloc) against at_select_batch, bit for bit.

Both run the same kernels; the no-alloc one keeps the partial reduction in
the library's fixed per-device scratch.  Two calls in a row, the second with
a smaller input, check that the scratch left by a call does not leak into
the next; the inputs need the partial reduction (more than 4096
candidates).  Sizes beyond the scratch limit are refused before anything is
enqueued.  Every call goes through the C ABI.
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
C12 = (1, 512, 7, 7, 512, 3, 3, 1, 1)


def say(msg):
    print(f"[gpu-noalloc] {msg}", flush=True)


@pytest.fixture(scope="module")
def P():
    import torch
    torch.cuda.set_device(0)
    import paper_1805_08166_amd
    return paper_1805_08166_amd


def to_dev(entries):
    import torch
    a = np.ascontiguousarray(entries).view(np.int32).reshape(*entries.shape, 4)
    return torch.from_numpy(a.copy()).to(DEV)


def select(P, fn, sp, cand_dev, pool, n_greedy, alpha, n_random, seed):
    import torch
    out = torch.full((n_greedy + n_random, 4), -1, dtype=torch.int32, device=DEV)
    fn(sp, cand_dev, pool, n_greedy, alpha, n_random, seed, out)
    torch.cuda.synchronize()
    return P.entries(out)


def same(a, b):
    return (np.array_equal(a["flag"], b["flag"]) and np.array_equal(a["cfg"], b["cfg"])
            and np.array_equal(a["score"].view(np.uint32), b["score"].view(np.uint32)))


def test_noalloc_equals_select_batch_two_calls_shrinking(P):
    sp = P.at_space_create(W.CONV2D, C12)
    osp = oracle.Space(W.CONV2D, C12)
    # first call: best lists of 8192 chains x 32 (262144 candidates, two
    # reduction levels at pool 128); second: 6000 x 16 (96000, one level,
    # pool 300) with another seed
    for n_lists, per, pool, n_greedy, n_random, seed in [(8192, 32, 128, 61, 3, 11), (6000, 16, 300, 200, 40, 12)]:
        say(f"noalloc vs select_batch: {n_lists} x {per}, pool {pool}")
        cand = W.make_candidates(n_lists, per, sp.n_configs, seed)
        d = to_dev(cand)
        got = select(P, P.at_select_batch_noalloc, sp, d, pool, n_greedy, 1.0, n_random, seed)
        want = select(P, P.at_select_batch, sp, d, pool, n_greedy, 1.0, n_random, seed)
        assert same(got, want)
        assert (got["flag"][:n_greedy] == 1).all()
        # and the oracle agrees with both
        ref = oracle.select_batch(osp, cand.view(oracle.TOP_DTYPE), pool, n_greedy, 1.0, n_random, seed)
        assert np.array_equal(got["cfg"], ref["cfg"]) and np.array_equal(got["flag"], ref["valid"])


def test_noalloc_small_input_and_limit(P):
    import torch
    sp = P.at_space_create(W.CONV2D, C12)
    # at most 4096 candidates: no scratch used
    cand = W.make_candidates(100, 16, sp.n_configs, 3)
    d = to_dev(cand)
    assert same(select(P, P.at_select_batch_noalloc, sp, d, 64, 30, 0.5, 2, 5),
                select(P, P.at_select_batch, sp, d, 64, 30, 0.5, 2, 5))
    # ceil(n / 4096) * pool above the scratch limit: refused, nothing enqueued
    big = torch.zeros((600000, 4), dtype=torch.int32, device=DEV)
    out = torch.zeros((64, 4), dtype=torch.int32, device=DEV)
    with pytest.raises(P.ATError) as ei:
        P.at_select_batch_noalloc(sp, big, 1024, 60, 1.0, 4, 1, out)
    assert ei.value.status == -2 and "scratch" in str(ei.value)
