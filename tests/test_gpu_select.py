"""GPU parity of the batch selection (Algorithm 1 after the annealing,
Section 3.3, Eq. 3): at_select_batch against the oracle, entry for entry
(configuration index, score bits, flag).  Candidate lists come from the
seeded generator or from oracle annealing runs, never from the GPU."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(f"[gpu-select] {msg}", flush=True)


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


def run_both(P, tmpl, shape, cand, pool, n_greedy, alpha, n_random, seed):
    import torch
    sp = P.at_space_create(tmpl, shape)
    osp = oracle.Space(tmpl, shape)
    out = torch.full((n_greedy + n_random, 4), -1, dtype=torch.int32, device=DEV)
    d = to_dev(cand) if cand.size else None
    P.at_select_batch(sp, d, pool, n_greedy, alpha, n_random, seed, out)
    torch.cuda.synchronize()
    got = P.entries(out)
    want = oracle.select_batch(osp, cand.view(oracle.TOP_DTYPE), pool, n_greedy, alpha, n_random, seed)
    assert np.array_equal(got["flag"], want["valid"]), "flags differ"
    assert np.array_equal(got["cfg"], want["cfg"]), "picks differ"
    assert np.array_equal(got["score"].view(np.uint32), want["score"].view(np.uint32)), "scores differ"
    return got


C2 = (1, 64, 56, 56, 64, 3, 3, 1, 1)
C12 = (1, 512, 7, 7, 512, 3, 3, 1, 1)


def test_select_after_annealing_c2(P):
    """Best lists of an oracle annealing run on conv2d C2 (64 chains x 150
    steps, top-16), the paper's batch b = 64 with epsilon = 0.05: 61 greedy
    picks from the top 2b = 128, 3 random."""
    say("select: oracle best lists of conv2d C2")
    wl = W.WORKLOADS["conv_c2_sa"]
    osp = oracle.Space(W.CONV2D, C2)
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    n, steps, k, seed = 64, 150, 16, wl["sa_seed"]
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps))
    cand = och.top.view(W.ENTRY_DTYPE)
    got = run_both(P, W.CONV2D, C2, cand, pool=128, n_greedy=61, alpha=1.0, n_random=3, seed=77)
    assert (got["flag"][:61] == 1).all() and (got["flag"][61:] == 2).all()


@pytest.mark.parametrize("n_lists,per_list,pool,n_greedy,alpha", [
    (8192, 32, 128, 61, 1.0),     # the C12 search's lists: two levels of partial reduction
    (1024, 16, 1024, 1024, 0.5),  # the largest pool, every candidate picked
    (128, 16, 128, 61, 0.0),      # 2048 candidates: one workgroup, no partial level
    (2049, 1, 64, 32, 2.0),       # one past a workgroup's slice
    (256, 16, 128, 61, 0.0),      # 4096 candidates: one partial level
    (300, 7, 200, 150, -0.25),    # negative alpha
    (6000, 16, 300, 200, 1.0),    # pool not a power of two: runs of 512
    (4096, 64, 1000, 300, 0.3),   # 262144 candidates, runs of 1024: seven partial levels
])
def test_select_synthetic_candidates(P, n_lists, per_list, pool, n_greedy, alpha):
    say(f"select: {n_lists}x{per_list} synthetic, pool {pool}, greedy {n_greedy}, alpha {alpha}")
    osp = oracle.Space(W.CONV2D, C12)
    cand = W.make_candidates(n_lists, per_list, osp.n_configs, seed=n_lists + per_list)
    run_both(P, W.CONV2D, C12, cand, pool=pool, n_greedy=n_greedy, alpha=alpha, n_random=5, seed=n_lists)


def in_list_order(cand):
    """Each list in best-list order: valid entries by score descending, then
    index ascending, empty slots last."""
    out = cand.copy()
    for i in range(len(out)):
        row = out[i]
        out[i] = row[np.lexsort((row["cfg"], -row["score"].astype(np.float64), row["flag"] == 0))]
    return out


def test_select_lists_in_list_order_through_reduction(P):
    # lists that are already ordered runs (as best lists are): the first
    # merge levels of every reduction workgroup find their runs in order
    say("select: 512x32 lists in best-list order")
    osp = oracle.Space(W.CONV2D, C12)
    cand = in_list_order(W.make_candidates(512, 32, osp.n_configs, seed=91))
    run_both(P, W.CONV2D, C12, cand, pool=128, n_greedy=61, alpha=1.0, n_random=3, seed=9)


def repeats_and_ties(kind, n_lists, per_list, n_configs, seed):
    """Candidate lists that stress the pool stage: exact repeats, the same
    index with different scores, ties, signed zeros, outlying scores."""
    rng = np.random.default_rng(seed)
    cand = W.make_candidates(n_lists, per_list, n_configs, seed=seed).reshape(-1)
    valid = np.flatnonzero(cand["flag"] == 1)
    if kind == "few_configs":
        # every entry one of 40 configurations, a score per configuration
        cfgs = rng.choice(n_configs, 40, replace=False).astype(np.uint64)
        scores = rng.normal(0.0, 1.0, 40).astype(np.float32)
        pick = rng.integers(0, 40, len(valid))
        cand["cfg"][valid] = cfgs[pick]
        cand["score"][valid] = scores[pick]
    elif kind == "same_index_other_score":
        # a quarter of the entries take another entry's index, keeping
        # their own score (outside what at_select_batch asks of its input;
        # the library still drops exactly what the oracle drops)
        idx = rng.choice(valid, len(valid) // 4, replace=False)
        cand["cfg"][idx] = cand["cfg"][rng.choice(valid, len(idx))]
    elif kind == "all_tied":
        cand["score"][valid] = np.float32(1.5)
    elif kind == "signed_zero":
        # scores +0.0 and -0.0 (equal in the order), repeats of an index
        # with either sign, and a few nonzero scores
        z = np.where(rng.random(len(valid)) < 0.5, np.float32(0.0), np.float32(-0.0))
        cand["score"][valid] = z
        few = rng.choice(valid, len(valid) // 50, replace=False)
        cand["score"][few] = rng.normal(0.0, 1.0, len(few)).astype(np.float32)
    elif kind == "outliers":
        # most scores in one histogram bin next to a handful of huge ones
        few = rng.choice(valid, 5, replace=False)
        cand["score"][few] = np.float32([1e30, -1e30, 3e29, -2e25, 1e20])
    return cand.reshape(n_lists, per_list)


@pytest.mark.parametrize("kind", ["few_configs", "same_index_other_score", "all_tied", "signed_zero", "outliers"])
@pytest.mark.parametrize("n_lists,per_list", [(100, 16), (8192, 32)])
def test_select_repeats_and_ties(P, kind, n_lists, per_list):
    say(f"select: {kind}, {n_lists}x{per_list}")
    osp = oracle.Space(W.CONV2D, C12)
    cand = repeats_and_ties(kind, n_lists, per_list, osp.n_configs, seed=len(kind) + n_lists)
    run_both(P, W.CONV2D, C12, cand, pool=128, n_greedy=61, alpha=1.0, n_random=3, seed=17)


@pytest.mark.parametrize("kind", ["empty", "all_invalid", "pool_smaller", "pool_zero", "exhaust_space", "one_pick"])
def test_select_edge_cases(P, kind):
    gemm = (2, 2, 2)   # 192 configurations
    if kind == "empty":
        cand = np.zeros((0,), W.ENTRY_DTYPE)
        run_both(P, W.GEMM, gemm, cand, pool=16, n_greedy=8, alpha=1.0, n_random=4, seed=1)
    elif kind == "all_invalid":
        cand = W.make_candidates(10, 8, 192, seed=3)
        cand["flag"] = 0
        run_both(P, W.GEMM, gemm, cand, pool=16, n_greedy=8, alpha=1.0, n_random=4, seed=2)
    elif kind == "pool_smaller":
        cand = W.make_candidates(20, 8, 192, seed=4)
        got = run_both(P, W.GEMM, gemm, cand, pool=10, n_greedy=30, alpha=1.0, n_random=6, seed=3)
        assert (got["flag"][:10] == 1).all() and (got["flag"][10:16] == 2).all() and (got["flag"][16:] == 0).all()
    elif kind == "pool_zero":
        cand = W.make_candidates(20, 8, 192, seed=5)
        run_both(P, W.GEMM, gemm, cand, pool=0, n_greedy=5, alpha=1.0, n_random=6, seed=4)
    elif kind == "exhaust_space":
        cand = W.make_candidates(40, 8, 192, seed=6, dup_frac=0.0)
        got = run_both(P, W.GEMM, gemm, cand, pool=100, n_greedy=100, alpha=0.5, n_random=150, seed=5)
        picked = got["cfg"][got["flag"] != 0]
        assert len(set(int(x) for x in picked)) == len(picked) == 192
    else:
        cand = W.make_candidates(3, 5, 192, seed=7)
        run_both(P, W.GEMM, gemm, cand, pool=1, n_greedy=1, alpha=3.0, n_random=0, seed=6)


def test_select_batch_on_two_streams(P):
    """The allocating call keeps one scratch per device and orders its calls
    through an event: calls on two streams, started so that their kernels
    would interleave, each give the oracle's batch."""
    import torch
    osp = oracle.Space(W.CONV2D, C12)
    sp = P.at_space_create(W.CONV2D, C12)
    cands = [W.make_candidates(4096, 16, osp.n_configs, seed=s) for s in (301, 302)]
    wants = [oracle.select_batch(osp, c.view(oracle.TOP_DTYPE), 128, 61, 1.0, 3, 11 + i) for i, c in enumerate(cands)]
    dev = [to_dev(c) for c in cands]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [torch.full((64, 4), -1, dtype=torch.int32, device=DEV) for _ in range(2)]
    torch.cuda.synchronize()
    for rep in range(6):
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                torch.cuda._sleep(200000 + 30000 * i)
                P.at_select_batch(sp, dev[i], 128, 61, 1.0, 3, 11 + i, outs[i], stream=streams[i])
        torch.cuda.synchronize()
        for i in range(2):
            got = P.entries(outs[i])
            assert np.array_equal(got["cfg"], wants[i]["cfg"]) and np.array_equal(got["flag"], wants[i]["valid"])
            assert np.array_equal(got["score"].view(np.uint32), wants[i]["score"].view(np.uint32))


def test_select_argument_errors(P):
    INVALID, UNSUPPORTED = -1, -2
    sp = P.at_space_create(W.GEMM, (8, 8, 8))
    sel = P.lib().at_select_batch
    assert sel(sp.h, None, 5, 4, 2, 1.0, 1, 0, None, None) == INVALID          # NULL candidates
    assert sel(sp.h, None, 0, 2000, 2, 1.0, 1, 0, None, None) == UNSUPPORTED    # pool above 1024
    assert sel(sp.h, None, 0, 4, 2000, 1.0, 100, 0, None, None) == UNSUPPORTED  # more than 2048 picks
    assert sel(sp.h, None, 0, 4, 2, float("inf"), 1, 0, None, None) == INVALID
    assert sel(sp.h, None, 0, 4, 2, 1.0, 1, 0, None, None) == INVALID          # NULL output
    assert sel(sp.h, None, 0, 4, 0, 1.0, 0, 0, None, None) == 0                # nothing to pick
    sets = P.at_spaceset_create([sp, sp], np.array([0, 1, 2], np.int64))
    assert sel(sets.h, None, 0, 4, 2, 1.0, 1, 0, None, None) == INVALID         # a set, not a space
