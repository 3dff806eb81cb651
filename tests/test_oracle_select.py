"""Pins of the oracle's batch selection (Algorithm 1 after the annealing,
Section 3.3, Eq. 3): greedy submodular picks from the top of the candidate
pool, then epsilon-greedy random configurations."""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_worked_example.json")


def entries(cfgs, scores, valid=None):
    e = np.zeros(len(cfgs), dtype=oracle.TOP_DTYPE)
    e["cfg"] = cfgs
    e["score"] = scores
    e["valid"] = 1 if valid is None else valid
    return e


def objective(vals, scores, S, alpha):
    """Eq. 3 written out: sum of scores plus alpha times, per knob, the number
    of distinct values the picks use (exact rational arithmetic)."""
    from fractions import Fraction
    tot = sum(Fraction(float(scores[i])) for i in S)
    for j in range(vals.shape[1]):
        tot += Fraction(float(alpha)) * len({int(vals[i, j]) for i in S})
    return tot


def pool_of(sp, cand, pool):
    """Distinct valid candidates ordered by score (higher first), then index."""
    seen = {}
    for e in cand:
        if e["valid"]:
            seen[int(e["cfg"])] = float(e["score"])
    order = sorted(seen.items(), key=lambda kv: (-kv[1], kv[0]))[:pool]
    cfgs = np.array([c for c, _ in order], np.uint64)
    scores = np.array([s for _, s in order], np.float32)
    vals = np.array([sp.decode(int(c)) for c in cfgs]) if len(cfgs) else np.zeros((0, sp.n_knobs), np.int64)
    return cfgs, scores, vals


def random_candidates(sp, n, rng, dyadic=True, nonneg=False):
    cfgs = rng.integers(0, sp.n_configs, n).astype(np.uint64)
    if dyadic:
        scores = rng.integers(0 if nonneg else -32, 32, n) / 8.0
    else:
        scores = rng.normal(0, 1, n)
    sc = {}
    for c, s in zip(cfgs, scores):       # one score per configuration, as the model gives
        sc.setdefault(int(c), np.float32(s))
    return entries(cfgs, [sc[int(c)] for c in cfgs])


def test_golden_worked_example():
    g = json.load(open(GOLDEN))
    sp = oracle.Space(W.GEMM, g["space"]["shape"])
    assert list(sp.knob_sizes) == g["knob_sizes"]
    cand = g["candidates"]
    for c in cand:
        assert sp.encode(c["knobs"]) == c["cfg"]
    e = entries([c["cfg"] for c in cand], [c["score"] for c in cand])
    out = oracle.select_batch(sp, e, pool=len(cand), n_greedy=g["n_greedy"], alpha=g["alpha"], n_random=0, seed=0)
    assert list(out["cfg"]) == g["picks_cfg"]
    assert np.array_equal(out["score"], np.array(g["picks_score"], np.float32))
    assert (out["valid"] == 1).all()


def test_alpha_zero_picks_the_best_scores():
    sp = oracle.Space(W.CONV2D, (1, 8, 8, 8, 16, 3, 3, 1, 1))
    rng = np.random.default_rng(3)
    cand = random_candidates(sp, 500, rng, dyadic=False)
    cfgs, scores, _ = pool_of(sp, cand, 64)
    out = oracle.select_batch(sp, cand, pool=64, n_greedy=40, alpha=0.0, n_random=0, seed=1)
    assert np.array_equal(out["cfg"], cfgs[:40])


@pytest.mark.parametrize("alpha", [0.25, 0.5, 1.0, 3.0])
def test_each_greedy_pick_maximises_eq3(alpha):
    """With dyadic scores and alpha every fp32 gain is exact, so each pick
    must be the maximiser of L(S + {s}) - L(S) recomputed from the
    definition, ties going to the earlier candidate in pool order."""
    sp = oracle.Space(W.GEMM, (16, 16, 8))
    rng = np.random.default_rng(int(alpha * 8))
    cand = random_candidates(sp, 300, rng)
    pool = 48
    cfgs, scores, vals = pool_of(sp, cand, pool)
    out = oracle.select_batch(sp, cand, pool=pool, n_greedy=20, alpha=alpha, n_random=0, seed=0)
    pos = {int(c): i for i, c in enumerate(cfgs)}
    S = []
    for pick in out["cfg"]:
        base = objective(vals, scores, S, alpha)
        gains = [(objective(vals, scores, S + [i], alpha) - base, -i) for i in range(len(cfgs)) if i not in S]
        best = max(gains)
        assert pos[int(pick)] == -best[1]
        S.append(pos[int(pick)])


def test_gains_never_increase():
    sp = oracle.Space(W.CONV2D, (1, 4, 8, 8, 8, 3, 3, 1, 1))
    rng = np.random.default_rng(11)
    cand = random_candidates(sp, 400, rng)
    cfgs, scores, vals = pool_of(sp, cand, 64)
    out = oracle.select_batch(sp, cand, pool=64, n_greedy=30, alpha=1.0, n_random=0, seed=0)
    pos = {int(c): i for i, c in enumerate(cfgs)}
    S, prev = [], None
    for pick in out["cfg"]:
        i = pos[int(pick)]
        g = objective(vals, scores, S + [i], 1.0) - objective(vals, scores, S, 1.0)
        assert prev is None or g <= prev
        prev = g
        S.append(i)


def test_within_one_minus_one_over_e_of_the_optimum():
    """Nonnegative scores make L monotone submodular, so the greedy value is
    at least (1 - 1/e) of the best subset (Nemhauser, Wolsey, Fisher 1978)."""
    sp = oracle.Space(W.GEMM, (8, 8, 4))
    worst = 1.0
    for seed in range(12):
        rng = np.random.default_rng(100 + seed)
        cand = random_candidates(sp, 9, rng, nonneg=True)
        cfgs, scores, vals = pool_of(sp, cand, 9)
        kk = 3
        out = oracle.select_batch(sp, cand, pool=9, n_greedy=kk, alpha=0.5, n_random=0, seed=0)
        pos = {int(c): i for i, c in enumerate(cfgs)}
        got = objective(vals, scores, [pos[int(c)] for c in out["cfg"]], 0.5)
        opt = max(objective(vals, scores, list(S), 0.5) for S in itertools.combinations(range(len(cfgs)), kk))
        assert got <= opt
        worst = min(worst, float(got / opt) if opt > 0 else 1.0)
    assert worst >= 1 - 1 / math.e


def test_pool_dedupes_ignores_invalid_and_truncates():
    sp = oracle.Space(W.GEMM, (8, 8, 8))
    cfgs = np.array([5, 9, 5, 7, 11, 3, 9, 13], np.uint64)
    scores = np.array([1.0, 0.75, 1.0, 0.5, 3.0, 0.25, 0.75, -1.0], np.float32)
    valid = np.array([1, 1, 1, 1, 0, 1, 1, 1], np.uint32)
    out = oracle.select_batch(sp, entries(cfgs, scores, valid), pool=3, n_greedy=8, alpha=0.0, n_random=0, seed=0)
    # distinct valid: 5 (1.0), 9 (0.75), 7 (0.5), 3 (0.25), 13 (-1); the pool keeps three
    assert list(out["cfg"][:3]) == [5, 9, 7]
    assert (out["valid"][:3] == 1).all() and (out["valid"][3:] == 0).all()


def test_random_picks_are_new_distinct_and_uniform():
    sp = oracle.Space(W.GEMM, (2, 2, 2))     # 192 configurations
    n = int(sp.n_configs)
    cand = entries(np.arange(0, 40, dtype=np.uint64), np.linspace(2, 1, 40, dtype=np.float32))
    counts = np.zeros(n, np.int64)
    for seed in range(600):
        out = oracle.select_batch(sp, cand, pool=40, n_greedy=10, alpha=0.5, n_random=5, seed=seed)
        g, r = out[:10], out[10:]
        assert (g["valid"] == 1).all() and (r["valid"] == 2).all()
        allc = [int(x) for x in out["cfg"]]
        assert len(set(allc)) == 15 and max(allc) < n
        assert not set(int(x) for x in r["cfg"]) & set(int(x) for x in g["cfg"])
        counts[r["cfg"].astype(np.int64)] += 1
    # greedy picks come from the first 40 configurations; random ones from the
    # rest, and also from the 30 pool members that were not picked
    from scipy.stats import chisquare
    free = counts[40:]
    assert chisquare(free).pvalue > 1e-3


def test_random_picks_exhaust_a_tiny_space():
    sp = oracle.Space(W.GEMM, (2, 2, 2))
    n = int(sp.n_configs)
    out = oracle.select_batch(sp, entries(np.array([], np.uint64), np.array([], np.float32)),
                              pool=0, n_greedy=0, alpha=1.0, n_random=n + 5, seed=4)
    assert sorted(int(x) for x in out["cfg"][:n]) == list(range(n))
    assert (out["valid"][:n] == 2).all() and (out["valid"][n:] == 0).all()
