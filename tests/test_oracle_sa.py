"""Oracle pins: parallel simulated annealing (Section 3.3, Algorithm 1).

Invariants checked against the trajectory trace, re-derived here without the
oracle's code: Metropolis acceptance, per-chain top-k, one-knob proposals,
zero/infinite temperatures, persistence and chain independence, and the
exhaustive-search check on a space small enough to enumerate.
"""
import numpy as np
import pytest

import oracle
import workloads

GEMM4 = (workloads.GEMM, (4, 4, 4))


def small_run(steps=120, n=8, seed=5, thr=None, topk=6, tmpl=GEMM4, depth=5, trees=20):
    sp = oracle.Space(*tmpl)
    ens = workloads.make_ensemble(trees, depth, sp.n_features, 17)
    ch = oracle.Chains([sp], [0, n], seed=seed, chain0=0, topk=topk)
    if thr is None:
        thr = oracle.thresholds(seed, 0, n, 0, steps)
    tr = ch.run(ens, steps, thr, trace=True)
    return sp, ens, ch, tr, thr


def score_of(sp, ens, cfgs):
    return oracle.predict(*ens, sp.features(np.asarray(cfgs, np.uint64)))


def replay(ch0_cfg, ch0_score, tr, thr):
    """Re-derive accept flags and current state from the trace (fp32 Metropolis)."""
    cur_c, cur_s = ch0_cfg, np.float32(ch0_score)
    for s in range(len(tr)):
        delta = np.float32(tr["score"][s]) - cur_s
        acc = bool(delta >= thr[s])
        assert acc == bool(tr["valid"][s]), s
        if acc:
            cur_c, cur_s = int(tr["cfg"][s]), np.float32(tr["score"][s])
    return cur_c, cur_s


def init_state(sp, ens, seed, chain):
    fresh = oracle.Chains([sp], [0, 1], seed=seed, chain0=chain, topk=4)
    fresh.run(ens, 0, np.zeros((1, 0), np.float32))
    return int(fresh.cur_cfgs()[0]), np.float32(fresh.score[0])


def test_accept_rule_scores_and_final_state():
    sp, ens, ch, tr, thr = small_run()
    for c in range(ch.n):
        c0, s0 = init_state(sp, ens, 5, c)
        assert s0 == score_of(sp, ens, [c0])[0]
        cur_c, cur_s = replay(c0, s0, tr[c], thr[c])
        assert ch.cur_cfgs()[c] == cur_c and ch.score[c] == cur_s
        # every proposal's score is the model's prediction of its features
        assert (score_of(sp, ens, tr["cfg"][c]) == tr["score"][c]).all()


def test_proposals_change_exactly_one_knob():
    sp, ens, ch, tr, thr = small_run(thr=np.full((8, 120), -np.inf, np.float32))
    for c in range(ch.n):
        prev = sp.decode(init_state(sp, ens, 5, c)[0])
        for s in range(120):
            v = sp.decode(int(tr["cfg"][c, s]))
            assert (v != prev).sum() == 1
            prev = v   # threshold -inf: every move accepted (pure random walk)
        assert tr["valid"][c].all()


def test_random_walk_is_uniform_over_knobs_and_values():
    n, steps = 64, 200
    sp, ens, ch, tr, thr = small_run(steps=steps, n=n, thr=np.full((n, steps), -np.inf, np.float32))
    counts = np.zeros(sp.n_knobs)
    for c in range(n):
        prev = sp.decode(init_state(sp, ens, 5, c)[0])
        for s in range(steps):
            v = sp.decode(int(tr["cfg"][c, s]))
            counts[np.nonzero(v != prev)[0][0]] += 1
            prev = v
    exp = n * steps / sp.n_knobs
    chi2 = ((counts - exp) ** 2 / exp).sum()
    assert chi2 < 20   # 4 dof


def test_infinite_threshold_never_moves():
    sp, ens, ch, tr, thr = small_run(thr=np.full((8, 120), np.inf, np.float32))
    assert not tr["valid"].any()
    for c in range(ch.n):
        assert ch.cur_cfgs()[c] == init_state(sp, ens, 5, c)[0]


def test_zero_temperature_never_decreases():
    n, steps = 16, 150
    thr = np.full((n, steps), -0.0, np.float32)
    sp, ens, ch, tr, _ = small_run(steps=steps, n=n, thr=thr)
    for c in range(n):
        c0, s0 = init_state(sp, ens, 5, c)
        cur = s0
        best = s0
        for s in range(steps):
            if tr["valid"][c, s]:
                assert tr["score"][c, s] >= cur
                cur = tr["score"][c, s]
            best = max(best, tr["score"][c, s])
            assert cur <= best
        assert ch.top["score"][c, 0] == best


def test_topk_is_k_best_distinct_visited():
    sp, ens, ch, tr, thr = small_run(steps=200, topk=7)
    for c in range(ch.n):
        c0, s0 = init_state(sp, ens, 5, c)
        seen = {c0: s0}
        for s in range(200):
            seen[int(tr["cfg"][c, s])] = np.float32(tr["score"][c, s])
        ranked = sorted(seen.items(), key=lambda kv: (-float(kv[1]), kv[0]))[:7]
        got = [(int(e["cfg"]), np.float32(e["score"])) for e in ch.top[c] if e["valid"]]
        assert got == [(k, np.float32(v)) for k, v in ranked]


def test_persistence_split_run_equals_full_run():
    n, steps = 6, 100
    sp = oracle.Space(*GEMM4)
    ens = workloads.make_ensemble(20, 5, sp.n_features, 3)
    thr = oracle.thresholds(9, 0, n, 0, steps)
    a = oracle.Chains([sp], [0, n], seed=9, chain0=0, topk=5)
    ta = a.run(ens, steps, thr, trace=True)
    b = oracle.Chains([sp], [0, n], seed=9, chain0=0, topk=5)
    tb1 = b.run(ens, 40, thr[:, :40].copy(), trace=True)
    tb2 = b.run(ens, 60, thr[:, 40:].copy(), trace=True)
    assert np.array_equal(ta, np.concatenate([tb1, tb2], axis=1))
    assert np.array_equal(a.top, b.top) and np.array_equal(a.knobs, b.knobs)
    assert (a.step_abs == 100).all() and (b.step_abs == 100).all()


def test_chain_independence_subset_is_slice():
    n, steps = 12, 60
    sp = oracle.Space(*GEMM4)
    ens = workloads.make_ensemble(20, 5, sp.n_features, 3)
    thr = oracle.thresholds(4, 0, n, 0, steps)
    full = oracle.Chains([sp], [0, n], seed=4, chain0=0, topk=3)
    tf = full.run(ens, steps, thr, trace=True)
    part = oracle.Chains([sp], [0, 5], seed=4, chain0=4, topk=3)
    tp = part.run(ens, steps, thr[4:9].copy(), trace=True)
    assert np.array_equal(tf[4:9], tp) and np.array_equal(full.top[4:9], part.top)


def test_spaceset_equals_separate_runs():
    spaces = [oracle.Space(workloads.CONV2D, s) for s in
              [(1, 2, 4, 4, 2, 3, 3, 1, 1), (1, 2, 6, 6, 2, 1, 1, 0, 2), (1, 1, 8, 8, 2, 7, 7, 3, 2)]]
    ens = workloads.make_ensemble(30, 6, 176, 8)
    off = workloads.chain_offsets(3, 4)
    steps = 40
    thr = oracle.thresholds(21, 100, 12, 0, steps)
    ss = oracle.Chains(spaces, off, seed=21, chain0=100, topk=4)
    t_all = ss.run(ens, steps, thr, trace=True)
    for w, sp in enumerate(spaces):
        one = oracle.Chains([sp], [0, 4], seed=21, chain0=100 + 4 * w, topk=4)
        t1 = one.run(ens, steps, thr[4 * w: 4 * w + 4].copy(), trace=True)
        assert np.array_equal(t1, t_all[4 * w: 4 * w + 4])


def test_one_by_one_kernels_have_unmutable_window_knobs():
    sp = oracle.Space(workloads.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2))
    assert sp.knob_sizes[4] == 1 and sp.knob_sizes[5] == 1
    ens = workloads.make_ensemble(10, 4, 176, 8)
    ch = oracle.Chains([sp], [0, 4], seed=3, chain0=0, topk=4)
    tr = ch.run(ens, 50, np.full((4, 50), -np.inf, np.float32), trace=True)
    for c in range(4):
        for s in range(50):
            v = sp.decode(int(tr["cfg"][c, s]))
            assert v[4] == 0 and v[5] == 0


def test_best_by_score_matches_exhaustive_search():
    # GEMM 4x4x4 has 1800 configurations: enumerate them, score each, and check
    # that the pooled top-k of 64 chains x 500 steps is the exhaustive top-k
    sp = oracle.Space(*GEMM4)
    ens = workloads.make_ensemble(40, 6, sp.n_features, 1000)
    allc = np.arange(sp.n_configs, dtype=np.uint64)
    sc = oracle.predict(*ens, sp.features(allc))
    order = sorted(range(sp.n_configs), key=lambda i: (-float(sc[i]), i))
    n, steps, k = 64, 500, 8
    thr = oracle.thresholds(2000, 0, n, 0, steps)
    ch = oracle.Chains([sp], [0, n], seed=2000, chain0=0, topk=k)
    ch.run(ens, steps, thr)
    pool = {}
    for c in range(n):
        for e in ch.top[c]:
            if e["valid"]:
                pool[int(e["cfg"])] = np.float32(e["score"])
    pooled = sorted(pool.items(), key=lambda kv: (-float(kv[1]), kv[0]))[:k]
    assert [c for c, _ in pooled] == order[:k]
    assert all(np.float32(sc[c]) == s for c, s in pooled)


def test_initial_configurations_uniform_and_distinct_across_chains():
    # chain initialisation draws each knob uniformly over its values from the
    # chain's own random stream: per-knob chi-square over 8192 chains, a
    # contingency chi-square between the two largest knobs, and distinct
    # starting configurations (a draw that ignored the chain id would give
    # every chain the same start)
    sp = oracle.Space(*workloads.WORKLOADS["conv_c2_sa"]["spaces"][0])
    ens = workloads.make_ensemble(1, 1, sp.n_features, 5)
    n = 8192
    ch = oracle.Chains([sp], [0, n], seed=2001, chain0=0, topk=1)
    ch.run(ens, 0, np.zeros((n, 0), np.float32))
    kv = ch.knobs[:, : sp.n_knobs]
    for j, size in enumerate(sp.knob_sizes):
        size = int(size)
        assert kv[:, j].min() >= 0 and kv[:, j].max() < size
        if size == 1:
            continue
        counts = np.bincount(kv[:, j], minlength=size)
        exp = n / size
        chi2 = ((counts - exp) ** 2 / exp).sum()
        dof = size - 1
        assert chi2 < dof + 6 * np.sqrt(2 * dof), (j, chi2, dof)
    # knobs 0 and 1 (84 and 80 values) binned into quarters: independent
    a, b = kv[:, 0] * 4 // int(sp.knob_sizes[0]), kv[:, 1] * 4 // int(sp.knob_sizes[1])
    table = np.zeros((4, 4))
    np.add.at(table, (a, b), 1)
    expt = table.sum(1, keepdims=True) * table.sum(0, keepdims=True) / n
    chi2 = ((table - expt) ** 2 / expt).sum()
    assert chi2 < 9 + 6 * np.sqrt(18)
    # 8192 draws from 90 M configurations: almost surely all distinct
    cfgs = ch.cur_cfgs()
    assert len(np.unique(cfgs)) >= n - 2
    # a chain's start depends on its global id only: chains 100.. started alone agree
    part = oracle.Chains([sp], [0, 16], seed=2001, chain0=100, topk=1)
    part.run(ens, 0, np.zeros((16, 0), np.float32))
    assert np.array_equal(part.knobs, ch.knobs[100:116])
