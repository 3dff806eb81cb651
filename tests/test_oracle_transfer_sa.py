"""Oracle pins: annealing whose energy is the transfer model of Section 4,
Eq. 4, f_hat = f_hat_global + f_hat_local, with the global model over the
context relation features and the local model over the loop-context
features (Section 3.3 annealing otherwise unchanged).

Pinned against things other than the annealing code itself:
  - a global model whose leaves are all +0.0 leaves every trajectory equal
    to a plain run with the local model alone (+0.0 + x == x in fp32, and a
    fold from +0.0 never yields -0.0);
  - a fold-order case: constant stumps with leaves (1e8, 1) in the global
    model and (-1e8, 1) in the local one give exactly 0 for every candidate
    (each model folded on its own, then added), while one fold over the
    concatenated trees would give 1;
  - every traced score equals the separately pinned predictions of the two
    models on the candidate's relation and loop features, added global
    first; the accept decisions follow the fp32 Metropolis rule.
"""
import numpy as np

import oracle
import workloads as W

SHAPE = (W.CONV2D, (1, 2, 6, 6, 4, 3, 3, 1, 1))
REL = 192


def models(seed=3, trees=(25, 30), depth=(5, 6)):
    sp = oracle.Space(*SHAPE)
    glob = W.make_ensemble(trees[0], depth[0], REL, seed)
    loc = W.make_ensemble(trees[1], depth[1], sp.n_features, seed + 1)
    return sp, glob, loc


def run(sp, loc, glob, n=12, steps=60, seed=7, thr=None):
    ch = oracle.Chains([sp], [0, n], seed=seed, chain0=0, topk=5)
    thr = oracle.thresholds(seed, 0, n, 0, steps) if thr is None else thr
    tr = ch.run(loc, steps, thr, trace=True, global_model=glob)
    return ch, tr, thr


def test_zero_global_model_equals_plain_run():
    sp, glob, loc = models()
    zero = (glob[0], glob[1], np.zeros_like(glob[2]))
    a, ta, thr = run(sp, loc, zero)
    b = oracle.Chains([sp], [0, 12], seed=7, chain0=0, topk=5)
    tb = b.run(loc, 60, thr, trace=True)
    assert np.array_equal(ta, tb)
    assert np.array_equal(a.top, b.top) and np.array_equal(a.knobs, b.knobs)
    assert np.array_equal(a.score.view(np.uint32), b.score.view(np.uint32))


def stumps(values, n_features):
    """Depth-1 trees whose two leaves both hold the given value."""
    T = len(values)
    fid = np.zeros((T, 1), np.uint8)
    thr = np.zeros((T, 1), np.uint8)
    leaf = np.repeat(np.asarray(values, np.float32)[:, None], 2, axis=1)
    del n_features
    return fid, thr, leaf


def test_fold_order_each_model_folded_on_its_own():
    sp = oracle.Space(*SHAPE)
    glob = stumps([1e8, 1.0], REL)
    loc = stumps([-1e8, 1.0], sp.n_features)
    ch, tr, _ = run(sp, loc, glob, n=4, steps=20)
    # fp32: (1e8 + 1) + (-1e8 + 1) = 1e8 + -1e8 = 0, not 1
    assert (tr["score"] == 0.0).all() and (ch.score == 0.0).all()
    one_fold = np.float32(0.0)
    for v in [1e8, 1.0, -1e8, 1.0]:
        one_fold = np.float32(one_fold + np.float32(v))
    assert one_fold == 1.0


def test_scores_are_global_plus_local_and_accepts_follow_metropolis():
    sp, glob, loc = models(seed=11)
    n, steps = 10, 80
    ch, tr, thr = run(sp, loc, glob, n=n, steps=steps, seed=5)
    for c in range(n):
        cfgs = tr["cfg"][c]
        want = oracle.predict_global_local(glob, sp.relation_features(cfgs), loc, sp.features(cfgs))
        assert np.array_equal(tr["score"][c].view(np.uint32), want.view(np.uint32))
    # initial state: chain c started alone, scored with both models
    for c in range(n):
        one = oracle.Chains([sp], [0, 1], seed=5, chain0=c, topk=2)
        one.run(loc, 0, np.zeros((1, 0), np.float32), global_model=glob)
        cur_s = np.float32(one.score[0])
        c0 = int(one.cur_cfgs()[0])
        want0 = oracle.predict_global_local(glob, sp.relation_features([c0]), loc, sp.features([c0]))[0]
        assert cur_s == want0
        for s in range(steps):
            acc = bool(np.float32(tr["score"][c, s] - cur_s) >= thr[c, s])
            assert acc == bool(tr["valid"][c, s])
            if acc:
                cur_s = np.float32(tr["score"][c, s])
        assert cur_s == ch.score[c]

