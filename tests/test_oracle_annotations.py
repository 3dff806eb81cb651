"""Oracle pins: the templates with vectorize and vthread knobs (Section 2
lists unrolling and vectorization among the annotations of its search space)
and the one-hot form of the annotation column (Appendix A.2 loop-context
table).

Pinned against:
  - the hand-worked annotation columns in tests/golden (Appendix A.3 GEMM and
    Appendix A.1 conv2d schedules under every vectorize/vthread setting);
  - the base templates: with both new knobs at 0, an annotated template's
    rows equal the base template's rows (those are pinned by hand-worked
    rows and brute-force nests), and only annotation columns ever differ;
  - the full Appendix A.2 rows: a one-hot row is the full row with the
    annotation id spread over 12 columns (exactly one 1, at the id);
  - counts: four times the base template's configurations, knob sizes 2, 2;
  - annealing invariants on an annotated space: one knob per proposal,
    uniform knob choice, and the exhaustive-search match on a small space.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "annotation_knobs_worked_example.json")
GEMM_VT, CONV_VT = 2, 3
KINDS = 12


def ann_cols(sp, cfg):
    return list(sp.features([cfg]).reshape(sp.n_loops, 11)[:, 1])


@pytest.mark.parametrize("name,base,vt", [("gemm_512_unroll", W.GEMM, GEMM_VT),
                                          ("conv_c2k2_h4_3x3", W.CONV2D, CONV_VT)])
def test_hand_worked_annotation_columns(name, base, vt):
    g = json.load(open(GOLDEN))[name]
    sp = oracle.Space(vt, g["shape"])
    for key, want in g["annotations"].items():
        vec, vth = int(key[0]), int(key[1])
        cfg = g["base_cfg"] * 4 + vec * 2 + vth
        assert list(sp.decode(cfg)[-2:]) == [vec, vth]
        assert ann_cols(sp, cfg) == want, key


@pytest.mark.parametrize("base,vt,shape", [(W.GEMM, GEMM_VT, (4, 4, 4)), (W.GEMM, GEMM_VT, (512, 512, 512)),
                                           (W.CONV2D, CONV_VT, (1, 2, 6, 6, 4, 3, 3, 1, 1)),
                                           (W.CONV2D, CONV_VT, W.conv_shape("C12"))])
def test_annotated_template_extends_the_base(base, vt, shape):
    b, a = oracle.Space(base, shape), oracle.Space(vt, shape)
    assert a.n_configs == 4 * b.n_configs
    assert list(a.knob_sizes) == list(b.knob_sizes) + [2, 2]
    assert a.n_loops == b.n_loops and a.n_features == b.n_features
    cfgs = W.make_configs(300, b.n_configs, seed=len(shape))
    fb = b.features(cfgs).reshape(-1, b.n_loops, 11)
    for vec in (0, 1):
        for vth in (0, 1):
            fa = a.features(cfgs * 4 + vec * 2 + vth).reshape(-1, a.n_loops, 11)
            # only the annotation column can differ
            assert (np.delete(fa, 1, axis=2) == np.delete(fb, 1, axis=2)).all()
            if vec == 0 and vth == 0:
                assert (fa == fb).all()
            # the innermost loop is vectorized exactly when vectorize is on
            assert ((fa[:, -1, 1] == 10) == bool(vec)).all()
            # vthread marks exactly the third-level spatial loops
            n_vt = (fa[:, :, 1] == 9).sum(axis=1)
            assert (n_vt == (2 if base == W.GEMM else 3) * vth).all()


@pytest.mark.parametrize("tmpl,shape", [(W.GEMM, (4, 4, 4)), (GEMM_VT, (8, 4, 16)), (W.CONV2D, (1, 2, 4, 4, 2, 3, 3, 1, 1)),
                                        (CONV_VT, (1, 2, 6, 6, 2, 1, 1, 0, 2)), (CONV_VT, W.conv_shape("C2"))])
def test_onehot_rows_are_full_rows_with_the_annotation_spread(tmpl, shape):
    sp = oracle.Space(tmpl, shape)
    n = min(sp.n_configs, 2000)
    cfgs = np.arange(n, dtype=np.uint64) if sp.n_configs <= 2000 else W.make_configs(n, sp.n_configs, 5)
    full = sp.features_full(cfgs).reshape(n, sp.n_loops, 13)
    oh = sp.features_onehot(cfgs).reshape(n, sp.n_loops, 3 + KINDS + 9)
    assert sp.n_features_onehot == sp.n_loops * 24
    assert (oh[:, :, 0] == full[:, :, 0]).all()
    hot = oh[:, :, 1:1 + KINDS]
    assert ((hot == 0) | (hot == 1)).all() and (hot.sum(axis=2) == 1).all()
    assert (hot.argmax(axis=2) == full[:, :, 1]).all()
    assert (oh[:, :, 1 + KINDS:] == full[:, :, 2:]).all()


def test_annealing_on_an_annotated_space_moves_every_knob_uniformly():
    sp = oracle.Space(CONV_VT, (1, 2, 6, 6, 4, 3, 3, 1, 1))
    ens = W.make_ensemble(20, 5, sp.n_features, 4)
    n, steps = 48, 150
    ch = oracle.Chains([sp], [0, n], seed=3, chain0=0, topk=4)
    tr = ch.run(ens, steps, np.full((n, steps), -np.inf, np.float32), trace=True)
    counts = np.zeros(sp.n_knobs)
    mutable = [j for j, k in enumerate(sp.knob_sizes) if k >= 2]
    for c in range(n):
        first = oracle.Chains([sp], [0, 1], seed=3, chain0=c, topk=1)
        first.run(ens, 0, np.zeros((1, 0), np.float32))
        prev = sp.decode(int(first.cur_cfgs()[0]))
        for s in range(steps):
            v = sp.decode(int(tr["cfg"][c, s]))
            d = np.nonzero(v != prev)[0]
            assert len(d) == 1
            counts[d[0]] += 1
            prev = v
    exp = n * steps / len(mutable)
    chi2 = ((counts[mutable] - exp) ** 2 / exp).sum()
    dof = len(mutable) - 1
    assert chi2 < dof + 6 * np.sqrt(2 * dof)
    assert counts[-1] > 0 and counts[-2] > 0


def test_best_by_score_matches_exhaustive_search_on_annotated_gemm():
    sp = oracle.Space(GEMM_VT, (4, 4, 4))
    ens = W.make_ensemble(40, 6, sp.n_features, 77)
    allc = np.arange(sp.n_configs, dtype=np.uint64)
    sc = oracle.predict(*ens, sp.features(allc))
    order = sorted(range(sp.n_configs), key=lambda i: (-float(sc[i]), i))
    n, steps, k = 64, 600, 8
    ch = oracle.Chains([sp], [0, n], seed=2002, chain0=0, topk=k)
    ch.run(ens, steps, oracle.thresholds(2002, 0, n, 0, steps))
    pool = {}
    for c in range(n):
        for e in ch.top[c]:
            if e["valid"]:
                pool[int(e["cfg"])] = np.float32(e["score"])
    pooled = sorted(pool.items(), key=lambda kv: (-float(kv[1]), kv[0]))[:k]
    assert [c for c, _ in pooled] == order[:k]
