"""Feature tiles of the tree-partitioned path.

The tree kernel's LDS tiles hold only the loop-context features that vary
over the space (or space set); a tree node that tests a feature constant over
it has a known outcome and is settled when the trees are relocated.  These
tests count the varying features by brute force with the oracle (every
configuration of each space), check that the tile size the run reports
matches that count, and compare the runs with the oracle bit for bit, so a
node settled the wrong way, a feature left out of the tile or a wrong tile
position shows up as a different trajectory.  The set case holds features
that are constant within each member but differ between them: those stay in
the tile.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from test_gpu_parity import DEV, P, assert_same_run, export, gpu_sa, mk_chains, say  # noqa: F401

pytestmark = pytest.mark.gpu
CONV_VT, GEMM_VT = 3, 2


def feature_range(spaces):
    """Per loop-context feature: (lowest, highest) over every configuration
    of every space."""
    lo = hi = None
    for osp in spaces:
        f = osp.features(np.arange(osp.n_configs, dtype=np.uint64))
        a, b = f.min(axis=0), f.max(axis=0)
        lo = a if lo is None else np.minimum(lo, a)
        hi = b if hi is None else np.maximum(hi, b)
    return lo, hi


def slot_bytes(quads):
    s = 256
    while s < quads * 256:
        s *= 2
    return s


def expected_tile_quads(spaces):
    """The varying features only when that makes the tile's slot (a power of
    two) smaller, else every feature."""
    lo, hi = feature_range(spaces)
    n_var = int((lo != hi).sum())
    full = (len(lo) + 3) // 4
    compact = max(1, (n_var + 3) // 4)
    return compact if slot_bytes(compact) < slot_bytes(full) else full, n_var


CASES = {
    "conv": [(W.CONV2D, (1, 2, 6, 6, 2, 3, 3, 1, 1))],
    # 125 varying features: a 32-quad tile fills its 8 KB slot, with eight
    # waves a workgroup (the counter then goes after the trees)
    "conv_full_slot": [(W.CONV2D, (1, 2, 6, 6, 2, 3, 3, 1, 1))],
    "conv_1x1_s2": [(W.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2))],
    "conv_7x7_s2": [(W.CONV2D, (1, 1, 8, 8, 2, 7, 7, 3, 2))],
    # 74 of 110 features vary: 19 quads take the same 8 KB slot as 28, so
    # the tile keeps every feature
    "gemm": [(W.GEMM, (4, 4, 4))],
    "gemm_annotated": [(GEMM_VT, (4, 4, 4))],
    "conv_annotated": [(CONV_VT, (1, 2, 6, 6, 2, 1, 1, 0, 2))],
    # a set whose members fix some features at different values (128 vary
    # over the set: 32 quads)
    "set": [(W.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2)), (W.CONV2D, (1, 2, 4, 4, 2, 1, 1, 0, 1))],
    # 145 vary over this set: 37 quads, a 16 KB slot as for all 44
    "set_wide": [(W.CONV2D, (1, 2, 6, 6, 2, 1, 1, 0, 2)), (W.CONV2D, (1, 2, 6, 6, 2, 3, 3, 1, 1))],
    # degenerate spaces: six configurations (only the unroll knobs move),
    # 10 features vary, 3 quads in a 1 KB slot; twelve configurations, 29
    # vary, 8 quads in a 2 KB slot
    "tiny_six": [(W.CONV2D, (1, 1, 1, 1, 1, 1, 1, 0, 1))],
    "tiny_twelve": [(W.CONV2D, (1, 2, 1, 1, 1, 1, 1, 0, 1))],
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_tile_holds_the_varying_features_and_runs_match_oracle(P, case):
    members = CASES[case]
    say(f"feature tiles {case}")
    ospaces = [oracle.Space(t, s) for t, s in members]
    want_q, n_var = expected_tile_quads(ospaces)
    n_feat = ospaces[0].n_features
    assert n_var < n_feat          # every case has constant features
    spaces = [P.at_space_create(t, s) for t, s in members]
    n_per, trees, steps = (1024, 1000, 8) if case == "conv_full_slot" else (96, 120, 40)
    off = np.arange(len(members) + 1, dtype=np.int64) * n_per
    sp = spaces[0] if len(spaces) == 1 else P.at_spaceset_create(spaces, off)
    fid, thr, leaf = W.make_ensemble(trees, 7, n_feat, 61)
    ens = P.at_ensemble_create(fid, thr, leaf, n_feat)
    n, seed, k = int(off[-1]), 17, 5
    ch = mk_chains(P, sp, 0, n, k, seed, "trees")
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    say(f"  {n_var} of {n_feat} features vary: plan {plan}")
    assert plan["path"] == P.AT_SA_PATH_TREES and plan["tile_quads"] == want_q
    if case == "conv_full_slot":
        assert want_q == 32 and plan["waves"] >= 2
    och = oracle.Chains(ospaces, off, seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_set_keeps_features_fixed_at_different_values_per_member():
    # the set case is only meaningful if such features exist, and if its
    # tile is the compact one
    a, b = [oracle.Space(t, s) for t, s in CASES["set"]]
    (lo_a, hi_a), (lo_b, hi_b) = feature_range([a]), feature_range([b])
    fixed_apart = (lo_a == hi_a) & (lo_b == hi_b) & (lo_a != lo_b)
    assert fixed_apart.sum() > 0
    q_set, n_set = expected_tile_quads([a, b])
    assert n_set == int(((lo_a != hi_a) | (lo_b != hi_b) | fixed_apart).sum())
    assert q_set == 32 < (a.n_features + 3) // 4


def test_c12_tile_and_plan(P):
    # the C12 search's space: 124 of its 176 loop-context features vary
    # (exhaustive count over its 844,800 configurations), so a tile takes 31
    # quads and twelve waves' tiles fit beside eight trees of depth 10
    wl = W.WORKLOADS["conv_c12_sa"]
    t, s = wl["spaces"][0]
    sp = P.at_space_create(t, s)
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, steps, seed, k = 8192, 2, wl["sa_seed"], wl["topk"]
    ch = P.at_chains_create(sp, 0, n, k, seed)
    gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps), traced=False)
    plan = P.at_chains_last_plan(ch)
    say(f"C12 plan {plan}")
    assert plan["path"] == P.AT_SA_PATH_TREES
    assert plan["tile_quads"] == 31 and plan["trees_per_wg"] == 8 and plan["waves"] == 12


def test_space_past_the_scan_limit_keeps_whole_tiles(P):
    # the annotated C2 space holds 361,267,200 configurations, more than the
    # 2^28 a space creation scans: its tiles keep all 44 quads
    shape = W.conv_shape("C2")
    osp = oracle.Space(CONV_VT, shape)
    assert osp.n_configs > 1 << 28
    sp = P.at_space_create(CONV_VT, shape)
    fid, thr, leaf = W.make_ensemble(60, 6, 176, 62)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, steps, seed, k = 128, 12, 23, 4
    ch = mk_chains(P, sp, 0, n, k, seed, "trees")
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    assert plan["path"] == P.AT_SA_PATH_TREES and plan["tile_quads"] == 44
    och = oracle.Chains([osp], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_set_with_an_unscanned_member_keeps_whole_tiles(P):
    # one member past the scan limit: nothing is known constant over the
    # set, so its tiles keep all 44 quads; chains on both members compared
    members = [(CONV_VT, (1, 2, 6, 6, 2, 1, 1, 0, 2)), (CONV_VT, W.conv_shape("C2"))]
    ospaces = [oracle.Space(t, s) for t, s in members]
    assert ospaces[1].n_configs > 1 << 28
    spaces = [P.at_space_create(t, s) for t, s in members]
    off = np.array([0, 64, 128], np.int64)
    sset = P.at_spaceset_create(spaces, off)
    fid, thr, leaf = W.make_ensemble(60, 6, 176, 63)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, steps, seed, k = 128, 12, 29, 4
    ch = mk_chains(P, sset, 0, n, k, seed, "trees")
    best, tr = gpu_sa(P, sset, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    assert plan["path"] == P.AT_SA_PATH_TREES and plan["tile_quads"] == 44
    och = oracle.Chains(ospaces, off, seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))
