"""GPU parity of the production launches of the tree-partitioned path.

The C12 search (2000 trees of depth 10, 8192 chains x 1000 steps) and the
twelve-workload set (1000 trees of depth 8, 6144 chains x 500 steps) are run
exactly as the bench runs them: default path, full chain count, full step
count.  The oracle recomputes slices of chains (a chain's trajectory depends
only on its global id, Section 3.3), so every slice of the GPU run must equal
an oracle run over those chains alone.

The launch plan is read back to check what these runs exercise: a wave that
walks more than one 64-chain block (the block claiming and tile refill of the
tree kernel), and sixteen trees per workgroup (two groups of eight).  Smaller
cases force the same plans with every chain compared.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from test_gpu_parity import DEV, P, assert_same_run, export, gpu_sa, mk_chains, say  # noqa: F401

pytestmark = pytest.mark.gpu


def oracle_slice(wl_spaces, offsets, ens_t, seed, topk, steps, lo, hi, global_model=None):
    """Oracle run of global chains [lo, hi) of a (possibly ragged) space set
    (with global_model: the Eq. 4 energy, global model first)."""
    offsets = np.asarray(offsets, np.int64)
    sp_lo = int(np.searchsorted(offsets, lo, side="right") - 1)
    sp_hi = int(np.searchsorted(offsets, hi - 1, side="right") - 1)
    spaces = [oracle.Space(t, s) for t, s in wl_spaces[sp_lo:sp_hi + 1]]
    off = [0] + [int(offsets[w + 1]) - lo for w in range(sp_lo, sp_hi)] + [hi - lo]
    och = oracle.Chains(spaces, off, seed=seed, chain0=lo, topk=topk)
    otr = och.run(ens_t, steps, oracle.thresholds(seed, lo, hi - lo, 0, steps), trace=True,
                  global_model=global_model)
    return och, otr


def run_workload(P, name, n_per_space, steps):
    wl = W.WORKLOADS[name]
    spaces = [P.at_space_create(t, s) for t, s in wl["spaces"]]
    off = W.chain_offsets(len(spaces), n_per_space)
    sp = spaces[0] if len(spaces) == 1 else P.at_spaceset_create(spaces, off)
    fid, thr, leaf = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, seed, k = int(off[-1]), wl["sa_seed"], wl["topk"]
    ch = P.at_chains_create(sp, 0, n, k, seed)
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    say(f"{name} {n} chains x {steps} steps: plan {plan}")
    return wl, off, (fid, thr, leaf), ch, best, tr, plan


def check_slices(P, wl, off, ens_t, ch, best, tr, steps, slices, global_model=None):
    cur = export(P, ch)
    for lo, hi in slices:
        say(f"oracle slice [{lo}, {hi})")
        och, otr = oracle_slice(wl["spaces"], off, ens_t, wl["sa_seed"], wl["topk"], steps, lo, hi, global_model)
        assert_same_run(best, tr, och, otr, rows=slice(lo, hi), cur=cur)


def test_c12_production_launch_sliced_oracle(P):
    # the bench's C12 search: default path, 8192 chains x 1000 steps
    wl, off, ens_t, ch, best, tr, plan = run_workload(P, "conv_c12_sa", 8192, 1000)
    assert plan["path"] == P.AT_SA_PATH_TREES
    # a wave walks several blocks: the claimed blocks refill its tile
    assert plan["slice_blocks"] > plan["waves"]
    check_slices(P, wl, off, ens_t, ch, best, tr, 1000, [(0, 32), (4096, 4128), (8160, 8192)])


def test_twelve_conv_production_launch_sliced_oracle(P):
    # the bench's twelve-workload set: default path, 12 x 512 chains x 500 steps
    wl, off, ens_t, ch, best, tr, plan = run_workload(P, "resnet18_12conv_sa", 512, 500)
    assert plan["path"] == P.AT_SA_PATH_TREES
    assert plan["trees_per_wg"] == 16 and plan["slice_blocks"] > plan["waves"]
    # eight chains around every space boundary, the first and the last chains
    slices = [(0, 4)] + [(int(b) - 4, int(b) + 4) for b in off[1:-1]] + [(int(off[-1]) - 4, int(off[-1]))]
    check_slices(P, wl, off, ens_t, ch, best, tr, 500, slices)


def test_c12_ensemble_block_claiming_every_chain(P):
    # 1024 chains: 16 blocks per slice against fewer waves, so every wave
    # claims and refills; every chain compared for a few steps
    wl, off, ens_t, ch, best, tr, plan = run_workload(P, "conv_c12_sa", 1024, 4)
    assert plan["path"] == P.AT_SA_PATH_TREES and plan["slice_blocks"] > plan["waves"]
    check_slices(P, wl, off, ens_t, ch, best, tr, 4, [(0, 1024)])


def test_one_group_form_with_ragged_trees_and_chains(P):
    # eight trees a workgroup, the form in which a block's leaf values are
    # stored after the next block's fill is issued: 2005 trees leave a last
    # workgroup of five (its values go out at once), 1000 chains a last
    # block of 40 active lanes, and 16 blocks against the waves make every
    # wave carry values over from one block to the next
    t, s = W.WORKLOADS["conv_c12_sa"]["spaces"][0]
    sp = P.at_space_create(t, s)
    fid, thr, leaf = W.make_ensemble(2005, 10, 176, 71)
    ens = P.at_ensemble_create(fid, thr, leaf, 176)
    n, steps, seed, k = 1000, 4, 31, 8
    ch = mk_chains(P, sp, 0, n, k, seed, "trees")
    best, tr = gpu_sa(P, sp, ens, ch, steps, P.at_sa_thresholds(seed, 0, n, 0, steps))
    plan = P.at_chains_last_plan(ch)
    say(f"2005 trees, {n} chains: plan {plan}")
    assert plan["path"] == P.AT_SA_PATH_TREES and plan["trees_per_wg"] == 8
    assert plan["slice_blocks"] > plan["waves"]
    och = oracle.Chains([oracle.Space(t, s)], [0, n], seed=seed, chain0=0, topk=k)
    otr = och.run((fid, thr, leaf), steps, oracle.thresholds(seed, 0, n, 0, steps), trace=True)
    assert_same_run(best, tr, och, otr, cur=export(P, ch))


def test_twelve_conv_sixteen_trees_every_chain(P):
    # the production plan of the twelve-workload set (sixteen trees per
    # workgroup, claimed blocks) with every chain compared for a few steps
    wl, off, ens_t, ch, best, tr, plan = run_workload(P, "resnet18_12conv_sa", 512, 3)
    assert plan["path"] == P.AT_SA_PATH_TREES and plan["trees_per_wg"] == 16
    assert plan["slice_blocks"] > plan["waves"]
    check_slices(P, wl, off, ens_t, ch, best, tr, 3, [(0, int(off[-1]))])


def test_twelve_conv_transfer_production_launch_sliced_oracle(P):
    # the bench's Eq. 4 leg: the twelve-workload set, 12 x 512 chains x 500
    # steps, a 1000-tree global model over the relation features beside the
    # 1000-tree local model (two tree launches a step, the two folds
    # interleaved in the chain kernel)
    import torch
    wl = W.WORKLOADS["resnet18_12conv_sa"]
    spaces = [P.at_space_create(t, s) for t, s in wl["spaces"]]
    off = W.chain_offsets(12, 512)
    sset = P.at_spaceset_create(spaces, off)
    loc = W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"])
    glob = W.make_ensemble(wl["trees"], wl["depth"], P.RELATION_FEATURES, wl["ens_seed"] + 50)
    n, steps, seed, k = int(off[-1]), wl["steps"], wl["sa_seed"], wl["topk"]
    ch = P.at_chains_create(sset, 0, n, k, seed)
    thr = torch.from_numpy(P.at_sa_thresholds(seed, 0, n, 0, steps)).to(DEV)
    best = torch.zeros((n, k, 4), dtype=torch.int32, device=DEV)
    trace = torch.zeros((n, steps, 4), dtype=torch.int32, device=DEV)
    P.at_sa_run_global_local(sset, P.at_ensemble_create(*glob, P.RELATION_FEATURES), P.at_ensemble_create(*loc, 176),
                             ch, steps, thr, best, trace)
    torch.cuda.synchronize()
    plan = P.at_chains_last_plan(ch)
    say(f"transfer {n} chains x {steps} steps: plan {plan}")
    assert plan["path"] == P.AT_SA_PATH_TREES
    slices = [(0, 4)] + [(int(b) - 2, int(b) + 2) for b in off[1:-1:3]] + [(n - 4, n)]
    check_slices(P, wl, off, loc, ch, P.entries(best), P.entries(trace), steps, slices, global_model=glob)
