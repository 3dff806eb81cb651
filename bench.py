"""Benchmark of the annealing hot path on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-extra] [--no-cpu]

A step is one at_sa_run over the whole workload: every chain anneals for the
workload's step count; each annealing step proposes, featurises, scores,
offers and accepts.  The headline workload is the largest single-GPU search,
C12 (8192 chains x 1000 steps, 2000 trees of depth 10); the other workloads
are reported under "extra".  One chains handle serves every run of a
workload: the warm-up runs initialise its chains and take its one-time
workspace allocation, and each timed run continues the chains for the
workload's step count with thresholds computed beforehand for its steps.
Inputs (ensemble tables, thresholds) are resident on the GPU before the
timed region, which holds kernel launches only.

Prints one JSON line.  Run times come from HIP events on the stream the
kernels run on.  The roofline object is for the dominant kernel, the tree
walk: one further run of each workload attaches start/stop events to every
kernel launch (at_sa_set_profiling), and the roofline divides the walk's
algorithmic LDS bytes per launch, (2d+1) x 4 bytes per tree evaluation
times chains times trees, by its average launch duration; "whole_run" does
the same for the whole run.  Fractions are given against 128 bytes per clock
per compute unit (4-byte accesses) and against the 202 measured for 16-byte
reads.  Its HBM traffic comes from the committed rocprofv3 counter summary
while the kernel source it was taken from is unchanged (null otherwise).  A
256 MiB device copy runs once before the timed region; its FETCH_SIZE /
WRITE_SIZE readings scale the counters.

The CPU baseline is the oracle on the first chains of the workload, on one
core and as P single-threaded processes at once (P = the host cores this
process may use, at most 16), run before the GPU is touched.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

METRIC = "SA candidate evals/sec (features+GBT+accept); GBT scores/sec, 1M cfg×1000 trees"

# MI355X: 256 CUs at 2.4 GHz; LDS serves 128 bytes per clock per CU.
N_CU, CLOCK_HZ = 256, 2.4e9
LDS_PEAK_BPS = 128 * N_CU * CLOCK_HZ          # 78.6 TB/s (4-byte accesses)
# ds_read_b128 measured 202 bytes per clock per CU on gfx950: the denominator
# for wide reads (every fraction against it is about 0.63 of the other)
LDS_B128_BPS = 202 * N_CU * CLOCK_HZ          # 124 TB/s
# the largest single-GPU annealing workload: the C12 search
HEADLINE = "conv_c12_sa"
HBM_PEAK_BPS = 8.0e12


def tree_eval_bytes(depth: int) -> int:
    """Algorithmic LDS bytes of one tree evaluation: depth node reads, depth
    feature reads and one leaf read, 4 bytes each."""
    return (2 * depth + 1) * 4


KERNEL_SOURCES = {"k_trees": os.path.join(ROOT, "paper_1805_08166_amd", "csrc", "at_sa_tp.hip"),
                  "k_local": os.path.join(ROOT, "paper_1805_08166_amd", "csrc", "at_sa_local.hip")}
COPY_BYTES = 256 << 20


def calibration_copy():
    """One device-to-device copy of known size (for scaling HBM counters)."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()


def committed_traffic(kernel: str, workload: str):
    """HBM bytes per launch of the walk kernel from the committed counter
    summary, or None when there is none or the kernel source has changed
    since."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    sha = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not val:
        return None
    cur = hashlib.sha256(open(KERNEL_SOURCES[kernel], "rb").read()).hexdigest()
    return float(val.group(1)) if sha.group(1) == cur else None


def describe(name: str) -> str:
    wl = W.WORKLOADS[name]
    if wl["kind"] == "score":
        return (f"{name}: {wl['n_cfgs']} random configs of conv2d C2, features + {wl['trees']} trees "
                f"depth {wl['depth']}")
    sp = wl["spaces"]
    what = "GEMM 512^3" if sp[0][0] == W.GEMM else (
        "12 ResNet-18 conv2d workloads" if len(sp) > 1 else f"conv2d {sp[0][1]}")
    return (f"{name}: {what}, {wl['trees']} trees depth {wl['depth']}, "
            f"{wl['chains_per_space'] * len(sp)} chains x {wl['steps']} steps, top-{wl['topk']}")


class SaWorkload:
    """One annealing workload on one chains handle.  transfer: the energy is
    Eq. 4's global model (as many trees, of the same depth, over the 192
    relation features) plus the workload's ensemble as the local model."""

    def __init__(self, P, name, transfer=False):
        import torch
        self.P, self.name, self.transfer = P, name, transfer
        wl = self.wl = W.WORKLOADS[name]
        self.spaces = [P.at_space_create(t, s) for t, s in wl["spaces"]]
        F = self.spaces[0].n_features
        if len(self.spaces) > 1:
            off = W.chain_offsets(len(self.spaces), wl["chains_per_space"])
            self.space = P.at_spaceset_create(self.spaces, off)
        else:
            self.space = self.spaces[0]
        self.n = wl["chains_per_space"] * len(self.spaces)
        self.steps, self.topk, self.seed = wl["steps"], wl["topk"], wl["sa_seed"]
        t0 = time.perf_counter()
        self.ens_tables = W.make_ensemble(wl["trees"], wl["depth"], F, wl["ens_seed"])
        self.ens = P.at_ensemble_create(*self.ens_tables, F)
        if transfer:
            self.glob = P.at_ensemble_create(*W.make_ensemble(wl["trees"], wl["depth"], P.RELATION_FEATURES,
                                                              wl["ens_seed"] + 50), P.RELATION_FEATURES)
        self.t_pack = time.perf_counter() - t0
        self.t_thr = None
        self.best = torch.zeros((self.n, self.topk, 4), dtype=torch.int32, device="cuda")
        self.evals = self.n * self.steps
        self.tree_evals = self.evals * wl["trees"] * (2 if transfer else 1)
        self.lds_bytes = self.tree_evals * tree_eval_bytes(wl["depth"])
        self.chains = P.at_chains_create(self.space, 0, self.n, self.topk, self.seed)

    def thresholds(self, runs):
        """Device threshold tables of the next `runs` runs of the chains
        (each run continues from where the previous one stopped)."""
        import torch
        base = self.P.at_chains_step(self.chains)
        out = []
        for r in range(runs):
            t0 = time.perf_counter()
            thr = self.P.at_sa_thresholds(self.seed, 0, self.n, base + r * self.steps, self.steps)
            if self.t_thr is None:
                self.t_thr = time.perf_counter() - t0
            out.append(torch.from_numpy(thr).cuda())
        return out

    def run(self, thr):
        if self.transfer:
            self.P.at_sa_run_global_local(self.space, self.glob, self.ens, self.chains, self.steps, thr, self.best)
        else:
            self.P.at_sa_run(self.space, self.ens, self.chains, self.steps, thr, self.best)


def time_events(fn, reps):
    """Per-call durations (s) from HIP events on the current stream."""
    import torch
    out = []
    for r in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn(r)
        b.record()
        b.synchronize()
        out.append(a.elapsed_time(b) / 1e3)
    return out


def bench_sa(P, name, steps, warmup, transfer=False):
    """Annealing runs of a workload on one chains handle.  The warm-up runs
    initialise the chains and take the handle's one-time workspace
    allocation; every timed run then continues the same chains for the
    workload's step count with thresholds precomputed for its steps, so the
    timed region holds kernel launches only."""
    import torch
    w = SaWorkload(P, name, transfer)
    warmup = max(1, warmup)
    thr = w.thresholds(warmup)
    for i in range(warmup):
        w.run(thr[i])
    thr = w.thresholds(steps + 1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev = time_events(lambda r: w.run(thr[r]), steps)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    t = float(np.mean(ev))
    # one more run, profiled: average launch durations of the kernels.  The
    # walk kernel is k_local on the chain-local path (one launch per run, a
    # scoring round per step) and k_trees on the tree-partitioned path (one
    # launch per scoring round).
    P.at_sa_set_profiling(w.chains, True)
    w.run(thr[steps])
    kt = P.at_sa_kernel_times(w.chains)
    P.at_sa_set_profiling(w.chains, False)
    local = P.at_chains_last_path(w.chains) == P.AT_SA_PATH_LOCAL
    plan = P.at_chains_last_plan(w.chains)
    tree_s = kt["tree_ms"] / kt["tree_launches"] * 1e-3
    rounds_per_launch = w.steps if local else 1
    tree_bytes = w.n * w.wl["trees"] * rounds_per_launch * tree_eval_bytes(w.wl["depth"])
    if transfer:
        name += " (Eq. 4: global model on the relation features + local model on the loop features, "
        name += f"{w.wl['trees']} trees depth {w.wl['depth']} each; two tree launches per step)"
    return w, dict(
        path="chain-local" if local else "tree-partitioned", plan=plan,
        walk_kernel="k_local" if local else "k_trees",
        workload=describe(name.split(" ")[0]) + name[len(name.split(" ")[0]):], ms_per_run=t * 1e3, ms_min=float(np.min(ev)) * 1e3, wall_s=wall,
        evals_per_s=w.evals / t, tree_evals_per_s=w.tree_evals / t,
        run_lds_bytes=w.lds_bytes, run_lds_TBps=w.lds_bytes / t / 1e12,
        run_lds_frac=w.lds_bytes / t / LDS_PEAK_BPS, run_lds_frac_b128=w.lds_bytes / t / LDS_B128_BPS,
        host_threshold_s=w.t_thr, host_ensemble_pack_s=w.t_pack,
        tree_kernel_us=tree_s * 1e6, tree_kernel_launches=kt["tree_launches"],
        chain_kernel_us=(kt["chain_ms"] / kt["chain_launches"] * 1e3) if kt["chain_launches"] else None,
        tree_lds_bytes_per_launch=tree_bytes, tree_lds_TBps=tree_bytes / tree_s / 1e12,
        tree_lds_frac=tree_bytes / tree_s / LDS_PEAK_BPS, tree_lds_frac_b128=tree_bytes / tree_s / LDS_B128_BPS)


def bench_score(P, reps, warmup):
    import torch
    name = "conv_c2_score1m"
    wl = W.WORKLOADS[name]
    tmpl, shape = wl["spaces"][0]
    sp = P.at_space_create(tmpl, shape)
    ens = P.at_ensemble_create(*W.make_ensemble(wl["trees"], wl["depth"], 176, wl["ens_seed"]), 176)
    n = wl["n_cfgs"]
    cfgs = torch.from_numpy(W.make_configs(n, sp.n_configs, wl["cfg_seed"]).view(np.int64)).cuda()
    feats = torch.empty((n, 176), dtype=torch.int32, device="cuda")
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    for _ in range(warmup):
        P.at_extract_features(sp, cfgs, feats)
        P.at_gbt_predict(ens, feats, scores)
    torch.cuda.synchronize()
    te = time_events(lambda r: P.at_extract_features(sp, cfgs, feats), reps)
    tp = time_events(lambda r: P.at_gbt_predict(ens, feats, scores), reps)
    te, tp = float(np.mean(te)), float(np.mean(tp))
    # context relation features of the same configurations (192 int32 a row)
    rel = torch.empty((n, P.RELATION_FEATURES), dtype=torch.int32, device="cuda")
    P.at_extract_relation_features(sp, cfgs, rel)
    tr = float(np.mean(time_events(lambda r: P.at_extract_relation_features(sp, cfgs, rel), reps)))
    rel_bytes = n * (8 + P.RELATION_FEATURES * 4)
    # Eq. 4: a 1000-tree global model on the relation features plus the
    # workload's local model on the loop features
    glob = P.at_ensemble_create(*W.make_ensemble(wl["trees"], wl["depth"], P.RELATION_FEATURES, wl["ens_seed"] + 50),
                                P.RELATION_FEATURES)
    tg = float(np.mean(time_events(lambda r: P.at_gbt_predict_global_local(glob, rel, ens, feats, scores), reps)))
    del rel
    # full Appendix A.2 rows (208 int32: top-down and bottom-up added)
    full = torch.empty((n, 13 * sp.n_loops), dtype=torch.int32, device="cuda")
    P.at_extract_features_full(sp, cfgs, full)
    tf = float(np.mean(time_events(lambda r: P.at_extract_features_full(sp, cfgs, full), reps)))
    full_bytes = n * (8 + 13 * sp.n_loops * 4)
    del full
    feat_bytes = n * (8 + 176 * 4)              # cfg in, feature row out
    score_lds = n * wl["trees"] * tree_eval_bytes(wl["depth"])
    return dict(
        workload=describe(name),
        extract_ms=te * 1e3, features_per_s=n / te, extract_hbm_GBps=feat_bytes / te / 1e9,
        extract_hbm_frac=feat_bytes / te / HBM_PEAK_BPS,
        predict_ms=tp * 1e3, scores_per_s=n / tp, tree_evals_per_s=n * wl["trees"] / tp,
        predict_lds_TBps=score_lds / tp / 1e12, predict_lds_frac=score_lds / tp / LDS_PEAK_BPS,
        predict_hbm_GBps=n * (176 * 4 + 4) / tp / 1e9,
        relation_ms=tr * 1e3, relation_rows_per_s=n / tr, relation_hbm_GBps=rel_bytes / tr / 1e9,
        relation_hbm_frac=rel_bytes / tr / HBM_PEAK_BPS,
        full_extract_ms=tf * 1e3, full_rows_per_s=n / tf, full_extract_hbm_GBps=full_bytes / tf / 1e9,
        full_extract_hbm_frac=full_bytes / tf / HBM_PEAK_BPS,
        global_local_ms=tg * 1e3, global_local_scores_per_s=n / tg,
        global_local_lds_frac=2 * score_lds / tg / LDS_PEAK_BPS)


def bench_select(P, w, reps=20):
    """Batch selection after an annealing run (Algorithm 1, Eq. 3) on the
    run's best lists: the paper's batch b = 64 with epsilon = 0.05 (61
    greedy picks, 3 random) from the top 2b = 128, alpha = 1."""
    import torch
    sp = w.spaces[0]
    out = torch.zeros((64, 4), dtype=torch.int32, device="cuda")
    fn = lambda r: P.at_select_batch(sp, w.best, 128, 61, 1.0, 3, 4000 + r, out)
    fn_na = lambda r: P.at_select_batch_noalloc(sp, w.best, 128, 61, 1.0, 3, 4000 + r, out)
    for r in range(2):
        fn(r)
        fn_na(r)
    torch.cuda.synchronize()
    t = float(np.median(time_events(fn, reps)))
    t_na = float(np.median(time_events(fn_na, reps)))
    n_cand = w.best.numel() // 4
    return dict(workload=f"{w.name}: best lists {w.n} x {w.topk}, pool 128, 61 greedy + 3 random, alpha 1",
                candidates=n_cand, ms=t * 1e3, ms_noalloc=t_na * 1e3, candidates_per_s=n_cand / t,
                read_GBps=n_cand * 16 / t / 1e9)


def oracle_sa_sample(name, chain0, n_chains):
    """The oracle on chains [chain0, chain0 + n_chains) of a single-space
    annealing workload, all of its steps; returns (evals, seconds)."""
    import oracle
    wl = W.WORKLOADS[name]
    spaces = [oracle.Space(t, s) for t, s in wl["spaces"][:1]]
    ens = W.make_ensemble(wl["trees"], wl["depth"], spaces[0].n_features, wl["ens_seed"])
    steps, seed, k = wl["steps"], wl["sa_seed"], wl["topk"]
    ch = oracle.Chains(spaces, [0, n_chains], seed=seed, chain0=chain0, topk=k)
    thr = oracle.thresholds(seed, chain0, n_chains, 0, steps)
    t0 = time.perf_counter()
    ch.run(ens, steps, thr)
    return n_chains * steps, time.perf_counter() - t0


def host_cores() -> int:
    """Host cores this process may use, capped at the one-GPU share of 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_baseline(name, chains):
    """The single-threaded oracle on a bounded sample of the workload: the
    first `chains` chains, all steps, on one core; then P = host_cores()
    single-threaded oracle processes at once, shard p taking chains
    [p * chains, (p + 1) * chains), for the all-cores rate (total evals over
    the slowest shard's time).  Runs before the GPU is touched."""
    import subprocess
    evals, t1 = oracle_sa_sample(name, 0, chains)
    P = host_cores()
    procs = [subprocess.Popen([sys.executable, os.path.abspath(__file__), "--oracle-shard", name, str(p * chains),
                               str(chains)], stdout=subprocess.PIPE, text=True) for p in range(P)]
    outs = [json.loads(p.communicate()[0].strip().splitlines()[-1]) for p in procs]
    if any(p.returncode != 0 for p in procs):
        raise RuntimeError("an oracle shard failed")
    total = sum(o["evals"] for o in outs)
    slowest = max(o["s"] for o in outs)
    steps = W.WORKLOADS[name]["steps"]
    return dict(value=total / slowest, unit="evals/s", cores=P, kind="oracle",
                sample=(f"{P} single-threaded oracle processes at once, each {chains} chains x {steps} steps of "
                        f"{name} (chains 0..{P * chains - 1}, {total} evals, slowest {slowest:.1f} s)"),
                one_core=dict(value=evals / t1, unit="evals/s", cores=1,
                              sample=f"first {chains} chains x {steps} steps of {name} ({evals} evals, {t1:.1f} s)"))


def oracle_shard_main(argv):
    """Child process of the all-cores CPU baseline: one oracle shard."""
    name, chain0, n = argv[0], int(argv[1]), int(argv[2])
    evals, secs = oracle_sa_sample(name, chain0, n)
    print(json.dumps({"evals": evals, "s": secs}), flush=True)


def main():
    if len(sys.argv) > 1 and sys.argv[1] == "--oracle-shard":
        oracle_shard_main(sys.argv[2:])
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--no-extra", action="store_true")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--cpu-chains", type=int, default=64,
                    help="chains per oracle sample (the C12 workload: 64 chains x 1000 steps, about 9 s a core)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU; --gpus {args.gpus} is not supported "
              "(chains are keyed by global chain id, so N GPUs would each run a contiguous block of chains "
              "and give the same results as one GPU)", file=sys.stderr)
        sys.exit(2)
    # the oracle baseline runs first, in this process and in child processes,
    # before anything touches the GPU
    cpu = None if args.no_cpu else cpu_baseline(args.workload, args.cpu_chains)

    import torch
    import paper_1805_08166_amd as P
    torch.cuda.set_device(0)

    calibration_copy()
    head, r = bench_sa(P, args.workload, args.steps, args.warmup)
    extra = {}
    if not args.no_extra:
        extra["select_" + args.workload] = bench_select(P, head)
        extra["conv_c2_score1m"] = bench_score(P, reps=5, warmup=1)
        for name in ["conv_c2_sa", "gemm512_sa", "conv_c12_sa", "resnet18_12conv_sa"]:
            if name == args.workload:
                continue
            reps = 2 if name == "conv_c12_sa" else 3
            w, extra[name] = bench_sa(P, name, reps, 1)
            if name in ("conv_c2_sa", "conv_c12_sa"):
                extra["select_" + name] = bench_select(P, w)
        _, extra["transfer_resnet18_12conv_sa"] = bench_sa(P, "resnet18_12conv_sa", 3, 1, transfer=True)
    depth = head.wl["depth"]
    line = {
        "metric": METRIC,
        "value": r["evals_per_s"],
        "unit": "evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_run"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32+f32",
        "data": "synthetic (seeded ensemble and configurations; Table 1 shapes)",
        "config": {"workload": r["workload"], "evals_per_step": head.evals,
                   "tree_evals_per_step": head.tree_evals, "path": r["path"], "plan": r["plan"]},
        "roofline": {"bound": "lds",
                     "kernel": (f"{r['walk_kernel']} ({r['path']} path: "
                                + ("one launch runs every step" if r["path"] == "chain-local"
                                   else "tree walk of one annealing step") + ")"),
                     "achieved": r["tree_lds_TBps"] * 1e3, "peak": LDS_PEAK_BPS / 1e9, "unit": "GB/s",
                     "frac": r["tree_lds_frac"], "traffic": committed_traffic(r["walk_kernel"], args.workload),
                     "launch_us": r["tree_kernel_us"],
                     "per_unit": f"{tree_eval_bytes(depth)} B LDS per tree evaluation, "
                                 f"{head.n} chains x {head.wl['trees']} trees x "
                                 f"{head.steps if r['path'] == 'chain-local' else 1} rounds per launch",
                     "peak_b128": LDS_B128_BPS / 1e9, "frac_b128": r["tree_lds_frac_b128"],
                     "whole_run": {"achieved": r["run_lds_TBps"] * 1e3, "frac": r["run_lds_frac"],
                                   "frac_b128": r["run_lds_frac_b128"],
                                   "per_unit": f"{tree_eval_bytes(depth)} B LDS per tree evaluation, "
                                               f"{head.n} chains x {head.steps} steps x {head.wl['trees']} trees "
                                               "per run"}},
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
