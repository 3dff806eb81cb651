"""Seeded synthetic inputs shared by the tests, the bench and the smoke check.

This module holds the workload recipes (template shapes, ensemble sizes, chain
counts) and the seeded generators of the *inputs* the method consumes: the
tree-ensemble arrays and the uniformly random configuration indices of the
batched-scoring workload.  It performs none of the method's arithmetic: no
knob decoding, no loop features, no tree traversal, no annealing.  Neither the
HIP library nor the CPU oracle imports it; callers pass its arrays to both.

Shapes follow the paper: the GEMM expression of Section 2 and the twelve
ResNet-18 conv2d operators of Table 1.  The trained XGBoost models of the
paper are not available, so a synthetic ensemble of full-depth trees stands in
for them: split feature uniform over [0, F), integer threshold uniform over
[0, 33), leaf value float32(N(0,1) * 0.05).
"""
from __future__ import annotations

import numpy as np

GEMM = 0
CONV2D = 1

# Table 1: (H/W, IC, OC, kernel, stride) of the conv2d operators of ResNet-18.
TABLE1 = {
    "C1": (224, 3, 64, 7, 2),
    "C2": (56, 64, 64, 3, 1),
    "C3": (56, 64, 64, 1, 1),
    "C4": (56, 64, 128, 3, 2),
    "C5": (56, 64, 128, 1, 2),
    "C6": (28, 128, 128, 3, 1),
    "C7": (28, 128, 256, 3, 2),
    "C8": (28, 128, 256, 1, 2),
    "C9": (14, 256, 256, 3, 1),
    "C10": (14, 256, 512, 3, 2),
    "C11": (14, 256, 512, 1, 2),
    "C12": (7, 512, 512, 3, 1),
}


def conv_shape(name: str) -> tuple:
    """Conv shape tuple (N, C, H, W, K, KH, KW, pad, stride) for a Table 1 row.

    Padding is (kernel-1)/2 (same padding), the reading that yields the output
    sizes 112/56/28/14/7 of the ResNet-18 stages.
    """
    hw, ic, oc, k, s = TABLE1[name]
    return (1, ic, hw, hw, oc, k, k, (k - 1) // 2, s)


GEMM_512 = (512, 512, 512)

# The five synthetic workloads.  "sa" workloads run annealing chains; "score"
# scores a batch of random configurations.  Seeds: ensemble 1000+i,
# annealing 2000+i, random configurations 3000+i.
WORKLOADS = {
    "gemm512_sa": dict(
        index=0, kind="sa", spaces=[(GEMM, GEMM_512)], trees=100, depth=6,
        chains_per_space=64, steps=500, topk=8, ens_seed=1000, sa_seed=2000),
    "conv_c2_sa": dict(
        index=1, kind="sa", spaces=[(CONV2D, conv_shape("C2"))], trees=500,
        depth=8, chains_per_space=1024, steps=500, topk=16, ens_seed=1001,
        sa_seed=2001),
    "conv_c2_score1m": dict(
        index=2, kind="score", spaces=[(CONV2D, conv_shape("C2"))], trees=1000,
        depth=8, n_cfgs=1 << 20, ens_seed=1002, cfg_seed=3002),
    "conv_c12_sa": dict(
        index=3, kind="sa", spaces=[(CONV2D, conv_shape("C12"))], trees=2000,
        depth=10, chains_per_space=8192, steps=1000, topk=32, ens_seed=1003,
        sa_seed=2003),
    "resnet18_12conv_sa": dict(
        index=4, kind="sa",
        spaces=[(CONV2D, conv_shape(f"C{i}")) for i in range(1, 13)],
        trees=1000, depth=8, chains_per_space=512, steps=500, topk=16,
        ens_seed=1004, sa_seed=2004),
}


def n_features_of(template: int) -> int:
    """Loop-context feature count: 10 GEMM loops or 16 conv loops, 11 each."""
    return 110 if template == GEMM else 176


def make_ensemble(n_trees: int, depth: int, n_features: int, seed: int):
    """Synthetic full-depth tree ensemble, heap-ordered nodes.

    Returns (fid uint8 [T, 2^d-1], thr uint8 [T, 2^d-1], leaf float32 [T, 2^d]).
    """
    if not (1 <= depth <= 15 and 1 <= n_features <= 256 and n_trees >= 1):
        raise ValueError("unsupported ensemble size")
    rng = np.random.default_rng(seed)
    n_int = (1 << depth) - 1
    fid = rng.integers(0, n_features, size=(n_trees, n_int), dtype=np.int64)
    thr = rng.integers(0, 33, size=(n_trees, n_int), dtype=np.int64)
    leaf = (rng.standard_normal(size=(n_trees, 1 << depth)) * 0.05).astype(np.float32)
    return fid.astype(np.uint8), thr.astype(np.uint8), leaf


def make_node_trees(n_trees: int, max_depth: int, n_features: int, seed: int, p_leaf: float = 0.25,
                    shuffle: bool = True) -> dict:
    """Synthetic trees of varying shape in node-list form, as a trained
    gradient-boosting library writes them: tree t owns nodes offsets[t] ..
    offsets[t+1]-1, its root first, children indexed from the tree's first
    node; left < 0 marks a leaf.  A node below the root becomes a leaf with
    probability p_leaf, and every node at max_depth is one.  Split features
    are uniform over [0, n_features); thresholds are float32, mostly integers
    and half-integers in [0, 33), a few negative or above 255; leaf values are
    fp32(N(0,1) * 0.05).  shuffle permutes each tree's non-root nodes."""
    rng = np.random.default_rng(seed)
    offs, L, R, Fe, Th, V = [0], [], [], [], [], []
    for _ in range(n_trees):
        # breadth-first growth: (level) per node, children filled in later
        lev, left, right = [0], [-1], [-1]
        i = 0
        while i < len(lev):
            if lev[i] < max_depth and (i == 0 or rng.random() >= p_leaf):
                left[i], right[i] = len(lev), len(lev) + 1
                lev += [lev[i] + 1, lev[i] + 1]
                left += [-1, -1]
                right += [-1, -1]
            i += 1
        m = len(lev)
        perm = np.arange(m)
        if shuffle and m > 2:
            perm[1:] = 1 + rng.permutation(m - 1)
        pos = np.empty(m, np.int64)
        pos[perm] = np.arange(m)            # node i is written at pos[i]
        l2, r2 = np.full(m, -1, np.int64), np.full(m, -1, np.int64)
        for i_ in range(m):
            if left[i_] >= 0:
                l2[pos[i_]], r2[pos[i_]] = pos[left[i_]], pos[right[i_]]
        kind = rng.random(m)
        th = rng.integers(0, 33, size=m).astype(np.float64) + np.where(kind < 0.5, 0.0, 0.5)
        th = np.where(kind > 0.97, rng.uniform(-40.0, -0.25, size=m), th)
        th = np.where((kind > 0.94) & (kind <= 0.97), rng.uniform(255.5, 1e6, size=m), th)
        L.append(l2)
        R.append(r2)
        Fe.append(np.where(l2 >= 0, rng.integers(0, n_features, size=m), 0))
        Th.append(np.where(l2 >= 0, th, 0.0))
        V.append(np.where(l2 < 0, rng.standard_normal(size=m) * 0.05, 0.0))
        offs.append(offs[-1] + m)
    return {"offsets": np.asarray(offs, np.int32), "left": np.concatenate(L).astype(np.int32),
            "right": np.concatenate(R).astype(np.int32), "feature": np.concatenate(Fe).astype(np.int32),
            "threshold": np.concatenate(Th).astype(np.float32), "value": np.concatenate(V).astype(np.float32)}


def make_configs(n: int, n_configs: int, seed: int) -> np.ndarray:
    """n configuration indices drawn uniformly from [0, n_configs) (uint64)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, n_configs, size=n, dtype=np.uint64)


def chain_offsets(n_spaces: int, chains_per_space: int) -> np.ndarray:
    """Contiguous chain ranges per space: space w owns [w*c, (w+1)*c)."""
    return np.arange(n_spaces + 1, dtype=np.int64) * chains_per_space


ENTRY_DTYPE = np.dtype([("cfg", "<u8"), ("score", "<f4"), ("flag", "<u4")])


def make_candidates(n_lists: int, per_list: int, n_configs: int, seed: int, dup_frac: float = 0.2,
                    invalid_frac: float = 0.05) -> np.ndarray:
    """Synthetic best lists [n_lists, per_list] of (cfg, score, flag) entries
    for the batch selection: uniformly random configuration indices, a share
    of them repeated across lists (with the same score, as a deterministic
    model gives), a share of empty slots, scores float32(N(0, 1))."""
    rng = np.random.default_rng(seed)
    n = n_lists * per_list
    base = rng.integers(0, n_configs, n, dtype=np.uint64)
    rep = rng.random(n) < dup_frac
    base[rep] = base[rng.integers(0, n, int(rep.sum()))]
    uniq, inv = np.unique(base, return_inverse=True)
    sc = rng.normal(0.0, 1.0, len(uniq)).astype(np.float32)
    out = np.zeros(n, dtype=ENTRY_DTYPE)
    out["cfg"] = base
    out["score"] = sc[inv]
    out["flag"] = (rng.random(n) >= invalid_frac).astype(np.uint32)
    out["cfg"][out["flag"] == 0] = 0
    out["score"][out["flag"] == 0] = 0.0
    return out.reshape(n_lists, per_list)
