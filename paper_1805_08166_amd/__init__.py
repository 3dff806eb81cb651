"""Python binding of libautotensor (HIP, gfx950): argument marshalling only.

Every function has the name of the C entry point it calls (include/autotensor.h)
and does nothing but check argument types, pass raw device pointers and the
current HIP stream, and turn a non-OK status into an exception.  All of the
method's work runs in the library's HIP kernels.  PyTorch provides device
memory and streams.

The library must have been built (``python -m paper_1805_08166_amd.build`` or
``__graft_entry__.build()``); importing this package without it raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libautotensor.so")

AT_TMPL_GEMM = 0
AT_TMPL_CONV2D_NCHW = 1
AT_TMPL_GEMM_VT = 2
AT_TMPL_CONV2D_NCHW_VT = 3

STATUS = {0: "AT_OK", -1: "AT_E_INVALID", -2: "AT_E_UNSUPPORTED", -3: "AT_E_OOM", -4: "AT_E_HIP",
          -5: "AT_E_RANGE", -6: "AT_E_MISMATCH"}

# at_entry: {uint64 cfg; float score; uint32 flag}
ENTRY_DTYPE = np.dtype([("cfg", "<u8"), ("score", "<f4"), ("flag", "<u4")])

EXPORTED = [
    "at_space_create", "at_space_info", "at_spaceset_create", "at_space_destroy",
    "at_extract_features", "at_extract_features_full", "at_extract_features_onehot", "at_extract_relation_features", "at_space_errors", "at_ensemble_create", "at_ensemble_destroy",
    "at_trees_depth", "at_trees_pad", "at_ensemble_import",
    "at_gbt_predict", "at_gbt_predict_global_local", "at_chains_create", "at_chains_destroy", "at_chains_step",
    "at_sa_thresholds", "at_sa_run", "at_sa_run_traced", "at_sa_run_global_local", "at_chains_export", "at_sa_set_profiling",
    "at_sa_kernel_times", "at_chains_set_path", "at_chains_last_path", "at_chains_last_plan", "at_select_batch", "at_select_batch_noalloc", "at_last_error",
]

# at_sa_path
AT_SA_PATH_AUTO = 0
AT_SA_PATH_TREES = 1
AT_SA_PATH_LOCAL = 2


class ATError(RuntimeError):
    def __init__(self, func: str, status: int, msg: str):
        super().__init__(f"{func} -> {STATUS.get(status, status)}: {msg}")
        self.status = status


def _load():
    from . import build as _build
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    if _build.stale():
        raise ImportError(f"{LIB_PATH} was built from other sources than those under csrc/; "
                          "run __graft_entry__.build() again")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64
    sig = {
        "at_space_create": [i32, vp, i32, vp],
        "at_space_info": [vp, vp, vp, vp, vp, vp],
        "at_spaceset_create": [vp, i32, vp, vp],
        "at_space_destroy": [vp],
        "at_extract_features": [vp, vp, i64, vp, vp],
        "at_extract_relation_features": [vp, vp, i64, vp, vp],
        "at_extract_features_full": [vp, vp, i64, vp, vp],
        "at_extract_features_onehot": [vp, vp, i64, vp, vp],
        "at_space_errors": [vp, vp],
        "at_ensemble_create": [i32, i32, i32, vp, vp, vp, vp],
        "at_ensemble_destroy": [vp],
        "at_trees_depth": [i32, vp, vp, vp, vp],
        "at_trees_pad": [i32, vp, vp, vp, vp, vp, vp, i32, i32, vp, vp, vp],
        "at_ensemble_import": [i32, vp, vp, vp, vp, vp, vp, i32, vp],
        "at_gbt_predict": [vp, vp, i64, vp, vp, vp],
        "at_gbt_predict_global_local": [vp, vp, vp, vp, i64, vp, vp],
        "at_chains_create": [vp, i64, i64, i32, u64, vp],
        "at_chains_destroy": [vp],
        "at_chains_step": [vp, vp],
        "at_sa_thresholds": [u64, i64, i64, u64, i32, vp],
        "at_sa_run": [vp, vp, vp, i32, vp, vp, vp],
        "at_sa_run_traced": [vp, vp, vp, i32, vp, vp, vp, vp],
        "at_sa_run_global_local": [vp, vp, vp, vp, i32, vp, vp, vp, vp],
        "at_chains_export": [vp, vp, vp, vp],
        "at_sa_set_profiling": [vp, i32],
        "at_sa_kernel_times": [vp, vp, vp, vp, vp],
        "at_chains_set_path": [vp, i32],
        "at_chains_last_path": [vp, vp],
        "at_chains_last_plan": [vp, vp],
        "at_select_batch": [vp, vp, i64, i32, i32, ctypes.c_float, i32, u64, vp, vp],
        "at_select_batch_noalloc": [vp, vp, i64, i32, i32, ctypes.c_float, i32, u64, vp, vp],
        "at_last_error": [],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    for name in ("at_space_destroy", "at_ensemble_destroy", "at_chains_destroy"):
        getattr(L, name).restype = None
    L.at_last_error.restype = ctypes.c_char_p
    return L


_lib = _load()


def lib():
    return _lib


def _check(func: str, st: int):
    if st != 0:
        raise ATError(func, st, _lib.at_last_error().decode())


def _np(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dev(t, dtype=None, name="tensor"):
    """Raw device pointer of a CUDA/HIP torch tensor (contiguous)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class _Handle:
    _destroy = None

    def __init__(self, h):
        self.h = h

    def close(self):
        if self.h:
            getattr(_lib, self._destroy)(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Space(_Handle):
    _destroy = "at_space_destroy"

    def info(self):
        return at_space_info(self)


class Ensemble(_Handle):
    _destroy = "at_ensemble_destroy"


class Chains(_Handle):
    _destroy = "at_chains_destroy"


def at_space_create(tmpl: int, shape) -> Space:
    sh = np.ascontiguousarray(shape, dtype=np.int64)
    h = ctypes.c_void_p()
    _check("at_space_create", _lib.at_space_create(int(tmpl), _np(sh), len(sh), ctypes.byref(h)))
    sp = Space(h)
    sp.n_knobs, sp.knob_sizes, sp.n_loops, sp.n_features, sp.n_configs = at_space_info(sp)
    return sp


def at_space_info(space: Space):
    nk, nl, nf = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    nc = ctypes.c_uint64()
    sizes = np.zeros(16, dtype=np.int32)
    _check("at_space_info", _lib.at_space_info(space.h, ctypes.byref(nk), _np(sizes), ctypes.byref(nl),
                                               ctypes.byref(nf), ctypes.byref(nc)))
    return nk.value, sizes[: nk.value].copy(), nl.value, nf.value, nc.value


def at_spaceset_create(spaces, chain_offsets) -> Space:
    arr = (ctypes.c_void_p * len(spaces))(*[s.h.value for s in spaces])
    off = np.ascontiguousarray(chain_offsets, dtype=np.int64)
    if len(off) != len(spaces) + 1:
        raise ValueError("chain_offsets must have len(spaces) + 1 entries")
    h = ctypes.c_void_p()
    _check("at_spaceset_create", _lib.at_spaceset_create(arr, len(spaces), _np(off), ctypes.byref(h)))
    sp = Space(h)
    sp.n_knobs, sp.knob_sizes, sp.n_loops, sp.n_features, sp.n_configs = at_space_info(sp)
    sp.chain_offsets = off.copy()
    return sp


def at_extract_features(space: Space, cfgs, feats, stream=None):
    """cfgs: device uint64 [n] (torch.int64 storage); feats: device int32 [n, F]."""
    import torch
    n = cfgs.numel()
    if feats.shape != (n, space.n_features):
        raise ValueError("feats must be [n, n_features]")
    _check("at_extract_features", _lib.at_extract_features(
        space.h, _dev(cfgs, torch.int64, "cfgs"), n, _dev(feats, torch.int32, "feats"), _stream(stream)))


def at_extract_features_full(space: Space, cfgs, feats, stream=None):
    """Full Appendix A.2 rows (13 per loop: loop-context columns with
    bitlen(top-down) and bitlen(bottom-up) after the annotation).
    cfgs: device uint64 [n] (torch.int64 storage); feats: device int32
    [n, 13 * n_loops]."""
    import torch
    n = cfgs.numel()
    if feats.shape != (n, 13 * space.n_loops):
        raise ValueError("feats must be [n, 13 * n_loops]")
    _check("at_extract_features_full", _lib.at_extract_features_full(
        space.h, _dev(cfgs, torch.int64, "cfgs"), n, _dev(feats, torch.int32, "feats"), _stream(stream)))


ONEHOT_PER_LOOP = 24


def at_extract_features_onehot(space: Space, cfgs, feats, stream=None):
    """Appendix A.2 rows with a one-hot annotation (24 per loop: length,
    12 annotation columns, top-down, bottom-up, touch/reuse/stride per
    buffer).  cfgs: device uint64 [n] (torch.int64 storage); feats: device
    int32 [n, 24 * n_loops]."""
    import torch
    n = cfgs.numel()
    if feats.shape != (n, ONEHOT_PER_LOOP * space.n_loops):
        raise ValueError("feats must be [n, 24 * n_loops]")
    _check("at_extract_features_onehot", _lib.at_extract_features_onehot(
        space.h, _dev(cfgs, torch.int64, "cfgs"), n, _dev(feats, torch.int32, "feats"), _stream(stream)))


RELATION_FEATURES = 192


def at_extract_relation_features(space: Space, cfgs, feats, stream=None):
    """cfgs: device uint64 [n] (torch.int64 storage); feats: device int32 [n, 192]."""
    import torch
    n = cfgs.numel()
    if feats.shape != (n, RELATION_FEATURES):
        raise ValueError("feats must be [n, 192]")
    _check("at_extract_relation_features", _lib.at_extract_relation_features(
        space.h, _dev(cfgs, torch.int64, "cfgs"), n, _dev(feats, torch.int32, "feats"), _stream(stream)))


def at_space_errors(space: Space) -> int:
    v = ctypes.c_uint64()
    _check("at_space_errors", _lib.at_space_errors(space.h, ctypes.byref(v)))
    return v.value


def at_ensemble_create(fid, thr, leaf, n_features: int) -> Ensemble:
    """fid, thr: host uint8 [T, 2^d-1]; leaf: host float32 [T, 2^d]."""
    fid = np.ascontiguousarray(fid, dtype=np.uint8)
    thr = np.ascontiguousarray(thr, dtype=np.uint8)
    leaf = np.ascontiguousarray(leaf, dtype=np.float32)
    T, n_int = fid.shape
    depth = int(n_int + 1).bit_length() - 1
    if thr.shape != fid.shape or leaf.shape != (T, 1 << depth) or (1 << depth) - 1 != n_int:
        raise ValueError("inconsistent ensemble tables")
    h = ctypes.c_void_p()
    _check("at_ensemble_create", _lib.at_ensemble_create(T, depth, int(n_features), _np(fid), _np(thr), _np(leaf),
                                                         ctypes.byref(h)))
    e = Ensemble(h)
    e.n_trees, e.depth, e.n_features = T, depth, int(n_features)
    return e


def _node_lists(trees):
    keys = ("offsets", "left", "right", "feature", "threshold", "value")
    dt = (np.int32,) * 4 + (np.float32,) * 2
    arr = [np.ascontiguousarray(trees[k], dtype=d) for k, d in zip(keys, dt)]
    m = len(arr[1])
    if len(arr[0]) < 2 or any(len(a) != m for a in arr[1:]) or arr[0][0] < 0 or arr[0][-1] > m:
        raise ValueError("inconsistent node lists")
    return arr


def at_trees_depth(trees) -> int:
    """Level of the deepest leaf of node-list trees (dict of offsets, left,
    right, feature, threshold, value; host arrays)."""
    off, left, right, _, _, _ = _node_lists(trees)
    d = ctypes.c_int()
    _check("at_trees_depth", _lib.at_trees_depth(len(off) - 1, _np(off), _np(left), _np(right), ctypes.byref(d)))
    return d.value


def at_trees_pad(trees, n_features: int, depth: int):
    """Full-tree tables (fid, thr uint8 [T, 2^d-1], leaf float32 [T, 2^d]) of
    node-list trees, padded to `depth`."""
    off, left, right, feat, th, val = _node_lists(trees)
    T = len(off) - 1
    dd = depth if 1 <= depth <= 12 else 1      # the library rejects other depths
    fid = np.zeros((T, (1 << dd) - 1), np.uint8)
    thr = np.zeros((T, (1 << dd) - 1), np.uint8)
    leaf = np.zeros((T, 1 << dd), np.float32)
    _check("at_trees_pad", _lib.at_trees_pad(T, _np(off), _np(left), _np(right), _np(feat), _np(th), _np(val),
                                             int(n_features), int(depth), _np(fid), _np(thr), _np(leaf)))
    return fid, thr, leaf


def at_ensemble_import(trees, n_features: int) -> Ensemble:
    """Ensemble from node-list trees of any shape, padded on the host to the
    deepest leaf's depth."""
    off, left, right, feat, th, val = _node_lists(trees)
    T = len(off) - 1
    h = ctypes.c_void_p()
    _check("at_ensemble_import", _lib.at_ensemble_import(T, _np(off), _np(left), _np(right), _np(feat), _np(th),
                                                         _np(val), int(n_features), ctypes.byref(h)))
    e = Ensemble(h)
    e.n_trees, e.depth, e.n_features = T, max(1, at_trees_depth(trees)), int(n_features)
    return e


def at_gbt_predict(ens: Ensemble, feats, scores, leaves=None, stream=None):
    """feats: device int32 [n, F]; scores: device float32 [n]; leaves: device int16 [n, T] or None."""
    import torch
    n = feats.shape[0]
    if feats.dim() != 2 or feats.shape[1] != ens.n_features or scores.numel() != n:
        raise ValueError("shape mismatch")
    if leaves is not None and leaves.shape != (n, ens.n_trees):
        raise ValueError("leaves must be [n, n_trees]")
    _check("at_gbt_predict", _lib.at_gbt_predict(
        ens.h, _dev(feats, torch.int32, "feats"), n, _dev(scores, torch.float32, "scores"),
        _dev(leaves, torch.int16, "leaves"), _stream(stream)))


def at_gbt_predict_global_local(glob: Ensemble, feats_global, local: Ensemble, feats_local, scores, stream=None):
    """Eq. 4: scores = global(feats_global) + local(feats_local), device tensors."""
    import torch
    n = scores.numel()
    if feats_global.shape != (n, glob.n_features) or feats_local.shape != (n, local.n_features):
        raise ValueError("shape mismatch")
    _check("at_gbt_predict_global_local", _lib.at_gbt_predict_global_local(
        glob.h, _dev(feats_global, torch.int32, "feats_global"), local.h, _dev(feats_local, torch.int32, "feats_local"),
        n, _dev(scores, torch.float32, "scores"), _stream(stream)))


def at_chains_create(space: Space, chain0: int, n_chains: int, topk: int, seed: int) -> Chains:
    h = ctypes.c_void_p()
    _check("at_chains_create", _lib.at_chains_create(space.h, int(chain0), int(n_chains), int(topk), int(seed),
                                                     ctypes.byref(h)))
    c = Chains(h)
    c.chain0, c.n_chains, c.topk, c.seed = int(chain0), int(n_chains), int(topk), int(seed)
    return c


def at_chains_step(chains: Chains) -> int:
    v = ctypes.c_uint64()
    _check("at_chains_step", _lib.at_chains_step(chains.h, ctypes.byref(v)))
    return v.value


def at_chains_set_path(chains: Chains, path: int):
    _check("at_chains_set_path", _lib.at_chains_set_path(chains.h, int(path)))


def at_chains_last_path(chains: Chains) -> int:
    v = ctypes.c_int()
    _check("at_chains_last_path", _lib.at_chains_last_path(chains.h, ctypes.byref(v)))
    return v.value


PLAN_KEYS_LOCAL = ["chains_per_wg", "threads", "workgroups", "trees_per_chunk", "chunks", "gather", "lds_bytes",
                   "stream_bytes_per_step"]
PLAN_KEYS_TREES = ["trees_per_wg", "waves", "workgroups", "slices", "slice_blocks", "chain_workgroups",
                   "tile_quads", "v_bytes_per_step"]


def at_chains_last_plan(chains: Chains) -> dict:
    """Launch plan of the last run, keyed by the layout of the path it took
    (PLAN_KEYS_LOCAL or PLAN_KEYS_TREES), plus "path"."""
    v = np.zeros(8, np.int64)
    _check("at_chains_last_plan", _lib.at_chains_last_plan(chains.h, _np(v)))
    path = at_chains_last_path(chains)
    keys = PLAN_KEYS_TREES if path == AT_SA_PATH_TREES else PLAN_KEYS_LOCAL
    plan = dict(zip(keys, (int(x) for x in v)))
    plan["path"] = path
    return plan


def _select(name, space: Space, cand, pool, n_greedy, alpha, n_random, seed, out, stream):
    import torch
    n_cand = cand.numel() // 4 if cand is not None else 0
    if cand is not None and (cand.dtype != torch.int32 or cand.shape[-1] != 4 or not cand.is_contiguous()):
        raise ValueError("cand must be a contiguous int32 [..., 4] at_entry tensor")
    if out.shape != (n_greedy + n_random, 4):
        raise ValueError("out must be [n_greedy + n_random, 4] int32")
    _check(name, getattr(_lib, name)(
        space.h, _dev(cand, torch.int32, "cand") if n_cand else None, int(n_cand), int(pool), int(n_greedy),
        float(alpha), int(n_random), int(seed), _dev(out, torch.int32, "out"), _stream(stream)))


def at_select_batch(space: Space, cand, pool: int, n_greedy: int, alpha: float, n_random: int, seed: int, out,
                    stream=None):
    """cand: device int32 [..., 4] (at_entry, any leading shape); out: device
    int32 [n_greedy + n_random, 4] (at_entry)."""
    _select("at_select_batch", space, cand, pool, n_greedy, alpha, n_random, seed, out, stream)


def at_select_batch_noalloc(space: Space, cand, pool: int, n_greedy: int, alpha: float, n_random: int, seed: int,
                            out, stream=None):
    """at_select_batch without device allocation (the library's fixed
    per-device scratch; calls that overlap on one device race)."""
    _select("at_select_batch_noalloc", space, cand, pool, n_greedy, alpha, n_random, seed, out, stream)


def at_sa_thresholds(seed: int, chain0: int, n_chains: int, step_base: int, steps: int) -> np.ndarray:
    out = np.zeros((n_chains, steps), dtype=np.float32)
    _check("at_sa_thresholds", _lib.at_sa_thresholds(int(seed), int(chain0), int(n_chains), int(step_base),
                                                     int(steps), _np(out)))
    return out


def at_sa_run(space: Space, ens: Ensemble, chains: Chains, steps: int, thr, best, stream=None):
    """thr: device float32 [n_chains, steps]; best: device int32 [n_chains, topk, 4] (at_entry)."""
    import torch
    _check_sa(chains, steps, thr, best)
    _check("at_sa_run", _lib.at_sa_run(space.h, ens.h, chains.h, int(steps), _dev(thr, torch.float32, "thr"),
                                       _dev(best, torch.int32, "best"), _stream(stream)))


def at_sa_run_traced(space: Space, ens: Ensemble, chains: Chains, steps: int, thr, best, trace, stream=None):
    """as at_sa_run; trace: device int32 [n_chains, steps, 4] (at_entry)."""
    import torch
    _check_sa(chains, steps, thr, best)
    if trace.shape != (chains.n_chains, steps, 4):
        raise ValueError("trace must be [n_chains, steps, 4] int32")
    _check("at_sa_run_traced", _lib.at_sa_run_traced(
        space.h, ens.h, chains.h, int(steps), _dev(thr, torch.float32, "thr"), _dev(best, torch.int32, "best"),
        _dev(trace, torch.int32, "trace"), _stream(stream)))


def at_sa_run_global_local(space: Space, glob: Ensemble, local: Ensemble, chains: Chains, steps: int, thr, best,
                           trace=None, stream=None):
    """Annealing with Eq. 4's energy: glob over the 192 relation features
    plus local over the loop features.  thr: device float32 [n_chains,
    steps]; best: device int32 [n_chains, topk, 4]; trace: device int32
    [n_chains, steps, 4] or None."""
    import torch
    _check_sa(chains, steps, thr, best)
    if trace is not None and trace.shape != (chains.n_chains, steps, 4):
        raise ValueError("trace must be [n_chains, steps, 4] int32")
    _check("at_sa_run_global_local", _lib.at_sa_run_global_local(
        space.h, glob.h, local.h, chains.h, int(steps), _dev(thr, torch.float32, "thr"),
        _dev(best, torch.int32, "best"), _dev(trace, torch.int32, "trace"), _stream(stream)))


def _check_sa(chains, steps, thr, best):
    if thr is not None and thr.numel() != chains.n_chains * steps:
        raise ValueError("thr must hold n_chains * steps values")
    if best.shape != (chains.n_chains, chains.topk, 4):
        raise ValueError("best must be [n_chains, topk, 4] int32")


def at_chains_export(chains: Chains, cur_cfg=None, cur_score=None, stream=None):
    import torch
    _check("at_chains_export", _lib.at_chains_export(
        chains.h, _dev(cur_cfg, torch.int64, "cur_cfg"), _dev(cur_score, torch.float32, "cur_score"),
        _stream(stream)))


def at_sa_set_profiling(chains: Chains, enable: bool):
    _check("at_sa_set_profiling", _lib.at_sa_set_profiling(chains.h, 1 if enable else 0))


def at_sa_kernel_times(chains: Chains) -> dict:
    """Device time of the last profiled run's launches (waits for the run)."""
    tms, cms = ctypes.c_double(0), ctypes.c_double(0)
    tn, cn = ctypes.c_int64(0), ctypes.c_int64(0)
    _check("at_sa_kernel_times", _lib.at_sa_kernel_times(chains.h, ctypes.byref(tms), ctypes.byref(tn),
                                                         ctypes.byref(cms), ctypes.byref(cn)))
    return {"tree_ms": tms.value, "tree_launches": tn.value, "chain_ms": cms.value, "chain_launches": cn.value}


def entries(t) -> np.ndarray:
    """Host structured view (cfg, score, flag) of a device at_entry tensor [..., 4] int32."""
    a = t.detach().cpu().contiguous().numpy()
    return a.view(ENTRY_DTYPE).reshape(a.shape[:-1])
