"""CPU oracle -- TEST INFRASTRUCTURE ONLY.

ctypes wrapper around ``liboracle.so`` (built from ``oracle.cpp`` with g++).
Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never loads it.

Every routine follows the paper "Learning to Optimize Tensor Programs":
templates and knobs (Section 2), loop-context features (Appendix A.2), the
gradient-boosted tree model (Section 3.1), parallel simulated annealing
(Section 3.3, Algorithm 1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")


def build() -> str:
    """Compile the oracle (single-threaded, no FMA contraction, no fast-math)."""
    cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-o", _LIB + ".tmp", _SRC]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64
        L.or_space_create.argtypes = [i32, vp, i32, ctypes.POINTER(vp)]
        L.or_space_destroy.argtypes = [vp]
        L.or_space_destroy.restype = None
        L.or_space_info.argtypes = [vp, vp, vp, vp, vp, vp]
        L.or_knob_split.argtypes = [vp, i32, i64, vp]
        L.or_decode.argtypes = [vp, u64, vp]
        L.or_encode.argtypes = [vp, vp, vp]
        L.or_loop_quantities.argtypes = [vp, u64, vp]
        L.or_features.argtypes = [vp, vp, i64, vp]
        L.or_features_full.argtypes = [vp, vp, i64, vp]
        L.or_features_onehot.argtypes = [vp, vp, i64, vp]
        L.or_predict.argtypes = [i32, i32, i32, vp, vp, vp, vp, i64, vp, vp]
        L.or_predict_nodes.argtypes = [i32, vp, vp, vp, vp, vp, vp, i32, vp, i64, vp]
        L.or_philox.argtypes = [u64, vp, vp]
        L.or_philox.restype = None
        L.or_thresholds.argtypes = [u64, i64, i64, u64, i32, vp]
        L.or_relation_features.argtypes = [vp, vp, i64, vp]
        L.or_select_batch.argtypes = [vp, vp, i64, i32, i32, ctypes.c_float, i32, u64, vp]
        L.or_sa_run.argtypes = [vp, i32, vp, i32, i32, i32, vp, vp, vp, u64, i64, i64, i32,
                                i32, vp, i32, vp, vp, vp, vp, vp, vp]
        L.or_sa_run_global_local.argtypes = [vp, i32, vp, i32, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, vp,
                                             u64, i64, i64, i32, i32, vp, i32, vp, vp, vp, vp, vp, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(st: int, what: str):
    if st != 0:
        raise ValueError(f"oracle {what} failed with status {st}")


TOP_DTYPE = np.dtype([("cfg", "<u8"), ("score", "<f4"), ("valid", "<u4")])


class Space:
    """A schedule space: template + shape (Section 2)."""

    def __init__(self, template: int, shape):
        self.template = int(template)
        self.shape = tuple(int(s) for s in shape)
        sh = np.asarray(self.shape, dtype=np.int64)
        h = ctypes.c_void_p()
        _check(lib().or_space_create(self.template, _p(sh), len(sh), ctypes.byref(h)), "space_create")
        self._h = h
        nk, nl, nf = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        nc = ctypes.c_uint64()
        sizes = np.zeros(16, dtype=np.int64)
        lib().or_space_info(h, ctypes.byref(nk), _p(sizes), ctypes.byref(nl), ctypes.byref(nf), ctypes.byref(nc))
        self.n_knobs = nk.value
        self.knob_sizes = sizes[: nk.value].copy()
        self.n_loops = nl.value
        self.n_features = nf.value
        # full Appendix A.2 rows add top-down and bottom-up: 4 + 3 per buffer (3) per loop
        self.n_features_full = self.n_loops * 13
        # one-hot rows: length, 12 annotation columns, top-down, bottom-up, 3 per buffer
        self.n_features_onehot = self.n_loops * (3 + 12 + 9)
        self.n_configs = nc.value

    def __del__(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            _lib.or_space_destroy(self._h)
            self._h = None

    def split(self, knob: int, idx: int) -> tuple:
        f = np.zeros(8, dtype=np.int64)
        k = lib().or_knob_split(self._h, knob, idx, _p(f))
        if k < 0:
            raise ValueError("not a split knob value")
        return tuple(int(x) for x in f[:k])

    def decode(self, cfg: int) -> np.ndarray:
        v = np.zeros(self.n_knobs, dtype=np.int64)
        _check(lib().or_decode(self._h, int(cfg), _p(v)), "decode")
        return v

    def encode(self, values) -> int:
        v = np.ascontiguousarray(values, dtype=np.int64)
        out = ctypes.c_uint64()
        _check(lib().or_encode(self._h, _p(v), ctypes.byref(out)), "encode")
        return out.value

    def loop_quantities(self, cfg: int) -> np.ndarray:
        """[n_loops, 3 + 3*n_buffers] raw quantities: ext, ann, bottom_up,
        then (touched, reuse, stride) per buffer."""
        out = np.zeros(self.n_loops * 12, dtype=np.int64)
        _check(lib().or_loop_quantities(self._h, int(cfg), _p(out)), "loop_quantities")
        return out.reshape(self.n_loops, 12)

    RELATION_THRESHOLDS = 32

    def relation_features(self, cfgs) -> np.ndarray:
        """Context relation features (Section 4, Appendix A.2): [n, 2, 3, 32]
        flattened to [n, 192]: per pair (reuse, top-down) and buffer, the
        largest bitlen over the loops touching fewer than 2^t elements."""
        c = np.ascontiguousarray(cfgs, dtype=np.uint64)
        out = np.zeros((len(c), 2 * 3 * self.RELATION_THRESHOLDS), dtype=np.int32)
        _check(lib().or_relation_features(self._h, _p(c), len(c), _p(out)), "relation_features")
        return out

    def features_full(self, cfgs) -> np.ndarray:
        """Rows with the top-down and bottom-up columns of Appendix A.2:
        per loop bitlen(length), annotation, bitlen(top-down),
        bitlen(bottom-up), then per buffer touch, reuse, stride bitlens."""
        c = np.ascontiguousarray(cfgs, dtype=np.uint64)
        out = np.zeros((len(c), self.n_features_full), dtype=np.int32)
        _check(lib().or_features_full(self._h, _p(c), len(c), _p(out)), "features_full")
        return out

    ANNOTATION_KINDS = 12

    def features_onehot(self, cfgs) -> np.ndarray:
        """Appendix A.2 rows with a one-hot annotation: per loop
        bitlen(length), 12 one-hot annotation columns (ids 0..11),
        bitlen(top-down), bitlen(bottom-up), then per buffer touch, reuse,
        stride bitlens."""
        c = np.ascontiguousarray(cfgs, dtype=np.uint64)
        out = np.zeros((len(c), self.n_features_onehot), dtype=np.int32)
        _check(lib().or_features_onehot(self._h, _p(c), len(c), _p(out)), "features_onehot")
        return out

    def features(self, cfgs) -> np.ndarray:
        c = np.ascontiguousarray(cfgs, dtype=np.uint64)
        out = np.zeros((len(c), self.n_features), dtype=np.int32)
        _check(lib().or_features(self._h, _p(c), len(c), _p(out)), "features")
        return out


def predict(fid, thr, leaf, feats, want_leaves=False):
    """fp32 ensemble scores (left fold in tree order) and optionally leaf indices."""
    fid = np.ascontiguousarray(fid, dtype=np.uint8)
    thr = np.ascontiguousarray(thr, dtype=np.uint8)
    leaf = np.ascontiguousarray(leaf, dtype=np.float32)
    feats = np.ascontiguousarray(feats, dtype=np.int32)
    T, n_int = fid.shape
    depth = int(n_int + 1).bit_length() - 1
    n, F = feats.shape
    scores = np.zeros(n, dtype=np.float32)
    leaves = np.zeros((n, T), dtype=np.uint16) if want_leaves else None
    _check(lib().or_predict(T, depth, F, _p(fid), _p(thr), _p(leaf), _p(feats), n, _p(scores),
                            _p(leaves) if want_leaves else None), "predict")
    return (scores, leaves) if want_leaves else scores


def predict_nodes(trees, feats):
    """fp32 scores of trees in node-list form (left fold in tree order).
    trees: dict of offsets [T+1], left, right, feature (int32), threshold,
    value (float32), as written by trained gradient-boosting libraries."""
    off = np.ascontiguousarray(trees["offsets"], dtype=np.int32)
    left = np.ascontiguousarray(trees["left"], dtype=np.int32)
    right = np.ascontiguousarray(trees["right"], dtype=np.int32)
    feat = np.ascontiguousarray(trees["feature"], dtype=np.int32)
    th = np.ascontiguousarray(trees["threshold"], dtype=np.float32)
    val = np.ascontiguousarray(trees["value"], dtype=np.float32)
    feats = np.ascontiguousarray(feats, dtype=np.int32)
    n, F = feats.shape
    scores = np.zeros(n, dtype=np.float32)
    _check(lib().or_predict_nodes(len(off) - 1, _p(off), _p(left), _p(right), _p(feat), _p(th), _p(val), F,
                                  _p(feats), n, _p(scores)), "predict_nodes")
    return scores


def predict_global_local(global_model, feats_global, local_model, feats_local):
    """Eq. 4 (Section 4): f_hat = f_hat_global + f_hat_local.  Each model's
    score is its own fp32 left fold over its trees (predict); the two are
    added once in fp32, the global one first.  A model is (fid, thr, leaf)."""
    g = predict(*global_model, feats_global)
    l = predict(*local_model, feats_local)
    return (g + l).astype(np.float32)


def philox(seed: int, ctr) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().or_philox(int(seed), _p(c), _p(out))
    return out


def thresholds(seed: int, chain0: int, n_chains: int, step_base: int, steps: int) -> np.ndarray:
    out = np.zeros((n_chains, steps), dtype=np.float32)
    _check(lib().or_thresholds(int(seed), chain0, n_chains, step_base, steps, _p(out)), "thresholds")
    return out


class Chains:
    """Persistent annealing chain state (Section 3.3)."""

    MAX_KNOBS = 12

    def __init__(self, spaces, offsets, seed: int, chain0: int, topk: int):
        self.spaces = list(spaces)
        self.offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        self.n = int(self.offsets[-1])
        self.seed, self.chain0, self.topk = int(seed), int(chain0), int(topk)
        self.knobs = np.zeros((self.n, self.MAX_KNOBS), dtype=np.int64)
        self.score = np.zeros(self.n, dtype=np.float32)
        self.initialised = np.zeros(self.n, dtype=np.uint8)
        self.step_abs = np.zeros(self.n, dtype=np.uint64)
        self.top = np.zeros((self.n, self.topk), dtype=TOP_DTYPE)

    def cur_cfgs(self) -> np.ndarray:
        out = np.zeros(self.n, dtype=np.uint64)
        for w, sp in enumerate(self.spaces):
            for c in range(int(self.offsets[w]), int(self.offsets[w + 1])):
                out[c] = sp.encode(self.knobs[c, : sp.n_knobs])
        return out

    @staticmethod
    def _model(ensemble):
        fid, thr_nodes, leaf = (np.ascontiguousarray(a) for a in ensemble)
        fid = fid.astype(np.uint8, copy=False)
        thr_nodes = thr_nodes.astype(np.uint8, copy=False)
        leaf = leaf.astype(np.float32, copy=False)
        T, n_int = fid.shape
        depth = int(n_int + 1).bit_length() - 1
        return fid, thr_nodes, leaf, T, depth

    def run(self, ensemble, steps: int, thr, trace=False, global_model=None):
        """`steps` annealing steps of every chain.  With global_model (a
        (fid, thr, leaf) ensemble over the 192 context relation features) the
        energy is Eq. 4's global + local model, `ensemble` being the local
        one over the loop-context features."""
        fid, thr_nodes, leaf, T, depth = self._model(ensemble)
        F = self.spaces[0].n_features
        thr = np.ascontiguousarray(thr, dtype=np.float32).reshape(self.n, steps)
        handles = (ctypes.c_void_p * len(self.spaces))(*[s._h.value for s in self.spaces])
        tr = np.zeros((self.n, steps), dtype=TOP_DTYPE) if trace else None
        tail = (self.seed, self.chain0, self.n, self.topk, steps, _p(thr), self.MAX_KNOBS, _p(self.knobs),
                _p(self.score), _p(self.initialised), _p(self.step_abs), _p(self.top), _p(tr) if trace else None)
        if global_model is None:
            st = lib().or_sa_run(handles, len(self.spaces), _p(self.offsets), T, depth, F,
                                 _p(fid), _p(thr_nodes), _p(leaf), *tail)
        else:
            gfid, gthr, gleaf, gT, gdepth = self._model(global_model)
            st = lib().or_sa_run_global_local(handles, len(self.spaces), _p(self.offsets), gT, gdepth,
                                              Space.RELATION_THRESHOLDS * 6, _p(gfid), _p(gthr), _p(gleaf),
                                              T, depth, F, _p(fid), _p(thr_nodes), _p(leaf), *tail)
        _check(st, "sa_run")
        return tr


def select_batch(space: Space, cand, pool: int, n_greedy: int, alpha: float, n_random: int, seed: int) -> np.ndarray:
    """The batch to measure (Algorithm 1, Eq. 3): greedy picks from the top
    `pool` distinct candidates, then `n_random` uniform configurations.
    cand: TOP_DTYPE entries (any shape).  Returns n_greedy + n_random entries
    (valid 1 greedy, 2 random, 0 empty)."""
    c = np.ascontiguousarray(np.asarray(cand).reshape(-1).astype(TOP_DTYPE, copy=False))
    out = np.zeros(n_greedy + n_random, dtype=TOP_DTYPE)
    _check(lib().or_select_batch(space._h, _p(c), len(c), int(pool), int(n_greedy), float(alpha),
                                 int(n_random), int(seed), _p(out)), "select_batch")
    return out
