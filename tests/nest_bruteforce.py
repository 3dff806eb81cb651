"""Brute-force loop-nest enumeration used to pin the loop-context features.

Given a template, its shape and the per-level tile factors of one schedule,
this builds the generated loop nest literally, runs every iteration of the
sub-nest rooted at each loop, and counts:
  * bottom-up  -- iterations of the sub-nest (this loop and all inner loops),
  * touch count -- distinct flat addresses of each buffer the sub-nest reads
                   or writes (Appendix A.2 "number of touched elements"),
  * reuse ratio -- bottom-up // touch count,
  * stride     -- change of the buffer's flat address for one step of this
                  loop's variable from its first iteration (the coefficient of
                  the variable in the index expression),
  * annotation -- the loop's thread binding, else unrolled when the sub-nest
                  has at most auto_unroll_max_step iterations.
It shares nothing with the oracle's closed forms: no range products, no
distinct-count formula, no coefficient bookkeeping.
"""
from __future__ import annotations

import itertools

import numpy as np

SERIAL, UNROLL, UNROLL_EXPLICIT = 0, 1, 2
BLOCK_X, BLOCK_Y, BLOCK_Z, THREAD_X, THREAD_Y, THREAD_Z = 3, 4, 5, 6, 7, 8


def bitlen(x: int) -> int:
    return int(x).bit_length()


def ordered_splits(n: int, k: int):
    """All ordered k-tuples of positive integers with product n, sorted."""
    divs = [d for d in range(1, n + 1) if n % d == 0]
    out = [t for t in itertools.product(divs, repeat=k) if int(np.prod(t)) == n]
    return sorted(out)


class Nest:
    """A generated loop nest: loops (outer to inner) over tiled axes."""

    def __init__(self, axes, factors, loops, buffers, auto_unroll, explicit):
        self.axes = axes            # axis names
        self.factors = factors      # axis -> tuple of level extents (outer first)
        self.loops = loops          # list of (components [(axis, level)], binding)
        self.buffers = buffers      # list of (name, flat_index(axis values dict) -> ndarray)
        self.auto_unroll = auto_unroll
        self.explicit = explicit

    def loop_extent(self, p):
        comps, _ = self.loops[p]
        e = 1
        for a, l in comps:
            e *= self.factors[a][l]
        return e

    def _axis_values(self, level_vars):
        """level_vars[(axis, level)] -> array; returns axis -> value array."""
        vals = {}
        for a in self.axes:
            f = self.factors[a]
            v = 0
            for l in range(len(f)):
                inner = int(np.prod(f[l + 1:])) if l + 1 < len(f) else 1
                v = v + level_vars[(a, l)] * inner
            vals[a] = v
        return vals

    def _level_vars(self, loop_vars):
        """loop_vars[p] -> array (value of loop p's variable); split fused loops."""
        lv = {}
        for p, (comps, _) in enumerate(self.loops):
            r = loop_vars[p]
            if len(comps) == 1:
                lv[comps[0]] = r
            else:
                (ay, ly), (ax, lx) = comps
                inner = self.factors[ax][lx]
                lv[(ay, ly)] = r // inner
                lv[(ax, lx)] = r % inner
        return lv

    def quantities(self, outer=None):
        """Per loop: (ext, ann, bottom_up, [(touched, reuse, stride) per buffer])."""
        P = len(self.loops)
        outer = outer or [0] * P
        rows = []
        for p in range(P):
            exts = [self.loop_extent(q) for q in range(p, P)]
            grid = np.indices(exts).reshape(len(exts), -1)
            loop_vars = {q: np.full(grid.shape[1], outer[q], dtype=np.int64) for q in range(p)}
            for i, q in enumerate(range(p, P)):
                loop_vars[q] = grid[i].astype(np.int64)
            vals = self._axis_values(self._level_vars(loop_vars))
            bottom_up = grid.shape[1]
            # one step of loop p's variable from its first iteration, all
            # other variables at their first iteration (outer ones as given)
            base_vars = {q: np.array([outer[q] if q < p else 0], dtype=np.int64) for q in range(P)}
            step_vars = dict(base_vars)
            step_vars[p] = np.array([1], dtype=np.int64)
            v0 = self._axis_values(self._level_vars(base_vars))
            v1 = self._axis_values(self._level_vars(step_vars))
            bufs = []
            for name, flat in self.buffers:
                addrs = flat(vals)
                touched = len(np.unique(addrs))
                stride = int(flat(v1)[0] - flat(v0)[0])
                bufs.append((touched, bottom_up // touched, stride))
            comps, binding = self.loops[p]
            if binding != SERIAL:
                ann = binding
            elif self.auto_unroll > 0 and bottom_up <= self.auto_unroll:
                ann = UNROLL_EXPLICIT if self.explicit else UNROLL
            else:
                ann = SERIAL
            rows.append((self.loop_extent(p), ann, bottom_up, bufs))
        return rows

    def feature_rows(self, outer=None):
        out = []
        for ext, ann, _, bufs in self.quantities(outer):
            row = [bitlen(ext), ann]
            for t, r, s in bufs:
                row += [bitlen(t), bitlen(r), bitlen(s)]
            out.append(row)
        return np.array(out, dtype=np.int64)


def gemm_nest(M, N, K, ti, tj, tk, auto_unroll, explicit):
    """C[i,j] = sum_k A[k,i] B[k,j]; A [K][M], B [K][N], C [M][N]."""
    loops = [([("i", 0)], BLOCK_Y), ([("j", 0)], BLOCK_X), ([("i", 1)], THREAD_Y), ([("j", 1)], THREAD_X),
             ([("k", 0)], SERIAL), ([("i", 2)], SERIAL), ([("j", 2)], SERIAL), ([("k", 1)], SERIAL),
             ([("i", 3)], SERIAL), ([("j", 3)], SERIAL)]
    buffers = [("A", lambda v: v["k"] * M + v["i"]),
               ("B", lambda v: v["k"] * N + v["j"]),
               ("C", lambda v: v["i"] * N + v["j"])]
    return Nest(["i", "j", "k"], {"i": ti, "j": tj, "k": tk}, loops, buffers, auto_unroll, explicit)


def conv_nest(shape, toc, toh, tow, trc, try_, trx, auto_unroll, explicit):
    """out[k][oh][ow] = sum data_pad[c][oh*S+ry][ow*S+rx] * kernel[k][c][ry][rx]."""
    _, C, H, W, K, KH, KW, P, S = shape
    Hp, Wp = H + 2 * P, W + 2 * P
    OH, OW = (Hp - KH) // S + 1, (Wp - KW) // S + 1
    loops = [([("oc", 0)], BLOCK_Z), ([("oh", 0)], BLOCK_Y), ([("ow", 0)], BLOCK_X),
             ([("oc", 1)], THREAD_Z), ([("oh", 1)], THREAD_Y), ([("ow", 1)], THREAD_X),
             ([("rc", 0)], SERIAL), ([("ry", 0), ("rx", 0)], SERIAL),
             ([("oc", 2)], SERIAL), ([("oh", 2)], SERIAL), ([("ow", 2)], SERIAL),
             ([("rc", 1)], SERIAL), ([("ry", 1), ("rx", 1)], SERIAL),
             ([("oc", 3)], SERIAL), ([("oh", 3)], SERIAL), ([("ow", 3)], SERIAL)]
    buffers = [("data", lambda v: v["rc"] * Hp * Wp + (v["oh"] * S + v["ry"]) * Wp + (v["ow"] * S + v["rx"])),
               ("kernel", lambda v: ((v["oc"] * C + v["rc"]) * KH + v["ry"]) * KW + v["rx"]),
               ("output", lambda v: (v["oc"] * OH + v["oh"]) * OW + v["ow"])]
    factors = {"oc": toc, "oh": toh, "ow": tow, "rc": trc, "ry": try_, "rx": trx}
    return Nest(list(factors), factors, loops, buffers, auto_unroll, explicit)


def conv_out_hw(shape):
    _, C, H, W, K, KH, KW, P, S = shape
    return (H + 2 * P - KH) // S + 1, (W + 2 * P - KW) // S + 1
