"""A CPU model of the integer arithmetic celty_spmspv documents (include/celty.h).

TEST INFRASTRUCTURE.  It restates, in plain Python/numpy, the arithmetic the
header specifies for the product, so that its error bound can be checked on
the CPU against the exact definition (the oracle's fp64 product) on inputs
chosen to stress the grids:

* the row tile t (R rows) and column slice c (Kc columns) of a launch;
* kept columns of (t, c): active (|x_k| > tau in fp32) and storing at least
  one entry in tile t;
* B = n * max over the n kept columns of colmax[k] * |x_k| (fp32), and the
  slice grid 2^-s with s = clamp(30 - e, -64, 64) where 2^(e-1) <= B < 2^e;
* every product w * x_k, exact, rounded to the nearest multiple of 2^-s
  (ties upward) and summed exactly;
* one slice: y = fp16(fp32(q) * 2^-s);
* several slices: each partial p = q * 2^-s is clamped to +-4096 and put on
  the grid 2^-33 (ties upward); the excess of a clamped partial goes on the
  grid 2^-8; y = fp16(fp32(fine) * 2^-33 + fp32(excess) * 2^-8).

It is not the GPU path (it imports nothing of the library) and not the
oracle (it does not define what y should be: it reproduces how the kernel
rounds).  bound() gives the documented per-row bound on |sum - exact|.
"""
from __future__ import annotations

import math

import numpy as np


def _grid_scale(b: float, top: int) -> int:
    if not b > 0.0 or not math.isfinite(b):
        return 0
    _, e = math.frexp(b)          # b = f * 2^e, 0.5 <= f < 1
    return min(max(top - e, -64), 64)


def _round_half_up(v: float) -> int:
    return int(math.floor(v + 0.5))


def model(W: np.ndarray, mask, x: np.ndarray, tau: float, R: int, Kc: int):
    """Returns (y fp16 [M], sum_before_output_rounding fp64 [M], bound fp64 [M])."""
    M, K = W.shape
    keep = (np.abs(W.astype(np.float32)) > 0) if mask is None else ((np.asarray(mask) != 0) &
                                                                     (W.view(np.uint16) & 0x7FFF != 0))
    Wd = np.where(keep, W.astype(np.float64), 0.0)
    colmax = np.max(np.abs(Wd), axis=0) if M else np.zeros(K)
    xf = x.astype(np.float32)
    active = np.abs(xf) > np.float32(tau)
    T = -(-M // R)
    KC = -(-K // Kc)
    y = np.zeros(M, dtype=np.float16)
    total = np.zeros(M, dtype=np.float64)
    bound = np.zeros(M, dtype=np.float64)
    for t in range(T):
        r0, r1 = t * R, min(M, (t + 1) * R)
        fine = np.zeros(r1 - r0, dtype=object)
        excess = np.zeros(r1 - r0, dtype=object)
        for c in range(KC):
            k0, k1 = c * Kc, min(K, (c + 1) * Kc)
            cols = [k for k in range(k0, k1) if active[k] and keep[r0:r1, k].any()]
            terms = [np.float32(np.float32(abs(float(xf[k]))) * np.float32(colmax[k])) for k in cols]
            b = float(np.float32(len(cols)) * np.float32(max(terms))) if cols else 0.0
            s = _grid_scale(b, 30)
            q = np.zeros(r1 - r0, dtype=object)
            for k in cols:
                xs = float(xf[k]) * 2.0 ** s
                for r in np.flatnonzero(keep[r0:r1, k]):
                    q[r] += _round_half_up(float(Wd[r0 + r, k]) * xs)
            n = np.array([sum(1 for k in cols if keep[r0 + r, k]) for r in range(r1 - r0)], dtype=np.float64)
            bound[r0:r1] += n * 2.0 ** (-s - 1)
            if KC == 1:
                total[r0:r1] = [float(v) * 2.0 ** -s for v in q]
                y[r0:r1] = [np.float16(np.float32(np.float32(float(v)) * np.float32(2.0 ** -s))) for v in q]
                continue
            for r in range(r1 - r0):
                p = int(q[r])
                if abs(p) > 4096 * 2.0 ** s:               # clamped: the excess goes on the grid 2^-8
                    sign = 1 if p > 0 else -1
                    fine[r] += sign * (1 << 45)
                    excess[r] += _round_half_up(p * 2.0 ** (8 - s)) - sign * (1 << 20)
                    bound[r0 + r] += 2.0 ** -9
                else:
                    fine[r] += _round_half_up(p * 2.0 ** (33 - s)) if s > 33 else p * 2 ** (33 - s)
                    bound[r0 + r] += 2.0 ** -34 if s > 33 else 0.0
        if KC > 1:
            for r in range(r1 - r0):
                total[r0 + r] = float(fine[r]) * 2.0 ** -33 + float(excess[r]) * 2.0 ** -8
                v = np.float32(np.float32(float(fine[r])) * np.float32(2.0 ** -33))
                if excess[r]:
                    v = np.float32(v + np.float32(np.float32(float(excess[r])) * np.float32(2.0 ** -8)))
                y[r0 + r] = np.float16(v)
    return y, total, bound
