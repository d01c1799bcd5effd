"""Reference products for the dual-sparse SpMSpV (Sections 2.1, 3.1, 3.3, 5).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition (exact target).  With the active set A = {k : |x_k| > tau}
(runtime magnitude thresholding, Sections 1 and 2.1; the strict ">" and the
fp32 comparison of the exact fp16 magnitude are readings of an operator the
paper does not print; NaN activations are never active), the product is

    y*[r] = sum_{k in A} W[r, k] * Mask[r, k] * x_k        for every row r < M,

with W and x taken as their exact fp16 values and the sum in fp64.  The
method (column skipping for inactive x_k, Section 3.1; pruned weights are
never stored, Section 3.2) reaches the same value; its only deviations are
the fp32 accumulation of the fused multiply-adds (Section 5) and the final
rounding of y to fp16.

Activations must be finite: an infinite x_k makes the definition ill-posed
(0 * inf for pruned weights), and such inputs are outside the domain.

Parity status
-------------
select_active          pinned: numpy predicate on tiny hand cases + invariants.
spmspv_dense_fp64      pinned: brute force (tiny), CSC path (1e-12), closed
                       forms (one-hot x, identity pattern, all inactive, tau<0
                       == textbook dense GEMV), linearity, sign and scaling.
spmspv_csc_fp64        pinned: same pins, built from (W, Mask) directly.
spmspv_bruteforce      pinned: hand-computed 2x3 example.
spmspv_rlc_fp64        pinned: equals spmspv_dense_fp64 to 1e-12 on random cases.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

from . import rlc as _rlc


def active_flags(x: np.ndarray, tau: float) -> np.ndarray:
    """|x_k| > tau, compared in fp32 on the exact fp16 magnitude."""
    return np.abs(np.asarray(x).astype(np.float32)) > np.float32(tau)


def select_active(x: np.ndarray, tau: float) -> np.ndarray:
    """Ascending int32 indices of the active columns."""
    return np.flatnonzero(active_flags(x, tau)).astype(np.int32)


def _masked_weights_fp64(W: np.ndarray, mask) -> np.ndarray:
    Wd = np.asarray(W).astype(np.float64)
    if mask is None:
        return Wd
    return np.where(np.asarray(mask) != 0, Wd, 0.0)


def spmspv_dense_fp64(W: np.ndarray, mask, x: np.ndarray, tau: float) -> np.ndarray:
    """(O1) dense fp64 masked GEMV over the thresholded activation vector."""
    a = active_flags(x, tau)
    xa = np.where(a, np.asarray(x).astype(np.float64), 0.0)
    return _masked_weights_fp64(W, mask) @ xa


def spmspv_csc_fp64(W: np.ndarray, mask, x: np.ndarray, tau: float) -> np.ndarray:
    """(O2) fp64 CSC SpMSpV: only the kept entries of the active columns.

    The CSC matrix is built straight from (W, Mask); it does not go through
    the RLC-CSC arrays.
    """
    M, K = W.shape
    keep = np.ones((M, K), dtype=bool) if mask is None else (np.asarray(mask) != 0)
    r, c = np.nonzero(keep)
    vals = np.asarray(W)[r, c].astype(np.float64)
    A = sp.csc_matrix((vals, (r, c)), shape=(M, K))
    act = select_active(x, tau)
    if act.size == 0:
        return np.zeros(M, dtype=np.float64)
    return np.asarray(A[:, act] @ np.asarray(x)[act].astype(np.float64)).reshape(M)


def spmspv_bruteforce(W: np.ndarray, mask, x: np.ndarray, tau: float) -> np.ndarray:
    """Triple-loop definition for tiny shapes (pure Python floats)."""
    M, K = W.shape
    y = [0.0] * M
    for k in range(K):
        xk = float(np.float32(x[k]))
        if not abs(xk) > float(np.float32(tau)):
            continue
        for r in range(M):
            if mask is not None and mask[r, k] == 0:
                continue
            y[r] += float(W[r, k]) * xk
    return np.array(y, dtype=np.float64)


def spmspv_rlc_fp64(enc: "_rlc.RlcCsc", x: np.ndarray, tau: float) -> np.ndarray:
    """The kernel's walk in fp64: skip inactive columns, fetch each segment of
    an active column, reconstruct rows (prefix of runs + ordinal) and
    scatter-accumulate value * x_k.  Pins the storage format against O1."""
    y = np.zeros(enc.M, dtype=np.float64)
    xs = np.asarray(x)
    for k in select_active(xs, tau):
        xk = float(xs[k])
        for t in range(enc.T):
            s = t * enc.K + int(k)
            if enc.gptr[s] == enc.gptr[s + 1]:
                continue
            rows, vals = _rlc.segment_rows(enc, s)
            v = vals.view(np.float16).astype(np.float64)
            real = v != 0
            np.add.at(y, rows[real], v[real] * xk)
    return y


def rel_error(y, y_ref) -> float:
    """max_r |y - y*| / (max_r |y*| + 1e-6), the acceptance measure."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    return float(np.max(np.abs(y - y_ref)) / (np.max(np.abs(y_ref)) + 1e-6)) if y.size else 0.0
