"""The error bound celty_spmspv documents, checked on a CPU model of its arithmetic.

tests/fixed_point_model.py restates the kernel's rounding (slice grids from
n * max colmax*|x|, ties-upward rounding of each product, the clamped merge
on 2^-33 plus the excess word on 2^-8).  Here, against the exact fp64
definition (the oracle):

* |sum - y*| <= the documented bound, row by row, on every case;
* the fp16 result meets max|y - y*| / (max|y*| + 1e-6) <= 2e-3 on the
  cases that stress the grids: one large weight in an inactive column or in
  an active column with a small activation, activations scaled by 1e-3 and
  1e-4, and magnitudes whose slice partials exceed the merge clamp;
* rows with a single term on the grid are exact.
The GPU suite checks the library itself on the same kinds of inputs.
"""
import numpy as np
import pytest

import workloads
from oracle import spmspv as ref
from tests.fixed_point_model import model

TOL = 2e-3


def _base(seed, M=300, K=257):
    p = workloads.random_small(seed, M, K, ws=70, as_=70)
    return p.W.copy(), p.mask.copy(), p.x.copy(), p.tau


def _check(W, mask, x, tau, R=64, Kc=32):
    y, total, bound = model(W, mask, x, tau, R, Kc)
    want = ref.spmspv_dense_fp64(W, mask, x, tau)
    # the documented bound holds for the integer sum (before the output roundings)
    slack = 1e-12 * (np.max(np.abs(want)) + 1.0)
    assert np.all(np.abs(total - want) <= bound + slack), float(np.max(np.abs(total - want) - bound))
    err = ref.rel_error(y.astype(np.float64), want)
    assert err <= TOL, err
    return err, bound, want


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("R,Kc", [(64, 32), (300, 257), (37, 5)])
def test_plain_inputs(seed, R, Kc):
    W, mask, x, tau = _base(seed)
    _check(W, mask, x, tau, R, Kc)


@pytest.mark.parametrize("w", [512.0, 2048.0, 16384.0])
@pytest.mark.parametrize("where", ["inactive", "active_small_x"])
def test_one_large_weight(w, where):
    W, mask, x, tau = _base(10)
    ax = np.abs(x.astype(np.float32))
    act = ax > np.float32(tau)
    col = int(np.flatnonzero(~act)[0]) if where == "inactive" else int(np.flatnonzero(act)[np.argmin(ax[act])])
    W[100, col] = np.float16(w)
    mask[100, col] = 1
    err, bound, want = _check(W, mask, x, tau)
    if where == "inactive":
        # no product uses the outlier: the bound stays at the level of the plain input
        W2, m2, _, _ = _base(10)
        _, b2, _ = model(W2, m2, x, tau, 64, 32)
        assert np.max(bound) <= 2.0 * np.max(b2)


@pytest.mark.parametrize("c", [1e-3, 1e-4])
@pytest.mark.parametrize("outlier", [False, True])
def test_scaled_activations(c, outlier):
    W, mask, x, tau = _base(11)
    x = (x.astype(np.float32) * np.float32(c)).astype(np.float16)
    tau = workloads.tau_for_sparsity(x, 70)
    if outlier:
        inact = np.flatnonzero(~(np.abs(x.astype(np.float32)) > np.float32(tau)))
        W[5, int(inact[-1])] = np.float16(16384)
        mask[5, int(inact[-1])] = 1
    _check(W, mask, x, tau)


def test_partials_beyond_the_merge_clamp():
    # weights ~N(0, 4^2) and activations ~Laplace * 200: slice partials of
    # thousands, some beyond 4096, go through the excess word
    rng = np.random.default_rng(12)
    M, K = 200, 300
    W = (rng.standard_normal((M, K)) * 4).astype(np.float16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    x = (rng.laplace(size=K) * 200).astype(np.float16)
    tau = workloads.tau_for_sparsity(x, 40)
    y, total, bound = model(W, mask, x, tau, 64, 32)
    assert np.any(bound >= 2.0 ** -9)                     # at least one slice took the excess path
    want = ref.spmspv_dense_fp64(W, mask, x, tau)
    finite = np.abs(want) < 65504
    assert np.all(np.abs(total - want) <= bound + 1e-9 * np.max(np.abs(want)))
    assert np.all(np.isinf(y[~finite].astype(np.float32)) | (np.abs(want[~finite]) < 65520))
    err = ref.rel_error(y[finite].astype(np.float64), want[finite])
    assert err <= TOL, err


def test_single_terms_on_the_grid_are_exact():
    K = 200
    I = np.eye(K, dtype=np.float16)
    x = (np.round(np.random.default_rng(13).laplace(size=K) * 64) / 64).astype(np.float16)
    for tau, Kc in ((0.5, 32), (-1.0, 7), (0.5, 200)):
        y, _, _ = model(I, None, x, tau, 64, Kc)
        want = np.where(np.abs(x.astype(np.float32)) > tau, x, np.float16(0)).astype(np.float16)
        want = np.where(want == 0, np.float16(0), want).astype(np.float16)
        assert np.array_equal(y.view(np.uint16), want.view(np.uint16))
