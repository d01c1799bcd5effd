"""GPU accuracy where fixed-point scales could go wrong.

The product sums in integer fixed point on grids derived from the data of
the call (column maxima times |x| of the active columns).  These cases put
magnitudes where a grid derived from anything else would be too coarse:

* one large weight (|w| in {512, 2048, 16384}) in an inactive column: it must
  not coarsen any grid, since no product uses it;
* the same weight in an active column whose activation is small (the
  smallest active |x|; and with tau < 0, a tiny x_k), so that it meets a
  small factor;
* activations scaled by 1e-3 and 1e-4 (y shrinks with them), with and
  without the outlier weight;
* slice partials beyond the merge's clamp of 4096 (the excess word), with
  rows beyond fp16's range, which must come out infinite.

Each case runs at the benchmark's 4096 x 4096 ws70/as70 problem and at the
28672 x 8192 gate projection of the 70B-shaped configuration, in the
automatic launch shape, and must meet max|y - y*| / (max|y*| + 1e-6) <= 2e-3
against the fp64 definition.
"""
import numpy as np
import pytest

import workloads
from oracle import spmspv as ref

pytestmark = pytest.mark.gpu

TOL = 2e-3


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch, torch.device("cuda:0")


@pytest.fixture(scope="module")
def celty():
    import paper_2608_01536_amd as c
    return c


def _note(msg):
    print(msg, flush=True)


_BASE = {}


def _base(shape):
    """The unmodified problem of a shape (drawn once per module)."""
    if shape not in _BASE:
        if shape == "headline":
            _BASE[shape] = workloads.headline_problem(0)
        else:
            c = workloads.CONFIGS[5]
            proj = next(pp for pp in c["layers"] if pp.name == "gate")
            x = workloads.shared_x(5, 0, 0, proj.x_group, proj.K, c["xdist"])
            _BASE[shape] = workloads.make_problem(5, proj.M, proj.K, c["ws"], 60, c["xdist"], seed=0, layer=0,
                                                  proj=workloads.PROJ_IDS["gate"], x=x)
    return _BASE[shape]


def _run(celty, torch_dev, W, mask, x, tau):
    torch, dev = torch_dev
    R = celty.default_tile_rows(*W.shape)
    Wd = celty.celty_encode(W, mask, R).to_device(dev)
    xt = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(dev)
    y = torch.full((W.shape[0],), 0x7C01, dtype=torch.int16, device=dev)
    ws = celty.new_workspace(Wd, dev)
    celty.celty_spmspv(Wd, xt, tau, y, ws)
    torch.cuda.synchronize()
    assert int(ws.count_nonzero()) == 0
    return y.cpu().numpy().view(np.float16)


def _check(label, y, W, mask, x, tau):
    want = ref.spmspv_dense_fp64(W, mask, x, tau)
    err = ref.rel_error(y.astype(np.float64), want)
    _note(f"  {label}: rel_err={err:.3e} max|y*|={np.max(np.abs(want)):.4g}")
    assert np.all(np.isfinite(y))
    assert err <= TOL, err


def _plant(W, mask, row, col, value):
    W = W.copy()
    mask = mask.copy()
    W[row, col] = np.float16(value)
    mask[row, col] = 1
    return W, mask


@pytest.mark.parametrize("shape", ["headline", "gate28672x8192"])
@pytest.mark.parametrize("w", [512.0, 2048.0, 16384.0])
@pytest.mark.parametrize("where", ["inactive", "active_small_x"])
def test_one_large_weight(celty, torch_dev, shape, w, where):
    p = _base(shape)
    ax = np.abs(p.x.astype(np.float32))
    active = ax > np.float32(p.tau)
    if where == "inactive":
        col = int(np.flatnonzero(~active)[0])
    else:
        cand = np.flatnonzero(active)
        col = int(cand[np.argmin(ax[cand])])       # the smallest active |x|
    row = p.W.shape[0] // 3
    W, mask = _plant(p.W, p.mask, row, col, w)
    _note(f"{shape}: |w|={w:g} in column {col} ({where}, |x|={ax[col]:.4g}, tau={p.tau:.4g})")
    y = _run(celty, torch_dev, W, mask, p.x, p.tau)
    _check(f"{shape} w={w:g} {where}", y, W, mask, p.x, p.tau)


@pytest.mark.parametrize("shape", ["headline", "gate28672x8192"])
@pytest.mark.parametrize("w", [2048.0, 16384.0])
def test_large_weight_meets_a_tiny_activation(celty, torch_dev, shape, w):
    # every column active (tau < 0, weight-only product); the outlier's column
    # carries x = 1e-3, so its product (2 to 16) is of the order of y itself
    p = _base(shape)
    x = p.x.copy()
    col = 5
    x[col] = np.float16(1e-3)
    W, mask = _plant(p.W, p.mask, p.W.shape[0] // 2, col, w)
    _note(f"{shape}: tau<0, |w|={w:g} with x={float(x[col]):.3g}")
    y = _run(celty, torch_dev, W, mask, x, -1.0)
    _check(f"{shape} w={w:g} tiny x", y, W, mask, x, -1.0)


@pytest.mark.parametrize("shape", ["headline", "gate28672x8192"])
@pytest.mark.parametrize("c", [1e-3, 1e-4])
@pytest.mark.parametrize("outlier", [False, True])
def test_scaled_activations(celty, torch_dev, shape, c, outlier):
    p = _base(shape)
    x = (p.x.astype(np.float32) * np.float32(c)).astype(np.float16)
    tau = workloads.tau_for_sparsity(x, p.meta["as_"])
    W, mask = p.W, p.mask
    if outlier:
        inactive = np.flatnonzero(~(np.abs(x.astype(np.float32)) > np.float32(tau)))
        W, mask = _plant(W, mask, 17, int(inactive[-1]), 16384.0)
    _note(f"{shape}: x * {c:g} (tau={tau:.4g}){' + inactive outlier' if outlier else ''}")
    y = _run(celty, torch_dev, W, mask, x, tau)
    _check(f"{shape} x*{c:g}{' outlier' if outlier else ''}", y, W, mask, x, tau)


@pytest.mark.parametrize("R,launch", [(256, None), (256, (32, 2, 1)), (256, (64, 4, 1)), (1024, (64, 2, 1)),
                                      (1024, (96, 4, 1))])
def test_partials_beyond_the_merge_clamp(celty, torch_dev, R, launch):
    # (tiles of 1024 rows on 128 or 256 lanes: each lane merges 4 or 8 rows)
    # weights ~N(0, 4^2) and activations ~Laplace * 200: slice partials of
    # thousands, some beyond the merge's clamp of 4096, whose excess goes
    # through the second merge word; rows beyond fp16's range become inf
    torch, dev = torch_dev
    rng = np.random.default_rng(12)
    M, K = 2000, 600
    W = (rng.standard_normal((M, K)) * 4).astype(np.float16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    x = (rng.laplace(size=K) * 200).astype(np.float16)
    tau = workloads.tau_for_sparsity(x, 40)
    Wd = celty.celty_encode(W, mask, R).to_device(dev)
    xt = torch.from_numpy(x.view(np.int16)).to(dev)
    y = torch.empty(M, dtype=torch.int16, device=dev)
    ws = celty.new_workspace(Wd, dev)
    want = ref.spmspv_dense_fp64(W, mask, x, tau)
    finite = np.abs(want) < 65504
    _note(f"excess path R={R} launch={launch}: {int((~finite).sum())} rows beyond fp16")
    for _ in range(2):   # twice: the excess words must be left zero as well
        celty.celty_spmspv_ex(Wd, xt, tau, y, ws, launch)
        torch.cuda.synchronize()
        assert int(ws.count_nonzero()) == 0
        got = y.cpu().numpy().view(np.float16)
        assert np.all(np.isinf(got[~finite].astype(np.float32)) | (np.abs(want[~finite]) < 65520))
        err = ref.rel_error(got[finite].astype(np.float64), want[finite])   # the finite rows on their own scale
        _note(f"  rel_err={err:.3e}")
        assert err <= TOL, err
