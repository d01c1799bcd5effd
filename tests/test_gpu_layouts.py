"""GPU parity of the product's other variants, through the C ABI.

* the 16-bit row layout (decode-free: rows loaded, not reconstructed);
* the lane-interleaved layout (Section 4.2's offline interleave; chunk-aligned
  passes and per-slot scans);
* the XOR-swizzled LDS tile (rows in a permuted slot order).

Each variant forms the same exact products on the same grids and sums them
exactly in integers, so its y must equal the RLC kernel's y bit for bit; it
is also checked against the fp64 definition (the oracle) within 2e-3.  Shapes
cover several tiles and a ragged last tile, one and several column slices,
segments of more than 64 groups (several interleave chunks, wavefront ranges
that start inside a segment), 2 to 16 wavefronts, tau < 0, NaN activations,
an all-inactive x, the identity pattern (single-term rows, bit-exact
against x itself), and the full-size 28672 x 8192 and 13824 x 5120 problems
in the automatic launch shape.
"""
import numpy as np
import pytest

import workloads
from oracle import spmspv as ref

pytestmark = pytest.mark.gpu

TOL = 2e-3
VARIANTS = ["rows16", "interleaved", "swizzle"]


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


def _layout(celty, variant):
    return {"rows16": celty.LAYOUT_ROWS16, "interleaved": celty.LAYOUT_INTERLEAVED}.get(variant, celty.LAYOUT_RLC)


def _run(celty, torch_dev, enc, x, tau, launch):
    torch, dev = torch_dev
    Wd = enc.to_device(dev)
    xt = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(dev)
    y = torch.full((enc.M,), 0x7C01, dtype=torch.int16, device=dev)   # NaN bits
    ws = celty.new_workspace(Wd, dev)
    for _ in range(2):   # twice: the merge words must be left zero
        celty.celty_spmspv_ex(Wd, xt, tau, y, ws, launch)
        torch.cuda.synchronize()
        assert int(ws.count_nonzero()) == 0
    return y.cpu().numpy().view(np.uint16)


def _both(celty, torch_dev, variant, W, mask, x, tau, R, cols=0, waves=0):
    """(variant's y bits, RLC kernel's y bits) for the same launch shape."""
    enc = celty.celty_encode(W, mask, R, layout=_layout(celty, variant))
    base = celty.celty_encode(W, mask, R)
    swz = 1 if variant == "swizzle" else 0
    y = _run(celty, torch_dev, enc, x, tau, (cols, waves, 1, swz))
    y0 = _run(celty, torch_dev, base, x, tau, (cols, waves, 1, 0))
    return y, y0


CASES = [
    # label, M, K, ws, as, R, cols, waves
    ("headline", 4096, 4096, 70, 70, 512, 0, 0),
    ("ragged", 1000, 777, 60, 50, 256, 0, 0),
    ("one_slice", 700, 300, 50, 50, 256, 512, 8),
    ("long_segments", 4096, 192, 0, 0, 2048, 64, 16),
    ("long_segments_8w", 2100, 130, 10, 20, 1024, 130, 8),
    ("waves2", 1500, 900, 70, 40, 512, 128, 2),
    ("waves4", 1500, 900, 50, 50, 512, 64, 4),
    ("tall_16w", 8192, 1024, 50, 60, 1024, 0, 0),
    ("r1", 37, 50, 30, 30, 1, 0, 0),
    ("eight_cols_per_lane", 3000, 4096, 60, 50, 512, 1024, 2),
    ("long_ranges_2w", 4096, 96, 0, 0, 2048, 96, 2),
]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("label,M,K,ws,as_,R,cols,waves", CASES)
def test_variant_matches_rlc_kernel_and_oracle(celty, torch_dev, variant, label, M, K, ws, as_, R, cols, waves):
    _note(f"{variant} {label}: {M}x{K} ws{ws} as{as_} R={R} launch=({cols},{waves})")
    p = workloads.make_problem(2, M, K, ws, as_, "laplace", seed=M + K + ws, proj=workloads.PROJ_IDS["w"])
    y, y0 = _both(celty, torch_dev, variant, p.W, p.mask, p.x, p.tau, R, cols, waves)
    assert np.array_equal(y, y0), f"{int(np.count_nonzero(y != y0))} rows differ from the RLC kernel"
    want = ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)
    err = ref.rel_error(y.view(np.float16).astype(np.float64), want)
    _note(f"  rel_err={err:.3e}")
    assert err <= TOL, err


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("M,K,ws,as_", [(28672, 8192, 50, 40), (13824, 5120, 60, 60)])
def test_variant_full_size_in_the_automatic_shape(celty, torch_dev, variant, M, K, ws, as_):
    # the variant study's largest problems, in the launch shape bench.py uses
    _note(f"{variant} full size {M}x{K} ws{ws} as{as_}")
    p = workloads.make_problem(2, M, K, ws, as_, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
    R = celty.default_tile_rows(M, K)
    y, y0 = _both(celty, torch_dev, variant, p.W, p.mask, p.x, p.tau, R)
    assert np.array_equal(y, y0), f"{int(np.count_nonzero(y != y0))} rows differ from the RLC kernel"
    want = ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)
    err = ref.rel_error(y.view(np.float16).astype(np.float64), want)
    _note(f"  rel_err={err:.3e}")
    assert err <= TOL, err


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("mode", ["tau_negative", "nan_x", "all_inactive"])
def test_variant_special_activations(celty, torch_dev, variant, mode):
    _note(f"{variant} {mode}")
    p = workloads.make_problem(2, 1200, 1000, 50, 50, "laplace", seed=7, proj=workloads.PROJ_IDS["w"])
    x, tau = p.x.copy(), p.tau
    if mode == "tau_negative":
        tau = -1.0
    elif mode == "nan_x":
        x[::7] = np.float16(np.nan)
    else:
        tau = float(np.max(np.abs(x.astype(np.float32)))) + 1.0
    y, y0 = _both(celty, torch_dev, variant, p.W, p.mask, x, tau, 256)
    assert np.array_equal(y, y0)
    if mode == "all_inactive":
        assert np.all(y == 0)
    else:
        want = ref.spmspv_dense_fp64(p.W, p.mask, x, tau)
        assert ref.rel_error(y.view(np.float16).astype(np.float64), want) <= TOL


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("K,R,launch", [(4096, 512, (0, 0)), (1000, 256, (1000, 2)), (4096, 1024, (4096, 16)),
                                        (300, 64, (64, 4))])
def test_variant_identity_is_exact(celty, torch_dev, variant, K, R, launch):
    # y = x on the active columns: single-term rows, bit-exact
    _note(f"{variant} identity K={K} R={R} launch={launch}")
    rng = np.random.default_rng(K)
    x = rng.laplace(size=K).astype(np.float16)
    tau = float(np.quantile(np.abs(x.astype(np.float32)), 0.5))
    I = np.eye(K, dtype=np.float16)
    enc = celty.celty_encode(I, None, R, layout=_layout(celty, variant))
    y = _run(celty, torch_dev, enc, x, tau, (launch[0], launch[1], 1, 1 if variant == "swizzle" else 0))
    want = np.where(np.abs(x.astype(np.float32)) > tau, x, np.float16(0)).astype(np.float16)
    assert np.array_equal(y.view(np.float16) == 0, want == 0)
    nz = want != 0
    assert np.array_equal(y[nz], want.view(np.uint16)[nz])


def test_variants_are_refused_where_unsupported(celty, torch_dev):
    torch, dev = torch_dev
    p = workloads.random_small(3, 300, 200, ws=50, as_=50)
    r16 = celty.celty_encode(p.W, p.mask, 64, layout=celty.LAYOUT_ROWS16).to_device(dev)
    xt = torch.from_numpy(p.x.view(np.int16)).to(dev)
    y = torch.empty(300, dtype=torch.int16, device=dev)
    ws = celty.new_workspace(r16, dev)
    for launch in [(0, 0, 2, 0), (0, 0, 0, 1)]:   # two groups per lane; swizzle with another layout
        with pytest.raises(celty.CeltyError):
            celty.celty_spmspv_ex(r16, xt, p.tau, y, ws, launch)
    base = celty.celty_encode(p.W, p.mask, 64).to_device(dev)
    with pytest.raises(celty.CeltyError):
        celty.celty_spmspv_ex(base, xt, p.tau, y, ws, (0, 0, 2, 1))
    # several products in one launch: RLC with the plain tile only
    y2 = torch.empty(300, dtype=torch.int16, device=dev)
    ws2 = celty.new_batch_workspace([r16, base], dev)
    with pytest.raises(celty.CeltyError):
        celty.celty_spmspv_batch([r16, base], [xt, xt], [p.tau, p.tau], [y, y2], ws2)
