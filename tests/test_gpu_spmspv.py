"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

* selection: the active index list is bit-exact;
* y: max|y - y*| / (max|y*| + 1e-6) <= 2e-3 with y* the fp64 definition;
* exact special cases (single-term rows): one-hot x, identity pattern,
  all-inactive x (every row +0), empty matrix;
* edge shapes: M < R, M % R != 0, K = 1, K not a multiple of 64, R = 1;
* every launch shape gives the same answer within tolerance;
* the workspace is left zero-filled by every call, also by calls queued
  back to back with no host synchronisation; y is fully overwritten;
* full-size runs of all five benchmark configurations, and of the paper's
  kernel shapes at 30/50/70 % dual sparsity, in the launch shape the
  benchmark uses.
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


def _run(celty, torch_dev, W, mask, x, tau, R, launch=None, check_ws=True, enc=None):
    torch, dev = torch_dev
    if enc is None:
        enc = celty.celty_encode(W, mask, R)
    Wd = enc.to_device(dev)
    xt = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(dev)
    y = torch.full((W.shape[0],), 0x7C01, dtype=torch.int16, device=dev)   # NaN bits
    ws = celty.new_workspace(Wd, dev)
    if launch is None:
        celty.celty_spmspv(Wd, xt, tau, y, ws)
    else:
        celty.celty_spmspv_ex(Wd, xt, tau, y, ws, launch)
    torch.cuda.synchronize()
    if check_ws:
        assert int(ws.count_nonzero()) == 0, "workspace not left zero-filled"
    return y.cpu().numpy().view(np.float16)


def _check(y, W, mask, x, tau):
    want = ref.spmspv_dense_fp64(W, mask, x, tau)
    err = ref.rel_error(y.astype(np.float64), want)
    assert np.all(np.isfinite(y)), "y has non-finite rows"
    assert err <= TOL, err
    return err


# --------------------------------------------------------------------------
# selection
# --------------------------------------------------------------------------
@pytest.mark.parametrize("K", [1, 63, 64, 65, 1000, 1024, 1025, 4096, 11008, 28672, 32767, 32768, 32769,
                               65600, 100000])
@pytest.mark.parametrize("mode", ["median", "neg", "zero", "max", "nan"])
def test_select_bit_exact(celty, torch_dev, K, mode):
    torch, dev = torch_dev
    _note(f"select K={K} mode={mode}")
    rng = np.random.default_rng(K)
    x = rng.laplace(size=K).astype(np.float16)
    x[rng.random(K) < 0.1] = 0
    if mode == "nan":
        x[rng.random(K) < 0.05] = np.nan
    tau = {"median": workloads.tau_for_sparsity(x, 50), "neg": -1.0, "zero": 0.0,
           "max": float(np.nanmax(np.abs(x.astype(np.float32)))), "nan": 0.3}[mode]
    xt = torch.from_numpy(x.view(np.int16)).to(dev)
    idx = torch.full((K,), -7, dtype=torch.int32, device=dev)
    cnt = torch.zeros(1, dtype=torch.int32, device=dev)
    celty.celty_select(xt, tau, idx, cnt)
    torch.cuda.synchronize()
    want = ref.select_active(x, tau)
    n = int(cnt.item())
    assert n == want.size
    got = idx.cpu().numpy()
    assert np.array_equal(got[:n], want)
    assert np.all(got[n:] == -7), "selection wrote past the active count"


@pytest.mark.parametrize("K", [1, 2, 1025, 28672, 32769])
def test_select_x_only_two_byte_aligned(celty, torch_dev, K):
    # x one element into a buffer: 2-byte but not 4-byte aligned (the path
    # without word loads)
    torch, dev = torch_dev
    _note(f"select misaligned K={K}")
    rng = np.random.default_rng(K + 7)
    x = rng.laplace(size=K + 1).astype(np.float16)
    tau = workloads.tau_for_sparsity(x[1:], 50)
    buf = torch.from_numpy(x.view(np.int16)).to(dev)
    xt = buf[1:]
    assert xt.data_ptr() % 4 == 2
    idx = torch.full((K,), -7, dtype=torch.int32, device=dev)
    cnt = torch.zeros(1, dtype=torch.int32, device=dev)
    celty.celty_select(xt, tau, idx, cnt)
    torch.cuda.synchronize()
    want = ref.select_active(x[1:], tau)
    n = int(cnt.item())
    got = idx.cpu().numpy()
    assert n == want.size and np.array_equal(got[:n], want) and np.all(got[n:] == -7)


# --------------------------------------------------------------------------
# small fuzz and edge shapes
# --------------------------------------------------------------------------
FUZZ = [(1, 1, 1), (1, 5, 8), (5, 1, 8), (3, 200, 1), (100, 100, 16), (257, 129, 256), (255, 1000, 256),
        (700, 513, 256), (1024, 64, 1024), (1500, 300, 512), (2049, 777, 128), (64, 4100, 64)]


@pytest.mark.parametrize("M,K,R", FUZZ)
@pytest.mark.parametrize("ws,as_", [(0, 0), (50, 50), (90, 30), (30, 90)])
@pytest.mark.parametrize("groups", [1, 4])
def test_spmspv_fuzz(celty, torch_dev, M, K, R, ws, as_, groups):
    _note(f"fuzz M={M} K={K} R={R} ws={ws} as={as_} groups={groups}")
    p = workloads.random_small(M * 13 + K * 7 + R + ws, M, K, ws=ws, as_=as_, zero_weights=3)
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, R, launch=(0, 0, groups))
    _check(y, p.W, p.mask, p.x, p.tau)


def _random_plan_cases(n=40, seed=2608):
    """Seeded shapes between the fixed lists: log-uniform M and K (at most
    3e7 entries, so that the oracle stays fast), the library's tile height or
    a random power of two, and sparsities from 30 to 85 %."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        M = int(np.exp(rng.uniform(np.log(48), np.log(30000))))
        K = int(np.exp(rng.uniform(np.log(48), np.log(30000))))
        if M * K > 30_000_000:
            continue
        R = int(2 ** rng.integers(6, 13)) if rng.random() < 0.5 else 0
        ws, as_ = (int(v) for v in rng.integers(30, 86, size=2))
        cases.append((M, K, R, ws, as_))
    return cases


@pytest.mark.parametrize("M,K,R,ws,as_", _random_plan_cases())
def test_automatic_plan_random_shapes(celty, torch_dev, M, K, R, ws, as_):
    """The automatic launch (workgroup count, slice width, wavefronts, ring
    depth) on seeded shapes that no other test names, against the oracle."""
    R = R or celty.default_tile_rows(M, K)
    _note(f"auto plan M={M} K={K} R={R} ws={ws} as={as_}")
    p = workloads.random_small(M + 3 * K + R, M, K, ws=ws, as_=as_)
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, R)
    _check(y, p.W, p.mask, p.x, p.tau)


# cols / (64 * waves) covers 1 to 8 columns per lane in the selection
@pytest.mark.parametrize("launch", [(40, 2, 1), (41, 4, 2), (64, 2, 4), (64, 4, 1), (128, 8, 2), (256, 16, 4),
                                    (1000, 4, 1), (1000, 4, 4), (2048, 4, 2), (4096, 16, 1), (700, 8, 4),
                                    (1024, 2, 4), (129, 2, 1), (4096, 8, 1)])
def test_launch_shapes_agree(celty, torch_dev, launch):
    _note(f"launch shape {launch}")
    p = workloads.random_small(77, 3000, 2500, ws=60, as_=50)
    enc = celty.celty_encode(p.W, p.mask, 256)
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, 256, launch=launch, enc=enc)
    _check(y, p.W, p.mask, p.x, p.tau)


def test_one_hot_returns_column_exactly(celty, torch_dev):
    rng = np.random.default_rng(3)
    M, K = 3000, 700
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    enc = celty.celty_encode(W, mask, 256)
    for k in (0, 1, 350, K - 1):
        _note(f"one-hot k={k}")
        x = np.zeros(K, dtype=np.float16)
        x[k] = 1
        y = _run(celty, torch_dev, W, mask, x, 0.5, 256, enc=enc)
        want = np.where(mask[:, k] != 0, W[:, k], np.float16(0)).astype(np.float16)
        assert np.array_equal(y.view(np.uint16), want.view(np.uint16))


def test_identity_pattern_returns_active_x(celty, torch_dev):
    K = 2000
    I = np.eye(K, dtype=np.float16)
    x = np.random.default_rng(4).laplace(size=K).astype(np.float16)
    tau = 0.8
    _note("identity pattern")
    y = _run(celty, torch_dev, I, None, x, tau, 128)
    want = np.where(np.abs(x.astype(np.float32)) > tau, x, np.float16(0)).astype(np.float16)
    assert np.array_equal(y.view(np.uint16), want.view(np.uint16))


def test_all_inactive_gives_positive_zero(celty, torch_dev):
    p = workloads.random_small(9, 1000, 900, ws=50, as_=50)
    tau = float(np.max(np.abs(p.x.astype(np.float32))))
    _note("all inactive")
    y = _run(celty, torch_dev, p.W, p.mask, p.x, tau, 256)
    assert np.all(y.view(np.uint16) == 0)


def test_empty_matrix(celty, torch_dev):
    W = np.zeros((300, 200), dtype=np.float16)
    x = np.ones(200, dtype=np.float16)
    _note("empty matrix")
    y = _run(celty, torch_dev, W, None, x, -1.0, 64)
    assert np.all(y.view(np.uint16) == 0)


def test_short_tensors_are_rejected_before_any_launch(celty, torch_dev):
    """x shorter than K or y shorter than M raise in the binding; y keeps its
    contents (nothing was launched) and a correct call afterwards still works."""
    torch, dev = torch_dev
    p = workloads.random_small(21, 300, 200, ws=50, as_=50)
    Wd = celty.celty_encode(p.W, p.mask, 64).to_device(dev)
    ws = celty.new_workspace(Wd, dev)
    xt = torch.from_numpy(np.ascontiguousarray(p.x).view(np.int16)).to(dev)
    y = torch.full((300,), 0x7C01, dtype=torch.int16, device=dev)
    _note("short x / short y rejected")
    with pytest.raises(ValueError):
        celty.celty_spmspv(Wd, xt[:199], p.tau, y, ws)
    with pytest.raises(ValueError):
        celty.celty_spmspv(Wd, xt, p.tau, y[:299], ws)
    with pytest.raises(ValueError):
        celty.celty_spmspv_batch([Wd, Wd], [xt, xt[:150]], [p.tau, p.tau], [y, y], celty.new_batch_workspace([Wd, Wd]))
    idx = torch.empty(199, dtype=torch.int32, device=dev)
    with pytest.raises(ValueError):
        celty.celty_select(xt, p.tau, idx, torch.empty(1, dtype=torch.int32, device=dev))
    torch.cuda.synchronize()
    assert bool((y == 0x7C01).all())
    celty.celty_spmspv(Wd, xt, p.tau, y, ws)
    torch.cuda.synchronize()
    got = y.cpu().numpy().view(np.float16).astype(np.float64)
    assert ref.rel_error(got, ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)) <= TOL


def test_weight_only_full_mask_is_dense_gemv(celty, torch_dev):
    rng = np.random.default_rng(12)
    M, K = 1024, 768
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float16)
    x = rng.standard_normal(K).astype(np.float16)
    _note("tau<0 full mask")
    y = _run(celty, torch_dev, W, None, x, -1.0, 256)
    want = W.astype(np.float64) @ x.astype(np.float64)
    assert ref.rel_error(y.astype(np.float64), want) <= TOL


def test_repeated_calls_share_a_workspace(celty, torch_dev):
    torch, dev = torch_dev
    p = workloads.random_small(10, 2500, 3000, ws=50, as_=50)
    enc = celty.celty_encode(p.W, p.mask, 256)
    Wd = enc.to_device(dev)
    ws = celty.new_workspace(Wd, dev)
    want = ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)
    xt = torch.from_numpy(p.x.view(np.int16)).to(dev)
    outs = []
    _note("repeated calls")
    for i in range(5):
        y = torch.empty(p.W.shape[0], dtype=torch.int16, device=dev)
        celty.celty_spmspv(Wd, xt, p.tau, y, ws)
        outs.append(y)
    torch.cuda.synchronize()
    assert int(ws.count_nonzero()) == 0
    for y in outs:
        assert ref.rel_error(y.cpu().numpy().view(np.float16).astype(np.float64), want) <= TOL


@pytest.mark.parametrize("M,K,ws,as_", [(4096, 4096, 70, 70), (8192, 8192, 50, 60)])
def test_queued_calls_share_a_workspace(celty, torch_dev, M, K, ws, as_):
    # calls enqueued while the GPU is still busy, so they run back to back
    # with no host synchronisation between them: each must find the merge
    # words the previous one left zero, and its y must equal a lone call's
    # bit for bit (the sums are exact integers, whatever the slices' order)
    torch, dev = torch_dev
    p = workloads.make_problem(2, M, K, ws, as_, "laplace", seed=3, proj=workloads.PROJ_IDS["w"])
    enc = celty.celty_encode(p.W, p.mask, celty.default_tile_rows(M, K))
    Wd = enc.to_device(dev)
    copies = [Wd, Wd.clone_to()]
    xt = torch.from_numpy(p.x.view(np.int16)).to(dev)
    ws_ = celty.new_workspace(Wd, dev)
    y0 = torch.empty(M, dtype=torch.int16, device=dev)
    celty.celty_spmspv(Wd, xt, p.tau, y0, ws_)
    torch.cuda.synchronize()
    ys = [torch.full((M,), 0x7C01, dtype=torch.int16, device=dev) for _ in range(32)]
    _note(f"queued calls {M}x{K} ws{ws} as{as_}")
    torch.cuda._sleep(2000000)   # about 1 ms of device time: the host enqueues every call meanwhile
    for i, y in enumerate(ys):
        celty.celty_spmspv(copies[i % 2], xt, p.tau, y, ws_)
    torch.cuda.synchronize()
    assert int(ws_.count_nonzero()) == 0
    assert all(torch.equal(y, y0) for y in ys)
    _check(y0.cpu().numpy().view(np.float16), p.W, p.mask, p.x, p.tau)


# --------------------------------------------------------------------------
# full-size benchmark configurations
# --------------------------------------------------------------------------
def _full(celty, torch_dev, p, label):
    from paper_2608_01536_amd import default_tile_rows
    R = default_tile_rows(p.W.shape[0], p.W.shape[1])
    _note(f"full {label} M={p.W.shape[0]} K={p.W.shape[1]} R={R}")
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, R)
    err = _check(y, p.W, p.mask, p.x, p.tau)
    _note(f"  rel_err={err:.3e}")
    return err


def test_config1(celty, torch_dev):
    c = workloads.CONFIGS[1]
    p = workloads.make_problem(1, 4096, 4096, c["ws"], c["as_"], c["xdist"], seed=0, proj=7)
    _full(celty, torch_dev, p, "config1")


@pytest.mark.parametrize("ws", [30, 50, 70])
@pytest.mark.parametrize("as_", [30, 50, 70])
def test_config2_sweep_seed0(celty, torch_dev, ws, as_):
    p = workloads.make_problem(2, 4096, 4096, ws, as_, "laplace", seed=0, proj=7)
    _full(celty, torch_dev, p, f"config2 ws{ws} as{as_}")


@pytest.mark.parametrize("seed", [0, 1, 2, 3, 4])
def test_config2_headline_seeds(celty, torch_dev, seed):
    p = workloads.headline_problem(seed)
    _full(celty, torch_dev, p, f"headline seed{seed}")


def test_config3_layer(celty, torch_dev):
    for p in workloads.layer_problems(3, 0, 0):
        _full(celty, torch_dev, p, f"config3 {p.meta['proj_name']}")


@pytest.mark.parametrize("layer", [0, 39])
def test_config4_layer(celty, torch_dev, layer):
    for p in workloads.layer_problems(4, 0, layer):
        _full(celty, torch_dev, p, f"config4 layer{layer} {p.meta['proj_name']}")


@pytest.mark.parametrize("as_", [40, 60, 80])
def test_config5_projections(celty, torch_dev, as_):
    # one of each distinct 70B shape: q (8192^2), k (1024x8192), gate (28672x8192), down (8192x28672)
    c = workloads.CONFIGS[5]
    for name in ("q", "k", "gate", "down"):
        proj = next(pp for pp in c["layers"] if pp.name == name)
        x = workloads.shared_x(5, 0, 0, proj.x_group, proj.K, c["xdist"])
        p = workloads.make_problem(5, proj.M, proj.K, c["ws"], as_, c["xdist"], seed=0, layer=0,
                                   proj=workloads.PROJ_IDS[name], x=x)
        _full(celty, torch_dev, p, f"config5 as{as_} {name}")


@pytest.mark.parametrize("pct", [30, 50, 70])
@pytest.mark.parametrize("M,K", [(4096, 11008), (5120, 5120), (5120, 13824), (7168, 7168), (7168, 28672)])
def test_paper_kernel_shapes(celty, torch_dev, M, K, pct):
    # the paper's kernel workloads (Section 5) at weight = activation sparsity,
    # the problems bench.py --paper-shapes times (4096^2 is config 2 above)
    p = workloads.make_problem(2, M, K, pct, pct, "laplace", seed=0, proj=workloads.PROJ_IDS["w"])
    _full(celty, torch_dev, p, f"paper shape {M}x{K} dual{pct}")


@pytest.mark.parametrize("M,K,R,ws,launch", [
    (4096, 40, 4096, 5, (40, 16, 1)),     # segments of ~490 groups: cuts more than 256 groups in
    (4096, 40, 4096, 5, (40, 16, 4)),
    (4096, 40, 4096, 5, (40, 2, 2)),
    (8192, 3, 8192, 2, (3, 16, 1)),       # three segments of ~1000 groups, 16 ranges
    (3000, 1, 3000, 10, (1, 16, 1)),      # one segment shared by every wavefront
    (64, 2, 64, 50, (2, 16, 1)),          # fewer groups than wavefronts: empty ranges
    (2000, 700, 1024, 20, (700, 8, 1)),   # several columns per lane, long segments
])
def test_wavefront_ranges_cut_inside_segments(celty, torch_dev, M, K, R, ws, launch):
    # a workgroup's groups are split into equal ranges, one per wavefront, so
    # a range can begin deep inside a segment and must start at the row that
    # the segment's earlier groups reach
    _note(f"ranges inside segments M={M} K={K} R={R} ws={ws} launch={launch}")
    p = workloads.random_small(871 + K, M, K, ws=ws, as_=0)
    y = _run(celty, torch_dev, p.W, p.mask, p.x, -1.0, R, launch=launch)
    _check(y, p.W, p.mask, p.x, -1.0)


@pytest.mark.parametrize("M,R,launch", [
    (22016, 2048, None),             # last tile 1536 rows: two rows per lane, the second past the tile for half
    (2 * 4096 + 3000, 4096, (256, 16, 1)),   # last tile 3000 rows: four rows per lane
    (5 * 2048 + 1025, 2048, (128, 16, 2)),
    (3 * 1024 + 700, 1024, (128, 8, 1)),
])
def test_partial_last_tile_taller_than_the_workgroup(celty, torch_dev, M, R, launch):
    # the merge takes several rows per lane; rows past a partial last tile must
    # neither change y nor leave the workspace dirty
    p = workloads.make_problem(2, M, 4096, 50, 50, "laplace", seed=3, proj=workloads.PROJ_IDS["w"])
    _note(f"partial tile M={M} R={R} launch={launch}")
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, R, launch=launch)
    _check(y, p.W, p.mask, p.x, p.tau)


@pytest.mark.parametrize("config,group", [(3, ("q", "k", "v")), (3, ("gate", "up")), (5, ("q", "k", "v"))])
def test_stacked_projections(celty, torch_dev, config, group):
    # projections reading one x stacked into one taller matrix at encode time
    # (the fused decode-step schedule): each block of y matches its own oracle
    probs = {p.meta["proj_name"]: p for p in workloads.layer_problems(config, 0, 0, as_=60 if config == 5 else None)}
    ps = [probs[n] for n in group]
    W = np.concatenate([p.W for p in ps])
    mask = np.concatenate([p.mask for p in ps])
    from paper_2608_01536_amd import default_tile_rows
    R = default_tile_rows(*W.shape)
    _note(f"stacked config{config} {group} {W.shape} R={R}")
    y = _run(celty, torch_dev, W, mask, ps[0].x, ps[0].tau, R)
    r0 = 0
    for p in ps:
        m = p.W.shape[0]
        _check(y[r0:r0 + m], p.W, p.mask, p.x, p.tau)
        r0 += m


@pytest.mark.parametrize("M,K,sigma", [(4096, 4096, 1.0), (4096, 11008, 1.0), (11008, 4096, 2.0),
                                         (28672, 8192, 1.0)])
def test_outlier_features(celty, torch_dev, M, K, sigma):
    # per-feature scales shared by W's columns and x: column densities from ~0
    # to ~95 %, magnitudes over several decades inside one column slice
    p = workloads.outlier_feature_problem(M, K, 50, 50, sigma)
    _full(celty, torch_dev, p, f"outlier features {M}x{K} sigma{sigma}")


# --------------------------------------------------------------------------
# several products in one launch
# --------------------------------------------------------------------------
def _batch_run(celty, torch_dev, probs, Rs, launch=None, shared_x=False):
    """Runs the products in one celty_spmspv_batch and, one by one, through
    celty_spmspv_ex with the same launch; returns both results."""
    torch, dev = torch_dev
    encs = [celty.celty_encode(p.W, p.mask, R) for p, R in zip(probs, Rs)]
    Wd = [e.to_device(dev) for e in encs]
    xt = [torch.from_numpy(np.ascontiguousarray(p.x).view(np.int16)).to(dev) for p in probs]
    if shared_x:
        xt = [xt[0]] * len(probs)
    ys = [torch.full((p.W.shape[0],), 0x7C01, dtype=torch.int16, device=dev) for p in probs]
    ws = celty.new_batch_workspace(Wd, dev)
    celty.celty_spmspv_batch(Wd, xt, [p.tau for p in probs], ys, ws, launch)
    torch.cuda.synchronize()
    assert int(ws.count_nonzero()) == 0, "batch workspace not left zero-filled"
    singles = []
    for W, x, p in zip(Wd, xt, probs):
        y = torch.empty(p.W.shape[0], dtype=torch.int16, device=dev)
        w1 = celty.new_workspace(W, dev)
        celty.celty_spmspv_ex(W, x, p.tau, y, w1, launch)
        singles.append(y)
    torch.cuda.synchronize()
    return ([y.cpu().numpy().view(np.float16) for y in ys], [y.cpu().numpy().view(np.float16) for y in singles])


def _batch_launch_for(celty, probs, Rs, launch):
    """The launch the batch resolves to, made explicit for the single calls
    (the batch takes 16 wavefronts if any product has R >= 1024)."""
    if launch is not None and len(launch) >= 2 and launch[1]:
        return launch
    waves = 16 if any(R >= 1024 for R in Rs) else 8
    cols = launch[0] if launch else 0
    groups = launch[2] if launch and len(launch) > 2 else 0
    return (cols, waves, groups)


@pytest.mark.parametrize("launch", [None, (256, 4, 1), (128, 8, 2)])
def test_batch_shared_x(celty, torch_dev, launch):
    _note(f"batch shared x launch={launch}")
    K = 1500
    p0 = workloads.random_small(501, 700, K, ws=60, as_=50)
    probs = [p0] + [workloads.random_small(502 + i, M, K, ws=ws, as_=50) for i, (M, ws) in
                    enumerate([(2049, 50), (3000, 70)])]
    probs = [workloads.Problem(p.W, p.mask, p0.x, p0.tau, p.meta) for p in probs]
    Rs = [256, 512, 128]
    L = _batch_launch_for(celty, probs, Rs, launch)
    yb, ys = _batch_run(celty, torch_dev, probs, Rs, L, shared_x=True)
    for p, a, b in zip(probs, yb, ys):
        _check(a, p.W, p.mask, p.x, p.tau)
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16)), "batch differs from single calls"


def test_batch_independent_mixed_shapes(celty, torch_dev):
    # different K, x and tau per product: one slice (K small), a tall tile,
    # an all-inactive x, an empty matrix and an identity
    _note("batch independent mixed shapes")
    probs = [workloads.random_small(601, 3000, 40, ws=50, as_=50),
             workloads.random_small(602, 5000, 2500, ws=70, as_=60),
             workloads.random_small(603, 1000, 900, ws=50, as_=50),
             workloads.random_small(604, 257, 129, ws=0, as_=0)]
    probs[2] = workloads.Problem(probs[2].W, probs[2].mask, probs[2].x,
                                 float(np.max(np.abs(probs[2].x.astype(np.float32)))), probs[2].meta)
    I = np.eye(600, dtype=np.float16)
    xi = np.random.default_rng(605).laplace(size=600).astype(np.float16)
    probs.append(workloads.Problem(I, None, xi, 0.8, {}))
    probs.append(workloads.Problem(np.zeros((300, 200), np.float16), None, np.ones(200, np.float16), -1.0, {}))
    Rs = [256, 1024, 256, 64, 128, 64]
    L = _batch_launch_for(celty, probs, Rs, None)
    yb, ys = _batch_run(celty, torch_dev, probs, Rs, L)
    for p, a, b in zip(probs, yb, ys):
        _check(a, p.W, p.mask, p.x, p.tau)
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
    assert np.all(yb[2].view(np.uint16) == 0)
    assert np.all(yb[5].view(np.uint16) == 0)
    want = np.where(np.abs(xi.astype(np.float32)) > 0.8, xi, np.float16(0)).astype(np.float16)
    assert np.array_equal(yb[4].view(np.uint16), want.view(np.uint16))


def test_batch_of_eight_repeated(celty, torch_dev):
    torch, dev = torch_dev
    _note("batch of eight, repeated")
    probs = [workloads.random_small(700 + i, 300 + 250 * i, 800 + 97 * i, ws=50, as_=50) for i in range(8)]
    Rs = [128, 256] * 4
    encs = [celty.celty_encode(p.W, p.mask, R) for p, R in zip(probs, Rs)]
    Wd = [e.to_device(dev) for e in encs]
    xt = [torch.from_numpy(p.x.view(np.int16)).to(dev) for p in probs]
    ws = celty.new_batch_workspace(Wd, dev)
    outs = []
    for rep in range(3):
        ys = [torch.empty(p.W.shape[0], dtype=torch.int16, device=dev) for p in probs]
        celty.celty_spmspv_batch(Wd, xt, [p.tau for p in probs], ys, ws)
        outs.append(ys)
    torch.cuda.synchronize()
    assert int(ws.count_nonzero()) == 0
    for ys in outs:
        for p, y in zip(probs, ys):
            _check(y.cpu().numpy().view(np.float16), p.W, p.mask, p.x, p.tau)


def test_config3_layer_batched(celty, torch_dev):
    # the 7B layer as four launches: q/k/v on one x, o, gate/up on one x, down
    torch, dev = torch_dev
    from paper_2608_01536_amd import default_tile_rows
    probs = {p.meta['proj_name']: p for p in workloads.layer_problems(3, 0, 0)}
    for group in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
        _note(f"config3 batched {group}")
        ps = [probs[g] for g in group]
        Rs = [default_tile_rows(*p.W.shape) for p in ps]
        encs = [celty.celty_encode(p.W, p.mask, R) for p, R in zip(ps, Rs)]
        Wd = [e.to_device(dev) for e in encs]
        x = torch.from_numpy(ps[0].x.view(np.int16)).to(dev)
        for p in ps[1:]:
            assert np.array_equal(p.x.view(np.uint16), ps[0].x.view(np.uint16)) and p.tau == ps[0].tau
        ys = [torch.empty(p.W.shape[0], dtype=torch.int16, device=dev) for p in ps]
        ws = celty.new_batch_workspace(Wd, dev)
        celty.celty_spmspv_batch(Wd, [x] * len(ps), [p.tau for p in ps], ys, ws)
        torch.cuda.synchronize()
        # each product alone, in the batch's launch shape, gives the same bits
        # (the batch of q/k/v runs a two-pass ring, the single calls three:
        # the fixed-point sums do not depend on the order of the adds)
        waves = 16 if any(R >= 1024 for R in Rs) else 8
        for p, y, W in zip(ps, ys, Wd):
            err = _check(y.cpu().numpy().view(np.float16), p.W, p.mask, p.x, p.tau)
            _note(f"  {p.meta['proj_name']} rel_err={err:.3e}")
            y1 = torch.empty_like(y)
            celty.celty_spmspv_ex(W, x, p.tau, y1, celty.new_workspace(W, dev), celty.celty_launch(0, waves, 1))
            torch.cuda.synchronize()
            assert torch.equal(y, y1), f"{p.meta['proj_name']}: batch and single call differ"


# --------------------------------------------------------------------------
# graph capture, concurrent streams, very wide K
# --------------------------------------------------------------------------
def test_graph_replays_match_eager(celty, torch_dev):
    # one single-product call and one batch captured in a HIP graph, replayed
    # several times with eager work between replays; every replay must equal
    # the eager result bit for bit and leave the workspaces zero
    torch, dev = torch_dev
    _note("graph replays")
    p = workloads.random_small(801, 2500, 3000, ws=60, as_=50)
    q = workloads.random_small(802, 1200, 3000, ws=50, as_=50)
    Wp = celty.celty_encode(p.W, p.mask, 512).to_device(dev)
    Wq = celty.celty_encode(q.W, q.mask, 256).to_device(dev)
    xp = torch.from_numpy(p.x.view(np.int16)).to(dev)
    xq = torch.from_numpy(q.x.view(np.int16)).to(dev)
    ws1 = celty.new_workspace(Wp, dev)
    wsb = celty.new_batch_workspace([Wp, Wq], dev)
    y1 = torch.empty(2500, dtype=torch.int16, device=dev)
    yb = [torch.empty(2500, dtype=torch.int16, device=dev), torch.empty(1200, dtype=torch.int16, device=dev)]
    e1 = torch.empty_like(y1)
    eb = [torch.empty_like(t) for t in yb]
    celty.celty_spmspv(Wp, xp, p.tau, e1, ws1)
    celty.celty_spmspv_batch([Wp, Wq], [xp, xq], [p.tau, q.tau], eb, wsb)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        celty.celty_spmspv(Wp, xp, p.tau, y1, ws1)
        celty.celty_spmspv_batch([Wp, Wq], [xp, xq], [p.tau, q.tau], yb, wsb)
    for rep in range(4):
        for t in [y1] + yb:
            t.fill_(0x7C01)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y1, e1), f"replay {rep}: single product differs"
        assert all(torch.equal(a, b) for a, b in zip(yb, eb)), f"replay {rep}: batch differs"
        assert int(ws1.count_nonzero()) == 0 and int(wsb.count_nonzero()) == 0
        celty.celty_spmspv(Wq, xq, q.tau, yb[1], celty.new_workspace(Wq, dev))   # eager work between replays
        torch.cuda.synchronize()
    _check(e1.cpu().numpy().view(np.float16), p.W, p.mask, p.x, p.tau)


@pytest.mark.parametrize("offset,size", [(0, 8), (1, 1), (3, 1001), (5, 7), (0, 2048 * 8 + 3),
                                         (7, 300000 * 8 + 5), (0, 1100000 * 8)])
def test_workspace_init_fills_exactly_its_bytes(celty, torch_dev, offset, size):
    torch, dev = torch_dev
    _note(f"workspace_init offset={offset} size={size}")
    buf = torch.full((offset + size + 16,), 0xAB, dtype=torch.uint8, device=dev)
    celty.celty_spmspv_workspace_init(buf[offset:offset + size])
    torch.cuda.synchronize()
    h = buf.cpu().numpy()
    assert np.all(h[offset:offset + size] == 0)
    assert np.all(h[:offset] == 0xAB) and np.all(h[offset + size:] == 0xAB)


def test_workspace_init_recorded_in_a_graph(celty, torch_dev):
    # the init and the product captured together; between replays the
    # workspace is overwritten with garbage by eager work, so every replay
    # depends on the captured fill
    torch, dev = torch_dev
    _note("workspace_init in a graph")
    p = workloads.random_small(803, 3000, 2000, ws=60, as_=50)
    Wp = celty.celty_encode(p.W, p.mask, 512).to_device(dev)
    xp = torch.from_numpy(p.x.view(np.int16)).to(dev)
    ws = celty.new_workspace(Wp, dev)
    want = torch.empty(3000, dtype=torch.int16, device=dev)
    celty.celty_spmspv(Wp, xp, p.tau, want, ws)
    torch.cuda.synchronize()
    y = torch.empty_like(want)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        celty.celty_spmspv_workspace_init(ws)
        celty.celty_spmspv(Wp, xp, p.tau, y, ws)
    for rep in range(4):
        ws.fill_(0x5A)
        y.fill_(0x7C01)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, want), f"replay {rep} differs"
        assert int(ws.count_nonzero()) == 0
    _check(want.cpu().numpy().view(np.float16), p.W, p.mask, p.x, p.tau)


def test_two_streams_with_own_workspaces(celty, torch_dev):
    torch, dev = torch_dev
    _note("two streams")
    probs = [workloads.random_small(811 + i, 3000, 2000, ws=50, as_=50) for i in range(2)]
    Ws = [celty.celty_encode(p.W, p.mask, 512).to_device(dev) for p in probs]
    xs = [torch.from_numpy(p.x.view(np.int16)).to(dev) for p in probs]
    wss = [celty.new_workspace(W, dev) for W in Ws]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[], []]
    for rep in range(6):
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                y = torch.empty(3000, dtype=torch.int16, device=dev)
                celty.celty_spmspv(Ws[i], xs[i], probs[i].tau, y, wss[i])
                outs[i].append(y)
    torch.cuda.synchronize()
    for i in range(2):
        assert int(wss[i].count_nonzero()) == 0
        first = outs[i][0].cpu()
        _check(first.numpy().view(np.float16), probs[i].W, probs[i].mask, probs[i].x, probs[i].tau)
        for y in outs[i][1:]:
            assert torch.equal(y.cpu(), first)


def test_very_wide_K_automatic_shape(celty, torch_dev):
    # K = 100000 puts more than one column on each selection lane under the
    # automatic shape (slices of ~1600 columns, at most 63 slices)
    torch, dev = torch_dev
    p = workloads.random_small(821, 300, 100000, ws=80, as_=60)
    enc = celty.celty_encode(p.W, p.mask, 256)
    plan = celty.celty_spmspv_plan(enc, None)
    _note(f"very wide K plan {plan}")
    assert plan['cols_per_block'] > 64 * plan['waves_per_block']
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, 256, enc=enc)
    _check(y, p.W, p.mask, p.x, p.tau)


def test_tall_tile_needs_more_than_64kb_of_lds(celty, torch_dev):
    # one tile of 30000 rows: about 120 KB of LDS, above the 64 KB default
    torch, dev = torch_dev
    p = workloads.random_small(831, 30000, 500, ws=70, as_=50)
    enc = celty.celty_encode(p.W, p.mask, 30000)
    plan = celty.celty_spmspv_plan(enc, None)
    _note(f"tall tile plan {plan}")
    assert plan['lds_bytes'] > 64 * 1024
    y = _run(celty, torch_dev, p.W, p.mask, p.x, p.tau, 30000, enc=enc)
    _check(y, p.W, p.mask, p.x, p.tau)
    q = workloads.random_small(832, 700, 500, ws=50, as_=50)
    yb, ys = _batch_run(celty, torch_dev, [p, q], [30000, 256], _batch_launch_for(celty, [p, q], [30000, 256], None))
    for pr, a, b in zip([p, q], yb, ys):
        _check(a, pr.W, pr.mask, pr.x, pr.tau)
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


# --------------------------------------------------------------------------
# numerical edge cases of x, tau and the weights
# --------------------------------------------------------------------------
def test_nan_x_is_never_active_and_inf_tau_selects_nothing(celty, torch_dev):
    p = workloads.random_small(841, 1500, 900, ws=50, as_=30)
    x = p.x.copy()
    rng = np.random.default_rng(841)
    x[rng.random(x.size) < 0.1] = np.float16(np.nan)
    _note("nan x")
    y = _run(celty, torch_dev, p.W, p.mask, x, p.tau, 256)
    _check(y, p.W, p.mask, x, p.tau)
    _note("tau = +inf")
    y = _run(celty, torch_dev, p.W, p.mask, x, float("inf"), 256)
    assert np.all(y.view(np.uint16) == 0)


def test_signed_zero_and_subnormal_activations(celty, torch_dev):
    # tau = 0: +-0 is inactive, every subnormal is active; the products are
    # ~1e-4, so the workgroups pick a large fixed-point scale.  (The weights
    # are scaled so that y stays in fp16's normal range: for subnormal outputs
    # the fp16 rounding of y alone, 2^-24 absolute, exceeds 2e-3 of max|y|.)
    rng = np.random.default_rng(851)
    M, K = 2000, 700
    W = (rng.standard_normal((M, K)) * 30).astype(np.float16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    bits = rng.integers(1, 0x03FF, size=K).astype(np.uint16)            # subnormal magnitudes
    bits |= (rng.integers(0, 2, size=K).astype(np.uint16) << np.uint16(15))
    bits[rng.random(K) < 0.2] = 0x0000
    bits[rng.random(K) < 0.1] = 0x8000
    x = bits.view(np.float16)
    _note("subnormal x")
    y = _run(celty, torch_dev, W, mask, x, 0.0, 256)
    _check(y, W, mask, x, 0.0)


def test_large_weights_and_activations(celty, torch_dev):
    # weights up to ~16 and activations up to ~1000: outputs of several
    # thousand, within fp16 range; the scales adapt to max|w| and max|x|
    rng = np.random.default_rng(861)
    M, K = 1800, 600
    W = (rng.standard_normal((M, K)) * 4).astype(np.float16)
    mask = (rng.random((M, K)) < 0.3).astype(np.uint8)
    x = (rng.laplace(size=K) * 100).astype(np.float16)
    tau = workloads.tau_for_sparsity(x, 50)
    _note("large magnitudes")
    y = _run(celty, torch_dev, W, mask, x, tau, 512)
    _check(y, W, mask, x, tau)


# --------------------------------------------------------------------------
# the fused selection where each lane scans several columns (Section 3.1's
# column skip, m = ceil(columns / lanes) of 2 to 8)
# --------------------------------------------------------------------------
def _identity_x(seed, K, nan_every=0, grid=None):
    rng = np.random.default_rng(seed)
    x = rng.laplace(size=K)
    if grid:
        x = np.round(x * grid) / grid          # every value a multiple of 1/grid
    x = x.astype(np.float16)
    if nan_every:
        x[::nan_every] = np.float16(np.nan)
    return x


@pytest.mark.parametrize("launch", [(1000, 2, 1), (4096, 8, 1), (4096, 16, 1), (300, 2, 1), (2048, 4, 1),
                                    (1000, 2, 2), (4096, 8, 4)])
@pytest.mark.parametrize("case", ["tau", "nan", "tau_negative"])
def test_identity_pattern_several_columns_per_lane(celty, torch_dev, launch, case):
    K = 4096
    I = np.eye(K, dtype=np.float16)
    lanes = 64 * launch[1]
    m = -(-min(launch[0], K) // lanes)
    tau = 0.8
    if case == "tau":
        x = _identity_x(11, K)
    elif case == "nan":
        x = _identity_x(12, K, nan_every=7)
    else:
        # every non-NaN column active, zeros included; the values sit on a
        # grid of 2^-6 so that each single-term row lands exactly on the
        # fixed-point grid
        x = _identity_x(13, K, nan_every=11, grid=64)
        tau = -1.0
    _note(f"identity K={K} launch={launch} ({m} columns per lane) {case}")
    assert 2 <= m <= 8
    y = _run(celty, torch_dev, I, None, x, tau, 512, launch=launch)
    xf = x.astype(np.float32)
    want = np.where(np.abs(xf) > tau, x, np.float16(0)).astype(np.float16)   # NaN fails the test
    # an active -0 contributes a zero: the row sums to +0 (as a sum started at
    # +0 would in any floating-point order), so zeros compare without sign
    want = np.where(want == 0, np.float16(0), want).astype(np.float16)
    assert np.array_equal(y.view(np.uint16), want.view(np.uint16))


# --------------------------------------------------------------------------
# the benchmark configurations at the remaining seeds and layers
# --------------------------------------------------------------------------
@pytest.mark.parametrize("seed", [1, 2, 3, 4])
@pytest.mark.parametrize("ws", [30, 50, 70])
@pytest.mark.parametrize("as_", [30, 50, 70])
def test_config2_sweep_other_seeds(celty, torch_dev, seed, ws, as_):
    p = workloads.make_problem(2, 4096, 4096, ws, as_, "laplace", seed=seed, proj=7)
    _full(celty, torch_dev, p, f"config2 seed{seed} ws{ws} as{as_}")


@pytest.mark.parametrize("layer", [1, 7, 13, 20, 26, 33, 38])
def test_config4_more_layers(celty, torch_dev, layer):
    for p in workloads.layer_problems(4, 0, layer):
        _full(celty, torch_dev, p, f"config4 layer{layer} {p.meta['proj_name']}")


@pytest.mark.parametrize("as_", [40, 60, 80])
def test_config5_last_layer(celty, torch_dev, as_):
    # layer 79 of the 80-layer step: every projection at as60, the distinct
    # shapes at as40 and as80
    names = ("q", "k", "v", "o", "gate", "up", "down") if as_ == 60 else ("q", "k", "gate", "down")
    for p in workloads.layer_problems(5, 0, 79, as_):
        if p.meta["proj_name"] in names:
            _full(celty, torch_dev, p, f"config5 layer79 as{as_} {p.meta['proj_name']}")


@pytest.mark.parametrize("M,K,R", [(3000, 2500, 256), (4096, 4097, 512), (1500, 33, 64)])
def test_x_only_two_byte_aligned(celty, torch_dev, M, K, R):
    # x at an odd 2-byte offset: the merge bound is summed one column per load
    # instead of two (the same terms, another order)
    torch, dev = torch_dev
    p = workloads.random_small(M + K, M, K, ws=50, as_=50)
    Wd = celty.celty_encode(p.W, p.mask, R).to_device(dev)
    buf = torch.zeros(K + 1, dtype=torch.int16, device=dev)
    buf[1:] = torch.from_numpy(p.x.view(np.int16)).to(dev)
    x = buf[1:]
    assert x.data_ptr() % 4 == 2
    y = torch.empty(M, dtype=torch.int16, device=dev)
    ws = celty.new_workspace(Wd, dev)
    _note(f"x 2-byte aligned M={M} K={K} R={R}")
    # automatic, and narrow slices (3 to 40 of them) so that the bound is summed
    for launch in (None, (max(16, -(-K // 40)), 2, 1)):
        celty.celty_spmspv_ex(Wd, x, p.tau, y, ws, launch)
        torch.cuda.synchronize()
        assert int(ws.count_nonzero()) == 0
        _check(y.cpu().numpy().view(np.float16), p.W, p.mask, p.x, p.tau)


# --------------------------------------------------------------------------
# the benchmark's read reference (celty_bench_stream_read)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("nbytes,blocks,threads", [(0, 4, 64), (16, 1, 64), (4096 * 16 + 48, 7, 192),
                                                   (3 << 20, 512, 512), (5 << 20, 256, 1024)])
def test_stream_read_reads_every_byte(celty, torch_dev, nbytes, blocks, threads):
    # each workgroup's word is the XOR of the 32-bit words it read; the XOR
    # of all workgroups' words is the XOR of the whole buffer
    torch, dev = torch_dev
    _note(f"stream read {nbytes} B, {blocks} x {threads}")
    rng = np.random.default_rng(nbytes + blocks)
    host = rng.integers(0, 2**32, size=max(4, nbytes // 4), dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).to(dev)
    sink = torch.full((blocks,), -1, dtype=torch.int32, device=dev)
    celty.celty_bench_stream_read(buf, nbytes, sink, blocks, threads)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host[:nbytes // 4]) if nbytes else np.uint32(0)
    assert int(got) == int(want)


def test_prepared_call_matches_spmspv_ex(celty, torch_dev):
    # PreparedSpMSpV checks its tensors once; each call passes only tau
    torch, dev = torch_dev
    p = workloads.headline_problem(0)
    Wd = celty.celty_encode(p.W, p.mask, 512).to_device(dev)
    xt = torch.from_numpy(p.x.view(np.int16)).to(dev)
    y1 = torch.empty(p.W.shape[0], dtype=torch.int16, device=dev)
    y2 = torch.empty_like(y1)
    ws1, ws2 = celty.new_workspace(Wd, dev), celty.new_workspace(Wd, dev)
    prep = celty.PreparedSpMSpV(Wd, xt, y2, ws2, (128, 4, 1))
    for tau in (p.tau, 0.5 * p.tau, -1.0):
        celty.celty_spmspv_ex(Wd, xt, tau, y1, ws1, (128, 4, 1))
        prep(tau)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2)
    assert int(ws2.count_nonzero()) == 0
    with pytest.raises(ValueError):
        celty.PreparedSpMSpV(Wd, xt[:-1], y2, ws2)       # short x is refused once, here
    with pytest.raises(celty.CeltyError):
        prep(float("nan"))                                # the C entry point still validates tau
