"""The C-ABI library loads, exports every declared entry point, and rejects bad
arguments with the documented status before touching the device.

The rejection checks pass fake (never dereferenced) device addresses; they run
only where no GPU is visible, so a validation bug can never launch a kernel on
garbage pointers.
"""
import ctypes
import glob
import math
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2608_01536_amd as celty
from paper_2608_01536_amd import (CELTY_EFORMAT, CELTY_EINVAL, CELTY_OK, celty_launch, celty_rlc_csc)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "celty.h")
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def _declared_functions():
    names = []
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names += re.findall(r"^[A-Za-z_][\w\s\*]*?\b(celty_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for want in ("celty_encode_plan", "celty_encode", "celty_decode", "celty_select", "celty_spmspv",
                 "celty_spmspv_ex", "celty_spmspv_plan", "celty_spmspv_workspace_bytes",
                 "celty_spmspv_workspace_init", "celty_status_string", "celty_default_tile_rows",
                 "celty_spmspv_batch", "celty_spmspv_batch_workspace_bytes", "celty_spmspv_noalloc",
                 "celty_bench_stream_read"):
        assert want in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(celty._LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", celty._LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (celty_\w+)", out))
    assert set(_declared_functions()) <= exported


def test_status_strings():
    for st in range(6):
        assert celty.celty_status_string(st).startswith("CELTY_")
    assert "unknown" in celty.celty_status_string(99)


def test_default_tile_rows():
    # largest power of two <= M / 8, clamped to [256, 2048] (K < 4 M)
    for M, want in [(1, 256), (1024, 256), (4096, 512), (4095, 256), (5120, 512), (8192, 1024), (11008, 1024),
                    (13824, 1024), (16384, 2048), (28672, 2048), (1 << 20, 2048)]:
        assert celty.default_tile_rows(M, 4096) == want, M
    # wide matrices (K >= 4 M): largest power of two <= M / 4
    for M, K, want in [(7168, 28672, 1024), (4096, 28672, 1024), (2048, 8192, 512), (1024, 8192, 256),
                       (8192, 28672, 1024), (5120, 13824, 512), (4096, 16383, 512), (4096, 16384, 1024)]:
        assert celty.default_tile_rows(M, K) == want, (M, K)
    assert celty._default_tile_rows(0, 5) == 0


def test_workspace_bytes():
    # two 64-bit merge words per output row, rounded to 256 bytes
    assert celty.celty_spmspv_workspace_bytes(4096, 4096, 256) == 4096 * 16
    assert celty.celty_spmspv_workspace_bytes(1000, 7, 300) == 16128
    assert celty.celty_spmspv_workspace_bytes(0, 1, 1) == 0


# --------------------------------------------------------------------------
# encoder / decoder error paths (pure host)
# --------------------------------------------------------------------------
def test_encode_plan_rejects_bad_arguments():
    W = np.ones((4, 5), dtype=np.float16).view(np.uint16)
    g, n, p = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    f = celty._encode_plan
    ok = f(W.ctypes.data, 5, None, 0, 4, 5, 2, 0, ctypes.byref(g), ctypes.byref(n), ctypes.byref(p))
    assert ok == CELTY_OK and n.value == 20 and p.value == 0 and g.value == 10
    assert f(None, 5, None, 0, 4, 5, 2, 0, ctypes.byref(g), ctypes.byref(n), ctypes.byref(p)) == CELTY_EINVAL
    assert f(W.ctypes.data, 4, None, 0, 4, 5, 2, 0, ctypes.byref(g), ctypes.byref(n),
             ctypes.byref(p)) == CELTY_EINVAL
    assert f(W.ctypes.data, 5, W.ctypes.data, 3, 4, 5, 2, 0, ctypes.byref(g), ctypes.byref(n),
             ctypes.byref(p)) == CELTY_EINVAL
    for M, K, R in ((0, 5, 2), (4, 0, 2), (4, 5, 0)):
        assert f(W.ctypes.data, 5, None, 0, M, K, R, 0, ctypes.byref(g), ctypes.byref(n),
                 ctypes.byref(p)) == CELTY_EINVAL
    assert f(W.ctypes.data, 5, None, 0, 4, 5, 2, 0, None, ctypes.byref(n), ctypes.byref(p)) == CELTY_EINVAL
    for layout in (-1, 3, 99):                                       # unknown layouts
        assert f(W.ctypes.data, 5, None, 0, 4, 5, 2, layout, ctypes.byref(g), ctypes.byref(n),
                 ctypes.byref(p)) == CELTY_EINVAL


def test_encode_rejects_bad_arguments():
    W = np.ones((4, 5), dtype=np.float16).view(np.uint16)
    gptr = celty._aligned_empty(3 * 5 + 1, np.uint32)
    vals = celty._aligned_empty(8 * 20, np.uint16)
    runs = celty._aligned_empty(20, np.uint32)
    cmax = celty._aligned_empty(6, np.uint16)
    d = celty_rlc_csc()
    f = celty._encode
    args = [W.ctypes.data, 5, None, 0, 4, 5, 2, 0, gptr.ctypes.data, vals.ctypes.data, runs.ctypes.data,
            cmax.ctypes.data]
    assert f(*args, 10, ctypes.byref(d), 1) == CELTY_OK
    assert cmax[:5].view(np.float16).tolist() == [1.0] * 5 and d.colmax == cmax.ctypes.data
    assert f(*args, 11, ctypes.byref(d), 1) == CELTY_EINVAL          # n_groups mismatch
    assert f(*args, 10, ctypes.byref(d), -1) == CELTY_EINVAL         # n_threads
    bad = list(args)
    bad[9] = vals.ctypes.data + 2                                    # values not 16-byte aligned
    assert f(*bad, 10, ctypes.byref(d), 1) == CELTY_EINVAL
    bad = list(args)
    bad[11] = cmax.ctypes.data + 2                                   # colmax not 4-byte aligned
    assert f(*bad, 10, ctypes.byref(d), 1) == CELTY_EINVAL
    bad[11] = None                                                   # no colmax
    assert f(*bad, 10, ctypes.byref(d), 1) == CELTY_EINVAL
    bad = list(args)
    bad[7] = 5                                                       # unknown layout
    assert f(*bad, 10, ctypes.byref(d), 1) == CELTY_EINVAL
    assert f(*args, 10, None, 1) == CELTY_EINVAL


def test_decode_rejects_corrupt_streams():
    rng = np.random.default_rng(0)
    W = (rng.standard_normal((40, 6)) * 0.02).astype(np.float16)
    enc = celty.celty_encode(W, (rng.random((40, 6)) < 0.5).astype(np.uint8), 16)
    d = enc.desc()
    out = np.empty((40, 6), np.uint16)
    m = np.empty((40, 6), np.uint8)
    assert celty._decode(ctypes.byref(d), out.ctypes.data, m.ctypes.data) == CELTY_OK
    g = enc.gptr.copy()
    g[3], g[4] = g[4] + 1, g[3]                                      # non-monotone
    d2 = enc.desc()
    d2.gptr = g.ctypes.data
    assert celty._decode(ctypes.byref(d2), out.ctypes.data, m.ctypes.data) == CELTY_EFORMAT
    d3 = enc.desc()
    d3.n_nnz += 1                                                    # header disagrees
    assert celty._decode(ctypes.byref(d3), out.ctypes.data, m.ctypes.data) == CELTY_EFORMAT
    d4 = enc.desc()
    d4.T += 1                                                        # inconsistent header
    assert celty._decode(ctypes.byref(d4), out.ctypes.data, m.ctypes.data) == CELTY_EINVAL
    d5 = enc.desc()
    d5.version = 1
    assert celty._decode(ctypes.byref(d5), out.ctypes.data, m.ctypes.data) == CELTY_EINVAL
    cm = enc.colmax.copy()
    cm[2] = np.uint16(int(cm[2]) + 1)                               # column maximum disagrees
    d6 = enc.desc()
    d6.colmax = cm.ctypes.data
    assert celty._decode(ctypes.byref(d6), out.ctypes.data, m.ctypes.data) == CELTY_EFORMAT
    d7 = enc.desc()
    d7.colmax = None
    assert celty._decode(ctypes.byref(d7), out.ctypes.data, m.ctypes.data) == CELTY_EINVAL


# --------------------------------------------------------------------------
# device entry points: validation before any launch (no GPU visible only)
# --------------------------------------------------------------------------
def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


host_only = pytest.mark.skipif(_gpu_visible(), reason="fake device addresses are only used without a GPU")

FAKE = 0x7F0000000000   # never dereferenced: every call below fails validation first


def _desc(M=4096, K=4096, R=256, G=1000):
    T = -(-M // R)
    return celty_rlc_csc(celty.FORMAT_VERSION, M, K, R, T, 4, G, 8 * G, 7 * G, G, 1.0, 0, FAKE, FAKE + 0x10000,
                         FAKE + 0x20000, FAKE + 0x30000)


@host_only
def test_automatic_plan_fills_the_compute_units_in_one_even_round():
    # 256 compute units, 16 wavefront slots each: the automatic shape never
    # starts a second round of workgroups; an 8-wavefront count between one
    # and 0.9 x two per unit is either widened to fill the slots or kept as
    # the rounded shape (64-column multiples) when its slices would be light
    def plan(M, K, G):
        R = celty.default_tile_rows(M, K)
        d = _desc(M, K, R, G)
        out, nb = celty_launch(), ctypes.c_int64()
        assert celty._plan(ctypes.byref(d), None, ctypes.byref(out), ctypes.byref(nb), None) == CELTY_OK
        return d, out, nb.value
    for M in (512, 1024, 3000, 4096, 5120, 7168, 8192, 10240, 11008, 13824, 15360, 22016, 28672, 57344):
        for K in (1000, 2048, 4096, 5120, 7168, 8192, 11008, 13824, 28672):
            for G in (1000, M * K // 16):
                d, out, n = plan(M, K, G)
                slots = 4096 // out.waves_per_block
                KC = -(-K // out.cols_per_block)
                assert n == d.T * KC <= slots, (M, K, G, n)
                if out.waves_per_block == 8 and 256 < n < 0.9 * slots:
                    assert out.cols_per_block % 64 == 0 or out.cols_per_block == K or KC == 63, (M, K, G, n)
    # 5120 x 13824 at half density: 10 tiles x 51 slices (two workgroups per
    # unit); 5120 x 5120 with light slices (under 80 KB of stored groups at
    # two per unit) takes one per unit, 10 x 25; with heavy slices 10 x 51
    assert plan(5120, 13824, 5120 * 13824 // 16)[2] == 510
    assert plan(5120, 5120, 1000)[2] == 250
    assert plan(5120, 5120, 5120 * 5120 // 16)[2] == 250
    assert plan(5120, 5120, 5120 * 5120 // 8)[2] == 510


@host_only
def test_spmspv_plan_is_host_only():
    d = _desc()
    out, nb, lds = celty_launch(), ctypes.c_int64(), ctypes.c_int64()
    assert celty._plan(ctypes.byref(d), None, ctypes.byref(out), ctypes.byref(nb), ctypes.byref(lds)) == CELTY_OK
    assert out.waves_per_block in (2, 4, 8, 16) and 1 <= out.cols_per_block <= 4096
    assert out.groups_per_lane in (1, 2, 4)
    assert nb.value == d.T * (-(-d.K // out.cols_per_block))
    assert 0 < lds.value <= 160 * 1024
    bad = celty_launch(66, 4, 3)                                      # groups per lane
    assert celty._plan(ctypes.byref(d), ctypes.byref(bad), ctypes.byref(out), None, None) == CELTY_EINVAL
    bad = celty_launch(64, 3)
    assert celty._plan(ctypes.byref(d), ctypes.byref(bad), ctypes.byref(out), None, None) == CELTY_EINVAL
    bad = celty_launch(5000, 4)
    assert celty._plan(ctypes.byref(d), ctypes.byref(bad), ctypes.byref(out), None, None) == CELTY_EINVAL
    big = _desc(M=100000, K=64, R=60000)                             # tile does not fit in LDS
    assert celty._plan(ctypes.byref(big), None, ctypes.byref(out), None, None) == CELTY_EINVAL
    many = celty_launch(64, 4)                                       # 64 slices of 4096 columns > 63
    assert celty._plan(ctypes.byref(d), ctypes.byref(many), ctypes.byref(out), None, None) == CELTY_EINVAL
    ok = celty_launch(66, 4)                                         # 63 slices
    assert celty._plan(ctypes.byref(d), ctypes.byref(ok), ctypes.byref(out), ctypes.byref(nb), None) == CELTY_OK
    assert nb.value == d.T * 63
    wide = _desc(K=200000)                                           # auto shape keeps <= 63 slices
    assert celty._plan(ctypes.byref(wide), None, ctypes.byref(out), ctypes.byref(nb), None) == CELTY_OK
    assert -(-200000 // out.cols_per_block) <= 63
    assert out.cols_per_block <= 512 * out.waves_per_block
    # at most 8 columns per lane in the selection: cols_per_block <= 512 * waves
    for cols, waves, want in [(1024, 2, CELTY_OK), (1025, 2, CELTY_EINVAL), (2048, 4, CELTY_OK),
                              (2049, 4, CELTY_EINVAL), (4096, 8, CELTY_OK), (4096, 4, CELTY_EINVAL)]:
        L = celty_launch(cols, waves)
        assert celty._plan(ctypes.byref(d), ctypes.byref(L), ctypes.byref(out), None, None) == want, (cols, waves)
    narrow = _desc(K=1000)                                           # columns beyond K are not counted
    L = celty_launch(4096, 2)
    assert celty._plan(ctypes.byref(narrow), ctypes.byref(L), ctypes.byref(out), None, None) == CELTY_OK
    assert out.cols_per_block == 1000


@host_only
@pytest.mark.parametrize("case", ["null_desc", "version", "run_bits", "T", "values_align", "runs_align",
                                  "null_x", "nan_tau", "x_align", "overlap", "short_ws", "null_ws",
                                  "ws_align", "waves", "max_abs_nan", "max_abs_inf", "max_abs_neg", "slices",
                                  "null_colmax", "colmax_align", "layout"])
def test_spmspv_rejects_bad_arguments(case):
    d = _desc()
    x, y, ws = FAKE + 0x100000, FAKE + 0x200000, FAKE + 0x300000
    tau = 0.5
    nws = celty.celty_spmspv_workspace_bytes(4096, 4096, 256)
    launch = None
    if case == "version":
        d.version = 1
    elif case == "run_bits":
        d.run_bits = 3
    elif case == "T":
        d.T += 1
    elif case == "values_align":
        d.values += 8
    elif case == "runs_align":
        d.runs += 2
    elif case == "null_x":
        x = None
    elif case == "nan_tau":
        tau = math.nan
    elif case == "x_align":
        x += 1
    elif case == "overlap":
        y = x + 100
    elif case == "short_ws":
        nws -= 1
    elif case == "null_ws":
        ws = None
    elif case == "ws_align":
        ws += 16
    elif case == "waves":
        launch = celty_launch(64, 5)
    elif case == "slices":
        launch = celty_launch(32, 4)
    elif case == "max_abs_nan":
        d.max_abs = math.nan
    elif case == "max_abs_inf":
        d.max_abs = math.inf
    elif case == "max_abs_neg":
        d.max_abs = -1.0
    elif case == "null_colmax":
        d.colmax = None
    elif case == "colmax_align":
        d.colmax += 2
    elif case == "layout":
        d.layout = 7
    pd = None if case == "null_desc" else ctypes.byref(d)
    st = celty._spmspv_ex(pd, x, tau, y, ws, nws, None if launch is None else ctypes.byref(launch), None)
    assert st == CELTY_EINVAL


def _batch_arrays(descs, xs, taus, ys):
    n = len(descs)
    arr = (ctypes.POINTER(celty_rlc_csc) * n)(*[ctypes.pointer(d) for d in descs])
    return (arr, (ctypes.c_void_p * n)(*xs), (ctypes.c_float * n)(*taus), (ctypes.c_void_p * n)(*ys))


def test_batch_workspace_bytes():
    descs = [_desc(M=4096), _desc(M=1000, K=300, R=128), _desc(M=11008, R=1024)]
    arr = (ctypes.POINTER(celty_rlc_csc) * 3)(*[ctypes.pointer(d) for d in descs])
    want = sum(celty.celty_spmspv_workspace_bytes(d.M, d.K, d.R) for d in descs)
    assert celty._batch_ws_bytes(3, arr) == want == 4096 * 16 + 16128 + 11008 * 16
    assert celty._batch_ws_bytes(0, arr) == 0
    assert celty._batch_ws_bytes(9, arr) == 0
    assert celty._batch_ws_bytes(2, None) == 0


@host_only
@pytest.mark.parametrize("case", ["n0", "n9", "null_W", "null_x", "null_tau", "null_y", "bad_header",
                                  "nan_tau", "y_over_other_x", "y_over_other_y", "y_over_ws", "x_over_ws",
                                  "short_ws", "slices"])
def test_batch_rejects_bad_arguments(case):
    descs = [_desc(M=4096), _desc(M=1000, K=4096, R=128), _desc(M=2048, K=300, R=512)]
    xs = [FAKE + 0x100000, FAKE + 0x100000, FAKE + 0x110000]      # products 0 and 1 share x
    ys = [FAKE + 0x200000, FAKE + 0x210000, FAKE + 0x220000]
    taus = [0.5, 0.5, 0.25]
    ws = FAKE + 0x400000
    n = 3
    arr, xp, tp, yp = _batch_arrays(descs, xs, taus, ys)
    nws = celty._batch_ws_bytes(n, arr)
    launch = None
    if case == "n0":
        n = 0
    elif case == "n9":
        n = 9
    elif case == "null_W":
        arr = None
    elif case == "null_x":
        xp = None
    elif case == "null_tau":
        tp = None
    elif case == "null_y":
        yp = None
    elif case == "bad_header":
        descs[2].version = 1
    elif case == "nan_tau":
        tp[2] = math.nan
    elif case == "y_over_other_x":
        yp[0] = xs[2] + 64
    elif case == "y_over_other_y":
        yp[2] = ys[1] + 100
    elif case == "y_over_ws":
        yp[1] = ws + 256
    elif case == "x_over_ws":
        xp[2] = ws + 512
    elif case == "short_ws":
        nws -= 1
    elif case == "slices":
        launch = celty_launch(32, 4)                                  # 128 slices of 4096 columns
    st = celty._batch(n, arr, xp, tp, yp, ws, nws, None if launch is None else ctypes.byref(launch), None)
    assert st == CELTY_EINVAL


@host_only
def test_select_rejects_bad_arguments():
    f = celty._select
    assert f(None, 10, 0.5, FAKE, FAKE + 64, None) == CELTY_EINVAL
    assert f(FAKE, 0, 0.5, FAKE + 64, FAKE + 128, None) == CELTY_EINVAL
    assert f(FAKE, 10, math.nan, FAKE + 64, FAKE + 128, None) == CELTY_EINVAL
    assert f(FAKE, 10, 0.5, FAKE + 66, FAKE + 128, None) == CELTY_EINVAL
    # x's byte size must fit the kernel's 32-bit buffer size
    assert f(FAKE, 2**30, 0.5, FAKE + 64, FAKE + 128, None) == CELTY_EINVAL


def test_stream_read_rejects_bad_arguments():
    f = celty._stream_read
    assert f(FAKE, 4096, None, 4, 256, None) == CELTY_EINVAL          # no sink
    assert f(FAKE, 4096, FAKE + 2, 4, 256, None) == CELTY_EINVAL      # misaligned sink
    assert f(FAKE + 8, 4096, FAKE, 4, 256, None) == CELTY_EINVAL      # misaligned buffer
    assert f(None, 4096, FAKE, 4, 256, None) == CELTY_EINVAL
    assert f(FAKE, 4100, FAKE, 4, 256, None) == CELTY_EINVAL          # not a multiple of 16
    for blocks, threads in ((0, 256), (65536, 256), (4, 32), (4, 100), (4, 2048)):
        assert f(FAKE, 4096, FAKE, blocks, threads, None) == CELTY_EINVAL


def test_single_hip_runtime_alongside_torch():
    """libcelty and torch must share one HIP runtime (torch bundles its own
    libamdhip64); two runtimes would make torch's streams invalid handles."""
    import torch  # noqa: F401
    maps = {l.split()[-1] for l in open("/proc/self/maps") if "libamdhip64" in l}
    assert len(maps) == 1, maps


def test_package_refuses_to_import_without_the_library(tmp_path):
    """With libcelty.so absent the binding raises at import: there is no
    fallback path to run instead of the HIP kernels."""
    import shutil
    pkg = os.path.join(ROOT, "paper_2608_01536_amd")
    dst = tmp_path / "paper_2608_01536_amd"
    dst.mkdir()
    for name in os.listdir(pkg):
        if name.endswith(".py"):
            shutil.copy(os.path.join(pkg, name), dst / name)
    env = dict(os.environ, PYTHONPATH=str(tmp_path))
    res = subprocess.run(["python3", "-c", "import paper_2608_01536_amd"], cwd=str(tmp_path), env=env,
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert res.returncode != 0
    assert "ImportError" in res.stderr and "is not built" in res.stderr


def test_product_path_does_not_use_the_oracle():
    """Neither the binding nor the native sources reference the CPU oracle."""
    pkg = os.path.join(ROOT, "paper_2608_01536_amd")
    for dirpath, _, files in os.walk(pkg):
        for name in files:
            if name.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, name)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, flags=re.M), name
                assert "oracle/" not in text and "oracle." not in text, name


class _FakeDeviceTensor:
    """Stands in for a contiguous CUDA tensor in the binding's argument checks
    (its address is never passed on: each case below fails a check first)."""

    is_cuda = True

    def __init__(self, numel, element_size, device="cuda:0", dtype=None):
        import torch
        self._n, self._e, self.device = numel, element_size, device
        self.dtype = dtype if dtype is not None else {1: torch.uint8, 2: torch.int16, 4: torch.int32}[element_size]

    def is_contiguous(self):
        return True

    def element_size(self):
        return self._e

    def numel(self):
        return self._n

    def data_ptr(self):
        return FAKE


class _FakeEncoded:
    def __init__(self, M, K, device="cuda:0"):
        self.M, self.K = M, K
        self.gptr = _FakeDeviceTensor(1, 4, device)

    def desc(self):
        return celty_rlc_csc()


@host_only
@pytest.mark.parametrize("case", ["x_short", "y_short", "x_device", "y_device", "ws_device", "x_bf16", "y_bf16"])
def test_binding_rejects_short_or_misplaced_tensors(case):
    """The C ABI takes bare pointers and trusts x to hold K halves and y M, so
    the binding checks the tensors' sizes, dtype and device before calling it
    (a bfloat16 tensor has 2-byte elements too, but is not fp16)."""
    import torch
    M, K = 300, 200
    W = _FakeEncoded(M, K)
    x = _FakeDeviceTensor(K - 1 if case == "x_short" else K, 2, "cuda:1" if case == "x_device" else "cuda:0",
                          torch.bfloat16 if case == "x_bf16" else None)
    y = _FakeDeviceTensor(M - 1 if case == "y_short" else M, 2, "cuda:1" if case == "y_device" else "cuda:0",
                          torch.bfloat16 if case == "y_bf16" else None)
    ws = _FakeDeviceTensor(1 << 20, 1, "cuda:1" if case == "ws_device" else "cuda:0")
    with pytest.raises(ValueError):
        celty.celty_spmspv(W, x, 0.5, y, ws, stream=0)
    with pytest.raises(ValueError):
        celty.celty_spmspv_ex(W, x, 0.5, y, ws, (64, 4, 1), stream=0)
    W2 = _FakeEncoded(M // 2, K)
    x2 = _FakeDeviceTensor(K, 2)
    y2 = _FakeDeviceTensor(M // 2, 2)
    with pytest.raises(ValueError):   # the faulty pair second, so that every element is checked
        celty.celty_spmspv_batch([W2, W], [x2, x], [0.5, 0.5], [y2, y], ws, stream=0)


@host_only
@pytest.mark.parametrize("case", ["idx_short", "count_empty", "idx_device"])
def test_select_binding_rejects_short_or_misplaced_outputs(case):
    K = 1000
    x = _FakeDeviceTensor(K, 2)
    idx = _FakeDeviceTensor(K - 1 if case == "idx_short" else K, 4, "cuda:1" if case == "idx_device" else "cuda:0")
    count = _FakeDeviceTensor(0 if case == "count_empty" else 1, 4)
    with pytest.raises(ValueError):
        celty.celty_select(x, 0.5, idx, count, stream=0)


@pytest.mark.parametrize("dtype", [np.float32, np.float64, np.int16, np.int32])
def test_encoder_binding_accepts_only_fp16_weights(dtype):
    """A float32 W viewed as uint16 would encode an M x 2K matrix of bit
    halves; the binding refuses every dtype but float16 and uint16 bits."""
    W = np.ones((4, 6), dtype=dtype)
    with pytest.raises(ValueError):
        celty.celty_encode(W, None, 2)
    with pytest.raises(ValueError):
        celty.celty_encode_plan(W, None, 2)
    ok = celty.celty_encode(np.ones((4, 6), np.float16).view(np.uint16), None, 2)
    assert ok.n_nnz == 24
