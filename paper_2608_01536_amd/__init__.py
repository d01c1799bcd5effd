"""Dual-sparse SpMSpV for AMD MI355X: Python binding of libcelty (include/celty.h).

The functions below carry the C names and only marshal arguments: numpy
arrays for the host encoder/decoder, torch tensors for device memory and
``torch.cuda`` streams for ordering.  All arithmetic of the product runs in
the HIP kernels of libcelty.so; there is no fallback path.  Importing this
package fails loudly if the library has not been built
(``python paper_2608_01536_amd/build_lib.py``).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcelty.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is not built; run `python paper_2608_01536_amd/build_lib.py`")


def _share_torch_hip_runtime() -> None:
    """Make libcelty bind to the HIP runtime torch uses.

    torch ships its own libamdhip64 (same soname as the system one).  Loading
    it first, by path and globally, makes libcelty's dependency resolve to that
    copy whatever the import order, so streams and device memory handed over
    from torch belong to the runtime that launches the kernels."""
    import importlib.util
    spec = importlib.util.find_spec("torch")
    for d in (spec.submodule_search_locations or []) if spec else []:
        path = os.path.join(d, "lib", "libamdhip64.so")
        if os.path.exists(path):
            ctypes.CDLL(path, mode=ctypes.RTLD_GLOBAL)
            return


_share_torch_hip_runtime()
_lib = ctypes.CDLL(_LIB_PATH)

CELTY_OK, CELTY_EINVAL, CELTY_ENOMEM, CELTY_EOVERFLOW, CELTY_EFORMAT, CELTY_EHIP = range(6)
FORMAT_VERSION = 2
RUN_BITS = 4
GROUP = 8
LAYOUT_RLC = 0           # 4-bit run lengths (the paper's format)
LAYOUT_ROWS16 = 1        # 16-bit row offsets within the tile (decode-free)
LAYOUT_INTERLEAVED = 2   # RLC entries in lane-interleaved order within chunks of 64 groups

_p = ctypes.c_void_p
_i32, _i64, _f32, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t


class celty_rlc_csc(ctypes.Structure):
    _fields_ = [("version", _i32), ("M", _i32), ("K", _i32), ("R", _i32), ("T", _i32),
                ("run_bits", _i32), ("n_groups", _i64), ("n_entries", _i64), ("n_nnz", _i64),
                ("n_pad", _i64), ("max_abs", _f32), ("layout", _i32), ("gptr", _p), ("values", _p),
                ("runs", _p), ("colmax", _p)]


class celty_launch(ctypes.Structure):
    _fields_ = [("cols_per_block", _i32), ("waves_per_block", _i32), ("groups_per_lane", _i32),
                ("lds_swizzle", _i32)]


def _sig(name, res, *args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


_encode_plan = _sig("celty_encode_plan", ctypes.c_int, _p, _i64, _p, _i64, _i32, _i32, _i32, _i32,
                    ctypes.POINTER(_i64), ctypes.POINTER(_i64), ctypes.POINTER(_i64))
_encode = _sig("celty_encode", ctypes.c_int, _p, _i64, _p, _i64, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _i64,
               ctypes.POINTER(celty_rlc_csc), _i32)
_decode = _sig("celty_decode", ctypes.c_int, ctypes.POINTER(celty_rlc_csc), _p, _p)
_select = _sig("celty_select", ctypes.c_int, _p, _i32, _f32, _p, _p, _p)
_ws_bytes = _sig("celty_spmspv_workspace_bytes", _sz, _i32, _i32, _i32)
_ws_init = _sig("celty_spmspv_workspace_init", ctypes.c_int, _p, _sz, _p)
_stream_read = _sig("celty_bench_stream_read", ctypes.c_int, _p, _sz, _p, _i32, _i32, _p)
_spmspv = _sig("celty_spmspv", ctypes.c_int, ctypes.POINTER(celty_rlc_csc), _p, _f32, _p, _p, _sz, _p)
_spmspv_ex = _sig("celty_spmspv_ex", ctypes.c_int, ctypes.POINTER(celty_rlc_csc), _p, _f32, _p, _p, _sz,
                  ctypes.POINTER(celty_launch), _p)
_spmspv_noalloc = _sig("celty_spmspv_noalloc", ctypes.c_int, ctypes.POINTER(celty_rlc_csc), _p, _f32, _p,
                       ctypes.POINTER(celty_launch), _p)
_default_tile_rows = _sig("celty_default_tile_rows", _i32, _i32, _i32)
_desc_pp = ctypes.POINTER(ctypes.POINTER(celty_rlc_csc))
_batch = _sig("celty_spmspv_batch", ctypes.c_int, _i32, _desc_pp, ctypes.POINTER(_p), ctypes.POINTER(_f32),
              ctypes.POINTER(_p), _p, _sz, ctypes.POINTER(celty_launch), _p)
_batch_ws_bytes = _sig("celty_spmspv_batch_workspace_bytes", _sz, _i32, _desc_pp)
_plan = _sig("celty_spmspv_plan", ctypes.c_int, ctypes.POINTER(celty_rlc_csc), ctypes.POINTER(celty_launch),
             ctypes.POINTER(celty_launch), ctypes.POINTER(_i64), ctypes.POINTER(_i64))
_status_string = _sig("celty_status_string", ctypes.c_char_p, ctypes.c_int)


class CeltyError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {celty_status_string(status)}")


def celty_status_string(status: int) -> str:
    return _status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != CELTY_OK:
        raise CeltyError(status, where)


def _aligned_empty(n: int, dtype, align: int = 64) -> np.ndarray:
    dt = np.dtype(dtype)
    raw = np.empty(n * dt.itemsize + align, dtype=np.uint8)
    off = (-raw.ctypes.data) % align
    return raw[off:off + n * dt.itemsize].view(dt)


def _host_matrix(W: np.ndarray, mask):
    Wa = np.asarray(W)
    if Wa.dtype not in (np.float16, np.uint16):
        raise ValueError(f"W must hold fp16 values (float16, or their uint16 bit patterns), not {Wa.dtype}")
    Wb = np.ascontiguousarray(Wa).view(np.uint16)
    if Wb.ndim != 2:
        raise ValueError("W must be 2-D (M x K)")
    if mask is None:
        return Wb, None
    m = np.ascontiguousarray(np.asarray(mask)).astype(np.uint8, copy=False)
    if m.shape != Wb.shape:
        raise ValueError("mask must have W's shape")
    return Wb, m


# ---------------------------------------------------------------------------
# Host encoder / decoder
# ---------------------------------------------------------------------------
class HostRlcCsc:
    """The encoded arrays in host memory plus the header."""

    def __init__(self, desc: celty_rlc_csc, gptr: np.ndarray, values: np.ndarray, runs: np.ndarray,
                 colmax: np.ndarray):
        self.M, self.K, self.R, self.T = desc.M, desc.K, desc.R, desc.T
        self.n_groups, self.n_entries = int(desc.n_groups), int(desc.n_entries)
        self.n_nnz, self.n_pad = int(desc.n_nnz), int(desc.n_pad)
        self.max_abs = float(desc.max_abs)
        self.layout = int(desc.layout)
        self.gptr, self.values, self.runs, self.colmax = gptr, values, runs, colmax

    def desc(self) -> celty_rlc_csc:
        return celty_rlc_csc(FORMAT_VERSION, self.M, self.K, self.R, self.T, RUN_BITS, self.n_groups,
                             self.n_entries, self.n_nnz, self.n_pad, self.max_abs, self.layout,
                             self.gptr.ctypes.data,
                             self.values.ctypes.data if self.values.size else None,
                             self.runs.ctypes.data if self.runs.size else None, self.colmax.ctypes.data)

    def to_device(self, device=None) -> "DeviceRlcCsc":
        return DeviceRlcCsc(self, device)


def celty_encode_plan(W: np.ndarray, mask, R: int, layout: int = LAYOUT_RLC) -> Tuple[int, int, int]:
    Wb, m = _host_matrix(W, mask)
    M, K = Wb.shape
    g, n, p = _i64(), _i64(), _i64()
    _check(_encode_plan(Wb.ctypes.data, K, None if m is None else m.ctypes.data, K, M, K, int(R), int(layout),
                        ctypes.byref(g), ctypes.byref(n), ctypes.byref(p)), "celty_encode_plan")
    return g.value, n.value, p.value


def celty_encode(W: np.ndarray, mask, R: int, n_threads: int = 0, layout: int = LAYOUT_RLC) -> HostRlcCsc:
    """fp16 W (M x K) + keep-mask -> the encoded arrays, in fresh host arrays."""
    Wb, m = _host_matrix(W, mask)
    M, K = Wb.shape
    G, _, _ = celty_encode_plan(Wb, m, R, layout)
    T = -(-M // int(R))
    gptr = _aligned_empty(T * K + 1, np.uint32)
    values = _aligned_empty(GROUP * G, np.uint16)
    runs = _aligned_empty(4 * G if int(layout) == LAYOUT_ROWS16 else G, np.uint32)
    colmax = _aligned_empty(K, np.uint16)
    desc = celty_rlc_csc()
    _check(_encode(Wb.ctypes.data, K, None if m is None else m.ctypes.data, K, M, K, int(R), int(layout),
                   gptr.ctypes.data, values.ctypes.data, runs.ctypes.data, colmax.ctypes.data, G,
                   ctypes.byref(desc), int(n_threads)), "celty_encode")
    return HostRlcCsc(desc, gptr, values, runs, colmax)


def celty_decode(enc: HostRlcCsc) -> Tuple[np.ndarray, np.ndarray]:
    W = np.empty((enc.M, enc.K), dtype=np.uint16)
    mask = np.empty((enc.M, enc.K), dtype=np.uint8)
    d = enc.desc()
    _check(_decode(ctypes.byref(d), W.ctypes.data, mask.ctypes.data), "celty_decode")
    return W.view(np.float16), mask


# ---------------------------------------------------------------------------
# Device side (torch supplies memory and streams)
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream_handle(stream) -> Optional[int]:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _dev_ptr(t, nbytes_each: int, name: str, min_numel: int = 0, device=None, dtypes=None) -> int:
    """Device address of t after the checks the C ABI cannot make itself: the
    library takes bare pointers and trusts the sizes (x holds K halves, y M,
    idx K ints), so a short or misplaced tensor is rejected here, before any
    launch, rather than read or written out of bounds on the GPU."""
    if not t.is_cuda or not t.is_contiguous() or t.element_size() != nbytes_each:
        raise ValueError(f"{name} must be a contiguous CUDA tensor of {nbytes_each}-byte elements")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}; expected one of {', '.join(str(d) for d in dtypes)}")
    if t.numel() < min_numel:
        raise ValueError(f"{name} holds {t.numel()} elements, fewer than the {min_numel} the call uses")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the encoded matrix on {device}")
    return int(t.data_ptr())


def _half_dtypes():
    """Device tensors that may carry fp16 x or y: float16, or int16 bit patterns."""
    torch = _torch()
    return (torch.float16, torch.int16)


class DeviceRlcCsc:
    """The encoded arrays copied into device tensors, plus a device descriptor."""

    def __init__(self, host: HostRlcCsc, device=None):
        torch = _torch()
        device = torch.device("cuda") if device is None else torch.device(device)
        self.host_header = host
        self.M, self.K, self.R, self.T = host.M, host.K, host.R, host.T
        self.n_groups, self.n_entries = host.n_groups, host.n_entries
        self.n_nnz, self.n_pad = host.n_nnz, host.n_pad
        self.max_abs = host.max_abs
        self.layout = host.layout
        self.gptr = torch.from_numpy(host.gptr.view(np.int32)).to(device)
        # at least one element so that pointers are never null
        self.values = torch.from_numpy(host.values.view(np.int16) if host.values.size
                                       else np.zeros(8, np.int16)).to(device)
        self.runs = torch.from_numpy(host.runs.view(np.int32) if host.runs.size
                                     else np.zeros(1, np.int32)).to(device)
        self.colmax = torch.from_numpy(host.colmax.view(np.int16)).to(device)
        self._desc = self._make_desc()

    def _make_desc(self) -> celty_rlc_csc:
        return celty_rlc_csc(FORMAT_VERSION, self.M, self.K, self.R, self.T, RUN_BITS, self.n_groups,
                             self.n_entries, self.n_nnz, self.n_pad, self.max_abs, self.layout,
                             self.gptr.data_ptr(), self.values.data_ptr(), self.runs.data_ptr(),
                             self.colmax.data_ptr())

    def desc(self) -> celty_rlc_csc:
        return self._desc

    def clone_to(self, device=None) -> "DeviceRlcCsc":
        """A second copy of the arrays at new device addresses."""
        other = object.__new__(DeviceRlcCsc)
        other.__dict__.update(self.__dict__)
        other.gptr, other.values, other.runs = self.gptr.clone(), self.values.clone(), self.runs.clone()
        other.colmax = self.colmax.clone()
        other._desc = other._make_desc()
        return other


def celty_spmspv_workspace_bytes(M: int, K: int, R: int) -> int:
    return int(_ws_bytes(int(M), int(K), int(R)))


def celty_spmspv_workspace_init(workspace, stream=None) -> None:
    _check(_ws_init(_dev_ptr(workspace, 1, "workspace"), workspace.numel(), _stream_handle(stream)),
           "celty_spmspv_workspace_init")


def new_workspace(W: DeviceRlcCsc, device=None):
    """A zero-filled device workspace for W's shape (uint8 tensor)."""
    torch = _torch()
    n = celty_spmspv_workspace_bytes(W.M, W.K, W.R)
    return torch.zeros(n, dtype=torch.uint8, device=device if device is not None else W.gptr.device)


def celty_select(x, tau: float, idx, count, stream=None) -> None:
    K = x.numel()
    _check(_select(_dev_ptr(x, 2, "x", 0, None, _half_dtypes()), K, float(tau), _dev_ptr(idx, 4, "idx", K, x.device),
                   _dev_ptr(count, 4, "count", 1, x.device), _stream_handle(stream)), "celty_select")


def _launch_struct(launch) -> Optional[celty_launch]:
    if launch is None:
        return None
    if isinstance(launch, celty_launch):
        return launch
    cols, waves = launch[0], launch[1]
    groups = launch[2] if len(launch) > 2 else 0
    swizzle = launch[3] if len(launch) > 3 else 0
    return celty_launch(int(cols), int(waves), int(groups), int(swizzle))


def celty_spmspv(W: DeviceRlcCsc, x, tau: float, y, workspace, stream=None) -> None:
    d, dev = W.desc(), W.gptr.device
    hd = _half_dtypes()
    _check(_spmspv(ctypes.byref(d), _dev_ptr(x, 2, "x", W.K, dev, hd), float(tau), _dev_ptr(y, 2, "y", W.M, dev, hd),
                   _dev_ptr(workspace, 1, "workspace", 0, dev), workspace.numel(), _stream_handle(stream)),
           "celty_spmspv")


def celty_spmspv_ex(W: DeviceRlcCsc, x, tau: float, y, workspace, launch=None, stream=None) -> None:
    d, dev = W.desc(), W.gptr.device
    ls = _launch_struct(launch)
    hd = _half_dtypes()
    _check(_spmspv_ex(ctypes.byref(d), _dev_ptr(x, 2, "x", W.K, dev, hd), float(tau), _dev_ptr(y, 2, "y", W.M, dev, hd),
                      _dev_ptr(workspace, 1, "workspace", 0, dev), workspace.numel(),
                      None if ls is None else ctypes.byref(ls), _stream_handle(stream)), "celty_spmspv_ex")


class PreparedSpMSpV:
    """celty_spmspv_ex with its arguments checked and marshalled once.

    For eager serving loops, where the per-call tensor checks and argument
    conversion of celty_spmspv_ex cost more host time than the launch itself:
    the tensors (x, y, workspace) and the stream are fixed here and must stay
    alive and in place; each call passes only tau and goes straight to the C
    entry point (which still validates every argument before launching)."""

    def __init__(self, W: DeviceRlcCsc, x, y, workspace, launch=None, stream=None):
        dev, hd = W.gptr.device, _half_dtypes()
        self._keep = (W, x, y, workspace)
        self._desc = W.desc()
        self._ls = _launch_struct(launch)
        self._args = (ctypes.byref(self._desc), _dev_ptr(x, 2, "x", W.K, dev, hd),
                      _dev_ptr(y, 2, "y", W.M, dev, hd), _dev_ptr(workspace, 1, "workspace", 0, dev),
                      workspace.numel(), None if self._ls is None else ctypes.byref(self._ls),
                      _stream_handle(stream))

    def __call__(self, tau: float) -> None:
        d, x, y, ws, n, ls, st = self._args
        status = _spmspv_ex(d, x, tau, y, ws, n, ls, st)
        if status != CELTY_OK:
            raise CeltyError(status, "celty_spmspv_ex")


def celty_spmspv_noalloc(W: DeviceRlcCsc, x, tau: float, y, launch=None, stream=None) -> None:
    """As celty_spmspv_ex with the library's static merge array (no workspace, nothing allocated)."""
    d, dev = W.desc(), W.gptr.device
    ls = _launch_struct(launch)
    hd = _half_dtypes()
    _check(_spmspv_noalloc(ctypes.byref(d), _dev_ptr(x, 2, "x", W.K, dev, hd), float(tau),
                           _dev_ptr(y, 2, "y", W.M, dev, hd), None if ls is None else ctypes.byref(ls),
                           _stream_handle(stream)), "celty_spmspv_noalloc")


def _desc_array(Ws):
    descs = [W.desc() for W in Ws]
    arr = (ctypes.POINTER(celty_rlc_csc) * len(descs))(*[ctypes.pointer(d) for d in descs])
    return descs, arr


def celty_spmspv_batch_workspace_bytes(Ws) -> int:
    descs, arr = _desc_array(Ws)
    return int(_batch_ws_bytes(len(descs), arr))


def new_batch_workspace(Ws, device=None):
    """A zero-filled device workspace for celty_spmspv_batch over Ws."""
    torch = _torch()
    n = celty_spmspv_batch_workspace_bytes(Ws)
    return torch.zeros(n, dtype=torch.uint8, device=device if device is not None else Ws[0].gptr.device)


def celty_spmspv_batch(Ws, xs, taus, ys, workspace, launch=None, stream=None) -> None:
    """n products y_i = W_i x_i (threshold tau_i) in one launch."""
    n = len(Ws)
    if not (len(xs) == len(taus) == len(ys) == n):
        raise ValueError("Ws, xs, taus and ys must have the same length")
    descs, arr = _desc_array(Ws)
    hd = _half_dtypes()
    xp = (_p * n)(*[_dev_ptr(x, 2, f"xs[{i}]", W.K, W.gptr.device, hd) for i, (W, x) in enumerate(zip(Ws, xs))])
    yp = (_p * n)(*[_dev_ptr(y, 2, f"ys[{i}]", W.M, W.gptr.device, hd) for i, (W, y) in enumerate(zip(Ws, ys))])
    tp = (_f32 * n)(*[float(t) for t in taus])
    ls = _launch_struct(launch)
    dev = Ws[0].gptr.device if n else None
    _check(_batch(n, arr, xp, tp, yp, _dev_ptr(workspace, 1, "workspace", 0, dev), workspace.numel(),
                  None if ls is None else ctypes.byref(ls), _stream_handle(stream)), "celty_spmspv_batch")


def celty_spmspv_plan(W, launch=None) -> dict:
    d = W.desc()
    ls = _launch_struct(launch)
    out, nb, lds = celty_launch(), _i64(), _i64()
    _check(_plan(ctypes.byref(d), None if ls is None else ctypes.byref(ls), ctypes.byref(out),
                 ctypes.byref(nb), ctypes.byref(lds)), "celty_spmspv_plan")
    return dict(cols_per_block=out.cols_per_block, waves_per_block=out.waves_per_block,
                groups_per_lane=out.groups_per_lane, lds_swizzle=out.lds_swizzle, blocks=nb.value,
                lds_bytes=lds.value)


def celty_bench_stream_read(buf, nbytes: int, sink, blocks: int, threads: int, stream=None) -> None:
    """Measurement reference (include/celty_bench.h): one launch that streams
    nbytes of the device tensor buf; sink holds at least `blocks` int32."""
    if int(nbytes) > buf.numel() * buf.element_size():
        raise ValueError("nbytes exceeds the buffer")
    _check(_stream_read(_dev_ptr(buf, buf.element_size(), "buf"), int(nbytes),
                        _dev_ptr(sink, 4, "sink", int(blocks), buf.device), int(blocks), int(threads),
                        _stream_handle(stream)), "celty_bench_stream_read")


def default_tile_rows(M: int, K: int) -> int:
    """Tile height R for encoding an M x K matrix (celty_default_tile_rows)."""
    return int(_default_tile_rows(int(M), int(K)))


__all__ = [
    "FORMAT_VERSION", "LAYOUT_RLC", "LAYOUT_ROWS16", "LAYOUT_INTERLEAVED", "default_tile_rows",
    "celty_encode_plan", "celty_encode", "celty_decode", "celty_select", "celty_spmspv", "celty_spmspv_ex",
    "celty_spmspv_batch", "celty_spmspv_batch_workspace_bytes", "new_batch_workspace", "celty_spmspv_noalloc",
    "celty_spmspv_plan", "celty_spmspv_workspace_bytes", "celty_spmspv_workspace_init", "celty_status_string",
    "celty_bench_stream_read", "PreparedSpMSpV",
    "new_workspace", "HostRlcCsc", "DeviceRlcCsc", "CeltyError", "celty_rlc_csc", "celty_launch",
]
