"""The device path from a plain C process with no PyTorch in it.

``tests/c_spmspv_client.c`` (compiled by ``__graft_entry__.build()``) encodes
with the host encoder, copies the arrays into ``hipMalloc`` memory, fills the
workspace with ``celty_spmspv_workspace_init`` and runs ``celty_spmspv`` on the
null stream.  Its y must meet the same bound against the oracle as the
Python-driven parity tests.
"""
import os
import struct
import subprocess

import numpy as np
import pytest

import workloads
from oracle import spmspv as ref

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "tests", "_bin", "c_spmspv_client")
TOL = 2e-3


@pytest.mark.parametrize("M,K,R,ws,as_", [(700, 513, 256, 50, 50), (1500, 300, 64, 30, 90),
                                           (4096, 4096, 512, 70, 70), (11008, 4096, 1024, 50, 50)])
def test_c_client_matches_the_oracle(tmp_path, M, K, R, ws, as_):
    if not os.path.exists(CLIENT):
        pytest.fail(f"{CLIENT} is not built: run __graft_entry__.build()")
    p = workloads.random_small(M + K + R + ws, M, K, ws=ws, as_=as_)
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        f.write(struct.pack("<iiif", M, K, R, float(p.tau)))
        f.write(np.ascontiguousarray(p.W).view(np.uint16).tobytes())
        f.write(np.ascontiguousarray(p.mask).astype(np.uint8).tobytes())
        f.write(np.ascontiguousarray(p.x).view(np.uint16).tobytes())
    print(f"c client M={M} K={K} R={R} ws={ws} as={as_}", flush=True)
    run = subprocess.run([CLIENT, str(src), str(dst)], capture_output=True, text=True, timeout=90)
    assert run.returncode == 0, f"client exit {run.returncode}: {run.stderr[-2000:]}"
    y = np.fromfile(dst, dtype=np.float16)
    assert y.shape == (M,)
    assert np.all(np.isfinite(y))
    err = ref.rel_error(y.astype(np.float64), ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau))
    assert err <= TOL, err
