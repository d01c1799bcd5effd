"""celty_spmspv_noalloc (the entry point that allocates nothing) against
celty_spmspv_ex: the same kernels with the library's static merge array in
place of a caller workspace, so y must agree bit for bit.  Two calls in a
row, the second on a smaller problem (the array keeps the last call's
contents, which every completed call leaves zero); then one that needs more
rows than the array holds, refused before any launch.  Runs through the C
ABI (ctypes), alone in a fresh process or after the other GPU tests."""
import numpy as np
import pytest

import workloads
from oracle import spmspv as ref

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch, torch.device("cuda:0")


def _pair(celty, torch_dev, p, R, launch):
    torch, dev = torch_dev
    Wd = celty.celty_encode(p.W, p.mask, R).to_device(dev)
    x = torch.from_numpy(p.x.view(np.int16)).to(dev)
    y_ref = torch.full((Wd.M,), 0x7C01, dtype=torch.int16, device=dev)
    y = torch.full((Wd.M,), 0x7C01, dtype=torch.int16, device=dev)
    ws = celty.new_workspace(Wd, dev)
    celty.celty_spmspv_ex(Wd, x, p.tau, y_ref, ws, launch)
    celty.celty_spmspv_noalloc(Wd, x, p.tau, y, launch)
    torch.cuda.synchronize()
    a, b = y_ref.cpu().numpy(), y.cpu().numpy()
    assert np.array_equal(a, b)
    err = ref.rel_error(b.view(np.float16).astype(np.float64), ref.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau))
    print(f"noalloc {Wd.M}x{Wd.K} launch={launch}: rel_err={err:.3e}", flush=True)
    assert err <= 2e-3


def test_noalloc_matches_the_workspace_entry_point_twice(torch_dev):
    import paper_2608_01536_amd as celty
    big = workloads.headline_problem(0)                                  # 4096 x 4096, 32 column slices
    small = workloads.random_small(5, 1000, 777, ws=50, as_=50)          # smaller, after the big one
    _pair(celty, torch_dev, big, 512, None)
    _pair(celty, torch_dev, small, 256, None)
    _pair(celty, torch_dev, small, 256, (64, 2, 1))                      # 13 slices, the merge words reused


def test_noalloc_refuses_more_rows_than_the_array(torch_dev):
    import paper_2608_01536_amd as celty
    torch, dev = torch_dev
    M, K = 131073, 4
    W = np.zeros((M, K), dtype=np.float16)
    W[::1000, 1] = np.float16(1.0)
    Wd = celty.celty_encode(W, None, 2048).to_device(dev)
    x = torch.ones(K, dtype=torch.float16, device=dev)
    y = torch.empty(M, dtype=torch.float16, device=dev)
    with pytest.raises(celty.CeltyError) as e:
        celty.celty_spmspv_noalloc(Wd, x, 0.5, y)
    assert e.value.status == celty.CELTY_EINVAL
    Wd2 = celty.celty_encode(W[:131072], None, 2048).to_device(dev)   # exactly the array's rows
    y2 = torch.empty(131072, dtype=torch.float16, device=dev)
    celty.celty_spmspv_noalloc(Wd2, x, 0.5, y2, (1, 2, 1))             # 4 column slices: every merge word
    torch.cuda.synchronize()
    want = ref.spmspv_dense_fp64(W[:131072], None, x.cpu().numpy(), 0.5)
    assert np.array_equal(y2.cpu().numpy().astype(np.float64), want)
