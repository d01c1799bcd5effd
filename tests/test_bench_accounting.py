"""bench.py's byte count (from the encoded arrays) equals the oracle's
accounting (from the loop encoder's entry counts) on random problems."""
import numpy as np
import pytest

import bench
import paper_2608_01536_amd as celty
import workloads
from oracle import accounting, rlc, spmspv


@pytest.mark.parametrize("M,K,R,ws,as_", [(300, 200, 64, 50, 50), (1000, 77, 256, 90, 30),
                                          (129, 1000, 16, 20, 70), (50, 50, 1000, 0, 0)])
def test_bench_bytes_match_oracle(M, K, R, ws, as_):
    p = workloads.random_small(M + K + R, M, K, ws=ws, as_=as_, zero_weights=2)
    enc = celty.celty_encode(p.W, p.mask, R)
    b, e_a, g_a = bench.algorithmic_bytes_from_encoding(enc, p.x, p.tau)
    o = rlc.encode_matrix(p.W, p.mask, R)
    assert b == accounting.algorithmic_bytes(o, p.x, p.tau)
    act = spmspv.select_active(p.x, p.tau)
    assert e_a == accounting.active_entries(o, act)
    assert g_a == accounting.active_groups(o, act)
