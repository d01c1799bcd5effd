"""The library's host encoder is bit-exact with the oracle's encoder.

gptr, values, runs, colmax and the header counts must match exactly, for any tile
height R, thread count, odd shapes, kept +-0 weights, empty and full columns,
and at the full 4096 x 4096 / 11008 x 4096 sizes of the benchmark configs.
"""
import numpy as np
import pytest

import paper_2608_01536_amd as celty
import workloads
from oracle import rlc


def _assert_same(enc, ref):
    assert enc.M == ref.M and enc.K == ref.K and enc.R == ref.R and enc.T == ref.T
    assert enc.n_groups == ref.n_groups
    assert enc.n_nnz == ref.n_nnz and enc.n_pad == ref.n_pad
    assert enc.n_entries == ref.n_entries
    assert np.array_equal(enc.gptr, ref.gptr)
    assert np.array_equal(enc.values, ref.values)
    assert np.array_equal(enc.runs, ref.runs)
    assert np.array_equal(enc.colmax, ref.colmax)
    assert enc.max_abs == float(ref.colmax.view(np.float16).astype(np.float32).max(initial=0.0))


SHAPES = [(1, 1, 1), (1, 9, 4), (9, 1, 4), (7, 8, 3), (64, 64, 64), (65, 63, 16), (200, 31, 1000),
          (1023, 5, 256), (1025, 17, 256), (300, 40, 7)]


@pytest.mark.parametrize("M,K,R", SHAPES)
@pytest.mark.parametrize("ws", [0, 50, 95])
def test_encoder_matches_oracle_small(M, K, R, ws):
    p = workloads.random_small(M * 7 + K * 3 + R + ws, M, K, ws=ws, as_=50, zero_weights=3)
    enc = celty.celty_encode(p.W, p.mask, R)
    _assert_same(enc, rlc.encode_matrix(p.W, p.mask, R))


@pytest.mark.parametrize("n_threads", [1, 2, 3, 0])
def test_encoder_thread_count_does_not_matter(n_threads):
    p = workloads.random_small(4, 1500, 1100, ws=70, as_=50)
    enc = celty.celty_encode(p.W, p.mask, 128, n_threads=n_threads)
    _assert_same(enc, rlc.encode_matrix(p.W, p.mask, 128))


def test_encoder_null_mask_and_long_gaps():
    rng = np.random.default_rng(5)
    M, K = 700, 9
    W = np.zeros((M, K), dtype=np.float16)
    # a handful of entries with gaps far beyond 15 rows, plus a dense column
    for k in range(K - 1):
        rows = np.sort(rng.choice(M, size=4, replace=False))
        W[rows, k] = rng.standard_normal(4).astype(np.float16) + np.float16(2)
    W[:, K - 1] = np.float16(1.5)
    for R in (1, 16, 100, 700, 4096):
        enc = celty.celty_encode(W, None, R)
        _assert_same(enc, rlc.encode_matrix(W, None, R))
        Wd, m = celty.celty_decode(enc)
        assert np.array_equal(Wd.view(np.uint16), W.view(np.uint16))


def test_plan_matches_encode():
    p = workloads.random_small(8, 333, 222, ws=40, as_=50)
    g, n, pad = celty.celty_encode_plan(p.W, p.mask, 32)
    enc = celty.celty_encode(p.W, p.mask, 32)
    assert (g, n, pad) == (enc.n_groups, enc.n_nnz, enc.n_pad)


@pytest.mark.parametrize("M,K,R", [(200, 300, 64), (1000, 77, 256)])
def test_library_decoder_round_trip(M, K, R):
    p = workloads.random_small(M + K, M, K, ws=60, as_=50, zero_weights=6)
    enc = celty.celty_encode(p.W, p.mask, R)
    W2, m2 = celty.celty_decode(enc)
    stored = (p.mask != 0) & ((p.W.view(np.uint16) & 0x7FFF) != 0)
    assert np.array_equal(m2, stored.astype(np.uint8))
    assert np.array_equal(W2.view(np.uint16), np.where(stored, p.W.view(np.uint16), 0).astype(np.uint16))


@pytest.mark.slow
@pytest.mark.parametrize("ws,R", [(30, 256), (50, 1024), (70, 256)])
def test_encoder_full_size_4096(ws, R):
    p = workloads.make_problem(2, 4096, 4096, ws, 50, "laplace", seed=0)
    enc = celty.celty_encode(p.W, p.mask, R)
    _assert_same(enc, rlc.encode_matrix(p.W, p.mask, R))


@pytest.mark.slow
def test_encoder_full_size_row_magnitude_11008():
    # a gate/up-shaped projection with per-row magnitude pruning (config 3)
    p = workloads.make_problem(3, 11008, 4096, 50, 50, "student_t4", seed=0, proj=4,
                               mask_kind="row_magnitude")
    enc = celty.celty_encode(p.W, p.mask, 256)
    _assert_same(enc, rlc.encode_matrix(p.W, p.mask, 256))


@pytest.mark.parametrize("M,K,R", [(300, 200, 64), (77, 5, 16)])
def test_header_max_abs(M, K, R):
    p = workloads.random_small(M * K, M, K, ws=50, as_=50, zero_weights=2)
    enc = celty.celty_encode(p.W, p.mask, R)
    stored = (p.mask != 0) & ((p.W.view(np.uint16) & 0x7FFF) != 0)
    want = float(np.max(np.abs(p.W.astype(np.float32))[stored])) if stored.any() else 0.0
    assert enc.max_abs == want
    # subnormal-only matrix: exact conversion of fp16 subnormals
    Ws = np.zeros((4, 4), dtype=np.float16)
    Ws.view(np.uint16)[1, 2] = 0x0003
    Ws.view(np.uint16)[3, 0] = 0x8201
    e2 = celty.celty_encode(Ws, None, 2)
    assert e2.max_abs == float(np.abs(Ws.astype(np.float32)).max())
    assert celty.celty_encode(np.zeros((3, 3), np.float16), None, 2).max_abs == 0.0
