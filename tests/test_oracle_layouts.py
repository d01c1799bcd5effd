"""The oracle's two other row encodings (oracle/layouts.py), pinned.

* hand-worked fixtures (tests/golden/layouts_worked_cases.txt);
* rows16: round trip to the dense masked matrix, row order, alignment rows,
  group counts from the stored counts;
* interleaved: on a full 64-group chunk, group l holds the row-order entries
  l + 64 j (Section 4.2's pattern with a 64-lane wavefront); rows read
  straight from the interleaved arrays equal the tiled format's rows; round
  trip to the dense masked matrix, padding entries included.
"""
import os

import numpy as np
import pytest

import workloads
from oracle import layouts, rlc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "layouts_worked_cases.txt")


def _fixture():
    out = {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = line.split(":", 1)
            out[key.strip()] = val.strip()
    return out


def _segments(text, dtype=float):
    return [[dtype(v) for v in part.split()] for part in text.split(" - ")]


def _half_bits(vals):
    return np.array(vals, dtype=np.float16).view(np.uint16)


def test_rows16_fixture():
    fx = _fixture()
    M, K, R = (int(v) for v in fx["rows16.shape"].split())
    W = np.zeros((M, K), dtype=np.float16)
    for ent in fx["rows16.entries"].split("|"):
        r, k, v = ent.split()
        W[int(r), int(k)] = np.float16(float(v))
    enc = layouts.encode_rows16(W, None, R)
    assert enc.gptr.tolist() == [int(v) for v in fx["rows16.gptr"].split()]
    assert np.array_equal(enc.values, _half_bits(sum(_segments(fx["rows16.values"]), [])))
    assert enc.rows.tolist() == sum(_segments(fx["rows16.rows"], int), [])
    assert enc.n_nnz == 7
    assert enc.colmax.tolist() == _half_bits([2.0, 4.0]).tolist()


def test_interleaved_fixture():
    fx = _fixture()
    M, K, R = (int(v) for v in fx["interleaved.shape"].split())
    W = np.zeros((M, K), dtype=np.float16)
    for i in range(20):
        W[2 * i, 0] = np.float16(i + 1)
    enc = layouts.encode_interleaved(W, None, R)
    assert enc.gptr.tolist() == [0, 3]
    assert np.array_equal(enc.values, _half_bits(sum(_segments(fx["interleaved.values"]), [])))
    assert rlc.unpack_runs(enc.runs).tolist() == sum(_segments(fx["interleaved.runs"], int), [])
    rows, _ = layouts.interleaved_segment_rows(enc, 0)
    assert rows.tolist() == sum(_segments(fx["interleaved.rows"], int), [])


def _random(seed, M, K, ws):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((M, K)).astype(np.float16)
    mask = (rng.random((M, K)) >= ws).astype(np.uint8)
    W[rng.random((M, K)) < 0.01] = np.float16(0)          # kept zeros are not stored
    return W, mask


def _masked(W, mask):
    Wb = W.view(np.uint16)
    keep = rlc.stored_mask(Wb, mask)
    return np.where(keep, Wb, np.uint16(0)), keep


@pytest.mark.parametrize("seed,M,K,R,ws", [(0, 70, 9, 16, 0.5), (1, 100, 5, 37, 0.9), (2, 33, 4, 64, 0.0),
                                           (3, 1, 3, 1, 0.3), (4, 257, 3, 256, 0.97)])
def test_rows16_round_trip_and_invariants(seed, M, K, R, ws):
    W, mask = _random(seed, M, K, ws)
    enc = layouts.encode_rows16(W, mask, R)
    Wd, md = layouts.decode_rows16(enc)
    want, keep = _masked(W, mask)
    assert np.array_equal(Wd.view(np.uint16), want)
    assert np.array_equal(md != 0, keep)
    # groups from the stored counts, no padding entries
    assert enc.n_groups == int(np.sum(-(-enc.seg_n // 8)))
    assert int(enc.seg_n.sum()) == enc.n_nnz == int(keep.sum())
    for s in range(enc.T * enc.K):
        e0, e1 = 8 * int(enc.gptr[s]), 8 * int(enc.gptr[s + 1])
        n = int(enc.seg_n[s])
        rows = enc.rows[e0:e1].astype(np.int64)
        assert np.all(np.diff(rows[:n]) > 0)                      # stored rows strictly increase
        assert np.all(rows[n:] == (rows[n - 1] if n else 0))      # alignment repeats the last row
        assert np.all(enc.values[e0 + n:e1] == 0)
        assert np.all(rows < R)


def test_rows16_rejects_tall_tiles():
    with pytest.raises(ValueError):
        layouts.encode_rows16(np.ones((4, 2), dtype=np.float16), None, 65537)


def test_interleaved_full_chunk_is_lane_strided():
    # a dense column of 1024 rows: 128 groups, two full chunks of 64
    M = 1024
    W = (np.arange(M) % 2000 + 1).astype(np.float16).reshape(M, 1)
    v1 = rlc.encode_matrix(W, None, M)
    il = layouts.encode_interleaved(W, None, M)
    assert il.gptr.tolist() == v1.gptr.tolist() == [0, 128]
    for c in range(2):
        for lane in range(64):
            for j in range(8):
                stored = 8 * (64 * c + lane) + j
                row_order = 8 * 64 * c + lane + 64 * j
                assert il.values[stored] == v1.values[row_order]


@pytest.mark.parametrize("seed,M,K,R,ws", [(5, 600, 3, 600, 0.2), (6, 2100, 2, 1024, 0.5), (7, 90, 7, 45, 0.95),
                                           (8, 300, 4, 128, 0.0)])
def test_interleaved_rows_and_round_trip(seed, M, K, R, ws):
    W, mask = _random(seed, M, K, ws)
    v1 = rlc.encode_matrix(W, mask, R)
    il = layouts.encode_interleaved(W, mask, R)
    assert np.array_equal(il.gptr, v1.gptr) and il.n_pad == v1.n_pad and il.n_nnz == v1.n_nnz
    for s in range(v1.T * v1.K):
        if v1.gptr[s] == v1.gptr[s + 1]:
            continue
        rows_v1, vals_v1 = rlc.segment_rows(v1, s)
        rows_il, vals_il = layouts.interleaved_segment_rows(il, s)
        # the same (row, value) pairs, each once: a permutation within the segment
        a = sorted(zip(rows_v1.tolist(), vals_v1.tolist()))
        b = sorted(zip(rows_il.tolist(), vals_il.tolist()))
        assert a == b
    Wd, md = layouts.decode_interleaved(il)
    want, keep = _masked(W, mask)
    assert np.array_equal(Wd.view(np.uint16), want)
    assert np.array_equal(md != 0, keep)
    assert np.array_equal(layouts.deinterleave(il).values, v1.values)
    assert np.array_equal(layouts.deinterleave(il).runs, v1.runs)


def test_interleaved_with_padding_entries():
    # gaps of 40 and 100 rows need padding entries (0, 15): they are entries
    # of the sequence and are interleaved like any other
    M = 512
    W = np.zeros((M, 1), dtype=np.float16)
    W[[3, 44, 145, 146, 400, 511], 0] = np.float16(1.5)
    v1 = rlc.encode_matrix(W, None, M)
    assert v1.n_pad > 0
    il = layouts.encode_interleaved(W, None, M)
    Wd, _ = layouts.decode_interleaved(il)
    assert np.array_equal(Wd.view(np.uint16), W.view(np.uint16))


def test_encodings_of_a_benchmark_problem():
    p = workloads.random_small(3, 300, 200, ws=70, as_=70)
    r16 = layouts.encode_rows16(p.W, p.mask, 64)
    Wd, _ = layouts.decode_rows16(r16)
    want, _ = _masked(p.W, p.mask)
    assert np.array_equal(Wd.view(np.uint16), want)
    il = layouts.encode_interleaved(p.W, p.mask, 64)
    Wd, _ = layouts.decode_interleaved(il)
    assert np.array_equal(Wd.view(np.uint16), want)
