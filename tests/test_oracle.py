"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Every check here compares the oracle with something that is not the oracle:
the paper's worked RLC example, hand-derived gap cases, the plain per-column
loop encoder, numpy/scipy library routines, closed forms and invariants.
"""
import os

import numpy as np
import pytest

from oracle import accounting, rlc, spmspv
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_cases(name):
    cases, cur = [], {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, val = line.partition(":")
            cur[key.strip()] = val.strip()
            if key.strip() == "runs":
                cases.append(cur)
                cur = {}
    return cases


def _expand_column(spec):
    """'4:1 16:2 20:' -> 4 zeros, 1, 16 zeros, 2, 20 zeros."""
    col = []
    for tok in spec.split():
        z, _, v = tok.partition(":")
        col += [0] * int(z)
        if v:
            col.append(int(v))
    return col


def _ints(s):
    return [int(t) for t in s.split()]


# --------------------------------------------------------------------------
# Run-length coding of one column (Section 3.2)
# --------------------------------------------------------------------------
def test_paper_worked_example():
    (c,) = _read_cases("rlc_worked_example.txt")
    col = _ints(c["column"])
    vals, runs = rlc.rlc_encode_column(col, int(c["n_bits"]))
    assert vals == _ints(c["values"])
    assert runs == _ints(c["runs"])
    assert rlc.rlc_decode_column(vals, runs, len(col)) == col


def test_worked_example_rows_by_algorithm1():
    # rows = inclusive prefix of runs + ordinal: 4 at row 2, padding at 6, 2 at 7, 8 at 8
    rows = rlc.alg1_rows(np.array([2, 3, 0, 0]), per_lane=1)
    assert rows.tolist() == [2, 6, 7, 8]


@pytest.mark.parametrize("case", range(5))
def test_gap_cases_4bit(case):
    c = _read_cases("rlc_gap_cases.txt")[case]
    col = _expand_column(c["column"])
    vals, runs = rlc.rlc_encode_column(col, int(c["n_bits"]))
    assert vals == _ints(c["values"])
    assert runs == _ints(c["runs"])
    assert rlc.rlc_decode_column(vals, runs, len(col)) == col


@pytest.mark.parametrize("n_bits", [1, 2, 3, 4, 5])
def test_column_round_trip_and_slot_count(n_bits):
    rng = np.random.default_rng(n_bits)
    cap = (1 << n_bits) - 1
    for _ in range(50):
        L = int(rng.integers(1, 300))
        col = np.where(rng.random(L) < rng.random(), rng.integers(1, 9, L), 0).tolist()
        vals, runs = rlc.rlc_encode_column(col, n_bits)
        assert rlc.rlc_decode_column(vals, runs, L) == col
        assert all(0 <= r <= cap for r in runs)
        nz = [i for i, v in enumerate(col) if v]
        # every entry, padding included, occupies one row position
        if nz:
            assert sum(r + 1 for r in runs) == nz[-1] + 1
        # closed form for the number of padding entries
        gaps = np.diff([-1] + nz) - 1
        assert len(vals) - len(nz) == int(np.sum(gaps // (cap + 1)))


# --------------------------------------------------------------------------
# Algorithm 1 (intra-warp prefix sum) against numpy's cumsum
# --------------------------------------------------------------------------
@pytest.mark.parametrize("lanes,per", [(32, 8), (64, 8), (4, 2), (1, 8)])
def test_algorithm1_matches_cumsum(lanes, per):
    rng = np.random.default_rng(lanes * 10 + per)
    runs = rng.integers(0, 16, size=(lanes, per))
    pre = rlc.alg1_prefix(runs)
    assert np.array_equal(pre.reshape(-1), np.cumsum(runs.reshape(-1)))
    rows = rlc.alg1_rows(runs.reshape(-1), per_lane=per)
    assert np.array_equal(rows, np.cumsum(runs.reshape(-1)) + np.arange(runs.size))


# --------------------------------------------------------------------------
# Tiled RLC-CSC for a matrix
# --------------------------------------------------------------------------
def _encode_by_loop(W, mask, R):
    """Reference built from the plain per-column loop, segment by segment."""
    Wb = W.view(np.uint16)
    M, K = Wb.shape
    T = -(-M // R)
    vals_all, runs_all, gptr = [], [], [0]
    n_pad = 0
    for t in range(T):
        for k in range(K):
            seg = [int(Wb[r, k]) if (mask is None or mask[r, k]) and (int(Wb[r, k]) & 0x7FFF) else 0
                   for r in range(t * R, min(M, (t + 1) * R))]
            v, r = rlc.rlc_encode_column(seg, 4)
            n_pad += sum(1 for a in v if a == 0)
            while len(v) % 8:
                v.append(0)
                r.append(0)
            vals_all += v
            runs_all += r
            gptr.append(gptr[-1] + len(v) // 8)
    runs_words = []
    for g in range(len(runs_all) // 8):
        w = 0
        for j in range(8):
            w |= runs_all[8 * g + j] << (4 * j)
        runs_words.append(w)
    return (np.array(gptr, dtype=np.uint32), np.array(vals_all, dtype=np.uint16),
            np.array(runs_words, dtype=np.uint32), n_pad)


SMALL_SHAPES = [(1, 1, 1), (3, 7, 2), (8, 9, 8), (17, 5, 4), (65, 3, 16), (40, 6, 1000),
                (63, 64, 32), (130, 10, 64)]


@pytest.mark.parametrize("M,K,R", SMALL_SHAPES)
@pytest.mark.parametrize("density", [0.05, 0.5, 1.0])
def test_matrix_encoder_matches_loop(M, K, R, density):
    rng = np.random.default_rng(M * 1000 + K * 10 + R)
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float16)
    mask = (rng.random((M, K)) < density).astype(np.uint8)
    # plant kept +0 / -0 weights (not stored) and an all-kept column
    Wb = W.view(np.uint16)
    Wb[rng.random((M, K)) < 0.05] = 0
    Wb[rng.random((M, K)) < 0.05] = 0x8000
    mask[:, 0] = 1
    enc = rlc.encode_matrix(W, mask, R)
    gptr, vals, runs, n_pad = _encode_by_loop(W, mask, R)
    assert np.array_equal(enc.gptr, gptr)
    assert np.array_equal(enc.values, vals)
    assert np.array_equal(enc.runs, runs)
    assert enc.n_pad == n_pad
    stored = mask.astype(bool) & ((Wb & 0x7FFF) != 0)
    assert enc.n_nnz == int(stored.sum())


@pytest.mark.parametrize("M,K,R", SMALL_SHAPES + [(300, 40, 128), (1025, 3, 256)])
def test_matrix_round_trip(M, K, R):
    rng = np.random.default_rng(7 + M + K + R)
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float16)
    mask = (rng.random((M, K)) < 0.4).astype(np.uint8)
    W.view(np.uint16)[rng.random((M, K)) < 0.03] = 0x8000
    enc = rlc.encode_matrix(W, mask, R)
    W2, m2 = rlc.decode_matrix(enc)
    stored = (mask != 0) & ((W.view(np.uint16) & 0x7FFF) != 0)
    assert np.array_equal(m2, stored.astype(np.uint8))
    assert np.array_equal(W2.view(np.uint16), np.where(stored, W.view(np.uint16), 0).astype(np.uint16))
    # every segment starts on a group boundary, runs are 4-bit by construction
    assert enc.values.size == 8 * enc.n_groups


def test_decoder_rejects_bad_streams():
    rng = np.random.default_rng(3)
    W = (rng.standard_normal((20, 4)) * 0.02).astype(np.float16)
    enc = rlc.encode_matrix(W, None, 8)
    bad = rlc.RlcCsc(**{**enc.__dict__, "gptr": enc.gptr[::-1].copy()})
    with pytest.raises(ValueError):
        rlc.decode_matrix(bad)
    # a stored entry pushed past its tile by an inflated run
    runs = enc.runs.copy()
    runs[enc.gptr[1] - 1] |= np.uint32(0xF << 28)
    vals = enc.values.copy()
    vals[8 * enc.gptr[1] - 1] = 0x3C00
    with pytest.raises(ValueError):
        rlc.decode_matrix(rlc.RlcCsc(**{**enc.__dict__, "runs": runs, "values": vals}))


def test_empty_matrix_and_pruned_everything():
    W = np.zeros((5, 3), dtype=np.float16)
    enc = rlc.encode_matrix(W, None, 2)
    assert enc.n_groups == 0 and enc.gptr.tolist() == [0] * (3 * 3 + 1)
    W2, m2 = rlc.decode_matrix(enc)
    assert not m2.any()


# --------------------------------------------------------------------------
# Products
# --------------------------------------------------------------------------
def test_bruteforce_hand_example():
    W = np.array([[1, 2, 0], [0, -1, 3]], dtype=np.float16)
    x = np.array([1, 0.5, -2], dtype=np.float16)
    y = spmspv.spmspv_bruteforce(W, None, x, 0.6)     # column 1 is inactive
    assert y.tolist() == [1.0, -6.0]
    assert spmspv.spmspv_dense_fp64(W, None, x, 0.6).tolist() == [1.0, -6.0]
    assert spmspv.spmspv_csc_fp64(W, None, x, 0.6).tolist() == [1.0, -6.0]
    assert spmspv.select_active(x, 0.6).tolist() == [0, 2]
    assert spmspv.select_active(x, 0.5).tolist() == [0, 2]    # strict
    assert spmspv.select_active(x, -1).tolist() == [0, 1, 2]


TINY = [1, 2, 3, 7, 8, 9, 15, 16, 17, 63, 64, 65]


@pytest.mark.parametrize("M", TINY[::2] + [33])
@pytest.mark.parametrize("K", TINY[1::2])
def test_three_paths_agree(M, K):
    p = workloads.random_small(M * 100 + K, M, K, ws=50, as_=50, zero_weights=2)
    yb = spmspv.spmspv_bruteforce(p.W, p.mask, p.x, p.tau)
    yd = spmspv.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)
    yc = spmspv.spmspv_csc_fp64(p.W, p.mask, p.x, p.tau)
    scale = np.max(np.abs(yd)) + 1e-300
    assert np.max(np.abs(yd - yb)) <= 1e-12 * scale
    assert np.max(np.abs(yd - yc)) <= 1e-12 * scale


@pytest.mark.parametrize("R", [1, 7, 16, 64, 512])
def test_rlc_walk_equals_definition(R):
    p = workloads.random_small(R, 200, 57, ws=60, as_=40, zero_weights=5)
    enc = rlc.encode_matrix(p.W, p.mask, R)
    y1 = spmspv.spmspv_dense_fp64(p.W, p.mask, p.x, p.tau)
    y2 = spmspv.spmspv_rlc_fp64(enc, p.x, p.tau)
    assert np.max(np.abs(y1 - y2)) <= 1e-12 * (np.max(np.abs(y1)) + 1e-300)


def test_invariants():
    p = workloads.random_small(5, 90, 70, ws=50, as_=50)
    f = spmspv.spmspv_dense_fp64
    y = f(p.W, p.mask, p.x, p.tau)
    assert np.all(f(p.W, p.mask, np.zeros_like(p.x), p.tau) == 0)                  # x = 0
    assert np.all(f(p.W, p.mask, p.x, float(np.max(np.abs(p.x.astype(np.float32))))) == 0)
    assert np.allclose(f(p.W, p.mask, -p.x, p.tau), -y, rtol=0, atol=1e-15)        # sign
    x2 = (p.x.astype(np.float32) * 2).astype(np.float16)
    assert np.allclose(f(p.W, p.mask, x2, 2 * p.tau), 2 * y, rtol=0, atol=1e-15)  # scaling
    perm = np.random.default_rng(0).permutation(p.W.shape[1])                     # columns
    assert np.allclose(f(p.W[:, perm], p.mask[:, perm], p.x[perm], p.tau), y, rtol=1e-12, atol=1e-15)


def test_linearity_fixed_support():
    rng = np.random.default_rng(11)
    W = (rng.standard_normal((31, 45)) * 0.02).astype(np.float16)
    mask = (rng.random((31, 45)) < 0.5).astype(np.uint8)
    x1, x2 = rng.standard_normal(45), rng.standard_normal(45)
    f = spmspv.spmspv_dense_fp64
    lhs = f(W, mask, 3 * x1 - 0.5 * x2, -1.0)
    rhs = 3 * f(W, mask, x1, -1.0) - 0.5 * f(W, mask, x2, -1.0)
    assert np.max(np.abs(lhs - rhs)) <= 1e-12 * np.max(np.abs(lhs))


def test_special_cases():
    rng = np.random.default_rng(2)
    M, K = 37, 29
    W = (rng.standard_normal((M, K)) * 0.02).astype(np.float16)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    # one-hot x returns column k of W o Mask
    for k in (0, 13, K - 1):
        x = np.zeros(K, dtype=np.float16)
        x[k] = 1
        y = spmspv.spmspv_dense_fp64(W, mask, x, 0.5)
        assert np.array_equal(y, np.where(mask[:, k] != 0, W[:, k].astype(np.float64), 0.0))
    # identity pattern returns x on the active set
    I = np.eye(K, dtype=np.float16)
    x = rng.laplace(size=K).astype(np.float16)
    tau = 0.7
    y = spmspv.spmspv_csc_fp64(I, None, x, tau)
    assert np.array_equal(y, np.where(np.abs(x.astype(np.float32)) > tau, x.astype(np.float64), 0.0))
    # tau < 0: weight-only SpMV, equals scipy CSC SpMV and a textbook GEMV loop
    x = rng.standard_normal(K).astype(np.float16)
    y = spmspv.spmspv_dense_fp64(W, mask, x, -1.0)
    import scipy.sparse as sp
    A = sp.csc_matrix(np.where(mask != 0, W.astype(np.float64), 0.0))
    assert np.allclose(y, A @ x.astype(np.float64), rtol=1e-13, atol=1e-16)
    gemv = [sum(float(W[r, k]) * float(x[k]) for k in range(K)) for r in range(M)]
    assert np.allclose(spmspv.spmspv_dense_fp64(W, None, x, -1.0), gemv, rtol=1e-12, atol=1e-16)
    # NaN activations are never active
    xn = x.copy()
    xn[3] = np.nan
    assert 3 not in spmspv.select_active(xn, -1.0).tolist()


# --------------------------------------------------------------------------
# Accounting and the paper's size claims (Section 3.2)
# --------------------------------------------------------------------------
def test_algorithmic_bytes_counts_active_entries():
    p = workloads.random_small(21, 70, 50, ws=70, as_=50)
    R = 16
    enc = rlc.encode_matrix(p.W, p.mask, R)
    act = spmspv.select_active(p.x, p.tau)
    # independent count: loop-encode each active segment and count its entries
    Wb = p.W.view(np.uint16)
    e = 0
    for k in act:
        for t in range(enc.T):
            seg = [1 if p.mask[r, k] and (int(Wb[r, k]) & 0x7FFF) else 0
                   for r in range(t * R, min(70, (t + 1) * R))]
            e += len(rlc.rlc_encode_column(seg, 4)[0])
    assert accounting.active_entries(enc, act) == e
    assert accounting.algorithmic_bytes(enc, p.x, p.tau) == 2.5 * e + 2 * 50 + 2 * 70


@pytest.mark.slow
def test_compression_ratio_4096_at_50pct():
    rng = np.random.default_rng(0)
    M = K = 4096
    W = workloads.draw_weight(rng, M, K)
    mask = workloads.draw_mask_uniform(rng, M, K, 50)
    enc = rlc.encode_matrix(W, mask, 1024)
    dense = accounting.dense_bytes(M, K)
    ratio = accounting.rlc_csc_bytes(enc) / dense
    # the paper quotes ~63 % for 4-bit RLC-CSC at 50 % sparsity on 4096^2
    assert abs(ratio - 0.63) < 0.005, ratio
    assert abs(accounting.rlc_csc_entry_bytes(enc) / dense - 0.625) < 0.002
    # and ~56 % for a bitmap (theoretical); closed form (d*16 + 1)/16 at d = 0.5
    bm = accounting.bitmap_bytes(M, K, enc.n_nnz) / dense
    assert abs(bm - 0.5625) < 0.002
    assert round(bm * 100) == 56


# --------------------------------------------------------------------------
# Column maxima (the product's scale data) and the acceptance measure
# --------------------------------------------------------------------------
@pytest.mark.parametrize("M,K,R", [(1, 1, 1), (9, 5, 4), (70, 33, 16), (200, 57, 64)])
def test_column_maxima_against_a_loop(M, K, R):
    p = workloads.random_small(M * 31 + K, M, K, ws=60, as_=50, zero_weights=3)
    Wb = p.W.view(np.uint16)
    enc = rlc.encode_matrix(p.W, p.mask, R)
    for k in range(K):
        best = 0.0
        for r in range(M):
            if p.mask[r, k] and float(p.W[r, k]) != 0.0:
                best = max(best, abs(float(p.W[r, k])))
        assert float(enc.colmax[k:k + 1].view(np.float16)[0]) == best
        assert (int(enc.colmax[k]) & 0x8000) == 0
    assert int(enc.colmax.max()) == max([int(b) & 0x7FFF for b, m in zip(Wb.ravel(), p.mask.ravel()) if m], default=0)


def test_column_maxima_hand_case():
    W = np.array([[1, 0, -65504], [-3, 0.5, 2], [0, -0.0, 6.1e-5]], dtype=np.float16)
    mask = np.array([[1, 1, 0], [1, 1, 1], [1, 1, 1]], dtype=np.uint8)
    enc = rlc.encode_matrix(W, mask, 2)
    # column 0: |-3|; column 1: 0.5 (the kept -0 is not stored); column 2: the
    # masked -65504 does not count, 2 does
    assert enc.colmax.view(np.float16).tolist() == [3.0, 0.5, 2.0]
    assert rlc.encode_matrix(np.zeros((2, 2), np.float16), None, 1).colmax.tolist() == [0, 0]


@pytest.mark.parametrize("y,ref,want", [
    ([1, 2], [1, 2], 0.0),
    ([1.5, 2], [1, 2], 0.2499998750000625),              # 0.5 / (2 + 1e-6)
    ([-1, 0], [1, 0], 1.999998000002),                   # a sign slip counts twice the value
    ([0, 3e-9], [0, 0], 0.003),                          # all-zero reference: the 1e-6 floor
    ([0.1, 0, 0, 0], [0, 0, 0, 0.2], 0.9999950000249999),  # the largest deviation, not the mean
    ([0, -3], [0, -4], 0.24999993750001562),             # magnitude of a negative reference
    ([], [], 0.0),
])
def test_rel_error_hand_values(y, ref, want):
    # expected values computed in exact rational arithmetic from the criterion
    # max_r |y - y*| / (max_r |y*| + 1e-6)
    got = spmspv.rel_error(np.array(y, dtype=np.float64), np.array(ref, dtype=np.float64))
    assert got == pytest.approx(want, rel=1e-15, abs=0.0)
