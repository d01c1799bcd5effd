"""Run-length compressed CSC (RLC-CSC), Section 3.2 and Algorithm 1.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper facts used here
---------------------
* A column is stored as its non-zero values plus, per value, an n-bit run
  length: the count of zeros that precede that value (Section 3.2).
* A gap longer than 2^n - 1 is bridged with zero-valued padding entries; the
  worked 2-bit example maps [0,0,4,0,0,0,0,2,8] to values [4,0,2,8] and runs
  [2,3,0,0], so the padding goes first and carries the largest run 2^n - 1,
  and a padding entry itself takes one row position (Section 3.2).
* The absolute row of an entry is the inclusive prefix sum of the run lengths
  plus the entry's ordinal (Section 3.3, Algorithm 1).
* Celty uses n = 4 (Section 3.2); values are fp16 (Section 3.1).

Readings where the paper is silent (the same list is kept with the design notes):
* trailing zeros of a column are not encoded;
* a kept weight whose value is +0 or -0 is not stored (it is treated like a
  pruned one), so a zero value always means padding or alignment;
* the rows are cut into tiles of R rows and the runs restart at each tile;
  the segment (tile t, column k) is stored at position s = t*K + k;
* each segment is padded to a multiple of 8 entries with (value 0, run 0)
  "dead" entries so that every 8-entry group starts 16-byte aligned;
* values and runs are separate arrays; the 8 runs of a group are packed in one
  32-bit word, entry j of the group in bits [4j, 4j+4);
* colmax[k] holds the fp16 bit pattern of the largest |stored value| of column
  k (+0 when the column stores nothing).  It is not part of the paper's
  format; the GPU product derives its fixed-point scales from it, so the
  encoder must produce it bit for bit.
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

import numpy as np

GROUP = 8          # entries per aligned group (one 16-byte fp16 vector)
RUN_BITS = 4       # Celty's run-length width (Section 3.2)


# ---------------------------------------------------------------------------
# One column, any run width n (Section 3.2).  Deliberately a plain loop.
# Parity: pinned by the paper's worked 2-bit example and hand-derived 4-bit
# gap cases (tests/golden), and by the round trip through rlc_decode_column.
# ---------------------------------------------------------------------------
def rlc_encode_column(column: Sequence[float], n_bits: int) -> Tuple[List[float], List[int]]:
    """n-bit RLC of one sparse column given as plain numbers (0 = absent)."""
    cap = (1 << n_bits) - 1
    values: List[float] = []
    runs: List[int] = []
    zeros = 0
    for v in column:
        if v == 0:
            zeros += 1
            continue
        while zeros > cap:          # bridge the gap: padding entry (0, cap)
            values.append(0)
            runs.append(cap)
            zeros -= cap + 1        # cap zeros plus the padding's own slot
        values.append(v)
        runs.append(zeros)
        zeros = 0
    return values, runs


def rlc_decode_column(values: Sequence[float], runs: Sequence[int], length: int) -> List[float]:
    """Inverse of rlc_encode_column: row(i) = sum_{j<=i} run_j + i."""
    out = [0] * length
    pos = -1
    for v, r in zip(values, runs):
        pos += r + 1
        if v != 0:
            out[pos] = v
    return out


# ---------------------------------------------------------------------------
# Algorithm 1: intra-warp prefix sum over the run lengths of one chunk.
# Each of L lanes holds P consecutive runs; the lane sums its runs, an
# inclusive Hillis-Steele scan over lanes (shuffle-up by 1, 2, 4, ...) turns the
# sums into lane-inclusive totals, and a backward walk subtracts runs to give
# the inclusive prefix of every entry.  The absolute row adds the ordinal.
# Parity: pinned against numpy's cumsum (a library routine) in the tests.
# ---------------------------------------------------------------------------
def alg1_prefix(rlc_arrays: np.ndarray) -> np.ndarray:
    """rlc_arrays: int array [L, P] (lane-major).  Returns inclusive prefix [L, P]."""
    lanes, per = rlc_arrays.shape
    total = rlc_arrays.sum(axis=1).astype(np.int64)          # per-lane sum
    step = 1
    while step < lanes:                                       # log2(L) shuffle-up steps
        prev = np.zeros_like(total)
        prev[step:] = total[:-step]                           # value from lane - step
        total = total + prev                                  # lanes >= step add it
        step *= 2
    prefix = np.zeros((lanes, per), dtype=np.int64)
    s = total.copy()
    for i in range(per - 1, -1, -1):                          # back-subtract
        prefix[:, i] = s
        s = s - rlc_arrays[:, i]
    return prefix


def alg1_rows(runs_flat: np.ndarray, per_lane: int = 8) -> np.ndarray:
    """Rows of a chunk of entries (length multiple of per_lane): prefix + ordinal."""
    r = np.asarray(runs_flat, dtype=np.int64).reshape(-1, per_lane)
    return alg1_prefix(r).reshape(-1) + np.arange(r.size)


# ---------------------------------------------------------------------------
# Tiled RLC-CSC ("format v1") for a whole matrix.
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class RlcCsc:
    M: int
    K: int
    R: int
    T: int
    gptr: np.ndarray      # uint32 [T*K + 1], group offsets of segments s = t*K + k
    values: np.ndarray    # uint16 [8*G], fp16 bit patterns
    runs: np.ndarray      # uint32 [G], 8 packed 4-bit runs per group
    seg_n: np.ndarray     # int64 [T*K], entries per segment before alignment
    n_nnz: int
    n_pad: int
    colmax: np.ndarray    # uint16 [K], fp16 bits of the largest |stored value| per column

    @property
    def n_groups(self) -> int:
        return int(self.runs.shape[0])

    @property
    def n_entries(self) -> int:
        return self.n_nnz + self.n_pad


def stored_mask(W_bits: np.ndarray, mask) -> np.ndarray:
    """Entries that are stored: kept by the mask and not +-0 (reading of 3.2)."""
    nz = (W_bits & np.uint16(0x7FFF)) != 0
    if mask is None:
        return nz
    return nz & (np.asarray(mask) != 0)


def encode_matrix(W: np.ndarray, mask, R: int) -> RlcCsc:
    """Format v1 of fp16 W (M x K, out x in) under a keep-mask, tile height R.

    Steps, in order: (1) stored set per segment; (2) gap before each stored
    entry, counted from the tile start or the previous stored entry;
    (3) greedy padding: gap // 16 entries (0, 15) then the value with run
    gap % 16; (4) alignment of each segment to 8 entries; (5) packing;
    (6) the column maxima of the stored magnitudes.
    Vectorised over all stored entries; checked against a per-column call of
    rlc_encode_column in the tests.
    """
    Wb = np.ascontiguousarray(W).view(np.uint16)
    M, K = Wb.shape
    if R < 1:
        raise ValueError("R must be >= 1")
    T = -(-M // R)
    cap = (1 << RUN_BITS) - 1
    S = stored_mask(Wb, mask)

    # (1) stored entries, ordered by segment s = t*K + k, then by row
    r_idx, k_idx = np.nonzero(S)                       # row-major order
    t_idx = r_idx // R
    seg = t_idx.astype(np.int64) * K + k_idx
    order = np.lexsort((r_idx, seg))
    r_idx, seg = r_idx[order].astype(np.int64), seg[order]
    vals = Wb[r_idx, k_idx[order]]
    rel = r_idx - (seg // K) * R                       # row within its tile

    # (2) gaps: zeros since the previous stored entry of the same segment
    first = np.ones(seg.shape, dtype=bool)
    first[1:] = seg[1:] != seg[:-1]
    prev = np.empty_like(rel)
    prev[0:1] = -1
    prev[1:] = rel[:-1]
    prev[first] = -1
    gap = rel - prev - 1

    # (3) greedy padding
    n_padding = gap // (cap + 1)
    run_last = gap % (cap + 1)
    width = n_padding + 1                              # entries emitted per stored value
    nseg = T * K
    seg_n = np.bincount(seg, weights=width, minlength=nseg).astype(np.int64)

    # (4) alignment to 8-entry groups
    seg_g = (seg_n + GROUP - 1) // GROUP
    gptr = np.zeros(nseg + 1, dtype=np.int64)
    np.cumsum(seg_g, out=gptr[1:])
    G = int(gptr[-1])

    # (5) placement: padding (0, cap) everywhere first, then stored values
    values = np.zeros(GROUP * G, dtype=np.uint16)
    runs_e = np.zeros(GROUP * G, dtype=np.uint8)
    within = np.cumsum(width) - 1                      # global running position ...
    seg_start_pos = np.zeros(nseg, dtype=np.int64)
    np.cumsum(seg_n[:-1], out=seg_start_pos[1:])
    within = within - seg_start_pos[seg]               # ... made segment-relative
    base = gptr[seg] * GROUP
    pos = base + within
    # padding slots of each stored entry occupy pos - n_padding .. pos - 1
    if n_padding.size and n_padding.max() > 0:
        rep = np.repeat(pos, n_padding)
        back = np.repeat(n_padding, n_padding)
        inner = np.arange(rep.size) - np.repeat(np.cumsum(n_padding) - n_padding, n_padding)
        runs_e[rep - back + inner] = cap
    values[pos] = vals
    runs_e[pos] = run_last.astype(np.uint8)

    packed = np.zeros(G, dtype=np.uint32)
    re = runs_e.reshape(G, GROUP).astype(np.uint32)
    for j in range(GROUP):
        packed |= re[:, j] << np.uint32(4 * j)

    # (6) fp16 magnitudes order like their bit patterns with the sign cleared
    colmax = column_max_bits(Wb, S)

    if G >= (1 << 32):
        raise OverflowError("group count does not fit in uint32")
    return RlcCsc(M=M, K=K, R=R, T=T, gptr=gptr.astype(np.uint32), values=values, runs=packed,
                  seg_n=seg_n, n_nnz=int(S.sum()), n_pad=int(n_padding.sum()), colmax=colmax)


def column_max_bits(W_bits: np.ndarray, stored: np.ndarray) -> np.ndarray:
    """uint16 [K]: bits of max |W[r, k]| over the stored r of column k (0 if none)."""
    mag = np.where(stored, np.asarray(W_bits, dtype=np.uint16) & np.uint16(0x7FFF), np.uint16(0))
    if mag.shape[0] == 0:
        return np.zeros(mag.shape[1], dtype=np.uint16)
    return mag.max(axis=0).astype(np.uint16)


def unpack_runs(runs: np.ndarray) -> np.ndarray:
    """uint32 [G] -> uint8 [8G] run lengths (entry j of a group from bits 4j..4j+3)."""
    r = np.asarray(runs, dtype=np.uint32)
    out = np.empty((r.shape[0], GROUP), dtype=np.uint8)
    for j in range(GROUP):
        out[:, j] = (r >> np.uint32(4 * j)) & np.uint32(0xF)
    return out.reshape(-1)


def segment_rows(enc: RlcCsc, s: int) -> Tuple[np.ndarray, np.ndarray]:
    """Decode segment s: (absolute rows of all its entries, fp16 value bits)."""
    g0, g1 = int(enc.gptr[s]), int(enc.gptr[s + 1])
    runs = unpack_runs(enc.runs[g0:g1]).astype(np.int64)
    vals = enc.values[GROUP * g0:GROUP * g1]
    t = s // enc.K
    rows = t * enc.R + np.cumsum(runs) + np.arange(runs.size)   # prefix + ordinal
    return rows, vals


def decode_matrix(enc: RlcCsc) -> Tuple[np.ndarray, np.ndarray]:
    """Format v1 -> (W' fp16 with zeros canonical +0, mask' uint8).

    Raises ValueError for a malformed stream: gptr not monotone from 0, array
    sizes that disagree with gptr, a stored (non-zero) entry outside its tile,
    or a zero-valued entry after the last stored entry of a segment whose run
    is not 0 (alignment entries are (0, 0) by construction).
    """
    M, K, R, T = enc.M, enc.K, enc.R, enc.T
    gptr = enc.gptr.astype(np.int64)
    if gptr.shape[0] != T * K + 1 or gptr[0] != 0 or np.any(np.diff(gptr) < 0):
        raise ValueError("gptr is not a monotone offset array of length T*K+1 from 0")
    if gptr[-1] != enc.runs.shape[0] or enc.values.shape[0] != GROUP * gptr[-1]:
        raise ValueError("array sizes do not match gptr")
    Wout = np.zeros((M, K), dtype=np.uint16)
    mout = np.zeros((M, K), dtype=np.uint8)
    all_runs = unpack_runs(enc.runs)
    for s in range(T * K):
        if gptr[s] == gptr[s + 1]:
            continue
        rows, vals = segment_rows(enc, s)
        t, k = divmod(s, K)
        hi = min(M, (t + 1) * R)
        real = (vals & np.uint16(0x7FFF)) != 0
        if np.any(rows[real] >= hi):
            raise ValueError(f"segment {s}: stored entry beyond its tile")
        last = int(np.flatnonzero(real)[-1]) if real.any() else -1
        tail_runs = all_runs[GROUP * gptr[s] + last + 1:GROUP * gptr[s + 1]]
        if np.any(tail_runs != 0):
            raise ValueError(f"segment {s}: alignment entry with a non-zero run")
        Wout[rows[real], k] = vals[real]
        mout[rows[real], k] = 1
    return Wout.view(np.float16), mout
