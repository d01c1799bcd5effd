"""Two other encodings of the rows of the tiled RLC-CSC segments.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Both keep the segments, the 8-entry groups and the group pointers of the
tiled format (rlc.encode_matrix): segment s = t*K + k holds the stored entries
of column k within row tile t.  They differ in how an entry's row is found.

rows16 (a decode-free form, for measuring what reconstruction costs)
    Section 3.3 reconstructs each entry's absolute row from the run lengths
    with an intra-warp prefix sum (Algorithm 1), and Section 4.2 proposes a
    hardware decoder because that reconstruction can take a large share of
    the kernel's time (Figure decompression_latency).  Here each entry
    carries its row directly: a 16-bit row offset within its tile.  Steps,
    in order: (1) the stored entries of each segment (rlc.stored_mask), in
    row order; (2) each entry's row offset r - t*R; (3) alignment of each
    segment to 8 entries with (value 0, row offset of the segment's last
    stored entry); (4) group pointers; (5) the column maxima.  No padding
    entries: a row offset needs no gap bridging.  Requires R <= 65536.

interleaved (Section 4.2's lane-interleaved order)
    Section 4.2 has the offline compression interleave the non-zero values
    and their run lengths across threads, so that thread 0 of a warp loads
    entries 0, 32, 64, ... of the sequence (each thread's 8 entries are then
    one per stride of the warp width).  Here the unit is a 64-lane wavefront:
    each segment's groups are cut into chunks of up to 64 groups (64 per
    chunk, the last chunk of a segment holding the rest), and within a chunk
    of G_c groups the entry at row-order position e (0 <= e < 8*G_c) is
    stored in group e mod G_c, slot e // G_c.  Lane l of a wavefront that
    loads the chunk's group l thus holds entries l, l + G_c, l + 2*G_c, ...
    Values and runs move together; the runs keep their meaning (zeros before
    the entry in row order), so the segment's entry sequence, its padding
    and its alignment are those of the tiled RLC-CSC format.  Scatter-adds
    commute, so the order in which a kernel meets the entries does not
    change the product.

Parity: rows16 is pinned by a hand-written fixture (tests/golden), by the
round trip through decode_rows16 against the dense masked matrix, and by
its invariants; interleaved by a hand-written fixture, by its definition
checked on a full 64-group chunk (group l holds row-order entries l + 64*j),
and by the round trip through decode_interleaved.
"""
from __future__ import annotations

import dataclasses
from typing import Tuple

import numpy as np

from . import rlc

GROUP = rlc.GROUP
CHUNK = 64          # groups per interleave chunk: one per lane of a wavefront


# ---------------------------------------------------------------------------
# rows16
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Rows16:
    M: int
    K: int
    R: int
    T: int
    gptr: np.ndarray      # uint32 [T*K + 1], group offsets of segments s = t*K + k
    values: np.ndarray    # uint16 [8*G], fp16 bit patterns
    rows: np.ndarray      # uint16 [8*G], row offsets within the tile
    seg_n: np.ndarray     # int64 [T*K], stored entries per segment
    n_nnz: int
    colmax: np.ndarray    # uint16 [K]

    @property
    def n_groups(self) -> int:
        return int(self.gptr[-1])


def encode_rows16(W: np.ndarray, mask, R: int) -> Rows16:
    """rows16 form of fp16 W (M x K) under a keep-mask, tile height R.

    A plain loop over segments (small inputs only)."""
    Wb = np.ascontiguousarray(W).view(np.uint16)
    M, K = Wb.shape
    if not 1 <= R <= 65536:
        raise ValueError("rows16 needs 1 <= R <= 65536")
    T = -(-M // R)
    S = rlc.stored_mask(Wb, mask)
    seg_vals, seg_rows, seg_n = [], [], np.zeros(T * K, dtype=np.int64)
    for t in range(T):
        r0, r1 = t * R, min(M, (t + 1) * R)
        for k in range(K):
            rs = [r for r in range(r0, r1) if S[r, k]]                 # (1) row order
            v = [int(Wb[r, k]) for r in rs]
            o = [r - r0 for r in rs]                                    # (2) offsets
            n = len(rs)
            seg_n[t * K + k] = n
            aligned = -(-n // GROUP) * GROUP
            v += [0] * (aligned - n)                                    # (3) alignment
            o += [o[-1] if o else 0] * (aligned - n)
            seg_vals.append(v)
            seg_rows.append(o)
    gptr = np.zeros(T * K + 1, dtype=np.int64)                          # (4)
    gptr[1:] = np.cumsum([len(v) // GROUP for v in seg_vals])
    values = np.array([x for v in seg_vals for x in v], dtype=np.uint16)
    rows = np.array([x for o in seg_rows for x in o], dtype=np.uint16)
    return Rows16(M=M, K=K, R=R, T=T, gptr=gptr.astype(np.uint32), values=values, rows=rows, seg_n=seg_n,
                  n_nnz=int(S.sum()), colmax=rlc.column_max_bits(Wb, S))   # (5)


def decode_rows16(enc: Rows16) -> Tuple[np.ndarray, np.ndarray]:
    """rows16 -> (W' fp16 with zeros canonical +0, mask' uint8).

    Raises ValueError for a malformed stream: gptr not monotone from 0, sizes
    that disagree with gptr, a stored (non-zero) entry whose row is outside
    its tile, or stored entries out of row order."""
    M, K, R, T = enc.M, enc.K, enc.R, enc.T
    gptr = enc.gptr.astype(np.int64)
    if gptr.shape[0] != T * K + 1 or gptr[0] != 0 or np.any(np.diff(gptr) < 0):
        raise ValueError("gptr is not a monotone offset array of length T*K+1 from 0")
    if enc.values.shape[0] != GROUP * gptr[-1] or enc.rows.shape[0] != GROUP * gptr[-1]:
        raise ValueError("array sizes do not match gptr")
    Wout = np.zeros((M, K), dtype=np.uint16)
    mout = np.zeros((M, K), dtype=np.uint8)
    for s in range(T * K):
        t, k = divmod(s, K)
        e0, e1 = GROUP * int(gptr[s]), GROUP * int(gptr[s + 1])
        vals = enc.values[e0:e1]
        rows = enc.rows[e0:e1].astype(np.int64)
        real = (vals & np.uint16(0x7FFF)) != 0
        r = rows[real] + t * R
        if np.any(r >= min(M, (t + 1) * R)):
            raise ValueError(f"segment {s}: stored entry beyond its tile")
        if np.any(np.diff(r) <= 0):
            raise ValueError(f"segment {s}: stored entries out of row order")
        Wout[r, k] = vals[real]
        mout[r, k] = 1
    return Wout.view(np.float16), mout


# ---------------------------------------------------------------------------
# interleaved
# ---------------------------------------------------------------------------
def chunk_slot(e: int, n_groups: int) -> Tuple[int, int]:
    """(group, slot) within a chunk of n_groups groups of row-order entry e."""
    return e % n_groups, e // n_groups


def interleave_segment(values: np.ndarray, runs_e: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """One segment's entries (row order, length a multiple of 8) -> stored order."""
    n = values.shape[0] // GROUP
    out_v = np.zeros_like(values)
    out_r = np.zeros_like(runs_e)
    for c0 in range(0, n, CHUNK):
        gc = min(CHUNK, n - c0)
        for e in range(GROUP * gc):
            g, j = chunk_slot(e, gc)
            out_v[GROUP * (c0 + g) + j] = values[GROUP * c0 + e]
            out_r[GROUP * (c0 + g) + j] = runs_e[GROUP * c0 + e]
    return out_v, out_r


def deinterleave_segment(values: np.ndarray, runs_e: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Inverse of interleave_segment."""
    n = values.shape[0] // GROUP
    out_v = np.zeros_like(values)
    out_r = np.zeros_like(runs_e)
    for c0 in range(0, n, CHUNK):
        gc = min(CHUNK, n - c0)
        for e in range(GROUP * gc):
            g, j = chunk_slot(e, gc)
            out_v[GROUP * c0 + e] = values[GROUP * (c0 + g) + j]
            out_r[GROUP * c0 + e] = runs_e[GROUP * (c0 + g) + j]
    return out_v, out_r


def _pack(runs_e: np.ndarray) -> np.ndarray:
    re = runs_e.reshape(-1, GROUP).astype(np.uint32)
    packed = np.zeros(re.shape[0], dtype=np.uint32)
    for j in range(GROUP):
        packed |= re[:, j] << np.uint32(4 * j)
    return packed


def _map_segments(enc: rlc.RlcCsc, fn) -> rlc.RlcCsc:
    values = enc.values.copy()
    runs_e = rlc.unpack_runs(enc.runs)
    for s in range(enc.T * enc.K):
        e0, e1 = GROUP * int(enc.gptr[s]), GROUP * int(enc.gptr[s + 1])
        if e1 > e0:
            values[e0:e1], runs_e[e0:e1] = fn(values[e0:e1], runs_e[e0:e1])
    return dataclasses.replace(enc, values=values, runs=_pack(runs_e))


def encode_interleaved(W: np.ndarray, mask, R: int) -> rlc.RlcCsc:
    """Interleaved form: the tiled RLC-CSC encoding, then each segment's
    chunks put in lane-interleaved order (same arrays and sizes)."""
    return _map_segments(rlc.encode_matrix(W, mask, R), interleave_segment)


def deinterleave(enc: rlc.RlcCsc) -> rlc.RlcCsc:
    """The tiled RLC-CSC encoding an interleaved one was made from."""
    return _map_segments(enc, deinterleave_segment)


def decode_interleaved(enc: rlc.RlcCsc) -> Tuple[np.ndarray, np.ndarray]:
    """Interleaved form -> (W', mask') through the tiled format's decoder."""
    return rlc.decode_matrix(deinterleave(enc))


def interleaved_segment_rows(enc: rlc.RlcCsc, s: int) -> Tuple[np.ndarray, np.ndarray]:
    """Rows of segment s read straight from the interleaved arrays, in stored
    order: the entry in group g, slot j of a chunk of G_c groups is row-order
    entry e = j * G_c + g, whose row is the tile base plus the sum of
    (run + 1) over the segment's entries up to e, minus 1 (Algorithm 1's
    prefix plus ordinal, taken in row order)."""
    g0, g1 = int(enc.gptr[s]), int(enc.gptr[s + 1])
    n = g1 - g0
    runs_e = rlc.unpack_runs(enc.runs[g0:g1]).astype(np.int64)
    vals = enc.values[GROUP * g0:GROUP * g1]
    rows = np.zeros(GROUP * n, dtype=np.int64)
    base = (s // enc.K) * enc.R - 1
    for c0 in range(0, n, CHUNK):
        gc = min(CHUNK, n - c0)
        pos = base
        for e in range(GROUP * gc):          # row order within the chunk
            g, j = chunk_slot(e, gc)
            p = GROUP * (c0 + g) + j
            pos += runs_e[p] + 1
            rows[p] = pos
        base = pos
    return rows, vals
