"""Byte accounting for the roofline and the format-size claims (Section 3.2).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Algorithmic bytes of one SpMSpV call:

    B_alg = 2.5 * E_A + 2 K + 2 M

E_A counts the entries (stored values plus RLC padding, not the 8-entry
alignment) of every segment of every active column: 2 bytes of fp16 value
plus 4 bits of run each.  2K is x and 2M is y, both fp16.  This is the
"compressed bytes of the active columns plus x and y" the paper's speedup
rests on (Section 5: the advantage stems from the lower effective traffic).

Parity status
-------------
algorithmic_bytes   pinned: equals the closed form 2.5 * (nnz_A + pad_A) + 2K + 2M
                    computed from the mask by a separate count in the tests.
rlc_csc_bytes       pinned: ~63 % of dense at 50 % sparsity on 4096^2 (Section 3.2).
bitmap_bytes        pinned: (d*16 + 1)/16 of dense, ~56 % at 50 % (Section 3.2).
"""
from __future__ import annotations

import numpy as np

from . import rlc as _rlc
from .spmspv import select_active


def active_entries(enc: "_rlc.RlcCsc", active: np.ndarray) -> int:
    """E_A: entries (real + padding, no alignment) in the active columns."""
    seg_n = enc.seg_n.reshape(enc.T, enc.K)
    return int(seg_n[:, np.asarray(active, dtype=np.int64)].sum())


def active_groups(enc: "_rlc.RlcCsc", active: np.ndarray) -> int:
    g = np.diff(enc.gptr.astype(np.int64)).reshape(enc.T, enc.K)
    return int(g[:, np.asarray(active, dtype=np.int64)].sum())


def algorithmic_bytes(enc: "_rlc.RlcCsc", x: np.ndarray, tau: float) -> float:
    e_a = active_entries(enc, select_active(x, tau))
    return 2.5 * e_a + 2 * enc.K + 2 * enc.M


def rlc_csc_bytes(enc: "_rlc.RlcCsc") -> int:
    """Stored size: fp16 values, packed runs, group pointers."""
    return 2 * enc.values.size + 4 * enc.runs.size + 4 * enc.gptr.size


def rlc_csc_entry_bytes(enc: "_rlc.RlcCsc") -> float:
    """2.5 bytes per entry (real + padding), without pointers or alignment."""
    return 2.5 * enc.n_entries


def bitmap_bytes(M: int, K: int, nnz: int) -> float:
    """Theoretical bitmap format: 1 bit per position plus fp16 per non-zero."""
    return M * K / 8.0 + 2.0 * nnz


def dense_bytes(M: int, K: int) -> int:
    return 2 * M * K
