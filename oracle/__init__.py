"""CPU oracle for the dual-sparse SpMSpV y = W x (Celty, Sections 3.1-3.3).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links anything in this package: only the test suite, the smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the GPU library
(the C ABI, its encoder or its kernels) and does not import it.

Everything here is plain numpy/scipy in fp64 (the paper fixes fp16 storage of
weights and activations, Section 3.1; products and sums are taken in fp64 here,
so the oracle is the exact definition up to fp64 rounding).

Modules
-------
rlc      : n-bit run-length coding of one sparse column (Section 3.2) and the
           tiled RLC-CSC storage layout ("format v1") built from it, plus the
           decoder and Algorithm 1 (intra-warp prefix sum over run lengths).
spmspv   : activation selection by magnitude threshold and three independent
           evaluations of y = W (M o W) x_A: dense fp64, CSC fp64, brute force,
           plus a fp64 product that walks the RLC-CSC arrays the way the
           paper's kernel does.
layouts  : two other encodings of the segments' rows: 16-bit absolute row
           offsets (a decode-free form) and the lane-interleaved order of
           Section 4.2, with their decoders.
accounting: byte counts used for the roofline (algorithmic bytes per call)
           and the compression ratios the paper quotes (Section 3.2).

Parity status of every function is listed in its docstring.
"""
from . import rlc, spmspv, accounting, layouts  # noqa: F401
