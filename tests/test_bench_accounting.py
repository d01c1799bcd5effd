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


def test_kernel_code_hash_ignores_comments_only():
    # the counter profiles are keyed by the kernel's code: comments and
    # whitespace do not count, string literals (inline assembly) and code do
    src = 'int a = 1; // note\n/* block\n comment */ asm("ds_add_u32 %0 // x"); char c = \'"\';\n'
    code = bench.kernel_source_code(src)
    assert code == 'int a = 1; asm("ds_add_u32 %0 // x"); char c = \'"\';'
    assert bench.kernel_source_code(src.replace("// note", "// other note\n\n")) == code
    assert bench.kernel_source_code(src.replace("a = 1", "a = 2")) != code
    assert bench.kernel_source_code('s = "a\\"b // c";') == 's = "a\\"b // c";'


@pytest.mark.parametrize("ws,as_", [(70, 70), (50, 0), (30, 90)])
def test_cold_rotation_counts_the_bytes_a_call_reads(ws, as_):
    # a copy is read again only after COLD_BYTES of reads of the other
    # copies: the rotation is sized by the bytes one call reads (its active
    # columns), which at high activation sparsity is far below the copy's
    # stored size
    p = workloads.random_small(ws + as_, 600, 500, ws=ws, as_=as_)
    enc = celty.celty_encode(p.W, p.mask, 128)
    read = bench.algorithmic_bytes_from_encoding(enc, p.x, p.tau)[0]
    n = bench.cold_copies(enc, p)
    assert n * read >= bench.COLD_BYTES
    assert (n - 1) * read < bench.COLD_BYTES
    if as_ > 0:
        assert read < bench.stored_bytes(enc)
        assert n > -(-bench.COLD_BYTES // bench.stored_bytes(enc))
