"""Host check of the GEMV's thread -> (row, group) split.

The flat GEMV kernel (paper_2605_08755_amd/csrc/linear.hip) replaces the
integer quotient t / G of a thread index t < 1024 by a group count G by
trunc((t + 0.5) * fl32(1 / G)) in float32 arithmetic.  This checks that the
two agree for every thread index of a block (blocks have at most 1024
threads) and every group count the C ABI admits (K <= 2^24, so G <= 2^17),
in IEEE float32 with round-to-nearest (numpy float32), independently of the
kernel and of the oracle.
"""
import numpy as np

MAX_THREADS = 1024
MAX_G = (1 << 24) // 128


def test_float_quotient_equals_integer_quotient():
    t = np.arange(MAX_THREADS, dtype=np.int64)
    tf = t.astype(np.float32) + np.float32(0.5)
    for g0 in range(1, MAX_G + 1, 4096):
        G = np.arange(g0, min(g0 + 4096, MAX_G + 1), dtype=np.int64)
        inv = (np.float32(1.0) / G.astype(np.float32)).astype(np.float32)
        q = (tf[None, :] * inv[:, None]).astype(np.float32)
        got = np.trunc(q).astype(np.int64)
        want = t[None, :] // G[:, None]
        bad = np.argwhere(got != want)
        assert bad.size == 0, "G=%d t=%d" % (G[bad[0][0]], t[bad[0][1]])
