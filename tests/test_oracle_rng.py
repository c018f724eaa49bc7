"""Pins of the oracle's random numbers.

Philox-4x64-10 is checked word for word against numpy.random.Philox (an
independent implementation of Salmon et al.'s generator; numpy advances the
counter by one before each block, so numpy's block after counter c equals our
block at c + 1).  The uniform mapping is checked for range, exactness in fp32
and uniformity.
"""
import numpy as np
import pytest
from scipy import stats

import oracle

CASES = [
    ((1, 0, 0, 0), (0, 0)),
    ((5, 6, 7, 8), (11, 12)),
    ((123456789, 2048, 63, 2), (0xDEADBEEF, 77)),
    ((2**63, 2**40 + 3, 2**32 + 1, 1), (2**64 - 1, 2**63 + 5)),
]


@pytest.mark.parametrize("ctr,key", CASES)
def test_philox_matches_numpy(ctr, key):
    numpy_ctr = np.array([ctr[0] - 1, ctr[1], ctr[2], ctr[3]], dtype=np.uint64)
    g = np.random.Philox(counter=numpy_ctr, key=np.array(key, dtype=np.uint64))
    want = g.random_raw(4)
    got = oracle.philox(ctr, key)
    assert [int(x) for x in got] == [int(x) for x in want]


def test_philox_counter_carry_matches_numpy():
    # numpy's increment of word 0 = 2^64-1 carries into word 1
    g = np.random.Philox(counter=np.array([2**64 - 1, 9, 3, 1], dtype=np.uint64), key=[4, 5])
    want = g.random_raw(4)
    got = oracle.philox((0, 10, 3, 1), (4, 5))
    assert [int(x) for x in got] == [int(x) for x in want]


def test_consecutive_blocks_match_numpy_stream():
    g = np.random.Philox(counter=[0, 17, 2, 0], key=[42, 7])
    want = g.random_raw(4 * 6)
    got = np.concatenate([oracle.philox((b + 1, 17, 2, 0), (42, 7)) for b in range(6)])
    assert np.array_equal(got, want)


def test_uniform_mapping_from_numpy_words():
    # uniform i of a row comes from word (i % 8) // 2 of block i // 8, low half first
    seed, step, stream, slot, pos = 3, 9, 1, 5, 100
    u = oracle.uniform_row(seed, step, stream, slot, pos, 40)
    for blk in range(5):
        ctr = np.array([blk - 1 if blk else 2**64 - 1, pos - (0 if blk else 1), slot, stream], dtype=np.uint64)
        g = np.random.Philox(counter=ctr, key=[seed, step])
        words = g.random_raw(4)
        halves = []
        for w in words:
            halves += [int(w) & 0xFFFFFFFF, int(w) >> 32]
        want = [((h >> 9) + 0.5) / 2**23 for h in halves]
        assert np.array_equal(u[8 * blk: 8 * blk + 8], np.array(want, dtype=np.float32))


def test_uniforms_open_interval_exact_and_uniform():
    u = oracle.uniform_row(0, 0, 0, 0, 0, 200_000)
    assert u.min() > 0.0 and u.max() < 1.0
    k = u.astype(np.float64) * 2**23 - 0.5
    assert np.array_equal(k, np.round(k))          # exact in fp32: (k + 0.5) * 2^-23
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    # different streams / positions / slots / keys give different rows
    rows = [oracle.uniform_row(0, 0, s, sl, p, 64) for s, sl, p in [(0, 0, 1), (1, 0, 0), (0, 1, 0)]]
    rows.append(oracle.uniform_row(1, 0, 0, 0, 0, 64))
    for r in rows:
        assert not np.array_equal(r, u[:64])
