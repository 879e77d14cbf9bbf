"""Pins for the oracle's Philox4x64-10 streams and their uniform/Gaussian maps.

Philox is checked against numpy's independent C implementation of the same
published generator (numpy.random.Philox is Philox4x64-10); numpy increments
its counter before each block, so block c is read with numpy's counter at c-1.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import philox


def _numpy_block(counter, key):
    c = np.array(counter, dtype=np.uint64)
    c[0] = c[0] - np.uint64(1) if c[0] > 0 else np.uint64(2**64 - 1)
    if counter[0] == 0:  # borrow
        c[1] = c[1] - np.uint64(1)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=c)
    return [int(x) for x in bg.random_raw(4)]


@pytest.mark.parametrize("counter,key", [
    ((1, 0, 0, 0), (5, 0)),
    ((7, 3, 1, 0), (0xDEADBEEFCAFEF00D, 0)),
    ((12345, 17, 2, 0), (2**64 - 1, 0)),
    ((2**40 + 3, 2**63, 2, 9), (42, 0x0123456789ABCDEF)),
])
def test_philox_matches_numpy(counter, key):
    ref = _numpy_block(counter, key)
    vec = philox.philox4x64(*[np.uint64(c) for c in counter], np.uint64(key[0]), np.uint64(key[1]))
    assert [int(v) for v in vec] == ref
    assert philox.philox4x64_int(counter, key) == ref


def test_philox_vectorised_equals_scalar():
    idx = np.arange(64, dtype=np.uint64)
    vec = philox.philox4x64(idx, np.uint64(3), np.uint64(1), np.uint64(0), np.uint64(99), np.uint64(0))
    for i in (0, 1, 31, 63):
        assert [int(v[i]) for v in vec] == philox.philox4x64_int((i, 3, 1, 0), (99, 0))


def test_words32_split_order():
    w = philox.words32(7, 2, 1, 24)
    blk = philox.philox4x64_int((1, 2, 1, 0), (7, 0))
    got = [int(x) for x in w[8:16]]
    want = []
    for word in blk:
        want += [word & 0xFFFFFFFF, word >> 32]
    assert got == want


def test_uniform_range_and_distribution():
    u = philox.uniforms(11, 0, 2, 200000)
    assert np.all(u > 0.0) and np.all(u < 1.0)
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    assert abs(u.mean() - 0.5) < 5 * np.sqrt(1 / 12 / u.size)


def test_uniform_extremes_exact():
    # x = 0 and x = 2^32 - 1 map strictly inside (0, 1)
    assert (0 + 0.5) * 2.0**-32 > 0
    assert ((2**32 - 1) + 0.5) * 2.0**-32 < 1


def test_box_muller_is_standard_normal():
    z = philox.gaussians(3, 1, 0, 200000)
    assert stats.kstest(z, "norm").pvalue > 1e-3
    assert abs(z.mean()) < 5 / np.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * np.sqrt(2 / z.size)
    # pairs are independent: correlation of the cos and sin halves ~ 0
    pairs = z.reshape(-1, 2)
    assert abs(np.corrcoef(pairs[:, 0], pairs[:, 1])[0, 1]) < 5 / np.sqrt(pairs.shape[0])


def test_streams_differ_by_head_and_purpose():
    a = philox.words32(1, 0, 0, 64)
    b = philox.words32(1, 1, 0, 64)
    c = philox.words32(1, 0, 1, 64)
    assert not np.array_equal(a, b) and not np.array_equal(a, c)
