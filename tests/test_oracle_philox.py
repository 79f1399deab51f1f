"""Pins of the oracle's Philox4x64-10 (oracle/philox.py).

numpy ships an independent implementation of the same published generator
(numpy.random.Philox, 4x64, 10 rounds), which draws block c + 1 for a state
holding counter c; comparing against it on random keys and counters pins
every round constant, the key schedule and the word order.
"""
import numpy as np
from scipy import stats

from oracle import philox

M64 = (1 << 64) - 1


def numpy_block(ctr, key):
    cint = sum(int(v) << (64 * i) for i, v in enumerate(ctr))
    kint = int(key[0]) | (int(key[1]) << 64)
    bg = np.random.Philox(key=kint, counter=(cint - 1) % (1 << 256))
    return [int(x) for x in bg.random_raw(4)]


def test_matches_numpy_philox_on_random_counters():
    g = np.random.default_rng(123)
    for _ in range(200):
        ctr = [int(x) for x in g.integers(0, M64, size=4, dtype=np.uint64, endpoint=True)]
        key = [int(x) for x in g.integers(0, M64, size=2, dtype=np.uint64, endpoint=True)]
        got = philox.philox4x64_10(*[np.uint64(c) for c in ctr], key[0], key[1])
        assert [int(x) for x in got] == numpy_block(ctr, key)


def test_matches_numpy_philox_on_edge_counters():
    for ctr, key in [((0, 0, 0, 0), (0, 0)), ((M64, M64, M64, M64), (M64, M64)),
                     ((1, 0, 0, 0), (0, 1)), ((0, 0, 0, 1), (1, 0))]:
        got = philox.philox4x64_10(*[np.uint64(c) for c in ctr], key[0], key[1])
        assert [int(x) for x in got] == numpy_block(ctr, key)


def test_vectorised_equals_scalar():
    u = philox.uniforms(7, 3, philox.PURPOSE_ACCEPT, 4, 5)
    for b in range(4):
        for j in range(5):
            x0 = numpy_block((j, b, 3, philox.PURPOSE_ACCEPT), (7, 0))[0]
            assert u[b, j] == np.float32((x0 >> 40) * 2.0 ** -24)


def test_uniforms_on_grid_and_uniform():
    u = philox.uniforms(42, 0, philox.PURPOSE_DRAFT, 64, 1024).ravel()
    assert u.dtype == np.float32
    assert np.all((u >= 0) & (u < 1))
    m = u.astype(np.float64) * 2 ** 24
    assert np.all(m == np.floor(m))
    counts, _ = np.histogram(u, bins=64, range=(0, 1))
    assert stats.chisquare(counts).pvalue > 1e-4


def test_streams_differ_by_purpose_loop_and_index():
    a = philox.uniforms(1, 0, 0, 2, 8)
    assert not np.array_equal(a, philox.uniforms(1, 0, 1, 2, 8))
    assert not np.array_equal(a, philox.uniforms(1, 1, 0, 2, 8))
    assert not np.array_equal(a, philox.uniforms(2, 0, 0, 2, 8))
    assert not np.array_equal(a[0], a[1])
