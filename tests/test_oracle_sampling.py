"""Pins of oracle/sampling.py: fixed-point weights, the categorical draw and
softmax with temperature.

The categorical draw is checked by brute force over all 2^24 grid values of
the uniform: the count of grid values landing on index i must be within one
grid step of w_i / W (the law the draw is meant to have), and zero weights
must never be drawn. softmax is checked against torch's fp64 softmax.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import sampling

GRID = 1 << 24


def test_to_weights_exact_floor():
    g = np.random.default_rng(0)
    x = np.concatenate([g.random(2000, dtype=np.float32),
                        np.array([0.0, 1.0, 2.0, -0.5, np.nan, np.inf, 1e-30, 2.0 ** -32,
                                  2.0 ** -33, np.nextafter(np.float32(1), np.float32(0))],
                                 dtype=np.float32)])
    w = sampling.to_weights(x)
    for xi, wi in zip(x, w):
        xi = float(xi)
        if not xi > 0:
            want = 0
        elif xi >= 1:
            want = 1 << 32
        else:
            want = int(Fraction(xi) * (1 << 32))   # Fraction floor via int()
        assert int(wi) == want, (xi, int(wi), want)


def grid_histogram(w):
    """Index drawn for every grid value m, computed independently of the oracle
    with searchsorted on the integer prefix sums."""
    w = np.asarray(w, dtype=np.uint64)
    prefix = np.cumsum(w, dtype=np.uint64)
    total = int(prefix[-1])
    m = np.arange(GRID, dtype=np.uint64)
    # t = floor(m * total / 2^24) without overflow: total < 2^40 here.
    hi, lo = divmod(total, 1 << 24)
    t = m * np.uint64(hi) + ((m * np.uint64(lo)) >> np.uint64(24))
    idx = np.searchsorted(prefix, t, side="right")
    return np.bincount(idx, minlength=len(w))


@pytest.mark.parametrize("case", range(6))
def test_categorical_law_by_brute_force(case):
    g = np.random.default_rng(case)
    V = [2, 3, 5, 8, 17, 64][case]
    x = g.dirichlet(np.ones(V) * 0.5).astype(np.float32)
    x[g.integers(0, V)] = 0.0                       # a zero-weight index
    w = sampling.to_weights(x)
    counts = grid_histogram(w)
    W = int(w.sum(dtype=np.uint64))
    for i in range(V):
        assert abs(Fraction(int(counts[i]), GRID) - Fraction(int(w[i]), W)) < Fraction(1, GRID)
        if w[i] == 0:
            assert counts[i] == 0
    # the oracle's draw agrees with the grid histogram at every bucket edge and
    # at random grid points
    prefix = np.cumsum(w, dtype=np.uint64)
    hi, lo = divmod(W, 1 << 24)
    edges = []
    for c in [0] + [int(v) for v in prefix[:-1]]:
        m0 = -(-c * GRID // W)                          # first m with t >= c
        edges += [m0 - 1, m0, m0 + 1]
    ms = [m for m in edges if 0 <= m < GRID] + list(g.integers(0, GRID, 200))
    for m in ms:
        t = m * hi + ((m * lo) >> 24)
        want = int(np.searchsorted(prefix, np.uint64(t), side="right"))
        got, ok = sampling.categorical(w, np.float32(m * 2.0 ** -24))
        assert ok and got == want


def test_categorical_dyadic_law_is_exact():
    # probabilities c_i / 2^12 summing to one: W = 2^32 and every grid bucket
    # holds exactly c_i * 2^12 grid values, so the law is exactly c_i / 2^12.
    c = np.array([1, 7, 100, 3988], dtype=np.int64)
    x = (c / 4096.0).astype(np.float32)
    counts = grid_histogram(sampling.to_weights(x))
    assert list(counts) == list(c * 4096)


def test_categorical_all_zero_weights():
    assert sampling.categorical(np.zeros(5, np.uint64), 0.3) == (0, False)


def test_grid_index_clamps():
    assert sampling.grid_index(np.float32(0.0)) == 0
    assert sampling.grid_index(np.float32(-1.0)) == 0
    assert sampling.grid_index(np.float32(np.nan)) == 0
    assert sampling.grid_index(np.float32(1.0)) == GRID - 1
    assert sampling.grid_index(np.float32(0.5)) == GRID // 2
    assert sampling.grid_index(np.float32(1e-9)) == 0


@pytest.mark.parametrize("T", [1.0, 0.8, 2.5])
def test_softmax_matches_torch(T):
    z = np.random.default_rng(1).normal(0, 3, size=(4, 100))
    ref = torch.softmax(torch.from_numpy(z) / T, dim=-1).numpy()
    np.testing.assert_allclose(sampling.softmax(z, T), ref, rtol=1e-13, atol=1e-16)


def test_softmax_greedy_lowest_index_on_ties():
    z = np.array([[1.0, 3.0, 3.0, 0.0], [-1.0, -1.0, -2.0, -5.0]])
    q = sampling.softmax(z, 0.0)
    assert q.tolist() == [[0, 1, 0, 0], [1, 0, 0, 0]]


def test_nonfinite_logit_rows_are_one_hot_at_zero():
    """Rows with a NaN or +Inf logit, or whose fp32 quotient by T overflows,
    are one-hot at token 0 (the library's definition); -Inf logits are valid
    and get probability 0."""
    z = np.random.default_rng(3).normal(0, 2, (6, 10)).astype(np.float32)
    z[0, 4] = np.nan
    z[1, 2] = np.inf
    z[2, 7] = -np.inf
    z[3, 1] = 3e38                 # 3e38 / 0.5 overflows fp32
    for T in (1.0, 0.5, 0.0):
        bad = sampling.nonfinite_rows(z, T)
        want_bad = [True, True, False, T == 0.5, False, False]
        assert list(bad) == want_bad, T
        out = sampling.softmax(z, T)
        for r in range(6):
            if want_bad[r]:
                assert out[r, 0] == 1.0 and out[r, 1:].sum() == 0.0
            else:
                assert np.isfinite(out[r]).all() and abs(out[r].sum() - 1.0) < 1e-12
        assert out[2, 7] == 0.0
    ref = torch.softmax(torch.from_numpy(z[4:].astype(np.float64)), dim=-1).numpy()
    np.testing.assert_allclose(sampling.softmax(z[4:], 1.0), ref, rtol=1e-13)
