"""Pins of oracle/modifiers.py: top-k and nucleus modifiers of p and q.

The paper fixes no formula (Modified Rejection Sampling section, closing
paragraph), so the pins are what any reading of "keep the k most probable
tokens" / "keep the smallest set of most probable tokens holding mass p"
must satisfy, plus library routines on inputs where the fixed-point
ranking cannot differ from the exact one:

* a hand-derived dyadic example (tests/golden/modifiers_dyadic.json);
* top-k equals torch.topk's index set on rows with distinct weights;
* nucleus equals the set torch's fp64 sort + cumsum gives, on rows whose
  cumulative mass is not within 1e-6 of p at the cut;
* the nucleus set is the shortest prefix of the ranking reaching the
  threshold, ties go to the lower index, exactly k entries survive top-k;
* renormalisation keeps ratios and sums to 1 within fp32 rounding;
* the correctly rounded integer-to-fp32 conversion against exact rationals;
* modified draft + modified target through accept_resample: the first
  emitted token follows the modified target (chi-square), never a dropped
  entry.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
from scipy import stats

from oracle import accept, modifiers, sampling

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "modifiers_dyadic.json")


def random_probs(V, seed, sharp=2.0):
    g = np.random.default_rng(seed)
    z = g.normal(0.0, sharp, V)
    x = np.exp(z - z.max())
    return (x / x.sum()).astype(np.float32)


def test_golden_dyadic_example():
    d = json.load(open(GOLDEN))
    x = np.array(d["x"], dtype=np.float32)
    for c in d["cases"]:
        mask = modifiers.kept_mask(x, c["top_k"], c["top_p"])
        assert sorted(np.nonzero(mask)[0].tolist()) == c["kept"], c
        out = modifiers.modify(x, c["top_k"], c["top_p"])
        np.testing.assert_array_equal(out, np.array(c["out"], dtype=np.float32))


@pytest.mark.parametrize("k", [1, 2, 7, 50, 999])
def test_top_k_matches_torch_topk(k):
    for seed in range(5):
        x = random_probs(1000, seed)
        w = sampling.to_weights(x)
        if len(np.unique(w)) != len(w):
            continue                                   # ties: covered by the tie test
        got = set(np.nonzero(modifiers.kept_mask(x, k, 1.0))[0].tolist())
        want = set(torch.topk(torch.from_numpy(x.astype(np.float64)), k).indices.tolist())
        assert got == want
        assert len(got) == k


@pytest.mark.parametrize("p", [0.1, 0.5, 0.8, 0.95, 0.999])
def test_nucleus_matches_sorted_cumsum(p):
    checked = 0
    for seed in range(20):
        x = random_probs(500, 100 + seed)
        t = torch.from_numpy(x.astype(np.float64))
        vals, idx = torch.sort(t, descending=True, stable=True)
        cum = torch.cumsum(vals, 0) / vals.sum()
        n = int(torch.searchsorted(cum, torch.tensor([p], dtype=torch.float64)).item()) + 1
        if np.min(np.abs(cum.numpy() - p)) < 1e-6:
            continue                                   # the cut is too close to call in fp64
        got = set(np.nonzero(modifiers.kept_mask(x, 0, p))[0].tolist())
        assert got == set(idx[:n].tolist()), (p, seed)
        checked += 1
    assert checked >= 10


def test_nucleus_is_shortest_prefix_reaching_threshold():
    for seed in range(30):
        x = random_probs(300, 200 + seed, sharp=1.0 + seed % 4)
        p = float(np.float32(np.random.default_rng(seed).random()))
        k = int(np.random.default_rng(seed + 1).integers(0, 300))
        mask = modifiers.kept_mask(x, k, p)
        w = [int(v) for v in sampling.to_weights(x)]
        ranked = sorted(range(300), key=lambda i: (-w[i], i))
        topk = ranked[:k] if 1 <= k < 300 else ranked
        Wk = sum(w[i] for i in topk)
        target = (int(np.floor(np.float64(np.float32(p)) * 2 ** 24)) * Wk) // 2 ** 24
        kept = [i for i in ranked if mask[i]]
        assert kept == ranked[:len(kept)]              # a prefix of the ranking
        s = sum(w[i] for i in kept)
        assert s >= target
        assert len(kept) == 1 or s - w[kept[-1]] < target
        assert len(kept) <= len(topk)


def test_ties_go_to_lower_index():
    x = np.array([0.1, 0.3, 0.2, 0.3, 0.1], dtype=np.float32)
    assert np.nonzero(modifiers.kept_mask(x, 1, 1.0))[0].tolist() == [1]
    assert np.nonzero(modifiers.kept_mask(x, 3, 1.0))[0].tolist() == [1, 2, 3]
    assert np.nonzero(modifiers.kept_mask(x, 4, 1.0))[0].tolist() == [0, 1, 2, 3]


def test_inactive_is_identity_and_renormalisation():
    x = random_probs(777, 5)
    np.testing.assert_array_equal(modifiers.modify(x, 0, 1.0), x)
    np.testing.assert_array_equal(modifiers.modify(x, 777, 1.0), x)
    for k, p in [(10, 1.0), (0, 0.9), (50, 0.7), (0, 0.0)]:
        y = modifiers.modify(x, k, p)
        kept = y > 0
        assert abs(float(y.astype(np.float64).sum()) - 1.0) < 1e-5
        r = y[kept].astype(np.float64) / x[kept].astype(np.float64)
        assert np.ptp(r) <= 4e-7 * r.max()              # one common scale up to fp32 rounding
        if p == 0.0:
            assert kept.sum() == 1 and y[np.argmax(x)] > 0.99999


def test_fp32_of_int_is_correctly_rounded():
    g = np.random.default_rng(3)
    vals = [0, 1, 2 ** 24 - 1, 2 ** 24, 2 ** 24 + 1, 2 ** 25 + 1, 2 ** 25 + 2, 2 ** 25 + 3, 2 ** 57 - 1,
            (2 ** 24 + 1) << 30, ((2 ** 24 + 1) << 30) + 1, (2 ** 23 + 1) << 31 | (1 << 30)]
    vals += [int(v) for v in g.integers(0, 2 ** 62, 500, dtype=np.uint64)]
    for S in vals:
        got = modifiers.fp32_of_int(S)
        f = Fraction(int(S))
        # nearest fp32 by exact comparison with both neighbours of the candidate
        lo = np.nextafter(got, np.float32(0)) if got > 0 else got
        hi = np.nextafter(got, np.float32(np.inf))
        for nb in (lo, hi):
            assert abs(Fraction(float(got)) - f) <= abs(Fraction(float(nb)) - f)
        if S < 2 ** 53:
            assert got == np.float32(float(S))


def test_modified_sps_follows_modified_target():
    """Draft drawn from the modified p, accept/resample on modified p and q:
    the first token's law is the modified q (Theorem 1 applied to the
    modified distributions); dropped target entries never appear."""
    V, K, n = 8, 2, 20000
    g = np.random.default_rng(11)
    q = modifiers.modify_rows(np.stack([random_probs(V, 50 + t) for t in range(K + 1)]), 5, 0.9)
    p = modifiers.modify_rows(np.stack([random_probs(V, 60 + t) for t in range(K)]), 5, 0.9)
    counts = np.zeros(V)
    for i in range(n):
        u = g.random(2 * K + 1, dtype=np.float32)
        drafts = []
        for t in range(K):
            j, ok = sampling.categorical(sampling.to_weights(p[t]), u[K + 1 + t])
            drafts.append(j)
        toks, a, flags = accept.accept_resample_one(p, q, np.array(drafts), u[:K + 1])
        counts[toks[0]] += 1
    want = q[0].astype(np.float64) / q[0].astype(np.float64).sum()
    assert counts[want == 0].sum() == 0
    keep = want > 0
    chi2, pval = stats.chisquare(counts[keep], want[keep] * n)
    assert pval > 1e-4, (chi2, pval)
