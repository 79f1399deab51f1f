"""Pins of oracle/accept.py (modified rejection sampling).

1. Exact enumeration: for tiny vocabularies and prefix-dependent draft and
   target tables, the exact law of the first N tokens produced by repeated
   SpS loops (drafting with the oracle's sampler, then accept_resample_one)
   is computed in rational arithmetic by enumerating every draft path, every
   accept/reject pattern and every interval of the uniform grid on which the
   final draw is constant. Theorem 1 applied loop after loop says that law is
   prod_i q(y_i | y_<i). The implementation draws uniforms on a 2^-24 grid,
   so each uniform-driven decision is off by less than 2^-24 from its ideal
   probability; the comparison bound is derived from that.
2. Negative controls: planting the classic mistakes into the oracle (drawing
   the replacement from q instead of (q - p)_+, or testing p/q instead of
   q/p) must break the same check.
3. Statistics on random (non-dyadic) distributions: chi-square of the first
   emitted token against q_1, and the acceptance frequency of x~_1 against
   sum_x min(p(x), q(x)) (Theorem 1 proof).
4. Special cases and decision edges.
"""
import itertools
from collections import defaultdict
from fractions import Fraction as Fr

import numpy as np
import pytest
from scipy import stats

from oracle import accept, philox, sampling

GRID = 1 << 24


# ---------------------------------------------------------------- helpers --

def dyadic_table(V, seed, allow_zero):
    """Random distribution with entries c_i / 4096 summing exactly to one."""
    g = np.random.default_rng(seed)
    lo = 0 if allow_zero else 1
    while True:
        cuts = np.sort(g.integers(0, 4097, size=V - 1))
        c = np.diff(np.concatenate([[0], cuts, [4096]]))
        if c.min() >= lo and c.max() > 0:
            return c


def make_tables(V, seed):
    cache = {}

    def table(kind, prefix):
        key = (kind, tuple(prefix))
        if key not in cache:
            h = hash(key) % (1 << 30)
            cache[key] = dyadic_table(V, seed * 7919 + h, allow_zero=(kind == "q"))
        return cache[key]

    P = lambda pre: (table("p", pre) / 4096.0).astype(np.float32)
    Q = lambda pre: (table("q", pre) / 4096.0).astype(np.float32)
    Qfr = lambda pre: [Fr(int(c), 4096) for c in table("q", pre)]
    return P, Q, Qfr


def g_count(c, W):
    """Grid values m with floor(m W / 2^24) < c."""
    return min(GRID, -(-c * GRID // W))


def intervals(weight_vectors):
    """Maximal runs of grid values on which every candidate draw is constant."""
    bps = {0, GRID}
    for w in weight_vectors:
        W = int(sum(int(x) for x in w))
        if W == 0:
            continue
        acc = 0
        for wi in w:
            acc += int(wi)
            bps.add(g_count(acc, W))
    bps = sorted(bps)
    return [(a, b - a) for a, b in zip(bps[:-1], bps[1:]) if b > a]


def accept_count(pi, rho):
    """Grid values m with (m 2^-24) * pi < rho, counted exactly."""
    pi, rho = Fr(float(pi)), Fr(float(rho))
    if pi == 0:
        return GRID if rho > 0 else 0
    x = rho * GRID / pi
    return max(0, min(GRID, -(-x.numerator // x.denominator)))


def candidate_weights(p_rows, q_rows):
    out = [sampling.to_weights(q) for q in q_rows]
    for p, q in zip(p_rows, q_rows):
        wq = sampling.to_weights(q).astype(np.int64)
        wp = sampling.to_weights(p).astype(np.int64)
        out.append(np.maximum(wq - wp, 0))
    return out


def loop_law(prefix, K, P, Q):
    """Exact law of the tokens one SpS loop emits after `prefix`."""
    out = defaultdict(Fr)

    def draft(t, drafts, prob):
        if t == K:
            finish(drafts, prob)
            return
        w = sampling.to_weights(P(prefix + drafts))
        for m0, L in intervals([w]):
            x, ok = sampling.categorical(w, np.float32(m0 * 2.0 ** -24))
            assert ok
            draft(t + 1, drafts + [x], prob * Fr(L, GRID))

    def finish(drafts, prob):
        p_rows = [P(prefix + drafts[:t]) for t in range(K)]
        q_rows = [Q(prefix + drafts[:t]) for t in range(K + 1)]
        cands = candidate_weights(p_rows, q_rows)
        p_arr = np.array(p_rows, dtype=np.float32).reshape(K, -1)
        q_arr = np.array(q_rows, dtype=np.float32)
        for pattern in itertools.product([1, 0], repeat=K):
            wgt, r = Fr(1), []
            for t in range(K):
                A = accept_count(p_rows[t][drafts[t]], q_rows[t][drafts[t]])
                if pattern[t]:
                    wgt *= Fr(A, GRID)
                    r.append(0.0)
                else:
                    wgt *= Fr(GRID - A, GRID)
                    r.append((GRID - 1) * 2.0 ** -24)
            if wgt == 0:
                continue
            for m0, L in intervals(cands):
                unif = np.array(r + [m0 * 2.0 ** -24], dtype=np.float32)
                toks, a, flags = accept.accept_resample_one(p_arr, q_arr, drafts, unif)
                assert flags == 0 and len(toks) == a + 1
                out[tuple(toks)] += prob * wgt * Fr(L, GRID)

    draft(0, [], Fr(1))
    return out


def sequence_law(N, K, P, Q):
    memo = {}

    def law(prefix):
        if len(prefix) >= N:
            return {tuple(prefix[:N]): Fr(1)}
        key = tuple(prefix)
        if key not in memo:
            res = defaultdict(Fr)
            for toks, w in loop_law(list(prefix), K, P, Q).items():
                for seq, w2 in law(list(prefix) + list(toks)).items():
                    res[seq] += w * w2
            memo[key] = res
        return memo[key]

    return law([])


def target_law(seq, Qfr):
    pr = Fr(1)
    for i, y in enumerate(seq):
        pr *= Qfr(list(seq[:i]))[y]
    return pr


def check_law(V, K, N, seed):
    P, Q, Qfr = make_tables(V, seed)
    law = sequence_law(N, K, P, Q)
    assert sum(law.values()) == 1
    # each loop has at most 2K+1 uniform-driven decisions, each within 2^-24
    # of its ideal probability per outcome (V outcomes for a draw); at most N
    # loops produce the first N tokens.
    bound = Fr(N * (2 * K + 1) * (V + 1), GRID)
    worst = Fr(0)
    for seq in itertools.product(range(V), repeat=N):
        worst = max(worst, abs(law.get(seq, Fr(0)) - target_law(seq, Qfr)))
    return worst, bound


# ------------------------------------------------------------ enumeration --

@pytest.mark.parametrize("V,K,N,seed", [(2, 1, 3, 1), (2, 2, 3, 2), (3, 1, 3, 3),
                                        (2, 3, 4, 4), (3, 2, 3, 5)])
def test_exact_law_equals_target(V, K, N, seed):
    worst, bound = check_law(V, K, N, seed)
    assert worst <= bound, (float(worst), float(bound))


def test_negative_control_resample_from_q(monkeypatch):
    monkeypatch.setattr(accept, "residual_weights", lambda q, p: sampling.to_weights(q))
    worst, bound = check_law(3, 2, 3, 5)
    assert worst > 100 * bound


def test_negative_control_swapped_ratio(monkeypatch):
    orig = accept.accept_test
    monkeypatch.setattr(accept, "accept_test", lambda r, pi, rho: orig(r, rho, pi))
    worst, bound = check_law(3, 2, 3, 5)
    assert worst > 100 * bound


# ------------------------------------------------------------- statistics --

def run_many(p, q, n, seed, K):
    """n independent loops on fixed p [K][V], q [K+1][V]; drafts drawn with
    the oracle sampler from Philox purpose DRAFT (batch index = run)."""
    ud = philox.uniforms(seed, 0, philox.PURPOSE_DRAFT, n, K)
    unif = accept.philox_uniforms(seed, 0, n, K)
    wp = [sampling.to_weights(p[t]) for t in range(K)]
    first, acc1 = [], 0
    for i in range(n):
        drafts = [sampling.categorical(wp[t], ud[i, t])[0] for t in range(K)]
        toks, a, _ = accept.accept_resample_one(p, q, drafts, unif[i])
        first.append(toks[0])
        acc1 += a >= 1
    return np.bincount(first, minlength=q.shape[1]), acc1


def random_pair(V, K, seed):
    g = np.random.default_rng(seed)
    q = g.dirichlet(np.ones(V), size=K + 1).astype(np.float32)
    p = g.dirichlet(np.ones(V), size=K).astype(np.float32)
    return p, q


@pytest.mark.parametrize("K", [1, 2, 4])
def test_chi_square_first_token_and_acceptance_rate(K):
    V, n = 8, 30000
    p, q = random_pair(V, K, 10 + K)
    counts, acc1 = run_many(p, q, n, seed=77 + K, K=K)
    q64 = q[0].astype(np.float64)
    expected = q64 / q64.sum() * n
    assert stats.chisquare(counts, expected).pvalue > 1e-4
    alpha = np.minimum(p[0].astype(np.float64), q[0]).sum()
    assert stats.binomtest(acc1, n, alpha).pvalue > 1e-4


def test_chi_square_negative_control(monkeypatch):
    monkeypatch.setattr(accept, "residual_weights", lambda q, p: sampling.to_weights(q))
    V, K, n = 8, 2, 30000
    p, q = random_pair(V, K, 12)
    counts, _ = run_many(p, q, n, seed=79, K=K)
    q64 = q[0].astype(np.float64)
    expected = q64 / q64.sum() * n
    assert stats.chisquare(counts, expected).pvalue < 1e-6


# ---------------------------------------------------------- special cases --

def test_equal_distributions_accept_everything():
    g = np.random.default_rng(3)
    for _ in range(50):
        K, V = int(g.integers(1, 6)), int(g.integers(2, 50))
        q = g.dirichlet(np.ones(V), size=K + 1).astype(np.float32)
        p = q[:K].copy()
        drafts = [int(g.choice(V, p=p[t].astype(np.float64) / p[t].astype(np.float64).sum()))
                  for t in range(K)]
        unif = np.concatenate([np.full(K, (GRID - 1) * 2.0 ** -24), [g.random()]]).astype(np.float32)
        toks, a, flags = accept.accept_resample_one(p, q, drafts, unif)
        assert a == K and toks[:K] == drafts and flags == 0


def test_counts_and_padding():
    p, q, d = random_pair(16, 4, 5)[0], random_pair(16, 4, 5)[1], None
    g = np.random.default_rng(9)
    P = np.stack([p] * 6)
    Q = np.stack([q] * 6)
    drafts = g.integers(0, 16, size=(6, 4))
    unif = g.random((6, 5)).astype(np.float32)
    out, n_acc, flags = accept.accept_resample(P, Q, drafts, unif)
    for b in range(6):
        a = n_acc[b]
        assert 0 <= a <= 4
        assert list(out[b, :a]) == list(drafts[b, :a])
        assert 0 <= out[b, a] < 16 and all(out[b, a + 1:] == -1)


def test_k0_is_a_plain_draw_from_q():
    q = np.random.default_rng(2).dirichlet(np.ones(10), size=1).astype(np.float32)
    for u in np.linspace(0, 1, 37, endpoint=False).astype(np.float32):
        toks, a, _ = accept.accept_resample_one(np.zeros((0, 10), np.float32), q, [], np.array([u]))
        assert a == 0 and toks == [sampling.categorical(sampling.to_weights(q[0]), u)[0]]


def test_greedy_one_hot():
    V = 6
    onehot = lambda i: np.eye(V, dtype=np.float32)[i]
    # target argmaxes 2, 4, 1 ; draft proposes 2, 5
    q = np.stack([onehot(2), onehot(4), onehot(1)])
    p = np.stack([onehot(2), onehot(5)])
    toks, a, _ = accept.accept_resample_one(p, q, [2, 5], np.array([0.9, 0.0, 0.5], np.float32))
    assert a == 1 and toks == [2, 4]
    q2 = np.stack([onehot(2), onehot(5), onehot(1)])
    toks, a, _ = accept.accept_resample_one(p, q2, [2, 5], np.array([0.99, 0.99, 0.5], np.float32))
    assert a == 2 and toks == [2, 5, 1]


def test_decision_edges():
    V = 4
    q = np.array([[0.25, 0.25, 0.25, 0.25], [0.25, 0.25, 0.25, 0.25]], np.float32)
    p = np.array([[0.5, 0.5, 0.0, 0.0]], np.float32)
    # rho / pi = 0.5 exactly: r = 0.5 rejects (strict <), one grid step below accepts
    assert accept.accept_resample_one(p, q, [0], np.array([0.5, 0.0], np.float32))[1] == 0
    below = np.float32(0.5 - 2.0 ** -24)
    assert accept.accept_resample_one(p, q, [0], np.array([below, 0.0], np.float32))[1] == 1
    # p(x~) = 0 accepts iff q(x~) > 0
    assert accept.accept_resample_one(p, q, [2], np.array([0.999, 0.0], np.float32))[1] == 1
    qz = q.copy()
    qz[0, 2] = 0.0
    assert accept.accept_resample_one(p, qz, [2], np.array([0.0, 0.0], np.float32))[1] == 0
    # rejected: the replacement comes from (q - p)_+ = tokens 2, 3 only
    for u in np.linspace(0, 1, 50, endpoint=False).astype(np.float32):
        toks, a, _ = accept.accept_resample_one(p, q, [0], np.array([0.99, u], np.float32))
        assert a == 0 and toks[0] in (2, 3)


def test_zero_residual_falls_back_to_q():
    # q = p / 2 everywhere: (q - p)_+ has no mass, so a rejection draws from q
    p = np.array([[0.5, 0.25, 0.25]], np.float32)
    q = np.array([[0.25, 0.125, 0.125], [1 / 3, 1 / 3, 1 / 3]], np.float32)
    for u in np.linspace(0, 1, 20, endpoint=False).astype(np.float32):
        toks, a, flags = accept.accept_resample_one(p, q, [1], np.array([0.75, u], np.float32))
        assert a == 0 and flags == 0
        assert toks[0] == sampling.categorical(sampling.to_weights(q[0]), u)[0]


def test_bad_token_and_empty_distribution_flags():
    p = np.full((2, 3), 1 / 3, np.float32)
    q = np.full((3, 3), 1 / 3, np.float32)
    toks, a, flags = accept.accept_resample_one(p, q, [1, 7], np.array([0, 0, 0.5], np.float32))
    assert a == 1 and flags & accept.FLAG_BAD_TOKEN and toks[0] == 1
    qz = np.zeros((1, 3), np.float32)
    toks, a, flags = accept.accept_resample_one(np.zeros((0, 3), np.float32), qz, [], np.array([0.3], np.float32))
    assert toks == [0] and flags & accept.FLAG_EMPTY


def test_nonfinite_inputs_give_a_defined_outcome():
    """The library's definition for inputs that are not distributions (the
    paper assumes valid ones): a NaN or infinite gathered probability, or
    one in a row the final draw reads, or a target row marked as having
    non-finite logits, gives a = 0 and token 0 with FLAG_NONFINITE; a NaN in
    an entry nothing reads changes nothing."""
    g = np.random.default_rng(5)
    K, V = 4, 16
    p = g.dirichlet(np.ones(V), size=K).astype(np.float32)
    q = g.dirichlet(np.ones(V), size=K + 1).astype(np.float32)
    drafts = np.array([3, 5, 7, 9])
    q[0, 3] = 1e-4                             # x~_1 is rejected: the draw reads q_1 and p_1
    unif = np.array([0.99, 0.99, 0.99, 0.99, 0.4], np.float32)
    base, a0, f0 = accept.accept_resample_one(p, q, drafts, unif)
    assert f0 == 0 and a0 == 0
    for what in ("q_gather_late", "p_gather", "p_row", "q_row", "inf"):
        pp, qq = p.copy(), q.copy()
        if what == "q_gather_late":
            qq[3, 9] = np.nan                  # x~_4's q, read even though the scan stops at x~_1
        elif what == "p_gather":
            pp[1, 5] = np.nan
        elif what == "p_row":
            pp[0, 0] = np.nan                  # off the draft token, in the row of the residual draw
        elif what == "q_row":
            qq[0, 15] = np.nan
        else:
            qq[0, 14] = np.inf
        toks, a, flags = accept.accept_resample_one(pp, qq, drafts, unif)
        assert toks == [0] and a == 0 and flags & accept.FLAG_NONFINITE, what
    # an entry nothing reads: q row 3 off its draft token
    qq = q.copy()
    qq[3, 0] = np.nan
    assert accept.accept_resample_one(p, qq, drafts, unif) == (base, a0, f0)
    bad = np.zeros(K + 1, bool)
    bad[K] = True
    toks, a, flags = accept.accept_resample_one(p, q, drafts, unif, bad)
    assert toks == [0] and a == 0 and flags & accept.FLAG_NONFINITE
