"""Philox4x64-10 counter-based generator and the uniforms SpS draws from it.

Oracle (test infrastructure only).

The paper draws r ~ U[0,1] for each accept test and samples the resampled,
bonus and draft tokens (Algorithm 2). It does not say how the randomness is
produced; it only notes that ArS and SpS consume seeds differently (Results,
Evaluation on XSum and HumanEval). We use Philox4x64 with 10 rounds as defined
by Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers: As Easy as 1, 2,
3" (SC'11): a bijection of a 256-bit counter keyed by a 128-bit key, so each
uniform is a pure function of (seed, loop, purpose, sequence, position).

Counter layout (words c0..c3) = (j, b, loop, purpose); key = (seed, 0).
  purpose 0: draft sample at draft position j (x~_{j+1})
  purpose 1: accept test r for draft position j (x~_{j+1})
  purpose 2: resample / bonus token (j = 0)
The uniform is u = (x0 >> 40) * 2^-24, i.e. the top 24 bits of output word 0,
so u lies on the 2^-24 grid in [0, 1) and is exactly representable in fp32.

Pinned by tests against numpy.random.Philox, an independent implementation of
the same published generator (tests/test_oracle_philox.py).
"""
import numpy as np

_MASK64 = (1 << 64) - 1
# Round multipliers and Weyl key increments for the 4x64 variant, as given in
# the Philox definition (SC'11, Section 5).
_M0 = 0xD2E7470EE14C6C93
_M1 = 0xCA5A826395121157
_W0 = 0x9E3779B97F4A7C15
_W1 = 0xBB67AE8584CAA73B

PURPOSE_DRAFT = 0
PURPOSE_ACCEPT = 1
PURPOSE_RESAMPLE = 2


def _mulhilo(a, b):
    """64x64 -> 128-bit product of uint64 arrays, as (hi, lo) uint64 arrays."""
    a = np.asarray(a, dtype=np.uint64)
    b = np.uint64(b)
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a_lo, a_hi = a & m32, a >> s32
    b_lo, b_hi = b & m32, b >> s32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    lo = (ll & m32) | ((mid & m32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64_10(c0, c1, c2, c3, k0, k1):
    """Ten Philox4x64 rounds over (broadcastable) uint64 counter words.

    Each round multiplies words 0 and 2 by the round constants and mixes the
    high halves with words 1, 3 and the key; the key is bumped by the Weyl
    constants between rounds.
    """
    with np.errstate(over="ignore"):
        c = [np.asarray(x, dtype=np.uint64) for x in (c0, c1, c2, c3)]
        c = np.broadcast_arrays(*c)
        c = [x.copy() for x in c]
        k0 = int(k0) & _MASK64
        k1 = int(k1) & _MASK64
        for rnd in range(10):
            hi0, lo0 = _mulhilo(c[0], _M0)
            hi1, lo1 = _mulhilo(c[2], _M1)
            c = [hi1 ^ c[1] ^ np.uint64(k0), lo1, hi0 ^ c[3] ^ np.uint64(k1), lo0]
            if rnd < 9:
                k0 = (k0 + _W0) & _MASK64
                k1 = (k1 + _W1) & _MASK64
    return c


def uniforms(seed, loop, purpose, B, n):
    """fp32 uniforms u[b][j] = top 24 bits of Philox word 0 times 2^-24.

    Returns an array of shape [B][n].
    """
    b = np.arange(B, dtype=np.uint64)[:, None]
    j = np.arange(n, dtype=np.uint64)[None, :]
    x0, _, _, _ = philox4x64_10(j, b, np.uint64(loop), np.uint64(purpose),
                                seed & _MASK64, 0)
    m = (x0 >> np.uint64(40)).astype(np.float64)
    return (m * 2.0 ** -24).astype(np.float32)
