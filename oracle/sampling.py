"""Softmax with temperature and exact fixed-point categorical sampling.

Oracle (test infrastructure only).

Probability modifiers: the paper applies temperature (and nucleus / top-k)
to both the draft and target distributions before the rejection step
(Modified Rejection Sampling section, closing paragraphs). Greedy decoding
(Table 1, "Greedy" rows) is temperature 0: a one-hot distribution on the
argmax, lowest index on ties.

Categorical sampling: the paper does not say how a token is drawn from a
distribution. A float prefix sum depends on summation order, so a parallel
GPU scan and a serial CPU loop would not agree bit for bit. We therefore draw
through an integer inverse CDF that is order independent:

  weights    w_i = floor(x_i * 2^32) for a probability x_i (0 if x_i <= 0 or
             NaN, 2^32 if x_i >= 1), exact for fp32 x_i;
  total      W = sum_i w_i, exact in integers;
  threshold  m = floor(u * 2^24) for the uniform u, t = floor(m * W / 2^24);
  result     the smallest i whose inclusive prefix sum exceeds t.

A zero-weight index can never be selected. Each index i is selected by
exactly the grid values m with prefix_{i-1} <= floor(m W / 2^24) < prefix_i,
so P(i) differs from w_i / W by less than 2^-24
(tests/test_oracle_sampling.py counts this on every grid point).
"""
import numpy as np

TWO32 = 1 << 32


def nonfinite_rows(logits, temperature):
    """Rows that have no distribution: a NaN or +Inf logit, or (T > 0) a
    logit whose fp32 quotient by T, formed as z * fp32(1 / T) in fp32,
    overflows to +Inf. -Inf logits are valid (probability 0). The paper
    assumes valid distributions (Modified Rejection Sampling section); the
    library defines such a row as one-hot at token 0."""
    z = np.asarray(logits, dtype=np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        if temperature != 0.0:
            z = z * np.float32(np.float32(1.0) / np.float32(temperature))
        return ~np.all(z < np.float32(np.inf), axis=-1)


def softmax(logits, temperature):
    """Row-wise softmax(logits / T) in fp64; T == 0 gives one-hot argmax.
    Rows in nonfinite_rows are one-hot at index 0."""
    z = np.asarray(logits, dtype=np.float64)
    bad = nonfinite_rows(logits, temperature)
    z = np.where(bad[..., None], 0.0, z)
    if temperature == 0.0:
        out = np.zeros_like(z)
        idx = np.argmax(z, axis=-1)          # first index among equal maxima
        np.put_along_axis(out, idx[..., None], 1.0, axis=-1)
        return out
    z = z / float(temperature)
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    out = e / e.sum(axis=-1, keepdims=True)
    out[bad] = 0.0
    out[bad, ..., 0] = 1.0
    return out


def to_weights(x):
    """Fixed-point weights floor(x * 2^32) as uint64, for fp32 probabilities x.

    The product of an fp32 value with 2^32 is exact in fp64, so the floor is
    exact. Values <= 0 or NaN give 0; values >= 1 give 2^32.
    """
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    w = np.zeros(x.shape, dtype=np.uint64)
    pos = x > 0.0                             # False for NaN
    big = x >= 1.0
    mid = pos & ~big
    w[mid] = np.floor(x[mid] * float(TWO32)).astype(np.uint64)
    w[big] = np.uint64(TWO32)
    return w


def grid_index(u):
    """m = floor(u * 2^24) for an fp32 uniform in [0, 1) (exact in fp64).

    Out-of-range inputs are clamped: u <= 0 or NaN gives 0, u >= 1 gives
    2^24 - 1.
    """
    v = float(np.float32(u))
    if not v > 0.0:                           # also catches NaN
        return 0
    if v >= 1.0:
        return (1 << 24) - 1
    return int(np.floor(v * float(1 << 24)))


def categorical(w, u):
    """Draw an index from integer weights w with uniform u (see module doc).

    Returns (index, ok). ok is False when every weight is zero; index is
    then 0.
    """
    w = [int(v) for v in np.asarray(w, dtype=np.uint64).ravel()]
    total = sum(w)
    if total == 0:
        return 0, False
    t = (grid_index(u) * total) >> 24
    acc = 0
    for i, wi in enumerate(w):
        acc += wi
        if acc > t:
            return i, True
    raise AssertionError("unreachable: t < total")
