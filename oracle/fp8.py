"""Weight-only FP8 quantisation of the projection matrices.

Oracle (test infrastructure only). The paper remarks that speculative
sampling is compatible with quantisation (Introduction; the closing remarks of
the Modified Rejection Sampling section): the draft and target distributions
only have to be the ones the models compute. It fixes no format. We read a
weight-only FP8 model as:

  * every projection matrix W [out][in] (QKV, attention output, FFN, the
    unembedding) is stored as 8-bit codes in the OCP FP8 E4M3 format (1 sign
    bit, 4 exponent bits with bias 7, 3 mantissa bits, subnormals, no
    infinities, the all-ones exponent-and-mantissa pattern is NaN; largest
    finite 448) and one fp32 scale per output row;
  * the scale of row n is s_n = fp32(amax_n) / fp32(448) in fp32 arithmetic
    (correctly rounded), amax_n the largest |W[n][k]|; an all-zero row gets
    s_n = 1;
  * the code of W[n][k] is the E4M3 value nearest to x = fp32(W[n][k]) / s_n
    (fp32 division, correctly rounded), ties to the even code (even
    mantissa), |x| clamped to 448 first so that a quotient that rounding
    pushed just past 448 saturates instead of becoming NaN; the sign of x is
    kept, so a negative x that rounds to zero encodes -0;
  * the model computes with W'[n][k] = s_n * value(code), exactly (fp64 here);
    embedding rows stay bf16, norm gains fp32, and activations and the KV
    cache follow the bf16 model (see oracle/model.py).

Every quantity that decides a code (amax, s_n, x) is computed in fp32, as the
device does, so codes and scales match bit for bit; the code decision itself
is a search over the 127 non-negative finite E4M3 values.
"""
import numpy as np

E4M3_MAX = 448.0


def e4m3_value(code):
    """Value of the E4M3 code(s) (uint8), from the format's definition:
    exponent field e, mantissa field m: (-1)^s 2^(e-7) (1 + m/8) for e >= 1,
    (-1)^s 2^-6 (m/8) for e = 0; e = 15, m = 7 is NaN. Returned as fp64."""
    c = np.asarray(code, dtype=np.uint8).astype(np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, np.ldexp(m.astype(np.float64) / 8.0, -6),
                   np.ldexp(1.0 + m.astype(np.float64) / 8.0, (e - 7).astype(np.int64)))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(s == 1, -mag, mag)


def _positive_table():
    """The 127 non-negative finite values, codes 0x00..0x7E, increasing."""
    codes = np.arange(0x7F, dtype=np.uint8)
    return codes, e4m3_value(codes)


def e4m3_encode(x):
    """Nearest E4M3 code of fp32 values x, ties to the even code, |x| clamped
    to 448 first. x must be finite."""
    x = np.asarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("e4m3_encode: non-finite input")
    codes, vals = _positive_table()
    a = np.minimum(np.abs(x).astype(np.float64), E4M3_MAX)
    # index of the largest table value <= a, and its upper neighbour
    lo = np.searchsorted(vals, a, side="right") - 1
    hi = np.minimum(lo + 1, len(vals) - 1)
    d_lo = a - vals[lo]
    d_hi = vals[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi != lo) & ((codes[hi] & 1) == 0))
    c = np.where(pick_hi, codes[hi], codes[lo]).astype(np.uint8)
    neg = np.signbit(x)
    return np.where(neg, c | np.uint8(0x80), c).astype(np.uint8)


def quantize_rows(w):
    """Codes [N][K] (uint8) and scales [N] (fp32) of a matrix w [N][K] whose
    entries are fp32-representable (bf16 weights are)."""
    w32 = np.asarray(w, dtype=np.float32)
    amax = np.max(np.abs(w32), axis=1)
    s = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    x = (w32 / s[:, None]).astype(np.float32)
    return e4m3_encode(x), s


def dequantize_rows(codes, s):
    """W' = s_n * value(code) in fp64 (exact)."""
    return np.asarray(s, dtype=np.float64)[:, None] * e4m3_value(codes)


def fp8_weights(W):
    """The oracle weights of the FP8 model built from the canonical weights W
    (dict of oracle/model.py): every projection matrix replaced by its
    dequantised FP8 form; embedding and gains unchanged."""
    q = lambda a: dequantize_rows(*quantize_rows(a))
    out = {"embed": W["embed"], "final_norm": W["final_norm"], "unembed": q(W["unembed"]), "layers": []}
    for lw in W["layers"]:
        nl = {}
        for k, v in lw.items():
            nl[k] = v if k.endswith("_norm") else q(v)
        out["layers"].append(nl)
    return out
