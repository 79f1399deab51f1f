"""Pins of the FP8 (OCP E4M3) weight quantisation of the oracle.

The paper fixes no number format; the format is the OCP 8-bit floating point
specification's E4M3 (bias 7, subnormals, no infinities, max 448). The
oracle's decode is pinned to torch's independent float8_e4m3fn type and to the
values the specification tabulates; its encoder (a nearest-value search) to
torch's round-to-nearest-even conversion; the per-row quantiser to the
properties its definition implies."""
import numpy as np
import pytest
import torch

from oracle import fp8


def torch_decode(codes):
    return torch.from_numpy(np.asarray(codes, np.uint8)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def torch_encode(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_spec_values_and_torch():
    codes = np.arange(256, dtype=np.uint8)
    v = fp8.e4m3_value(codes)
    t = torch_decode(codes)
    nan = np.isnan(t)
    assert np.array_equal(np.isnan(v), nan)
    assert list(np.nonzero(nan)[0]) == [0x7F, 0xFF]
    assert np.array_equal(v[~nan], t[~nan])
    assert np.array_equal(np.signbit(v[~nan]), np.signbit(t[~nan]))
    # values the specification lists for E4M3
    assert v[0x7E] == 448.0 and v[0xFE] == -448.0          # max normal  S.1111.110
    assert v[0x08] == 2.0 ** -6                             # min normal  S.0001.000
    assert v[0x07] == 0.875 * 2.0 ** -6                     # max subnormal S.0000.111
    assert v[0x01] == 2.0 ** -9                             # min subnormal S.0000.001
    assert v[0x38] == 1.0 and v[0x00] == 0.0 and np.signbit(v[0x80])
    assert np.all(np.diff(v[:0x7F]) > 0)                    # codes 0..0x7E increase


def test_encode_matches_torch_rne():
    rng = np.random.default_rng(0)
    pos = fp8.e4m3_value(np.arange(0x7F, dtype=np.uint8))
    mids = (pos[:-1] + pos[1:]) / 2                          # exact ties (fp32-representable)
    mids32 = mids.astype(np.float32)
    assert np.array_equal(mids32.astype(np.float64), mids)
    xs = [pos.astype(np.float32), mids32,
          np.nextafter(mids32, np.float32(np.inf)), np.nextafter(mids32, np.float32(0)),
          (rng.standard_normal(20000) * 60).clip(-448, 448).astype(np.float32),
          (rng.standard_normal(20000) * 2.0 ** -7).astype(np.float32),    # subnormal range
          np.float32([0.0, -0.0, 1e-30, -1e-30, 2.0 ** -10, 3 * 2.0 ** -11, 448.0, 464.0, -464.0])]
    x = np.concatenate(xs)
    x = np.concatenate([x, -x])
    got = fp8.e4m3_encode(x)
    want = torch_encode(x)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (x[bad[:5]], got[bad[:5]], want[bad[:5]])
    # ties go to the even code: the midpoint of codes c, c+1 encodes to the even one
    c = fp8.e4m3_encode(mids32)
    assert np.all(c % 2 == 0)


def test_encode_saturates_instead_of_nan():
    x = np.float32([448.0, 449.0, 470.0, 479.9, 480.0, 1e6, 3e38])
    assert np.all(fp8.e4m3_encode(x) == 0x7E)
    assert np.all(fp8.e4m3_encode(-x) == 0xFE)
    with pytest.raises(ValueError):
        fp8.e4m3_encode(np.float32([np.inf]))


def test_quantize_rows_properties():
    rng = np.random.default_rng(1)
    w = (rng.standard_normal((64, 512)) * 0.02)
    w[3] = 0.0
    w[5, 7] = 0.5                                            # one outlier
    w = torch.from_numpy(w).to(torch.bfloat16).float().numpy()
    codes, s = fp8.quantize_rows(w)
    assert codes.dtype == np.uint8 and s.dtype == np.float32
    amax = np.abs(w).max(axis=1).astype(np.float32)
    assert np.array_equal(s[amax > 0], (amax[amax > 0] / np.float32(448)).astype(np.float32))
    assert s[3] == 1.0 and np.all(codes[3] == 0)
    # the largest entry of a row maps to +-448 (the quotient is within an ulp of 448)
    rows = np.nonzero(amax > 0)[0]
    arg = np.abs(w[rows]).argmax(axis=1)
    assert np.all((codes[rows, arg] & 0x7F) == 0x7E)
    # reconstruction error: half a step of the format at |x|
    wq = fp8.dequantize_rows(codes, s)
    x = np.abs(w / s[:, None].astype(np.float64))
    step = np.where(x < 2.0 ** -6, 2.0 ** -9, 2.0 ** (np.floor(np.log2(np.maximum(x, 2.0 ** -6))) - 3))
    assert np.all(np.abs(w - wq) <= step / 2 * s[:, None] * (1 + 1e-6))
    # signs are kept
    nz = np.abs(wq) > 0
    assert np.array_equal(np.sign(wq[nz]), np.sign(w[nz]))


def test_fp8_weights_replace_only_projections():
    rng = np.random.default_rng(2)
    W = {"embed": rng.standard_normal((10, 64)), "final_norm": rng.standard_normal(64),
         "unembed": rng.standard_normal((10, 64)) * 0.02,
         "layers": [{"attn_norm": np.ones(64), "ffn_norm": np.ones(64), "wq": rng.standard_normal((64, 64)) * 0.02}]}
    Q = fp8.fp8_weights(W)
    assert Q["embed"] is W["embed"] and Q["final_norm"] is W["final_norm"]
    assert Q["layers"][0]["attn_norm"] is W["layers"][0]["attn_norm"]
    c, s = fp8.quantize_rows(W["layers"][0]["wq"])
    assert np.array_equal(Q["layers"][0]["wq"], fp8.dequantize_rows(c, s))
    assert not np.array_equal(Q["unembed"], W["unembed"])
