"""Pins of oracle/model.py (the transformer forward used for scoring).

* bf16 rounding equals torch's fp32 -> bfloat16 conversion (library RNE).
* RMSNorm, tanh-GELU and SiLU equal torch's fp64 library routines.
* Rotate-half RoPE equals multiplication of the complex numbers
  x_i + i x_{i+Dh/2} by exp(i pos theta_i), and attention logits after RoPE
  depend only on the relative position.
* The whole forward equals a torch fp64 model built from library routines
  (F.linear, F.rms_norm, F.scaled_dot_product_attention with is_causal, F.gelu),
  for both FFN kinds, with and without bf16 rounding of the attention
  operands (q, k, v).
* Scoring K+1 new tokens against a KV cache equals a full causal recompute
  (the conditionals of the Conditional Scoring section are the same numbers),
  including after a rollback that overwrites uncommitted cache entries.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model
from oracle.model import ModelSpec
from paper_2302_01318_amd import configs, synth
from oracle_helpers import oracle_weights, spec_of


def test_round_bf16_matches_torch():
    g = np.random.default_rng(0)
    x = np.concatenate([g.normal(0, 1, 5000), g.normal(0, 1e-30, 100), [0.0, -0.0, 1.0 + 2 ** -8,
                        1.0 + 3 * 2 ** -8, 65504.0, 3.0e38]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(model.round_bf16(x), ref)


def test_blocks_match_torch_library():
    g = np.random.default_rng(1)
    h = g.normal(0, 2, (3, 5, 64))
    gain = g.normal(1, 0.1, 64)
    ref = F.rms_norm(torch.from_numpy(h), (64,), weight=torch.from_numpy(gain), eps=1e-5).numpy()
    np.testing.assert_allclose(model.rms_norm(h, gain, 1e-5), ref, rtol=1e-13)
    x = g.normal(0, 3, 1000)
    np.testing.assert_allclose(model.gelu_tanh(x), F.gelu(torch.from_numpy(x), approximate="tanh").numpy(),
                               rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(model.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-12, atol=1e-15)


def test_rope_is_complex_rotation():
    g = np.random.default_rng(2)
    Dh = 64
    x = g.normal(0, 1, (7, Dh))
    pos = np.array([0, 1, 2, 17, 100, 2047, 8191])
    z = x[:, :Dh // 2] + 1j * x[:, Dh // 2:]
    theta = 10000.0 ** (-np.arange(0, Dh, 2) / Dh)
    zr = z * np.exp(1j * pos[:, None] * theta[None, :])
    want = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(model.rope(x, pos, 10000.0), want, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(model.rope(x[:1], np.array([0]), 10000.0), x[:1])


def test_rope_relative_position():
    g = np.random.default_rng(3)
    q, k = g.normal(0, 1, 128), g.normal(0, 1, 128)
    d1 = model.rope(q, np.array(50), 1e4) @ model.rope(k, np.array(20), 1e4)
    d2 = model.rope(q, np.array(1030), 1e4) @ model.rope(k, np.array(1000), 1e4)
    assert abs(d1 - d2) < 1e-9
    assert abs(np.linalg.norm(model.rope(q, np.array(999), 1e4)) - np.linalg.norm(q)) < 1e-12


def torch_forward(spec, W, tokens):
    """Independent fp64 forward from torch library routines."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    rb = (lambda x: x.float().to(torch.bfloat16).double()) if spec.dtype == "bf16" else (lambda x: x)
    B, T = tokens.shape
    H, Dh, d = spec.n_heads, spec.head_dim, spec.d_model
    pos = torch.arange(T, dtype=torch.float64)
    theta = spec.rope_base ** (-torch.arange(0, Dh, 2, dtype=torch.float64) / Dh)
    rot = torch.polar(torch.ones(T, Dh // 2, dtype=torch.float64), pos[:, None] * theta[None, :])

    def rope(x):                               # x [B, T, H, Dh]
        z = torch.complex(x[..., :Dh // 2], x[..., Dh // 2:]) * rot[None, :, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    h = t(W["embed"])[torch.from_numpy(tokens).long()]
    for lw in W["layers"]:
        x = F.rms_norm(h, (d,), weight=t(lw["attn_norm"]), eps=spec.eps)
        q = rb(rope(F.linear(x, t(lw["wq"])).view(B, T, H, Dh)))
        k = rb(rope(F.linear(x, t(lw["wk"])).view(B, T, H, Dh)))
        v = rb(F.linear(x, t(lw["wv"])).view(B, T, H, Dh))
        o = F.scaled_dot_product_attention(q.transpose(1, 2), k.transpose(1, 2), v.transpose(1, 2),
                                           is_causal=True)
        o = o.transpose(1, 2).reshape(B, T, H * Dh)
        h = h + F.linear(o, t(lw["wo"]))
        x = F.rms_norm(h, (d,), weight=t(lw["ffn_norm"]), eps=spec.eps)
        if spec.ffn == "gelu":
            a = F.gelu(F.linear(x, t(lw["w1"])), approximate="tanh")
            h = h + F.linear(a, t(lw["w2"]))
        else:
            a = F.silu(F.linear(x, t(lw["wg"]))) * F.linear(x, t(lw["wu"]))
            h = h + F.linear(a, t(lw["wd"]))
    x = F.rms_norm(h, (d,), weight=t(W["final_norm"]), eps=spec.eps)
    return F.linear(x, t(W["unembed"])).numpy()


SMALL = configs.ModelShape("small", 64, 2, 2, 32, 96, 50, "gelu", "f32")


@pytest.mark.parametrize("ffn", ["gelu", "swiglu"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_matches_torch_model(ffn, dtype):
    shape = SMALL.with_(ffn=ffn, dtype=dtype)
    W = oracle_weights(shape, synth.weights(shape, seed=5, std=0.1))
    spec = spec_of(shape)
    toks = synth.tokens(6, 2, 9, shape.vocab)
    got = model.forward_full(spec, W, toks)
    want = torch_forward(spec, W, toks)
    np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_incremental_scoring_equals_full_recompute(dtype):
    shape = SMALL.with_(dtype=dtype, ffn="swiglu")
    W = oracle_weights(shape, synth.weights(shape, seed=7, std=0.1))
    spec = spec_of(shape)
    toks = synth.tokens(8, 3, 14, shape.vocab)
    full = model.forward_full(spec, W, toks)
    cache = model.new_cache(spec, 3, 32)
    model.forward_cached(spec, W, cache, toks[:, :9], np.zeros(3, int))
    # a rejected draft block: scored, then overwritten by the next call
    model.forward_cached(spec, W, cache, (toks[:, 9:14] + 1) % shape.vocab, np.full(3, 9))
    got = model.forward_cached(spec, W, cache, toks[:, 9:14], np.full(3, 9))
    np.testing.assert_allclose(got, full[:, 9:14], rtol=1e-9, atol=1e-9)
