"""Decoder-only transformer forward used for conditional scoring.

Oracle (test infrastructure only). Plain numpy in fp64, one sequence and one
head at a time, no blocking or fusion.

The paper scores the K+1 prefixes (x_1..x_n), (x_1..x_n, x~_1), ...,
(x_1..x_n, x~_1..x~_K) with one parallel call of the target (Algorithm 2;
Conditional Scoring section), keeping a cache of the keys and values of all
earlier tokens. It names the Chinchilla shapes (Hyperparams table: d_model,
heads, layers) but not the block design. We read the architecture as:

  * pre-norm decoder blocks, no biases, untied embedding and unembedding;
  * RMSNorm  y = h / sqrt(mean(h^2) + eps) * g, eps = 1e-5;
  * multi-head attention with rotary position encoding, rotate-half pairing
    (dims i and i + Dh/2 rotate by pos * base^(-2i/Dh), base 10000), scale
    1/sqrt(Dh), query at position P sees keys at positions <= P;
  * FFN either GELU (tanh form) with two matrices, or SwiGLU with three.

Weights are float32 arrays in nn.Linear orientation [out][in] (for bf16
models they hold bf16-representable values). Activations and accumulation
are fp64. A bf16 model is read as bf16 WEIGHTS and a bf16 KV CACHE: the
queries, keys and values of attention are rounded to bf16 (round to nearest
even) after the rotary encoding, which is what the cache stores and what
enters the score product; every other activation keeps full precision. (If
the normed activations, the attention output and the FFN hidden were also
rounded to bf16, a single last-bit difference upstream flips a large share
of those roundings downstream, so two faithful implementations with
different fp32 summation orders would disagree by about 1% of the logit
scale.) Parity against the GPU path is to a tolerance (1e-4 fp32, 2e-2 bf16
on logits); the paper prints no values to pin them, so the logits are
"parity unpinned" by the paper; the forward itself is pinned by the tests in
tests/test_oracle_model.py (incremental scoring equals full recompute; blocks
equal torch fp64 library routines; RoPE equals complex rotation).
"""
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ModelSpec:
    d_model: int
    n_layers: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    ffn: str = "gelu"          # "gelu" or "swiglu"
    dtype: str = "f32"         # "f32" or "bf16"
    eps: float = 1e-5
    rope_base: float = 10000.0


def round_bf16(x):
    """Round to the nearest bf16 value (ties to even), returned as fp64.

    fp64 is first rounded to fp32, then the low 16 bits of the fp32 pattern
    are rounded away.
    """
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16) << np.uint64(16)
    out = (u & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)
    nan = np.isnan(f)
    if np.any(nan):
        out = out.copy()
        out[nan] = np.nan
    return out.astype(np.float64)


def _store(spec, x):
    """What the KV cache (and the score product) sees: bf16 for bf16 models."""
    return round_bf16(x) if spec.dtype == "bf16" else np.asarray(x, dtype=np.float64)


def rms_norm(h, g, eps):
    h = np.asarray(h, dtype=np.float64)
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps) * np.asarray(g, np.float64)


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def silu(x):
    return x / (1.0 + np.exp(-x))


def rope(x, pos, base):
    """Rotate-half RoPE of x [..., Dh] at integer positions pos (shape x[..., 0])."""
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    inv_freq = base ** (-(2.0 * np.arange(half)) / dh)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def linear(x, w):
    """y = x W^T for W in [out][in] orientation."""
    return np.asarray(x, np.float64) @ np.asarray(w, np.float64).T


def new_cache(spec, B, T_cap):
    """KV cache: k, v of shape [L][B][H][T_cap][Dh] fp64 (k already rotated)."""
    shape = (spec.n_layers, B, spec.n_heads, T_cap, spec.head_dim)
    return {"k": np.zeros(shape), "v": np.zeros(shape)}


def _attend(q, K, V, scale):
    """Softmax attention of one query q [Dh] over keys/values [n][Dh]."""
    s = (K @ q) * scale
    s = s - s.max()
    w = np.exp(s)
    w = w / w.sum()
    return w @ V


def forward_cached(spec, W, cache, tokens, lengths):
    """Score tokens [B][M] placed at positions lengths[b] + j, j < M.

    Writes their keys/values into the cache (the caller decides whether the
    lengths advance) and returns logits [B][M][V] in fp64. Query j of
    sequence b attends to cache positions 0 .. lengths[b] + j.
    """
    tokens = np.asarray(tokens)
    B, M = tokens.shape
    H, Dh = spec.n_heads, spec.head_dim
    scale = 1.0 / np.sqrt(Dh)
    pos = np.asarray(lengths, dtype=np.int64)[:, None] + np.arange(M)[None, :]
    h = np.asarray(W["embed"], np.float64)[tokens]                     # [B][M][d]
    for li, lw in enumerate(W["layers"]):
        x = rms_norm(h, lw["attn_norm"], spec.eps)
        q = linear(x, lw["wq"]).reshape(B, M, H, Dh)
        k = linear(x, lw["wk"]).reshape(B, M, H, Dh)
        v = linear(x, lw["wv"]).reshape(B, M, H, Dh)
        q = _store(spec, rope(q, pos[:, :, None], spec.rope_base))
        k = _store(spec, rope(k, pos[:, :, None], spec.rope_base))
        v = _store(spec, v)
        o = np.zeros((B, M, H, Dh))
        for b in range(B):
            for j in range(M):
                cache["k"][li, b, :, pos[b, j]] = k[b, j]
                cache["v"][li, b, :, pos[b, j]] = v[b, j]
            for j in range(M):
                n = pos[b, j] + 1
                for hh in range(H):
                    o[b, j, hh] = _attend(q[b, j, hh], cache["k"][li, b, hh, :n],
                                          cache["v"][li, b, hh, :n], scale)
        o = o.reshape(B, M, H * Dh)
        h = h + linear(o, lw["wo"])
        x = rms_norm(h, lw["ffn_norm"], spec.eps)
        if spec.ffn == "gelu":
            a = gelu_tanh(linear(x, lw["w1"]))
            h = h + linear(a, lw["w2"])
        else:
            a = silu(linear(x, lw["wg"])) * linear(x, lw["wu"])
            h = h + linear(a, lw["wd"])
    x = rms_norm(h, W["final_norm"], spec.eps)
    return linear(x, W["unembed"])


def forward_full(spec, W, tokens):
    """Full causal recompute over tokens [B][T]: logits for every position."""
    tokens = np.asarray(tokens)
    B, T = tokens.shape
    cache = new_cache(spec, B, T)
    return forward_cached(spec, W, cache, tokens, np.zeros(B, dtype=np.int64))


def n_params(spec):
    """Parameter count (matrices and gains)."""
    d, F, V, HD = spec.d_model, spec.d_ff, spec.vocab, spec.n_heads * spec.head_dim
    ffn = (2 if spec.ffn == "gelu" else 3) * d * F
    per_layer = 3 * d * HD + HD * d + ffn + 2 * d
    return spec.n_layers * per_layer + 2 * V * d + d
