"""Seeded synthetic inputs.

This module only draws random numbers in the shapes and distributions of the
workloads; it holds none of the method's arithmetic. Both the GPU path and
the CPU oracle consume its outputs, so neither depends on the other.

Recipes:
  weights      N(0, std^2) per entry (std 0.02), stored in the model dtype
               (bf16 by round-to-nearest-even through torch; bf16 also for
               FP8 models, whose packer quantises them); RMSNorm gains
               1 + N(0, gain_std^2) in fp32. One numpy Generator per tensor,
               seeded by (seed, tensor id), so any single tensor can be
               regenerated on its own.
  tokens       uniform integers in [0, V).
  kv_prior     N(0, 1) keys and values in the model dtype (a synthetic prior
               context of the given length).
  accept_case  target logits z_q ~ N(0, sigma^2) per entry, draft logits
               z_p = z_q + N(0, sigma_pert^2); p and q are the normalised
               exponentials of those logits, rounded to fp32; draft token t
               is drawn from p_t with numpy's generic categorical sampler.
  coupled pair a target and a draft of different widths whose logits are
               the accept_case recipe realised in weights: both share token
               codes z_x ~ N(0, I_r) and output codes o_y ~ N(0, s^2 I_r)
               (rank r, one generator seeded by the pair seed); a model may
               perturb its copy, o'_y = o_y + code_pert n_y with
               n_y ~ N(0, I_r) from its own seed. Each model has its own
               orthonormal basis Q [d][r] (QR of an N(0, 1) matrix), embeds
               E[x] = sqrt(d) Q z_x and unembeds with W_U[y] = Q o'_y / sqrt(d);
               norm gains are 1. Through the skip path alone the final
               RMSNorm of E[x] is sqrt(d) Q z_x / |z_x|, so the logits are
               o'_y . z_x / |z_x|: N(0, s^2) per entry for the target and the
               same plus N(0, code_pert^2) for the draft. Attention and FFN
               weights are N(0, layer_std^2); at small layer_std they cost
               their full time but move the logits little.
"""
import numpy as np
import torch

W_NAMES = ("embed", "final_norm", "unembed", "attn_norm", "wq", "wk", "wv", "wo",
           "ffn_norm", "w1", "w3", "w2")


def _rng(seed, *ids):
    return np.random.default_rng([int(seed)] + [int(i) for i in ids])


def tensor_shapes(cfg):
    """Canonical shapes of every weight tensor: {(name, layer): shape}."""
    d, HD, F, V = cfg.d_model, cfg.n_heads * cfg.head_dim, cfg.d_ff, cfg.vocab
    out = {("embed", -1): (V, d), ("final_norm", -1): (d,), ("unembed", -1): (V, d)}
    for l in range(cfg.n_layers):
        out[("attn_norm", l)] = (d,)
        out[("wq", l)] = (HD, d)
        out[("wk", l)] = (HD, d)
        out[("wv", l)] = (HD, d)
        out[("wo", l)] = (d, HD)
        out[("ffn_norm", l)] = (d,)
        out[("w1", l)] = (F, d)
        if cfg.ffn == "swiglu":
            out[("w3", l)] = (F, d)
        out[("w2", l)] = (d, F)
    return out


def weight(cfg, name, layer, seed, std=0.02, gain_std=0.1):
    """One canonical weight tensor as a CPU torch tensor."""
    shape = tensor_shapes(cfg)[(name, layer)]
    g = _rng(seed, W_NAMES.index(name), layer + 1)
    if name.endswith("norm"):
        return torch.from_numpy(1.0 + gain_std * g.standard_normal(shape, dtype=np.float32))
    a = torch.from_numpy(g.standard_normal(shape, dtype=np.float32) * np.float32(std))
    return a.to(torch.bfloat16) if cfg.dtype in ("bf16", "fp8") else a


def weights(cfg, seed, std=0.02, gain_std=0.1):
    """Every weight tensor: {(name, layer): CPU torch tensor}."""
    return {key: weight(cfg, key[0], key[1], seed, std, gain_std) for key in tensor_shapes(cfg)}


def tokens(seed, B, n, V):
    return _rng(seed, 1).integers(0, V, size=(B, n), dtype=np.int64).astype(np.int32)


def kv_prior(cfg, seed, layer, B, T):
    """Keys and values [B][H][T][Dh] ~ N(0, 1) in the model dtype (CPU)."""
    g = _rng(seed, 2, layer)
    shape = (B, cfg.n_heads, T, cfg.head_dim)
    k = torch.from_numpy(g.standard_normal(shape, dtype=np.float32))
    v = torch.from_numpy(g.standard_normal(shape, dtype=np.float32))
    if cfg.dtype in ("bf16", "fp8"):
        k, v = k.to(torch.bfloat16), v.to(torch.bfloat16)
    return k, v


def _normalised_exp(z):
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def accept_case(seed, B, K, V, sigma=2.0, sigma_pert=0.5):
    """Draft/target distribution pairs for the accept/resample stage.

    Returns p [B][K][V] fp32, q [B][K+1][V] fp32, drafts [B][K] int32.
    """
    g = _rng(seed, 3, B, K, V)
    zq = g.normal(0.0, sigma, size=(B, K + 1, V))
    zp = zq[:, :K] + g.normal(0.0, sigma_pert, size=(B, K, V))
    q64 = _normalised_exp(zq)
    p64 = _normalised_exp(zp)
    drafts = np.zeros((B, K), dtype=np.int32)
    for b in range(B):
        for t in range(K):
            drafts[b, t] = g.choice(V, p=p64[b, t])
    return p64.astype(np.float32), q64.astype(np.float32), drafts


def accept_case_device(seed, B, K, V, sigma=2.0, sigma_pert=0.5, device="cuda"):
    """Large accept/resample inputs drawn on the device with torch's own
    generator (for timing; the oracle-checked cases use accept_case)."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    zq = torch.randn((B, K + 1, V), generator=gen, device=device) * sigma
    zp = zq[:, :K] + torch.randn((B, K, V), generator=gen, device=device) * sigma_pert
    q = torch.softmax(zq.double(), dim=-1).float()
    p = torch.softmax(zp.double(), dim=-1).float()
    drafts = torch.multinomial(p.reshape(B * K, V), 1, generator=gen).reshape(B, K).int() if K else \
        torch.zeros((B, 0), dtype=torch.int32, device=device)
    return p.contiguous(), q.contiguous(), drafts.contiguous()


def device_weights(cfg, seed, std=0.02, gain_std=0.1, device="cuda"):
    """Yield ((name, layer), tensor) for every weight, drawn on the device with
    torch's generator (same distributions as `weights`; for models too large
    to draw on the host, e.g. the 70B shape). One tensor is alive at a time."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    dt = torch.bfloat16 if cfg.dtype in ("bf16", "fp8") else torch.float32
    for key, shape in tensor_shapes(cfg).items():
        if key[0].endswith("norm"):
            t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32).mul_(gain_std).add_(1.0)
        else:
            t = torch.randn(shape, generator=gen, device=device, dtype=dt).mul_(std)
        yield key, t
        del t


def coupled_device_weights(cfg, pair_seed, model_seed, layer_std, code_pert=0.0, logit_std=2.0, rank=64,
                           device="cuda"):
    """Yield ((name, layer), tensor) for one model of a coupled pair (module
    doc): embedding and unembedding from the shared codes in this model's
    basis (output codes perturbed by code_pert), unit gains, N(0, layer_std^2)
    layer weights."""
    d, V = cfg.d_model, cfg.vocab
    dt = torch.bfloat16 if cfg.dtype in ("bf16", "fp8") else torch.float32
    pair = torch.Generator(device=device)
    pair.manual_seed(int(pair_seed))
    z = torch.randn((V, rank), generator=pair, device=device)
    o = torch.randn((V, rank), generator=pair, device=device) * logit_std
    q, _ = np.linalg.qr(_rng(model_seed, 4, d).standard_normal((d, rank)))
    Q = torch.from_numpy(q.astype(np.float32)).to(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(model_seed))
    if code_pert:
        o = o + torch.randn((V, rank), generator=gen, device=device) * code_pert
    for key, shape in tensor_shapes(cfg).items():
        if key[0] == "embed":
            t = (z @ Q.t()).mul_(float(np.sqrt(d))).to(dt)
        elif key[0] == "unembed":
            t = (o @ Q.t()).mul_(float(1.0 / np.sqrt(d))).to(dt)
        elif key[0].endswith("norm"):
            t = torch.ones(shape, device=device, dtype=torch.float32)
        else:
            t = torch.randn(shape, generator=gen, device=device, dtype=dt).mul_(layer_std)
        yield key, t
        del t
