"""Test helpers: turn synthetic inputs into the oracle's inputs."""
import numpy as np
import torch

from oracle.model import ModelSpec


def spec_of(shape, **kw):
    """oracle ModelSpec with the dimensions of a configs.ModelShape."""
    s = dict(d_model=shape.d_model, n_layers=shape.n_layers, n_heads=shape.n_heads,
             head_dim=shape.head_dim, d_ff=shape.d_ff, vocab=shape.vocab, ffn=shape.ffn,
             dtype="bf16" if shape.dtype == "fp8" else shape.dtype, eps=shape.eps,
             rope_base=shape.rope_base)
    s.update(kw)
    return ModelSpec(**s)


def oracle_weights(shape, wdict):
    """{(name, layer): torch tensor} -> the oracle's nested dict of fp32 arrays
    (for an FP8 model: the projections quantised and dequantised by the
    oracle's own FP8 quantiser)."""
    f = lambda t: t.float().numpy()
    W = {"embed": f(wdict[("embed", -1)]), "final_norm": f(wdict[("final_norm", -1)]),
         "unembed": f(wdict[("unembed", -1)]), "layers": []}
    for l in range(shape.n_layers):
        lw = {"attn_norm": f(wdict[("attn_norm", l)]), "wq": f(wdict[("wq", l)]),
              "wk": f(wdict[("wk", l)]), "wv": f(wdict[("wv", l)]), "wo": f(wdict[("wo", l)]),
              "ffn_norm": f(wdict[("ffn_norm", l)])}
        if shape.ffn == "gelu":
            lw["w1"] = f(wdict[("w1", l)])
            lw["w2"] = f(wdict[("w2", l)])
        else:
            lw["wg"] = f(wdict[("w1", l)])
            lw["wu"] = f(wdict[("w3", l)])
            lw["wd"] = f(wdict[("w2", l)])
        W["layers"].append(lw)
    if shape.dtype == "fp8":
        from oracle import fp8
        W = fp8.fp8_weights(W)
    return W
