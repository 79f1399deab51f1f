"""Helpers for GPU parity tests: build the same synthetic model / KV for the
HIP library and for the oracle."""
import numpy as np
import torch

from oracle import model as om
from paper_2302_01318_amd import synth
from oracle_helpers import oracle_weights, spec_of


def round_up(x, m):
    return (x + m - 1) // m * m


def build_pair(shape, seed, std=0.02, gain_std=0.1):
    from paper_2302_01318_amd import sps
    w = synth.weights(shape, seed, std, gain_std)
    gm = sps.Model(shape, w)
    W = oracle_weights(shape, w)
    del w
    return gm, W


def install_prior(shape, kv, ocache, seed, n_prior):
    """Random prior keys/values (N(0,1), model dtype) of length n_prior[b]."""
    B = len(n_prior)
    T = max(n_prior)
    for l in range(shape.n_layers):
        k, v = synth.kv_prior(shape, seed, l, B, T)
        for b in range(B):
            n = int(n_prior[b])
            if n == 0:
                continue
            kv.write(l, b, 0, k[b, :, :n].contiguous().cuda(), v[b, :, :n].contiguous().cuda())
            ocache["k"][l, b, :, :n] = k[b, :, :n].double().numpy()
            ocache["v"][l, b, :, :n] = v[b, :, :n].double().numpy()
    kv.lengths.copy_(torch.tensor(list(n_prior), dtype=torch.int32))
    torch.cuda.synchronize()


def new_cache(shape, B, T_cap):
    return om.new_cache(spec_of(shape), B, T_cap)


def install_oracle_prior(shape, ocache, seed, n_prior):
    """The oracle half of install_prior (the same random prior keys/values)."""
    B = len(n_prior)
    T = max(n_prior)
    for l in range(shape.n_layers):
        k, v = synth.kv_prior(shape, seed, l, B, T)
        for b in range(B):
            n = int(n_prior[b])
            ocache["k"][l, b, :, :n] = k[b, :, :n].double().numpy()
            ocache["v"][l, b, :, :n] = v[b, :, :n].double().numpy()
