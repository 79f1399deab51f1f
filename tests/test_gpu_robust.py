"""Robustness of the HIP path, through the C ABI:

* a draft step at a batch whose one-token forwards split K more ways than
  its two-token forward stays inside the workspace sps_workspace_bytes sized
  (a sentinel after the workspace is untouched);
* non-finite logits and probabilities (the library's definition: the row is
  one-hot at token 0, a sequence with such inputs gets a = 0 and token 0,
  and the device flag SPS_DEV_NONFINITE is raised) in sps_softmax,
  sps_accept_resample, the fused verify step and the draft step, bit-exact
  against the oracle's definition, with the other sequences of the batch
  unchanged;
* determinism: reruns give bit-identical logits and tokens; the same
  sequence through other launch configurations (single-tile GEMM against
  the split-K wide GEMM of a batch; 256-position attention partials
  against the 64-position partials of a prefill chunk) gives logits within
  the tolerance and identical tokens;
* resume at a loop boundary: 64 tokens in one run equal stopping at a loop
  boundary and resuming from prompt + tokens at the next loop index;
* the per-loop JSONL log of the SpS loop.
"""
import ctypes
import io
import json

import numpy as np
import pytest
import torch

from oracle import accept as oacc
from oracle import generate as ogen
from oracle import sampling as osamp
from paper_2302_01318_amd import configs, synth
from gpu_helpers import build_pair, install_prior, new_cache, round_up
from oracle_helpers import spec_of

pytestmark = pytest.mark.gpu

SMALL = configs.ModelShape("small", 192, 2, 3, 64, 320, 1000, "gelu", "bf16")


def cuda(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dt)


# ------------------------------------------------------------ workspace --

def test_draft_step_stays_inside_its_workspace(sps):
    """The 70B draft's width at B = 64: the first forward runs 128 rows, the
    later ones 64 rows, whose split-K partials are larger than those of the
    128-row launches. The workspace is the head of a larger buffer; the tail
    must keep its sentinel."""
    shape = configs.DRAFT_70B.with_(n_layers=1)
    B, K, T_cap, V = 64, 3, 64, configs.DRAFT_70B.vocab
    print("draft step workspace sentinel B", B, flush=True)
    gm = sps.Model(shape, synth.weights(shape, 40))
    kv = sps.KVCache(shape, B, T_cap)
    kv.buf.zero_()
    kv.lengths.fill_(8)
    need = sps.lib.sps_workspace_bytes(ctypes.byref(sps.config_of(shape)), B, 2, T_cap)
    assert need > 0
    buf = torch.empty(need + (32 << 20), dtype=torch.uint8, device="cuda")
    buf.fill_(0xA5)
    ws = buf[:need]
    ctx = cuda(synth.tokens(41, B, 2, V), torch.int32)
    tokens = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    p = torch.empty((B, K, V), dtype=torch.float32, device="cuda")
    sps.device_error()
    sps.draft_step(gm, kv, ctx, K, 1.0, (1, 0), tokens, p, ws)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    assert bool((buf[need:] == 0xA5).all()), "the draft step wrote past its workspace"
    assert bool(((tokens >= 0) & (tokens < V)).all())


@pytest.mark.parametrize("B,top_p", [(40, 1.0), (64, 1.0), (64, 0.9)])
def test_draft_draw_at_large_batch(sps, B, top_p):
    """The draft draw over 32000-token rows at B = 40 and 64, where a row is
    cut into 13 and 8 segments and the chosen segment is scanned in two
    rounds: every drawn token equals the oracle's integer inverse-CDF draw
    from the exported p row with the same Philox uniform, every exported row
    is a distribution, a rerun gives the same bits, and with nucleus 0.9 the
    first row of each sequence is the oracle's cut of the unmodified run's
    row, bit for bit."""
    from oracle import modifiers as omod
    from oracle import philox as ophil
    shape = configs.DRAFT_70B.with_(n_layers=1)
    K, T_cap, V = 3, 64, shape.vocab
    print("draft draw B", B, "top_p", top_p, flush=True)
    gm = sps.Model(shape, synth.weights(shape, 42))
    kv = sps.KVCache(shape, B, T_cap)
    ws = sps.workspace(shape, B, 2, T_cap)
    ctx = cuda(synth.tokens(43, B, 2, V), torch.int32)
    seed, loop = 44, 5

    def run(p_nuc):
        kv.buf.zero_()
        kv.lengths.fill_(8)
        tokens = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        p = torch.empty((B, K, V), dtype=torch.float32, device="cuda")
        sps.draft_step(gm, kv, ctx, K, 1.0, (seed, loop), tokens, p, ws, 0, p_nuc)
        torch.cuda.synchronize()
        assert sps.device_error() == 0
        return tokens.cpu().numpy(), p.cpu().numpy()

    got_t, got_p = run(top_p)
    np.testing.assert_array_equal(got_t[:, 0], ctx.cpu().numpy()[:, 1])
    # A rerun is bit-identical (the histograms' atomics add integers).
    again_t, again_p = run(top_p)
    np.testing.assert_array_equal(again_t, got_t)
    assert again_p.tobytes() == got_p.tobytes()
    ud = ophil.uniforms(seed, loop, ophil.PURPOSE_DRAFT, B, K)
    for b in range(B):
        for t in range(K):
            row = got_p[b, t]
            assert np.isfinite(row).all() and (row >= 0).all()
            assert abs(float(row.astype(np.float64).sum()) - 1.0) < 1e-4
            y, ok = osamp.categorical(osamp.to_weights(row), ud[b, t])
            assert ok and got_t[b, t + 1] == y, (b, t, y, got_t[b, t + 1])
    if top_p < 1.0:
        _, p_plain = run(1.0)
        np.testing.assert_array_equal(got_p[:, 0], omod.modify_rows(p_plain[:, 0], 0, top_p))


@pytest.mark.parametrize("B,K", [(40, 3), (64, 1)])
def test_verify_accept_at_large_batch(sps, B, K):
    """The verify step's fused accept / resample over 32000-token rows at
    B = 40 (K = 3) and B = 64 (K = 1), where the final draw's row is cut into
    13 and 8 segments and the chosen segment is scanned in two rounds: the
    tokens and counts equal the oracle's accept_resample on the GPU's own q
    rows, the drafts' p rows and the same uniforms, and a rerun gives the
    same outputs."""
    shape = configs.DRAFT_70B.with_(n_layers=1)
    V, T_cap = shape.vocab, 64
    print("verify accept B", B, "K", K, flush=True)
    gm = sps.Model(shape, synth.weights(shape, 45))
    kv = sps.KVCache(shape, B, T_cap)
    p, _, drafts = synth.accept_case(46, B, K, V, 2.0, 0.5)
    first = synth.tokens(47, B, 1, V)
    toks = cuda(np.concatenate([first, drafts], 1).astype(np.int32), torch.int32)
    ws = sps.workspace(shape, B, K + 1, T_cap)
    q = torch.empty((B, K + 1, V), dtype=torch.float32, device="cuda")

    def run():
        kv.buf.zero_()
        kv.lengths.fill_(8)
        out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        nacc = torch.empty(B, dtype=torch.int32, device="cuda")
        sps.verify_step(gm, kv, toks, K, 1.0, ws, q=q, p_draft=cuda(p, torch.float32), rng=(48, 2),
                        out_tokens=out, n_accepted=nacc)
        torch.cuda.synchronize()
        assert sps.device_error() == 0
        return out.cpu().numpy(), nacc.cpu().numpy()

    out, nacc = run()
    w_out, w_n, _ = oacc.accept_resample(p, q.cpu().numpy(), drafts, oacc.philox_uniforms(48, 2, B, K))
    np.testing.assert_array_equal(out, w_out)
    np.testing.assert_array_equal(nacc, w_n)
    out2, nacc2 = run()
    np.testing.assert_array_equal(out2, out)
    np.testing.assert_array_equal(nacc2, nacc)


def test_vocabulary_past_the_multi_cu_sampling(sps):
    """A 50257-token vocabulary, past the 32768 entries the multi-CU sampling
    paths take (rows this long go through the one-work-group kernels, whose
    statistics keep a running max and sum): the verify step's q rows equal
    the softmax of its logits, its fused accept / resample equals the
    oracle's on those rows, and the draft step's tokens are the oracle's
    integer inverse-CDF draws from its exported p rows."""
    from oracle import philox as ophil
    shape = configs.ModelShape("v50257", 128, 1, 2, 64, 256, 50257, "gelu", "bf16")
    V, T_cap, B = shape.vocab, 64, 2
    print("vocabulary", V, flush=True)
    gm = sps.Model(shape, synth.weights(shape, 49))
    kv = sps.KVCache(shape, B, T_cap)
    kv.buf.zero_()
    kv.lengths.fill_(8)
    # verify step, K = 4
    K = 4
    p, _, drafts = synth.accept_case(50, B, K, V, 2.0, 0.5)
    toks = cuda(np.concatenate([synth.tokens(51, B, 1, V), drafts], 1).astype(np.int32), torch.int32)
    ws = sps.workspace(shape, B, K + 1, T_cap)
    logits = torch.empty((B, K + 1, V), dtype=torch.float32, device="cuda")
    q = torch.empty_like(logits)
    out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    nacc = torch.empty(B, dtype=torch.int32, device="cuda")
    sps.verify_step(gm, kv, toks, K, 1.0, ws, logits=logits, q=q, p_draft=cuda(p, torch.float32), rng=(52, 1),
                    out_tokens=out, n_accepted=nacc)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    qg = q.cpu().numpy()
    np.testing.assert_allclose(qg, osamp.softmax(logits.cpu().numpy().astype(np.float64), 1.0), rtol=2e-5, atol=1e-9)
    w_out, w_n, _ = oacc.accept_resample(p, qg, drafts, oacc.philox_uniforms(52, 1, B, K))
    np.testing.assert_array_equal(out.cpu().numpy(), w_out)
    np.testing.assert_array_equal(nacc.cpu().numpy(), w_n)
    # draft step, K = 3
    Kd = 3
    kv.lengths.fill_(8)
    ctx = cuda(synth.tokens(53, B, 2, V), torch.int32)
    wsd = sps.workspace(shape, B, 2, T_cap)
    tokens = torch.empty((B, Kd + 1), dtype=torch.int32, device="cuda")
    pd = torch.empty((B, Kd, V), dtype=torch.float32, device="cuda")
    sps.draft_step(gm, kv, ctx, Kd, 1.0, (54, 2), tokens, pd, wsd)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    got_t, got_p = tokens.cpu().numpy(), pd.cpu().numpy()
    ud = ophil.uniforms(54, 2, ophil.PURPOSE_DRAFT, B, Kd)
    for b in range(B):
        for t in range(Kd):
            row = got_p[b, t]
            assert abs(float(row.astype(np.float64).sum()) - 1.0) < 1e-4
            y, ok = osamp.categorical(osamp.to_weights(row), ud[b, t])
            assert ok and got_t[b, t + 1] == y, (b, t)


# ----------------------------------------------------------- non-finite --

def test_softmax_nonfinite_rows(sps):
    g = np.random.default_rng(8)
    V = 1000
    z = g.normal(0, 2, size=(7, V)).astype(np.float32)
    z[1, 17] = np.nan
    z[2, 3] = np.inf
    z[3, 9] = -np.inf                   # valid: probability 0
    z[4, 500] = 3e38                    # overflows only when divided by T = 0.5
    z[5, :] = np.nan
    for T, k, pp in ((1.0, 0, 1.0), (0.5, 0, 1.0), (0.0, 0, 1.0), (1.0, 50, 0.9)):
        print("softmax non-finite T", T, k, pp, flush=True)
        sps.device_error()
        got = sps.softmax(cuda(z, torch.float32), T, k, pp).cpu().numpy()
        flags = sps.device_error()
        bad = osamp.nonfinite_rows(z, T)
        assert bool(flags & sps.DEV_NONFINITE) == bool(bad.any())
        for r in range(7):
            if bad[r]:
                assert got[r, 0] == 1.0 and not got[r, 1:].any(), r
            else:
                assert np.isfinite(got[r]).all()
                assert abs(got[r].sum(dtype=np.float64) - 1.0) < 1e-5
        assert got[3, 9] == 0.0
        if k == 0 and pp == 1.0:
            want = osamp.softmax(z.astype(np.float64), T)
            ok = ~bad
            if T == 0.0:
                np.testing.assert_array_equal(got[ok], want[ok].astype(np.float32))
            else:
                np.testing.assert_allclose(got[ok], want[ok], rtol=2e-5, atol=1e-10)


def test_accept_nonfinite_inputs_bit_exact(sps):
    """Sequences with a NaN / Inf among the values the accept tests or the
    final draw read get a = 0 and token 0; the others are untouched; all
    bit-exact against the oracle's definition."""
    B, K, V = 8, 4, 1000
    p, q, drafts = synth.accept_case(60, B, K, V, 2.0, 0.5)
    unif = np.random.default_rng(61).random((B, K + 1)).astype(np.float32)
    q[1, 3, drafts[1, 3]] = np.nan          # a late gathered q value
    p[2, 0, drafts[2, 0]] = np.inf          # a gathered p value
    q[3, :, 11] = np.nan                    # every q row (the draw reads one of them)
    p[4, :, 12] = -np.inf                   # every p row (a residual draw reads one)
    q[5, K, 0] = np.nan                     # the bonus row only
    drafts[6, 1] = V + 3                    # a bad token, not non-finite
    sps.device_error()
    out, nacc = sps.accept_resample(cuda(p, torch.float32), cuda(q, torch.float32), cuda(drafts, torch.int32),
                                    cuda(unif, torch.float32))
    flags = sps.device_error()
    w_out, w_n, w_f = oacc.accept_resample(p, q, drafts, unif)
    np.testing.assert_array_equal(out.cpu().numpy(), w_out)
    np.testing.assert_array_equal(nacc.cpu().numpy(), w_n)
    assert flags & sps.DEV_NONFINITE and (w_f & oacc.FLAG_NONFINITE).any()
    assert flags & sps.DEV_BAD_TOKEN
    for b in (1, 2, 3):
        assert list(w_out[b]) == [0] + [-1] * K and w_n[b] == 0
    clean = [b for b in range(B) if not w_f[b] & oacc.FLAG_NONFINITE]
    assert 0 in clean and 7 in clean


def _verify(sps, gm, kv, toks, K, T, ws, p, rng, top_k=0, top_p=1.0):
    B, V = toks.shape[0], gm.shape.vocab
    logits = torch.empty((B, K + 1, V), dtype=torch.float32, device="cuda")
    q = torch.empty_like(logits)
    out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    nacc = torch.empty(B, dtype=torch.int32, device="cuda")
    sps.verify_step(gm, kv, toks, K, T, ws, logits=logits, q=q, p_draft=p, rng=rng, out_tokens=out,
                    n_accepted=nacc, top_k=top_k, top_p=top_p)
    torch.cuda.synchronize()
    return logits.cpu().numpy(), q.cpu().numpy(), out.cpu().numpy(), nacc.cpu().numpy()


@pytest.mark.parametrize("top_k,top_p", [(0, 1.0), (20, 0.9)])
def test_verify_step_nonfinite_logits(sps, top_k, top_p):
    """A NaN embedding row makes the logits of one sequence NaN (attention is
    per sequence; later positions see the NaN key and value, earlier ones
    take 0 x NaN from the masked position in the score product): its
    exported q rows are one-hot at token 0, its outcome is a = 0 and token
    0, the flag is raised, and the other sequences are bit-identical to a
    clean run; with a top-k / nucleus cut too (the cut over several CUs
    leaves such a row uncut)."""
    shape = configs.TINY_TARGET
    B, K, V = 3, 4, shape.vocab
    w = synth.weights(shape, 70)
    toks = synth.tokens(71, B, K + 1, V)
    toks[1, 2] = 11
    toks[[0, 2]] = np.where(toks[[0, 2]] == 11, 12, toks[[0, 2]])
    p, _, _ = synth.accept_case(72, B, K, V, 2.0, 0.5)
    runs = []
    for poison in (False, True):
        ww = dict(w)
        if poison:
            e = w[("embed", -1)].clone()
            e[11] = float("nan")
            ww[("embed", -1)] = e
        gm = sps.Model(shape, ww)
        kv = sps.KVCache(shape, B, 64)
        kv.buf.zero_()
        kv.lengths.copy_(torch.tensor([5, 9, 2], dtype=torch.int32))
        ws = sps.workspace(shape, B, K + 1, 64)
        sps.device_error()
        runs.append(_verify(sps, gm, kv, cuda(toks, torch.int32), K, 1.0, ws, cuda(p, torch.float32), (3, 1),
                            top_k, top_p) + (sps.device_error(),))
    (l0, q0, o0, n0, f0), (l1, q1, o1, n1, f1) = runs
    assert f0 == 0 and f1 & sps.DEV_NONFINITE
    for b in (0, 2):
        np.testing.assert_array_equal(l1[b], l0[b])
        np.testing.assert_array_equal(q1[b], q0[b])
        np.testing.assert_array_equal(o1[b], o0[b])
        assert n1[b] == n0[b]
    assert list(o1[1]) == [0] + [-1] * K and n1[1] == 0
    for j in range(K + 1):
        assert np.isnan(l1[1, j]).any()
        assert q1[1, j, 0] == 1.0 and not q1[1, j, 1:].any()


@pytest.mark.parametrize("top_k,top_p", [(0, 1.0), (20, 0.9)])
def test_draft_step_nonfinite_logits(sps, top_k, top_p):
    """A draft whose logits are NaN for one sequence: its p rows are one-hot
    at token 0 (a valid draft distribution), its drafts are token 0, the
    flag is raised; the other sequence is bit-identical to a clean run (with
    or without a top-k / nucleus cut)."""
    shape = configs.TINY_DRAFT
    B, K, V = 2, 3, shape.vocab
    w = synth.weights(shape, 80)
    ctx = np.array([[5, 6], [11, 7]], np.int32)
    runs = []
    for poison in (False, True):
        ww = dict(w)
        if poison:
            e = w[("embed", -1)].clone()
            e[11] = float("nan")
            ww[("embed", -1)] = e
        gm = sps.Model(shape, ww)
        kv = sps.KVCache(shape, B, 64)
        kv.buf.zero_()
        kv.lengths.fill_(6)
        ws = sps.workspace(shape, B, 2, 64)
        tokens = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        p = torch.empty((B, K, V), dtype=torch.float32, device="cuda")
        sps.device_error()
        sps.draft_step(gm, kv, cuda(ctx, torch.int32), K, 1.0, (4, 2), tokens, p, ws, top_k, top_p)
        torch.cuda.synchronize()
        runs.append((tokens.cpu().numpy(), p.cpu().numpy(), sps.device_error()))
    (t0, p0, f0), (t1, p1, f1) = runs
    assert 11 not in t0[0], "the clean sequence drafts the poisoned token: pick another seed"
    assert f0 == 0 and f1 & sps.DEV_NONFINITE
    np.testing.assert_array_equal(t1[0], t0[0])
    np.testing.assert_array_equal(p1[0], p0[0])
    assert list(t1[1]) == [7, 0, 0, 0]
    assert (p1[1, :, 0] == 1.0).all() and not p1[1, :, 1:].any()


# ---------------------------------------------------------- determinism --

def _prior_case(sps, shape, B, K, n_prior, seed):
    gm, W = build_pair(shape, seed)
    T_cap = round_up(max(n_prior) + K + 1 + 32, 32)
    kv = sps.KVCache(shape, B, T_cap)
    ocache = new_cache(shape, B, T_cap)
    install_prior(shape, kv, ocache, seed + 1, n_prior)
    return gm, W, kv, ocache, T_cap


@pytest.mark.parametrize("shape", [SMALL, SMALL.with_(dtype="f32")], ids=["bf16", "f32"])
def test_verify_reruns_are_bit_identical(sps, shape):
    """Ten reruns of a batched verify step (B = 16, K = 8: the wide GEMM with
    split-K and its reduction kernel for bf16) give bit-identical logits,
    probabilities and tokens: every reduction runs in a fixed order."""
    B, K = 16, 8
    g = np.random.default_rng(90)
    gm, _, kv, _, T_cap = _prior_case(sps, shape, B, K, [int(x) for x in g.integers(10, 300, B)], 91)
    p, _, drafts = synth.accept_case(92, B, K, shape.vocab, 2.0, 0.5)
    toks = cuda(np.concatenate([synth.tokens(93, B, 1, shape.vocab), drafts], 1), torch.int32)
    ws = sps.workspace(shape, B, K + 1, T_cap)
    first = _verify(sps, gm, kv, toks, K, 1.0, ws, cuda(p, torch.float32), (5, 0))
    for _ in range(9):
        again = _verify(sps, gm, kv, toks, K, 1.0, ws, cuda(p, torch.float32), (5, 0))
        for a, b in zip(first, again):
            np.testing.assert_array_equal(a, b)
    assert sps.device_error() == 0


def test_launch_configurations_agree(sps):
    """One sequence (bf16, K = 4, 300 prior positions plus 16 scored by a
    forward) through three launch configurations:
      A. a B = 1 verify step: single-tile GEMMs, 256-position attention
         partials;
      B. sequence 0 of a B = 6 verify step: the wide GEMM with split-K;
      C. the last K + 1 rows of a 21-token forward chunk of the same batch:
         the wide GEMM at 126 rows and the prefill attention's 64-position
         partials.
    Logits agree within the bf16 tolerance and the accept / resample tokens
    (same uniforms, b = 0) are identical."""
    shape = SMALL.with_(ffn="swiglu")
    K, V, n_prior, extra = 4, SMALL.vocab, 300, 16
    gm, _ = build_pair(shape, 95)
    NB = 6
    p, _, drafts = synth.accept_case(96, NB, K, V, 2.0, 0.5)
    head = synth.tokens(97, NB, extra + 1, V)
    T_cap = round_up(n_prior + extra + K + 1 + 32, 32)
    kvb = sps.KVCache(shape, NB, T_cap)
    install_prior(shape, kvb, new_cache(shape, NB, T_cap), 98, [n_prior] * NB)
    # C: forward over extra + K + 1 tokens (writes the extra tokens' KV)
    chunk = np.concatenate([head, drafts], 1).astype(np.int32)          # [NB][extra + 1 + K]
    M = extra + 1 + K
    wsb = sps.workspace(shape, NB, M, T_cap)
    logits_c = torch.empty((NB, M, V), dtype=torch.float32, device="cuda")
    sps.forward(gm, kvb, cuda(chunk, torch.int32), M, 0, logits_c, wsb)
    torch.cuda.synchronize()
    lc = logits_c.cpu().numpy()[:, extra:]
    # B: verify of (x_n, drafts) at lengths n_prior + extra
    kvb.lengths.fill_(n_prior + extra)
    vt = cuda(chunk[:, extra:], torch.int32)
    lb, qb, ob, nb = _verify(sps, gm, kvb, vt, K, 1.0, wsb, cuda(p, torch.float32), (6, 2))
    # A: sequence 0 alone, its cache copied from the batch
    kv1 = sps.KVCache(shape, 1, T_cap)
    for l in range(shape.n_layers):
        k, v = kvb.read(l, 0, 0, n_prior + extra)
        kv1.write(l, 0, 0, k, v)
    kv1.lengths.fill_(n_prior + extra)
    ws1 = sps.workspace(shape, 1, K + 1, T_cap)
    la, qa, oa, na = _verify(sps, gm, kv1, vt[:1].contiguous(), K, 1.0, ws1, cuda(p[:1], torch.float32), (6, 2))
    assert sps.device_error() == 0
    for other, what in ((lb[0], "B"), (lc[0], "C")):
        err = np.abs(other - la[0]).max()
        print("  launch configuration %s: max |logits - A| = %.3g" % (what, err), flush=True)
        assert err <= 2e-2 and err <= 2e-3
    # tokens: A's fused accept, B's fused accept at b = 0, and C's logits
    # through the standalone softmax + accept with the same uniforms
    unif = oacc.philox_uniforms(6, 2, 1, K)
    qc = sps.softmax(cuda(lc[:1], torch.float32), 1.0)
    oc, nc = sps.accept_resample(cuda(p[:1], torch.float32), qc, cuda(drafts[:1], torch.int32),
                                 cuda(unif, torch.float32))
    np.testing.assert_array_equal(oa[0], ob[0])
    np.testing.assert_array_equal(oa[0], oc.cpu().numpy()[0])
    assert na[0] == nb[0] == int(nc.cpu()[0])


# --------------------------------------------------------------- resume --

def test_resume_at_a_loop_boundary_equals_one_run(sps):
    """Tiny fp32 pair, K = 4: 64 tokens in one run equal running loops until
    at least 32 tokens exist, then prefilling prompt + those tokens into a
    fresh generator and continuing at the next loop index."""
    tgt, drf = configs.TINY_TARGET, configs.TINY_DRAFT
    gt, Wt = build_pair(tgt, 100)
    gd, Wd = build_pair(drf, 101)
    prompt = torch.from_numpy(synth.tokens(110, 1, 32, tgt.vocab)).cuda()
    K, T, seed = 4, 1.0, 13
    full = sps.Generator(gt, gd, 1, 192, K).generate(prompt, 64, T, seed).cpu().numpy()[0]
    gen = sps.Generator(gt, gd, 1, 192, K)
    gen.prefill(prompt)
    seq = torch.zeros((1, 64), dtype=torch.int32, device="cuda")
    n_out = torch.zeros(1, dtype=torch.int32, device="cuda")
    loops = 0
    while int(n_out.item()) < 32:
        gen.loop(T, seed, loops, seq, n_out, 64)
        loops += 1
    n1 = int(n_out.item())
    first = seq[:, :n1]
    gen2 = sps.Generator(gt, gd, 1, 192, K)
    rest = gen2.generate(torch.cat([prompt, first], 1), 64 - n1, T, seed, loop0=loops).cpu().numpy()[0]
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    got = np.concatenate([first.cpu().numpy()[0], rest])
    np.testing.assert_array_equal(got, full)
    # and both equal the oracle's one run
    want, _ = ogen.sps_generate_one(spec_of(tgt), Wt, spec_of(drf), Wd, prompt.cpu().numpy()[0], 64, K, T, seed)
    assert list(full) == want


def test_per_loop_jsonl_log(sps):
    """The SpS loop's JSONL log: one record per loop with its loop time and
    the accepted / emitted tokens per sequence, and a run summary."""
    tgt, drf = configs.TINY_TARGET, configs.TINY_DRAFT
    gt, _ = build_pair(tgt, 100)
    gd, _ = build_pair(drf, 101)
    prompt = torch.from_numpy(synth.tokens(111, 2, 16, tgt.vocab)).cuda()
    gen = sps.Generator(gt, gd, 2, 160, 4)
    log, acc_log = io.StringIO(), []
    toks = gen.generate(prompt, 40, 1.0, 3, accepted_log=acc_log, log=log)
    torch.cuda.synchronize()
    lines = [json.loads(x) for x in log.getvalue().splitlines()]
    loops, summary = lines[:-1], lines[-1]["run"]
    assert len(loops) == len(acc_log) == gen.loops == summary["loops"]
    emitted = np.zeros(2, int)
    for rec, (a, done) in zip(loops, acc_log):
        assert rec["ms"] > 0
        for b in range(2):
            if bool(done[b]):
                assert rec["accepted"][b] == -1 and rec["emitted"][b] == 0
            else:
                assert rec["accepted"][b] == int(a[b])
                assert 1 <= rec["emitted"][b] <= int(a[b]) + 1
        emitted += rec["emitted"]
    assert list(emitted) == [40, 40] and summary["tokens"] == 80 and toks.shape == (2, 40)
    assert summary["tokens_per_s"] > 0 and 0 <= summary["mean_accepted"] <= 4
