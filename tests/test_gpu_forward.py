"""GPU parity of the verify step (Conditional Scoring + Modified Rejection
Sampling) against the oracle.

Logits must agree within 1e-4 (fp32 models) or 2e-2 (bf16 models) max-abs;
the exported q must be the softmax of the GPU logits; the fused accept /
resample outputs must equal the oracle's accept_resample run on the GPU's own
q (the decision is taken in the kernel's fp32 precision on both sides) bit
for bit; the appended keys / values must match the oracle's cache.
Shapes span several MFMA tiles, ragged vocabularies and ragged per-sequence
cache lengths; the full-width 7B- and 70B-shaped layers run in exactly the
launch configuration of the benchmarked step (the per-layer kernels do not
depend on the number of layers).
"""
import numpy as np
import pytest
import torch

from oracle import accept as oacc
from oracle import model as om
from oracle import sampling as osamp
from paper_2302_01318_amd import configs, synth
from gpu_helpers import build_pair, install_oracle_prior, install_prior, new_cache, round_up
from oracle_helpers import spec_of

pytestmark = pytest.mark.gpu


# Second, tighter bound on the measured logit error, relative to the logit
# scale (the benchmark spec's tolerance stays the pass criterion; this one catches
# regressions well below it). Measured: bf16 blocks 5e-5 to 4e-4 at logit
# std ~0.27; full-width 70B blocks (logit std 1.82) 9.5e-4 at ctx 2048,
# 4.1e-3 at ctx 8192, 3.6e-3 to 5.0e-3 batched; FP8 70B blocks 1.8e-3 to
# 8.4e-3 (B = 16, K = 8); fp32 4e-7 to 7e-7.
TIGHT = {"bf16": 5e-3, "fp8": 8e-3, "f32": 2e-5}


def tight_bound(dtype, logit_std):
    return TIGHT[dtype] * max(1.0, float(logit_std))


def verify_parity(sps, shape, B, K, n_prior, seed, tol, T=1.0, check_kv=True, built=None, want_out=None):
    print("verify parity", shape.name, shape.dtype, shape.ffn, "B", B, "K", K, "prior", n_prior, flush=True)
    V = shape.vocab
    gm, W = built if built is not None else build_pair(shape, seed)
    T_cap = round_up(max(n_prior) + K + 1, 32)
    kv = sps.KVCache(shape, B, T_cap)
    ocache = new_cache(shape, B, T_cap)
    install_prior(shape, kv, ocache, seed + 1, n_prior)
    p, _, drafts = synth.accept_case(seed + 2, B, K, V, 2.0, 0.5)
    first = synth.tokens(seed + 3, B, 1, V)
    toks = np.concatenate([first, drafts], axis=1).astype(np.int32)
    ws = sps.workspace(shape, B, K + 1, T_cap)
    logits = torch.empty((B, K + 1, V), dtype=torch.float32, device="cuda")
    q = torch.empty_like(logits)
    out = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    nacc = torch.empty(B, dtype=torch.int32, device="cuda")
    sps.verify_step(gm, kv, torch.from_numpy(toks).cuda(), K, T, ws, logits=logits, q=q,
                    p_draft=torch.from_numpy(p).cuda() if K else None, rng=(seed, 3), out_tokens=out,
                    n_accepted=nacc)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    if want_out is not None:       # the oracle's inputs, for negative controls
        want_out.update(toks=toks, n_prior=np.array(n_prior), T_cap=T_cap, seed=seed)
    want = om.forward_cached(spec_of(shape), W, ocache, toks, np.array(n_prior))
    got = logits.cpu().numpy()
    err = np.abs(got - want).max()
    tight = tight_bound(shape.dtype, want.std())
    print("  max |logits - oracle| = %.3g (tol %.1g, tight %.1g), logit std %.3g" % (err, tol, tight, want.std()),
          flush=True)
    assert err <= tol
    assert err <= tight
    qg = q.cpu().numpy()
    np.testing.assert_allclose(qg, osamp.softmax(got.astype(np.float64), T), rtol=2e-5, atol=1e-9)
    w_out, w_n, _ = oacc.accept_resample(p if K else np.zeros((B, 0, V), np.float32), qg, drafts,
                                         oacc.philox_uniforms(seed, 3, B, K))
    np.testing.assert_array_equal(out.cpu().numpy(), w_out)
    np.testing.assert_array_equal(nacc.cpu().numpy(), w_n)
    if check_kv:
        kt = tol if shape.dtype in ("bf16", "fp8") else 1e-4
        for l in range(shape.n_layers):
            for b in range(B):
                k, v = kv.read(l, b, n_prior[b], K + 1)
                np.testing.assert_allclose(k.float().cpu().numpy(),
                                           ocache["k"][l, b, :, n_prior[b]:n_prior[b] + K + 1], atol=kt, rtol=kt)
                np.testing.assert_allclose(v.float().cpu().numpy(),
                                           ocache["v"][l, b, :, n_prior[b]:n_prior[b] + K + 1], atol=kt, rtol=kt)
    return got


SMALL = configs.ModelShape("small", 192, 2, 3, 64, 320, 1000, "gelu", "bf16")


def test_tiny_fp32_verify(sps):
    verify_parity(sps, configs.TINY_TARGET, 1, 4, [32], 1, 1e-4)


def test_tiny_fp32_ragged_batch(sps):
    verify_parity(sps, configs.TINY_TARGET, 3, 4, [7, 40, 33], 2, 1e-4)


@pytest.mark.parametrize("ffn", ["gelu", "swiglu"])
def test_small_bf16_ragged(sps, ffn):
    verify_parity(sps, SMALL.with_(ffn=ffn), 3, 3, [5, 100, 257], 3, 2e-2)


def test_small_bf16_many_rows(sps):
    # 4 sequences x 9 positions = 36 rows: three 16-row MFMA tiles
    verify_parity(sps, SMALL.with_(ffn="swiglu"), 4, 8, [64, 1, 130, 33], 4, 2e-2)


@pytest.mark.parametrize("B,K", [(12, 8), (16, 8)])
def test_small_bf16_large_batch(sps, B, K):
    # 108 and 144 rows: the widest single GEMM launches (14 and 18 M tiles)
    g = np.random.default_rng(B)
    verify_parity(sps, SMALL.with_(ffn="gelu"), B, K, [int(x) for x in g.integers(0, 200, B)], 40 + B, 2e-2,
                  check_kv=False)


@pytest.mark.parametrize("B,K", [(16, 8), (25, 4), (4, 8), (12, 7), (11, 9), (8, 7), (16, 4)])
def test_small_bf16_odd_depth_wide(sps, B, K):
    """Contraction depths of 5, 6 and 9 k-tiles (d_model 160, three 64-wide
    heads, d_ff 288) at 144, 125, 36, 96, 110, 64 and 80 rows (18, 16, 5,
    12, 14, 8 and 10 M tiles: 4-wave groups, 8-wave groups with
    register-held weights, 8-wave groups with staged weights): wide-GEMM
    chunks whose last k-tile pair is half past the end."""
    g = np.random.default_rng(B + 900)
    verify_parity(sps, SMALL.with_(d_model=160, d_ff=288, ffn="swiglu"), B, K,
                  [int(x) for x in g.integers(0, 150, B)], 90 + B, 2e-2, check_kv=False)


def test_small_fp32_greedy(sps):
    verify_parity(sps, SMALL.with_(dtype="f32"), 2, 4, [20, 77], 5, 1e-4, T=0.0)


def test_head_dim_128_fp32(sps):
    verify_parity(sps, configs.ModelShape("dh128", 256, 1, 2, 128, 512, 300, "swiglu", "f32"), 2, 2,
                  [130, 3], 6, 1e-4)


def test_prefill_chunk_parity(sps):
    """A 64-token prefill chunk per sequence (QT = 4 query tiles, 128 rows)."""
    shape = SMALL.with_(ffn="swiglu")
    print("prefill chunk", flush=True)
    B, M = 2, 64
    gm, W = build_pair(shape, 8)
    kv = sps.KVCache(shape, B, 128)
    ocache = new_cache(shape, B, 128)
    install_prior(shape, kv, ocache, 9, [10, 30])
    toks = synth.tokens(10, B, M, shape.vocab)
    ws = sps.workspace(shape, B, M, 128)
    logits = torch.empty((B, M, shape.vocab), dtype=torch.float32, device="cuda")
    sps.forward(gm, kv, torch.from_numpy(toks).cuda(), M, 0, logits, ws)
    torch.cuda.synchronize()
    want = om.forward_cached(spec_of(shape), W, ocache, toks, np.array([10, 30]))
    assert np.abs(logits.cpu().numpy() - want).max() <= 2e-2


def test_capacity_overflow_is_flagged(sps):
    """Positions past the cache capacity: the writes are skipped, the device
    flag is raised, and nothing faults."""
    shape = configs.TINY_TARGET
    gm, _ = build_pair(shape, 12)
    kv = sps.KVCache(shape, 1, 64)
    kv.lengths.fill_(62)
    ws = sps.workspace(shape, 1, 5, 64)
    sps.device_error()
    sps.verify_step(gm, kv, torch.zeros((1, 5), dtype=torch.int32, device="cuda"), 4, 1.0, ws,
                    logits=torch.empty((1, 5, shape.vocab), device="cuda"))
    assert sps.device_error() & sps.DEV_CAPACITY
    toks = torch.tensor([[1, 2, 5000, 3, 4]], dtype=torch.int32, device="cuda")
    kv.lengths.fill_(10)
    sps.verify_step(gm, kv, toks, 4, 1.0, ws, logits=torch.empty((1, 5, shape.vocab), device="cuda"))
    assert sps.device_error() & sps.DEV_BAD_TOKEN
    assert sps.device_error() == 0


_BUILT = {}


def full_width_layer(shape, seed):
    """One full-width block of `shape` (weights and oracle copy), kept for
    the tests that share it; one such model is held at a time."""
    key = (shape.name, shape.dtype, seed)
    if key not in _BUILT:
        _BUILT.clear()
        _BUILT[key] = build_pair(shape.with_(n_layers=1), seed)
    return _BUILT[key]


@pytest.mark.parametrize("shape", [configs.SEVEN_B, configs.SEVENTY_B], ids=["7b", "70b"])
def test_full_width_layer(sps, shape):
    """One full-width block + unembedding at K = 4, B = 1 against a 2048-token
    prior context: the per-layer kernels in the benchmark's launch shapes."""
    verify_parity(sps, shape.with_(n_layers=1), 1, 4, [2048], 21, 2e-2, built=full_width_layer(shape, 21))


def _planted(kind):
    """Oracle forward with a plausible kernel mistake planted (CPU): the
    rotary angle one position late, or the last 32-position block of
    keys / values each query sees left out."""
    import contextlib

    @contextlib.contextmanager
    def ctx():
        if kind == "rope+1":
            orig = om.rope
            om.rope = lambda x, pos, base: orig(x, np.asarray(pos) + 1, base)
            try:
                yield
            finally:
                om.rope = orig
        else:
            orig = om._attend

            def drop_last_block(q, Kc, Vc, scale):
                last = (len(Kc) - 1) // 32 * 32
                return orig(q, Kc[:last], Vc[:last], scale) if last > 0 else orig(q, Kc, Vc, scale)
            om._attend = drop_last_block
            try:
                yield
            finally:
                om._attend = orig
    return ctx()


def test_full_width_layer_negative_controls(sps):
    """The parity check bites: the 70B block's GPU logits (ctx 2048, K = 4)
    fail the 2e-2 tolerance against the oracle with a rotary angle one
    position late, and with the last 32-position KV block left out."""
    shape = configs.SEVENTY_B.with_(n_layers=1)
    built = full_width_layer(configs.SEVENTY_B, 21)
    inp = {}
    got = verify_parity(sps, shape, 1, 4, [2048], 21, 2e-2, built=built, want_out=inp)
    _, W = built
    for kind in ("rope+1", "drop last block"):
        ocache = new_cache(shape, 1, inp["T_cap"])
        install_oracle_prior(shape, ocache, inp["seed"] + 1, list(inp["n_prior"]))
        with _planted(kind):
            bad = om.forward_cached(spec_of(shape), W, ocache, inp["toks"], inp["n_prior"])
        err = np.abs(got - bad).max()
        print("  planted %s: max |GPU logits - planted oracle| = %.3g" % (kind, err), flush=True)
        assert err > 10 * 2e-2


@pytest.mark.parametrize("B,priors", [(1, [8192]), (4, [8192, 8001, 7777, 8190])], ids=["B1", "B4"])
def test_full_width_layer_ctx8192(sps, B, priors):
    """The 70B block at the sweep's long context (ctx 8192, K = 4): 33
    attention partials per head in the combine, rotary angles and KV tile
    offsets past position 8000, ragged lengths at B = 4."""
    verify_parity(sps, configs.SEVENTY_B.with_(n_layers=1), B, 4, priors, 21, 2e-2,
                  built=full_width_layer(configs.SEVENTY_B, 21), check_kv=B == 1)


@pytest.mark.parametrize("shape,B,K", [(configs.SEVENTY_B, 4, 4), (configs.SEVENTY_B, 16, 8),
                                       (configs.SEVEN_B, 16, 1)], ids=["70b-B4K4", "70b-B16K8", "7b-B16K1"])
def test_full_width_layer_batched(sps, shape, B, K):
    """Batched full-width blocks: the wide GEMM in the sweep's launch shapes,
    split-K (partials + reduction kernel) on the d_model-wide outputs."""
    g = np.random.default_rng(100 * B + K)
    verify_parity(sps, shape.with_(n_layers=1), B, K, [int(x) for x in g.integers(200, 600, B)], 31 + B, 2e-2,
                  check_kv=False)


@pytest.mark.gpu
def test_stream_read_helper(sps):
    """The streaming-read measurement helper reads without writing: the sink
    keeps its value for a buffer whose folded words differ from the key."""
    buf = torch.ones(1 << 20, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    sps.stream_read(buf, 4 << 20, sink)
    sps.stream_read(buf, (4 << 20) - 48, sink)   # ragged tail past the unrolled loop
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
    with pytest.raises(ValueError):
        sps.stream_read(buf, (4 << 20) + 16, sink)


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_max_rows_one_launch(sps, dtype):
    """160 rows (32 sequences x 5 positions), the most one GEMM launch takes
    (20 M tiles), with ragged cache lengths."""
    g = np.random.default_rng(160)
    verify_parity(sps, SMALL.with_(dtype=dtype, ffn="swiglu", d_model=192, d_ff=320), 32, 4,
                  [int(x) for x in g.integers(0, 90, 32)], 160, 2e-2, check_kv=False)


def test_max_lookahead(sps):
    """K = 63, the largest lookahead: 64 positions of one sequence (8 M tiles,
    4 query tiles in attention)."""
    verify_parity(sps, SMALL, 1, 63, [100], 163, 2e-2)


@pytest.mark.parametrize("B,T", [(1, 1.0), (2, 0.8)])
def test_draft_step_full_width(sps, B, T):
    """The 70B draft's shape (d_model 3072, 24 heads of 128, GELU FFN 12288,
    vocab 32000, bf16) in the launch shapes the end-to-end runs use, with
    two layers (the per-layer kernels do not depend on the layer count): a
    K = 4 draft step against a 2048-token prior (ragged at B = 2). Per step,
    the oracle's forward of the same tokens gives the draft distribution
    p_t = softmax(logits / T), which the exported p rows match within the
    bf16 logit tolerance (as log-probabilities); each drawn token equals the
    oracle's integer inverse-CDF draw from the GPU's own p row (bit-exact);
    the appended keys and values match the oracle cache."""
    from oracle import philox as ophil
    shape = configs.DRAFT_70B.with_(n_layers=2)
    K, V, tol = 4, shape.vocab, 2e-2
    n_prior = [2048, 1500][:B]
    print("draft step full width B", B, "T", T, flush=True)
    gm, W = build_pair(shape, 51)
    T_cap = round_up(max(n_prior) + K + 1, 32)
    kv = sps.KVCache(shape, B, T_cap)
    ocache = new_cache(shape, B, T_cap)
    install_prior(shape, kv, ocache, 52, n_prior)
    ctx = synth.tokens(53, B, 2, V)
    ws = sps.workspace(shape, B, 2, T_cap)
    tokens = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    p_out = torch.empty((B, K, V), dtype=torch.float32, device="cuda")
    seed, loop = 54, 3
    sps.draft_step(gm, kv, torch.from_numpy(ctx).cuda(), K, T, (seed, loop), tokens, p_out, ws)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    got_t, got_p = tokens.cpu().numpy(), p_out.cpu().numpy()
    np.testing.assert_array_equal(got_t[:, 0], ctx[:, 1])
    ud = ophil.uniforms(seed, loop, ophil.PURPOSE_DRAFT, B, K)
    lens = np.array(n_prior)
    spec = spec_of(shape)
    worst = 0.0
    for t in range(K):
        if t == 0:   # the last committed token and the newest one, at positions len - 1 and len
            lg = om.forward_cached(spec, W, ocache, ctx, lens - 1)[:, -1]
        else:
            lg = om.forward_cached(spec, W, ocache, got_t[:, t:t + 1], lens + t)[:, 0]
        want_p = osamp.softmax(lg, T)
        for b in range(B):
            keep = want_p[b] > 1e-30
            dlog = np.log(got_p[b, t, keep].astype(np.float64)) - np.log(want_p[b, keep])
            worst = max(worst, np.abs(dlog).max())
            y, ok = osamp.categorical(osamp.to_weights(got_p[b, t]), ud[b, t])
            assert ok and got_t[b, t + 1] == y, (b, t)
    print("  max |log p - log p_oracle| = %.3g (tol %.2g)" % (worst, 2 * tol / T), flush=True)
    assert worst <= 2 * tol / T and worst <= tol / T
    for l in range(shape.n_layers):
        for b in range(B):
            k, v = kv.read(l, b, n_prior[b] - 1, K + 1)
            np.testing.assert_allclose(k.float().cpu().numpy(),
                                       ocache["k"][l, b, :, n_prior[b] - 1:n_prior[b] + K], atol=tol, rtol=tol)
            np.testing.assert_allclose(v.float().cpu().numpy(),
                                       ocache["v"][l, b, :, n_prior[b] - 1:n_prior[b] + K], atol=tol, rtol=tol)
