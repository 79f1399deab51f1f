"""GPU parity of the weight-only FP8 path against the oracle.

* decode: every E4M3 code converts, with the GEMM's conversion, to the value
  the oracle's table gives (bit for bit; the two NaN codes to NaN);
* pack: the packed codes and row scales of every projection kind (plain rows,
  the fused QKV with rotary partners side by side, SwiGLU gate / up
  interleaving, the padded unembedding) equal the oracle quantiser's, bit for
  bit;
* verify step: logits within 2e-2 max-abs of the oracle forward run on the
  oracle's own dequantised weights, q the softmax of the logits, the fused
  accept / resample outputs bit-exact against the oracle on the GPU's q; the
  appended keys and values within 2e-2. Cases: 5 rows (one M tile, the
  single-tile kernel), 12 to 144 rows (the wide kernel, register and LDS
  staged weights, with and without split-K), a 64-token prefill chunk, and full-width blocks of the 70B and 7B
  shapes in the benchmark's and the sweep's launch shapes;
* end to end: with the draft equal to the target every draft is accepted,
  and greedy SpS emits the same tokens as greedy ArS.
"""
import numpy as np
import pytest
import torch

from oracle import fp8
from oracle import model as om
from paper_2302_01318_amd import configs, synth
from gpu_helpers import build_pair, install_prior, new_cache
from oracle_helpers import spec_of
from test_gpu_forward import verify_parity

pytestmark = pytest.mark.gpu

SMALL8 = configs.ModelShape("small-fp8", 192, 2, 3, 64, 320, 1000, "gelu", "fp8")


def test_fp8_decode_every_code(sps):
    codes = torch.arange(256, dtype=torch.int32, device="cuda").to(torch.uint8)
    got = sps.fp8_decode(codes).cpu().numpy().astype(np.float64)
    want = fp8.e4m3_value(np.arange(256, dtype=np.uint8))
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


def _codes_at(buf, off, rows, cols):
    """Codes [rows][cols] of an FP8 slot, by packed row, from the documented
    tile layout: 16 x 64 tiles [n-tile][k-tile pair], lane l = row % 16 +
    16 * ((k % 32) / 8) holding 16 bytes (first k-tile of the pair, then the
    second)."""
    KT = cols // 32
    nf, k = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
    lane = nf % 16 + 16 * ((k % 32) // 8)
    byte = (((nf // 16) * (KT // 2) + k // 64) * 64 + lane) * 16 + ((k % 64) // 32) * 8 + k % 8
    return buf[off + byte]


def _rope_rows(HD, dh):
    """Packed row of canonical q / k row n: rotary partners side by side."""
    n = np.arange(HD)
    f, head = n % dh, n // dh
    half = dh // 2
    r = np.where(f < half, (f // 8) * 16 + f % 8, ((f - half) // 8) * 16 + 8 + (f - half) % 8)
    return head * dh + r


@pytest.mark.parametrize("ffn", ["gelu", "swiglu"])
def test_fp8_pack_matches_oracle_quantiser(sps, ffn):
    shape = SMALL8.with_(ffn=ffn, n_layers=1)
    print("fp8 pack", ffn, flush=True)
    w = synth.weights(shape, 50)
    gm = sps.Model(shape, w)
    torch.cuda.synchronize()
    buf = gm.packed.cpu().numpy()
    d, HD, F, V = shape.d_model, shape.n_heads * shape.head_dim, shape.d_ff, shape.vocab

    def check(name, canon, rows_packed, packed_of, cols):
        off, nbytes, soff = sps.weight_slot(shape, name, 0)
        assert nbytes == rows_packed * cols
        codes = _codes_at(buf, off, rows_packed, cols)
        scales = buf[soff:soff + 4 * rows_packed].view(np.float32)
        want_c, want_s = fp8.quantize_rows(canon.float().numpy())
        np.testing.assert_array_equal(codes[packed_of], want_c, err_msg=name)
        np.testing.assert_array_equal(scales[packed_of], want_s, err_msg=name)
        return codes, scales

    rope = _rope_rows(HD, shape.head_dim)
    check("wq", w[("wq", 0)], 3 * HD, rope, d)
    check("wk", w[("wk", 0)], 3 * HD, HD + rope, d)
    check("wv", w[("wv", 0)], 3 * HD, 2 * HD + np.arange(HD), d)
    check("wo", w[("wo", 0)], d, np.arange(d), HD)
    n = np.arange(F)
    if ffn == "swiglu":
        check("w1", w[("w1", 0)], 2 * F, (n // 8) * 16 + n % 8, d)
        check("w3", w[("w3", 0)], 2 * F, (n // 8) * 16 + 8 + n % 8, d)
    else:
        check("w1", w[("w1", 0)], F, n, d)
    check("w2", w[("w2", 0)], d, np.arange(d), F)
    NU = (V + 15) // 16 * 16
    codes, scales = check("unembed", w[("unembed", -1)], NU, np.arange(V), d)
    assert np.all(codes[V:] == 0) and np.all(scales[V:] == 1.0)   # padding rows


def test_fp8_verify_one_tile(sps):
    verify_parity(sps, SMALL8, 1, 4, [77], 61, 2e-2)


@pytest.mark.parametrize("ffn", ["gelu", "swiglu"])
def test_fp8_verify_ragged_wide(sps, ffn):
    # 3 sequences x 4 positions = 12 rows: the wide kernel at 2 M tiles
    verify_parity(sps, SMALL8.with_(ffn=ffn), 3, 3, [5, 100, 257], 62, 2e-2)


@pytest.mark.parametrize("B,K", [(12, 8), (16, 8), (16, 4), (7, 8)])
def test_fp8_verify_large_batch(sps, B, K):
    # 108, 144, 80 and 63 rows: 14, 18, 10 and 8 M tiles (the staged loop)
    g = np.random.default_rng(B + 500)
    verify_parity(sps, SMALL8, B, K, [int(x) for x in g.integers(0, 200, B)], 70 + B, 2e-2, check_kv=False)


def test_fp8_verify_greedy(sps):
    verify_parity(sps, SMALL8, 2, 2, [31, 9], 63, 2e-2, T=0.0)


def test_fp8_prefill_chunk(sps):
    shape = SMALL8.with_(ffn="swiglu")
    print("fp8 prefill chunk", flush=True)
    B, M = 2, 64
    gm, W = build_pair(shape, 64)
    kv = sps.KVCache(shape, B, 128)
    ocache = new_cache(shape, B, 128)
    install_prior(shape, kv, ocache, 65, [10, 30])
    toks = synth.tokens(66, B, M, shape.vocab)
    ws = sps.workspace(shape, B, M, 128)
    logits = torch.empty((B, M, shape.vocab), dtype=torch.float32, device="cuda")
    sps.forward(gm, kv, torch.from_numpy(toks).cuda(), M, 0, logits, ws)
    torch.cuda.synchronize()
    want = om.forward_cached(spec_of(shape), W, ocache, toks, np.array([10, 30]))
    assert np.abs(logits.cpu().numpy() - want).max() <= 2e-2


@pytest.mark.parametrize("shape", [configs.SEVENTY_B, configs.SEVEN_B], ids=["70b", "7b"])
def test_fp8_full_width_layer(sps, shape):
    """One full-width FP8 block + unembedding at K = 4, B = 1 against a
    2048-token prior: the per-layer kernels in the benchmark's launch shapes."""
    verify_parity(sps, shape.with_(n_layers=1, dtype="fp8"), 1, 4, [2048], 67, 2e-2)


@pytest.mark.parametrize("B,K", [(4, 4), (16, 8)], ids=["B4K4", "B16K8"])
def test_fp8_full_width_layer_batched(sps, B, K):
    """Batched full-width FP8 blocks of the 70B shape: the wide kernel with
    split-K on the 8192-wide outputs."""
    g = np.random.default_rng(200 * B + K)
    verify_parity(sps, configs.SEVENTY_B.with_(n_layers=1, dtype="fp8"), B, K,
                  [int(x) for x in g.integers(200, 600, B)], 80 + B, 2e-2, check_kv=False)


def test_fp8_e2e_properties(sps):
    """Draft = target accepts every draft; greedy SpS equals greedy ArS."""
    shape = SMALL8.with_(n_layers=2)
    gm, _ = build_pair(shape, 68)
    prompt = torch.from_numpy(synth.tokens(69, 2, 16, shape.vocab)).cuda()
    log = []
    sps.Generator(gm, gm, 2, 128, 4).generate(prompt, 40, 1.0, 5, accepted_log=log)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    flat = [int(a[b]) for a, done in log for b in range(2) if not bool(done[b])]
    assert sum(a == 4 for a in flat) >= 0.99 * len(flat)
    g1 = sps.Generator(gm, gm, 2, 128, 4).generate(prompt, 32, 0.0, 1)
    g0 = sps.Generator(gm, None, 2, 128, 0).generate(prompt, 32, 0.0, 1)
    torch.cuda.synchronize()
    assert torch.equal(g1, g0)


def test_bf16_target_fp8_draft(sps):
    """A bf16 target drafted by its own weights in weight-only FP8 (the pair
    the end-to-end benchmark also runs): greedy SpS emits exactly the
    target's greedy ArS tokens, since every emitted token is the target's
    argmax whatever the draft proposes; at T = 1 the quantised draft is
    accepted most of the time."""
    shape = SMALL8.with_(n_layers=2, dtype="bf16")
    w = synth.weights(shape, 71)
    gt = sps.Model(shape, w)
    gd = sps.Model(shape.with_(dtype="fp8"), w)
    del w
    prompt = torch.from_numpy(synth.tokens(72, 2, 16, shape.vocab)).cuda()
    print("bf16 target, fp8 draft", flush=True)
    g1 = sps.Generator(gt, gd, 2, 128, 4).generate(prompt, 32, 0.0, 1)
    g0 = sps.Generator(gt, None, 2, 128, 0).generate(prompt, 32, 0.0, 1)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    assert torch.equal(g1, g0)
    log = []
    sps.Generator(gt, gd, 2, 128, 4).generate(prompt, 40, 1.0, 5, accepted_log=log)
    torch.cuda.synchronize()
    assert sps.device_error() == 0
    flat = [int(a[b]) for a, done in log for b in range(2) if not bool(done[b])]
    assert sum(flat) >= 0.8 * 4 * len(flat)
