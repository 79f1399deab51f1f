"""ctypes binding of libsps.so, the HIP speculative-sampling library.

Argument marshalling only: torch tensors become device pointers, the current
torch stream becomes the hipStream_t, and every status code is checked. All
computation happens in the library's kernels. Importing this module fails
loudly when libsps.so has not been built.
"""
import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsps.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError("libsps.so is not built; run `python -m paper_2302_01318_amd.build` "
                      "(or __graft_entry__.build())")
lib = ctypes.CDLL(_LIB_PATH)

c_int32, c_uint64, c_float, c_size_t, c_void_p = (ctypes.c_int32, ctypes.c_uint64, ctypes.c_float,
                                                   ctypes.c_size_t, ctypes.c_void_p)

FFN = {"gelu": 0, "swiglu": 1}
DTYPE = {"f32": 0, "bf16": 1, "fp8": 2}
# Tensor type of the canonical matrices handed to the packer and of the KV
# cache: an FP8 model is packed from bf16 matrices and keeps a bf16 cache.
TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.bfloat16}
TENSOR_ID = {"embed": 0, "final_norm": 1, "unembed": 2, "attn_norm": 3, "wq": 4, "wk": 5, "wv": 6,
             "wo": 7, "ffn_norm": 8, "w1": 9, "w3": 10, "w2": 11}
PURPOSE_DRAFT, PURPOSE_ACCEPT, PURPOSE_RESAMPLE = 0, 1, 2
DEV_BAD_TOKEN, DEV_EMPTY, DEV_CAPACITY, DEV_NONFINITE = 1, 2, 4, 8


class Config(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("n_layers", c_int32), ("n_heads", c_int32),
                ("head_dim", c_int32), ("d_ff", c_int32), ("vocab", c_int32),
                ("ffn_kind", c_int32), ("dtype", c_int32), ("rms_eps", c_float),
                ("rope_base", c_float)]


class Philox(ctypes.Structure):
    _fields_ = [("seed", c_uint64), ("loop", c_uint64)]


class Sampling(ctypes.Structure):
    """Temperature, top-k and nucleus parameters (sps_sampling)."""
    _fields_ = [("temperature", c_float), ("top_k", c_int32), ("top_p", c_float)]


def sampling_of(temperature, top_k=0, top_p=1.0):
    return Sampling(float(temperature), int(top_k), float(top_p))


class AcceptIO(ctypes.Structure):
    _fields_ = [("p_draft", c_void_p), ("uniforms", c_void_p), ("rng", Philox),
                ("out_tokens", c_void_p), ("n_accepted", c_void_p)]


def _sig(name, res, args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = args
    return f


P = c_void_p
_sig("sps_status_string", ctypes.c_char_p, [c_int32])
_sig("sps_abi_version", c_int32, [])
_sig("sps_weight_bytes", c_size_t, [ctypes.POINTER(Config)])
_sig("sps_pack_weight", c_int32, [ctypes.POINTER(Config), c_int32, c_int32, P, P, P])
_sig("sps_model_create", c_int32, [ctypes.POINTER(Config), P, ctypes.POINTER(P)])
_sig("sps_model_destroy", None, [P])
_sig("sps_kv_bytes", c_size_t, [ctypes.POINTER(Config), c_int32, c_int32])
_sig("sps_kv_create", c_int32, [ctypes.POINTER(Config), c_int32, c_int32, P, P, ctypes.POINTER(P)])
_sig("sps_kv_destroy", None, [P])
_sig("sps_kv_write", c_int32, [P, c_int32, c_int32, c_int32, c_int32, P, P, P])
_sig("sps_kv_read", c_int32, [P, c_int32, c_int32, c_int32, c_int32, P, P, P])
_sig("sps_workspace_bytes", c_size_t, [ctypes.POINTER(Config), c_int32, c_int32, c_int32])
_sig("sps_forward", c_int32, [P, P, P, c_int32, c_int32, c_int32, c_int32, P, P, c_size_t, P])
_sig("sps_verify_step", c_int32, [P, P, P, c_int32, c_int32, Sampling, P, P, ctypes.POINTER(AcceptIO), P,
                                  c_size_t, P])
_sig("sps_verify_step_noalloc", c_int32, [P, P, P, c_int32, c_int32, Sampling, P, P, ctypes.POINTER(AcceptIO), P])
_sig("sps_accept_resample", c_int32, [P, P, P, P, Philox, c_int32, c_int32, c_int32, P, P, P])
_sig("sps_draft_step", c_int32, [P, P, P, c_int32, c_int32, Sampling, Philox, P, P, P, c_size_t, P])
_sig("sps_commit", c_int32, [P, P, P, P, c_int32, c_int32, P, P, P, c_int32, P])
_sig("sps_philox_uniforms", c_int32, [Philox, c_int32, c_int32, c_int32, P, P])
_sig("sps_softmax", c_int32, [P, c_int32, c_int32, Sampling, P, P])
_sig("sps_device_error", c_int32, [P, c_int32, ctypes.POINTER(c_int32)])
_sig("sps_profile_gemm_begin", c_int32, [c_int32])
_sig("sps_stream_read", c_int32, [P, c_size_t, P, P])
_sig("sps_fp8_decode", c_int32, [P, c_int32, P, P])
_sig("sps_weight_slot", c_int32, [ctypes.POINTER(Config), c_int32, c_int32, ctypes.POINTER(c_size_t),
                                  ctypes.POINTER(c_size_t), ctypes.POINTER(c_size_t)])
_sig("sps_profile_gemm_end", c_int32, [ctypes.POINTER(c_float), ctypes.POINTER(c_int32),
                                       ctypes.POINTER(ctypes.c_double)])

EXPORTS = ["sps_status_string", "sps_abi_version", "sps_weight_bytes", "sps_pack_weight",
           "sps_model_create", "sps_model_destroy", "sps_kv_bytes", "sps_kv_create", "sps_kv_destroy",
           "sps_kv_write", "sps_kv_read", "sps_workspace_bytes", "sps_forward", "sps_verify_step",
           "sps_accept_resample", "sps_draft_step", "sps_commit", "sps_philox_uniforms", "sps_softmax",
           "sps_device_error", "sps_profile_gemm_begin", "sps_profile_gemm_end",
           "sps_stream_read", "sps_fp8_decode", "sps_weight_slot", "sps_verify_step_noalloc"]


class SPSError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__("%s: %s (status %d)" % (what, lib.sps_status_string(status).decode(), status))


def check(status, what):
    if status != 0:
        raise SPSError(status, what)


def _stream():
    return c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t, dtype=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return c_void_p(t.data_ptr())


def config_of(shape):
    return Config(shape.d_model, shape.n_layers, shape.n_heads, shape.head_dim, shape.d_ff, shape.vocab,
                  FFN[shape.ffn], DTYPE[shape.dtype], shape.eps, shape.rope_base)


def weight_bytes(shape):
    return lib.sps_weight_bytes(ctypes.byref(config_of(shape)))


class Model:
    """Packed weights of one model on the device plus its library handle."""

    def __init__(self, shape, tensors=None, device="cuda"):
        self.shape = shape
        self.cfg = config_of(shape)
        nbytes = lib.sps_weight_bytes(ctypes.byref(self.cfg))
        if nbytes == 0:
            raise SPSError(2, "sps_weight_bytes(%s)" % shape.name)
        self.packed = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.handle = c_void_p()
        # __del__ may run at interpreter exit, after this module's globals
        # are cleared: keep the destructor on the instance.
        self._destroy = lib.sps_model_destroy
        check(lib.sps_model_create(ctypes.byref(self.cfg), _ptr(self.packed), ctypes.byref(self.handle)),
              "sps_model_create")
        if tensors is not None:
            for (name, layer), t in tensors.items():
                self.pack(name, layer, t)

    def pack(self, name, layer, t):
        want = torch.float32 if name.endswith("norm") else TORCH_DTYPE[self.shape.dtype]
        t = t.to(device=self.packed.device, dtype=want).contiguous()
        check(lib.sps_pack_weight(ctypes.byref(self.cfg), TENSOR_ID[name], layer, _ptr(t), _ptr(self.packed),
                                  _stream()), "sps_pack_weight(%s, %d)" % (name, layer))
        torch.cuda.current_stream().synchronize()   # t may be freed after return

    def __del__(self):
        h, destroy = getattr(self, "handle", None), getattr(self, "_destroy", None)
        if h is not None and h.value and destroy is not None:
            destroy(h)
        self.handle = None


class KVCache:
    """KV cache buffer, the shared device `lengths` [B] array and the handle."""

    def __init__(self, shape, B, T_cap, lengths=None, device="cuda"):
        self.shape, self.B, self.T_cap = shape, B, T_cap
        self.cfg = config_of(shape)
        nbytes = lib.sps_kv_bytes(ctypes.byref(self.cfg), B, T_cap)
        if nbytes == 0:
            raise SPSError(2, "sps_kv_bytes")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.lengths = lengths if lengths is not None else torch.zeros(B, dtype=torch.int32, device=device)
        self.handle = c_void_p()
        self._destroy = lib.sps_kv_destroy   # see Model.__init__
        check(lib.sps_kv_create(ctypes.byref(self.cfg), B, T_cap, _ptr(self.buf),
                                _ptr(self.lengths, torch.int32, "lengths"), ctypes.byref(self.handle)),
              "sps_kv_create")

    def write(self, layer, b, pos0, k, v):
        """k, v: [H][n][Dh] in the model dtype (keys already rotated)."""
        dt = TORCH_DTYPE[self.shape.dtype]
        n = k.shape[1]
        check(lib.sps_kv_write(self.handle, layer, b, pos0, n, _ptr(k, dt, "k"), _ptr(v, dt, "v"), _stream()),
              "sps_kv_write")

    def read(self, layer, b, pos0, n):
        dt = TORCH_DTYPE[self.shape.dtype]
        k = torch.empty((self.shape.n_heads, n, self.shape.head_dim), dtype=dt, device=self.buf.device)
        v = torch.empty_like(k)
        check(lib.sps_kv_read(self.handle, layer, b, pos0, n, _ptr(k), _ptr(v), _stream()), "sps_kv_read")
        return k, v

    def __del__(self):
        h, destroy = getattr(self, "handle", None), getattr(self, "_destroy", None)
        if h is not None and h.value and destroy is not None:
            destroy(h)
        self.handle = None


def workspace(shape, B, max_tokens_per_seq, T_cap, device="cuda"):
    n = lib.sps_workspace_bytes(ctypes.byref(config_of(shape)), B, max_tokens_per_seq, T_cap)
    if n == 0:
        raise SPSError(2, "sps_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def forward(model, kv, tokens, M, pos_offset=0, logits=None, ws=None, tok_stride=None):
    B = kv.B
    check(lib.sps_forward(model.handle, kv.handle, _ptr(tokens, torch.int32, "tokens"),
                          tok_stride if tok_stride is not None else tokens.shape[-1], B, M, pos_offset,
                          _ptr(logits, torch.float32, "logits"), _ptr(ws), ws.numel(), _stream()),
          "sps_forward")


def verify_step(model, kv, tokens, K, temperature, ws, logits=None, q=None, p_draft=None, uniforms=None,
                rng=(0, 0), out_tokens=None, n_accepted=None, top_k=0, top_p=1.0):
    acc = None
    if out_tokens is not None:
        acc = AcceptIO(_ptr(p_draft, torch.float32, "p_draft"), _ptr(uniforms, torch.float32, "uniforms"),
                       Philox(*rng), _ptr(out_tokens, torch.int32, "out_tokens"),
                       _ptr(n_accepted, torch.int32, "n_accepted"))
    check(lib.sps_verify_step(model.handle, kv.handle, _ptr(tokens, torch.int32, "tokens"), kv.B, K,
                              sampling_of(temperature, top_k, top_p), _ptr(logits, torch.float32, "logits"),
                              _ptr(q, torch.float32, "q"), ctypes.byref(acc) if acc else None, _ptr(ws),
                              ws.numel(), _stream()), "sps_verify_step")


def verify_step_noalloc(model, kv, tokens, K, temperature, logits=None, q=None, p_draft=None, uniforms=None,
                        rng=(0, 0), out_tokens=None, n_accepted=None, top_k=0, top_p=1.0):
    """verify_step with the library's own scratch (no workspace argument)."""
    acc = None
    if out_tokens is not None:
        acc = AcceptIO(_ptr(p_draft, torch.float32, "p_draft"), _ptr(uniforms, torch.float32, "uniforms"),
                       Philox(*rng), _ptr(out_tokens, torch.int32, "out_tokens"),
                       _ptr(n_accepted, torch.int32, "n_accepted"))
    check(lib.sps_verify_step_noalloc(model.handle, kv.handle, _ptr(tokens, torch.int32, "tokens"), kv.B, K,
                                      sampling_of(temperature, top_k, top_p), _ptr(logits, torch.float32, "logits"),
                                      _ptr(q, torch.float32, "q"), ctypes.byref(acc) if acc else None, _stream()),
          "sps_verify_step_noalloc")


def accept_resample(p_draft, q_target, draft_tokens, uniforms=None, rng=(0, 0), out_tokens=None,
                    n_accepted=None):
    B, K1, V = q_target.shape
    K = K1 - 1
    dev = q_target.device
    if out_tokens is None:
        out_tokens = torch.empty((B, K + 1), dtype=torch.int32, device=dev)
    if n_accepted is None:
        n_accepted = torch.empty(B, dtype=torch.int32, device=dev)
    check(lib.sps_accept_resample(_ptr(p_draft, torch.float32, "p_draft") if K else None,
                                  _ptr(q_target, torch.float32, "q_target"),
                                  _ptr(draft_tokens, torch.int32, "draft_tokens") if K else None,
                                  _ptr(uniforms, torch.float32, "uniforms"), Philox(*rng), B, K, V,
                                  _ptr(out_tokens), _ptr(n_accepted), _stream()), "sps_accept_resample")
    return out_tokens, n_accepted


def draft_step(model, kv, ctx, K, temperature, rng, tokens, p_out, ws, top_k=0, top_p=1.0):
    check(lib.sps_draft_step(model.handle, kv.handle, _ptr(ctx, torch.int32, "ctx"), kv.B, K,
                             sampling_of(temperature, top_k, top_p),
                             Philox(*rng), _ptr(tokens, torch.int32, "tokens"), _ptr(p_out, torch.float32, "p_out"),
                             _ptr(ws), ws.numel(), _stream()), "sps_draft_step")


def commit(kv, tokens, out_tokens, n_accepted, K, ctx, seq_out=None, n_out=None, cap=0):
    check(lib.sps_commit(kv.handle, _ptr(tokens, torch.int32), _ptr(out_tokens, torch.int32),
                         _ptr(n_accepted, torch.int32), kv.B, K, _ptr(ctx, torch.int32),
                         _ptr(seq_out, torch.int32), _ptr(n_out, torch.int32), cap, _stream()), "sps_commit")


def philox_uniforms(seed, loop, purpose, B, n, device="cuda"):
    out = torch.empty((B, n), dtype=torch.float32, device=device)
    check(lib.sps_philox_uniforms(Philox(seed, loop), purpose, B, n, _ptr(out), _stream()), "sps_philox_uniforms")
    return out


def softmax(logits, temperature, top_k=0, top_p=1.0, out=None):
    rows, V = logits.reshape(-1, logits.shape[-1]).shape
    if out is None:
        out = torch.empty_like(logits)
    elif out.shape != logits.shape:
        raise ValueError("out has shape %s, logits %s" % (tuple(out.shape), tuple(logits.shape)))
    check(lib.sps_softmax(_ptr(logits, torch.float32, "logits"), rows, V, sampling_of(temperature, top_k, top_p),
                          _ptr(out),
                          _stream()), "sps_softmax")
    return out


def device_error(clear=True):
    flags = c_int32(0)
    check(lib.sps_device_error(_stream(), 1 if clear else 0, ctypes.byref(flags)), "sps_device_error")
    return flags.value


def profile_gemm_begin(repeats=1):
    check(lib.sps_profile_gemm_begin(repeats), "sps_profile_gemm_begin")


def profile_gemm_end():
    """(total ms, launches, algorithmic bytes) of the GEMM launches since begin."""
    ms, n, b = c_float(0), c_int32(0), ctypes.c_double(0)
    check(lib.sps_profile_gemm_end(ctypes.byref(ms), ctypes.byref(n), ctypes.byref(b)), "sps_profile_gemm_end")
    return ms.value, n.value, b.value


def stream_read(buf, nbytes, sink):
    """One streaming read of the first `nbytes` of device tensor `buf`
    (measurement helper: the attainable HBM read rate)."""
    if nbytes > buf.numel() * buf.element_size():
        raise ValueError("stream_read: %d bytes exceed the buffer" % nbytes)
    check(lib.sps_stream_read(_ptr(buf), nbytes, _ptr(sink, torch.int32, "sink"), _stream()), "sps_stream_read")


def weight_slot(shape, name, layer=0):
    """(offset, bytes, scale offset) of a tensor's slot in the packed buffer."""
    o, n, sc = c_size_t(0), c_size_t(0), c_size_t(0)
    check(lib.sps_weight_slot(ctypes.byref(config_of(shape)), TENSOR_ID[name], layer, ctypes.byref(o),
                              ctypes.byref(n), ctypes.byref(sc)), "sps_weight_slot")
    return o.value, n.value, sc.value


def fp8_decode(codes):
    """fp32 values of E4M3 codes (uint8 device tensor, numel % 16 == 0) with
    the FP8-weight GEMM's conversion."""
    out = torch.empty(codes.numel(), dtype=torch.float32, device=codes.device)
    check(lib.sps_fp8_decode(_ptr(codes, torch.uint8, "codes"), codes.numel(), _ptr(out), _stream()),
          "sps_fp8_decode")
    return out


class Generator:
    """The SpS loop (Algorithm 2) on the device: prefill, then per loop one
    draft step, one verify step and one commit, with no host synchronisation
    except an end-of-output check every `check_every` loops. K = 0 without a
    draft model is auto-regressive sampling (Algorithm 1)."""

    def __init__(self, target, draft, B, T_cap, K, device="cuda", prefill_chunk=64):
        if draft is not None and draft.shape.vocab != target.shape.vocab:
            # p_t and q_t are distributions over one token space (the accept
            # ratio q(x)/p(x) of Algorithm 2); the draft's p rows are read at
            # the target's vocabulary stride.
            raise ValueError("draft vocabulary %d differs from the target's %d"
                             % (draft.shape.vocab, target.shape.vocab))
        self.target, self.draft, self.B, self.K, self.T_cap = target, draft, B, K, T_cap
        self.chunk = max(1, min(prefill_chunk, 160 // B, 64))
        mps = max(self.chunk, K + 1, 2)
        self.lengths = torch.zeros(B, dtype=torch.int32, device=device)
        self.kv_t = KVCache(target.shape, B, T_cap, self.lengths, device)
        self.ws_t = workspace(target.shape, B, mps, T_cap, device)
        if draft is not None:
            self.kv_d = KVCache(draft.shape, B, T_cap, self.lengths, device)
            self.ws_d = workspace(draft.shape, B, mps, T_cap, device)
        V = target.shape.vocab
        self.ctx = torch.zeros((B, 2), dtype=torch.int32, device=device)
        self.tokens = torch.zeros((B, K + 1), dtype=torch.int32, device=device)
        self.p = torch.zeros((B, max(K, 1), V), dtype=torch.float32, device=device)
        self.out = torch.zeros((B, K + 1), dtype=torch.int32, device=device)
        self.n_acc = torch.zeros(B, dtype=torch.int32, device=device)

    def prefill(self, prompt):
        """prompt: [B][P] int32 device tensor, P >= 2. Scores x_1..x_{P-1} into
        both caches; x_P is the first token the loop feeds."""
        B, Pn = prompt.shape
        prompt = prompt.contiguous()
        self.lengths.zero_()
        for c0 in range(0, Pn - 1, self.chunk):
            n = min(self.chunk, Pn - 1 - c0)
            view = prompt[:, c0:]
            for model, kv, ws in ((self.target, self.kv_t, self.ws_t),) + \
                    (((self.draft, self.kv_d, self.ws_d),) if self.draft is not None else ()):
                check(lib.sps_forward(model.handle, kv.handle, c_void_p(view.data_ptr()), Pn, B, n, c0, None,
                                      _ptr(ws), ws.numel(), _stream()), "sps_forward(prefill)")
        self.lengths.fill_(Pn - 1)
        self.ctx.copy_(prompt[:, Pn - 2:Pn])

    def loop(self, temperature, seed, loop_index, seq_out=None, n_out=None, cap=0, top_k=0, top_p=1.0):
        K = self.K
        rng = (seed, loop_index)
        if self.draft is not None and K > 0:
            draft_step(self.draft, self.kv_d, self.ctx, K, temperature, rng, self.tokens, self.p, self.ws_d,
                       top_k, top_p)
        else:
            check(lib.sps_draft_step(self.target.handle, self.kv_t.handle, _ptr(self.ctx), self.B, 0,
                                     sampling_of(temperature, top_k, top_p), Philox(*rng), _ptr(self.tokens), None,
                                     _ptr(self.ws_t), self.ws_t.numel(), _stream()), "sps_draft_step(K=0)")
        verify_step(self.target, self.kv_t, self.tokens, K, temperature, self.ws_t, p_draft=self.p if K else None,
                    rng=rng, out_tokens=self.out, n_accepted=self.n_acc, top_k=top_k, top_p=top_p)
        commit(self.kv_t, self.tokens, self.out, self.n_acc, K, self.ctx, seq_out, n_out, cap)

    def generate(self, prompt, n_new, temperature, seed, accepted_log=None, top_k=0, top_p=1.0, loop0=0,
                 log=None):
        """Prefill, then run(); returns [B][n_new] int32 tokens (device)."""
        self.prefill(prompt)
        return self.run(n_new, temperature, seed, accepted_log, top_k, top_p, loop0, log)

    def run(self, n_new, temperature, seed, accepted_log=None, top_k=0, top_p=1.0, loop0=0, log=None):
        """SpS loops until every sequence has n_new tokens. The host looks at
        the device-side output counts only between bursts of loops: every
        loop emits at most K + 1 tokens, so ceil(remaining / (K + 1)) loops
        can always run before the next look without overshooting the end.

        loop0 is the index of the first loop (the Philox loop counter): the
        SpS state at a loop boundary is the token sequence and the loop
        index, so a run resumes by prefilling prompt + the tokens so far and
        passing the loops done as loop0. self.loops is the index after the
        last loop.
        If accepted_log is a list, (n_accepted, done-before-loop) device
        tensors of every loop are appended to it. If log is a writable text
        file, one JSON line per loop -- {"loop", "ms" (HIP events around the
        loop on the stream), "accepted" and "emitted" per sequence, -1 / 0 for
        sequences already done} -- and one summary line at the end ({"run":
        tokens, loops, seconds, tokens per second, mean accepted per loop})
        are written (the paper logs the tokens each loop generates)."""
        import json
        import time
        dev = self.ctx.device
        seq = torch.zeros((self.B, n_new), dtype=torch.int32, device=dev)
        n_out = torch.zeros(self.B, dtype=torch.int32, device=dev)
        loop_index = loop0
        t0 = time.perf_counter()
        acc_sum, acc_n = 0, 0
        while True:
            remaining = n_new - int(n_out.min().item())
            if remaining <= 0:
                break
            burst = []
            for _ in range(max(1, -(-remaining // (self.K + 1)))):
                want = accepted_log is not None or log is not None
                done = (n_out >= n_new).clone() if want else None
                before = n_out.clone() if log is not None else None
                ev = None
                if log is not None:
                    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    ev[0].record()
                self.loop(temperature, seed, loop_index, seq, n_out, n_new, top_k, top_p)
                if log is not None:
                    ev[1].record()
                    burst.append((loop_index, ev, self.n_acc.clone(), done, before, n_out.clone()))
                if accepted_log is not None:
                    accepted_log.append((self.n_acc.clone(), done))
                loop_index += 1
            for li, ev, a, done, before, after in burst:   # resolved once the burst has run
                ev[1].synchronize()
                live = ~done
                acc = [int(x) if bool(l) else -1 for x, l in zip(a.tolist(), live.tolist())]
                emitted = (after - before).tolist()
                acc_sum += sum(x for x in acc if x >= 0)
                acc_n += sum(1 for x in acc if x >= 0)
                log.write(json.dumps({"loop": li, "ms": round(ev[0].elapsed_time(ev[1]), 4), "accepted": acc,
                                      "emitted": emitted}) + "\n")
        self.loops = loop_index
        if log is not None:
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            log.write(json.dumps({"run": {"tokens": n_new * self.B, "loops": loop_index - loop0,
                                          "seconds": round(wall, 6), "tokens_per_s": round(n_new * self.B / wall, 3),
                                          "mean_accepted": round(acc_sum / max(acc_n, 1), 4)}}) + "\n")
            log.flush()
        return seq
