/*
 * sps.h -- C ABI of libsps, the MI355X (gfx950) speculative-sampling library.
 *
 * Speculative sampling (SpS), Chen et al. 2023, "Accelerating Large Language
 * Model Decoding with Speculative Sampling". Notation follows the paper:
 * q is the TARGET model, p is the DRAFT model, K is the lookahead.
 *
 * Conventions shared by every entry point
 *  - Buffers named in the argument lists are DEVICE pointers unless a
 *    comment says "host". The caller owns and frees all of them; the library
 *    never frees a caller buffer and never allocates device memory.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Calls enqueue work on it and return without synchronising, except
 *    sps_device_error, which synchronises the stream.
 *  - Every call validates its host-side arguments before any HIP call and
 *    returns an sps_status; nothing aborts and nothing throws. Validation
 *    failures leave device memory untouched.
 *  - Errors that only the device can see (a token id outside [0, V), a KV
 *    position at or beyond the cache capacity, a distribution whose weights
 *    are all zero, a NaN or infinite logit or probability) set a sticky
 *    per-device flag read by sps_device_error. The kernels then write
 *    defined outputs and make no out-of-bounds access.
 *  - Handles (sps_model_t, sps_kv_t) are small host objects holding a
 *    configuration and non-owning device pointers. They are not thread safe.
 *  - Calls that share a workspace or a KV cache must not run concurrently.
 */
#ifndef SPS_H
#define SPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPS_OK = 0,
  SPS_E_INVALID = 1,      /* null pointer, negative size, bad enum value      */
  SPS_E_SHAPE = 2,        /* shape the kernels do not support (see sps_config) */
  SPS_E_CAPACITY = 3,     /* workspace / KV buffer too small                   */
  SPS_E_UNSUPPORTED = 4,  /* valid request the library does not implement     */
  SPS_E_HIP = 5           /* a HIP runtime call or kernel launch failed       */
} sps_status;

/* Device error flag bits reported by sps_device_error. */
#define SPS_DEV_BAD_TOKEN 1  /* token id outside [0, V)                        */
#define SPS_DEV_EMPTY 2      /* categorical draw with all weights zero         */
#define SPS_DEV_CAPACITY 4   /* KV write at a position >= T_cap (write skipped) */
/* A row of logits with a NaN or +Inf entry (or one that overflows to +Inf
 * when divided by the temperature) has no distribution: its probabilities
 * are defined as one-hot at token 0 (exported q / p rows, draft draws). In
 * modified rejection sampling a sequence with such a target row, or with a
 * NaN or infinite value among the probabilities the accept tests and the
 * final draw read, is given a = 0 accepted drafts and token 0. -Inf logits
 * are valid (probability 0). The paper's method assumes valid distributions
 * (Modified Rejection Sampling section); this is the library's definition
 * for inputs that are not. */
#define SPS_DEV_NONFINITE 8

enum { SPS_FFN_GELU = 0, SPS_FFN_SWIGLU = 1 };
enum { SPS_DTYPE_F32 = 0, SPS_DTYPE_BF16 = 1, SPS_DTYPE_FP8 = 2 };

/* Decoder-only transformer shape (Conditional Scoring section; Hyperparams
 * table). Pre-norm blocks, RMSNorm with learned gains, multi-head attention
 * with rotate-half rotary position encoding, FFN = GELU(tanh) with two
 * matrices or SwiGLU with three, untied embedding / unembedding, no biases.
 * Supported: d_model % 32 == 0, d_model <= 16384, head_dim in {64, 128},
 * (n_heads * head_dim) % 32 == 0, d_ff % 32 == 0, 2 <= vocab < 2^24,
 * 1 <= n_layers <= 4096, 1 <= n_heads <= 1024, d_ff <= 2^20.
 *
 * dtype SPS_DTYPE_FP8 is a weight-only FP8 model (the paper notes SpS is
 * compatible with quantisation: Introduction; Modified Rejection Sampling
 * section): the projection matrices (WQ, WK, WV, WO, W1, W3, W2, UNEMBED)
 * are OCP FP8 E4M3 codes (bias 7, subnormals, no infinities, max 448) with
 * one fp32 scale per output row; the embedding, the KV cache and the
 * activations are those of a bf16 model, the gains fp32. It needs d_model,
 * n_heads * head_dim and d_ff to be multiples of 64. */
typedef struct {
  int32_t d_model, n_layers, n_heads, head_dim, d_ff, vocab;
  int32_t ffn_kind; /* SPS_FFN_GELU or SPS_FFN_SWIGLU                         */
  int32_t dtype;    /* SPS_DTYPE_F32 / _BF16: weights, KV, GEMM inputs; _FP8 above */
  float rms_eps;    /* e.g. 1e-5                                                */
  float rope_base;  /* e.g. 10000                                               */
} sps_config;

/* Counter-based randomness: Philox4x64-10 (Salmon et al., SC'11) keyed by
 * (seed, 0) with counter (j, b, loop, purpose). The uniform is the top 24
 * bits of output word 0 times 2^-24. `loop` is the SpS loop index. */
typedef struct {
  uint64_t seed;
  uint64_t loop;
} sps_philox;

enum { SPS_PURPOSE_DRAFT = 0, SPS_PURPOSE_ACCEPT = 1, SPS_PURPOSE_RESAMPLE = 2 };

/* Probability modifiers applied alike to the draft and the target
 * distributions before modified rejection sampling (Modified Rejection
 * Sampling section, closing paragraph; Table 1 uses nucleus sampling):
 *  - temperature T >= 0: softmax(logits / T); T == 0 is greedy (one-hot
 *    argmax, lowest index on ties; top_k / top_p are then ignored);
 *  - top_k: keep the top_k highest-ranked entries (0 or >= V: off);
 *  - top_p in [0, 1]: nucleus -- among what top-k kept, keep the shortest
 *    prefix of the ranking whose mass reaches top_p, at least one entry
 *    (1: off).
 * Ranking is by the draw weight floor(x 2^32), larger first, ties by lower
 * index; masses are integer sums of those weights and the nucleus threshold
 * is floor(floor(top_p 2^24) W / 2^24) of the kept total W; kept entries are
 * renormalised as x / (fp32(S) 2^-32) with S their exact integer weight sum.
 * With either modifier on, V must be <= 32768 (SPS_E_UNSUPPORTED else). */
typedef struct {
  float temperature;
  int32_t top_k;
  float top_p;
} sps_sampling;

/* Weight tensors, in canonical row-major nn.Linear orientation [out][in] and
 * the model dtype (bf16 for every matrix of an FP8 model), except the gains
 * (always fp32):
 *   EMBED [V][d], FINAL_NORM [d], UNEMBED [V][d],
 *   per layer: ATTN_NORM [d], WQ/WK/WV [H*Dh][d], WO [d][H*Dh], FFN_NORM [d],
 *   W1 [F][d] (GELU up, or SwiGLU gate), W3 [F][d] (SwiGLU up only),
 *   W2 [d][F] (down). */
enum {
  SPS_W_EMBED = 0, SPS_W_FINAL_NORM = 1, SPS_W_UNEMBED = 2,
  SPS_W_ATTN_NORM = 3, SPS_W_Q = 4, SPS_W_K = 5, SPS_W_V = 6, SPS_W_O = 7,
  SPS_W_FFN_NORM = 8, SPS_W_1 = 9, SPS_W_3 = 10, SPS_W_2 = 11
};

typedef struct sps_model_s* sps_model_t;
typedef struct sps_kv_s* sps_kv_t;

const char* sps_status_string(int32_t status);
int32_t sps_abi_version(void);

/* ---- model weights --------------------------------------------------- */

/* Bytes of the packed weight buffer for cfg (0 if cfg is invalid). The packed
 * layout stores every projection as 16 x 32 tiles in the register order of
 * the gfx950 MFMA B operand, so each wavefront load is one contiguous KiB.
 * FP8 models store 16 x 64 tiles of one-byte codes (lane l: row l % 16,
 * columns 8 (l / 16) .. +7 of the tile's first 32 columns, then the same
 * columns of its second 32), each projection followed by its fp32 row
 * scales in packed row order. */
size_t sps_weight_bytes(const sps_config* cfg);

/* Pack one canonical tensor `src` (layout above) into its slot of the packed
 * buffer `packed` (sps_weight_bytes(cfg) bytes). `layer` is ignored for
 * EMBED, FINAL_NORM and UNEMBED. W3 is only valid for SwiGLU. Every tensor
 * of the model must be packed once before the model is used.
 * FP8 models quantise each bf16 matrix row n here: scale s_n = fp32(max_k
 * |w[n][k]|) / 448 (1 for an all-zero row), code = the E4M3 value nearest to
 * fp32(w[n][k]) / s_n (fp32 divisions, correctly rounded), ties to the even
 * code, |quotient| clamped to 448 first; the model computes with
 * s_n * value(code). */
sps_status sps_pack_weight(const sps_config* cfg, int32_t tensor, int32_t layer,
                           const void* src, void* packed, void* stream);

/* Where tensor `tensor` of layer `layer` lives in the packed buffer (host
 * outputs): its slot's byte offset and size, and for the projections of an
 * FP8 model the byte offset of their fp32 row scales (0 otherwise). WQ, WK
 * and WV share the fused QKV slot (packed rows: q and k heads with rotary
 * partners side by side, then v), W1 and W3 of a SwiGLU model the
 * interleaved gate / up slot (8 gate rows, then the matching 8 up rows). */
sps_status sps_weight_slot(const sps_config* cfg, int32_t tensor, int32_t layer, size_t* offset /*host*/,
                           size_t* bytes /*host*/, size_t* scale_offset /*host*/);

/* Create a host handle viewing `packed` (not copied, not owned). */
sps_status sps_model_create(const sps_config* cfg, void* packed, sps_model_t* out /*host*/);
void sps_model_destroy(sps_model_t model);

/* ---- KV cache -------------------------------------------------------- */

/* Bytes of a KV cache for B sequences of capacity T_cap positions
 * (T_cap % 32 == 0, 32 <= T_cap <= 2^22; 0 otherwise). Layout per (layer,
 * sequence, head): keys in 16-position x 32-dim MFMA tiles, values in
 * 32-position x 16-dim tiles, both in the register order of the attention
 * kernel's MFMA operands. */
size_t sps_kv_bytes(const sps_config* cfg, int32_t B, int32_t T_cap);

/* Create a handle over `kv_buf` (sps_kv_bytes bytes) and `lengths`, a device
 * int32 [B] array of committed lengths that the caller initialises. A draft
 * and a target cache of the same batch share one `lengths` array: positions
 * are the same token positions in both. SPS_E_SHAPE for a T_cap that is not
 * a multiple of 32 in [32, 2^22]. */
sps_status sps_kv_create(const sps_config* cfg, int32_t B, int32_t T_cap, void* kv_buf,
                         int32_t* lengths, sps_kv_t* out /*host*/);
void sps_kv_destroy(sps_kv_t kv);

/* Copy n positions starting at pos0 of sequence b, layer `layer`, between
 * canonical buffers k/v [H][n][Dh] (model dtype; keys already rotated) and
 * the cache. Used to install a synthetic prior context and by tests. */
sps_status sps_kv_write(sps_kv_t kv, int32_t layer, int32_t b, int32_t pos0, int32_t n,
                        const void* k_src, const void* v_src, void* stream);
sps_status sps_kv_read(sps_kv_t kv, int32_t layer, int32_t b, int32_t pos0, int32_t n,
                       void* k_dst, void* v_dst, void* stream);

/* ---- workspace ------------------------------------------------------- */

/* Bytes of scratch a forward / verify / draft call needs for B sequences of
 * up to max_tokens_per_seq new tokens each against a cache of capacity
 * T_cap: any call with B sequences and at most that many tokens per sequence
 * (a verify step takes K + 1, a draft step 2) fits. 0 for an invalid config,
 * T_cap outside [32, 2^22], or a request no call admits (max_tokens_per_seq > 64 or
 * B * max_tokens_per_seq > 160). */
size_t sps_workspace_bytes(const sps_config* cfg, int32_t B, int32_t max_tokens_per_seq,
                           int32_t T_cap);

/* ---- the SpS hot path -------------------------------------------------- */

/* Transformer forward over M new tokens per sequence (Conditional Scoring
 * section): tokens[b * tok_stride + j] sits at position
 * lengths[b] + pos_offset + j. Writes their keys/values into the cache
 * (lengths are NOT advanced) and, if logits_out != NULL, the fp32 logits
 * [B][M][V]. With logits_out == NULL the final norm and unembedding are
 * skipped (prompt prefill). */
sps_status sps_forward(sps_model_t model, sps_kv_t kv, const int32_t* tokens, int32_t tok_stride,
                       int32_t B, int32_t M, int32_t pos_offset, float* logits_out,
                       void* workspace, size_t ws_bytes, void* stream);

/* Outputs of the fused accept / resample stage (Modified Rejection Sampling). */
typedef struct {
  const float* p_draft; /* [B][K][V] fp32: the exact draft distributions the
                           draft tokens were sampled from                       */
  const float* uniforms;/* [B][K+1]: r_1..r_K then u; NULL = draw from rng     */
  sps_philox rng;       /* used when uniforms == NULL                           */
  int32_t* out_tokens;  /* [B][K+1]: x~_1..x~_a, then the resampled or bonus
                           token, then -1 padding                               */
  int32_t* n_accepted;  /* [B]: a in [0, K]; a + 1 tokens are emitted           */
} sps_accept_io;

/* The SpS verify step (Algorithm 2): one target forward over
 * tokens[b] = (x_n, x~_1..x~_K) ([B][K+1] int32) at positions
 * lengths[b]..lengths[b]+K, i.e. the K+1 conditionals q(.|x_1..x_n),
 * ..., q(.|x_1..x_n, x~_1..x~_K) in one call; then q = the modified
 * softmax(logits / T) of `sampling` and, if acc != NULL, the
 * modified rejection sampling of the drafts. K == 0 is auto-regressive
 * sampling (Algorithm 1): one token drawn from q. logits_out [B][K+1][V] and
 * q_out [B][K+1][V] are optional. KV entries are written but lengths are not
 * advanced (see sps_commit). */
sps_status sps_verify_step(sps_model_t target, sps_kv_t kv, const int32_t* tokens, int32_t B,
                           int32_t K, sps_sampling sampling, float* logits_out, float* q_out,
                           const sps_accept_io* acc, void* workspace, size_t ws_bytes,
                           void* stream);

/* sps_verify_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). The library keeps the scratch in a
 * device array of 64 MiB per device, reserved when the library's code is
 * loaded on that device and held until the process ends; the call itself
 * allocates nothing. Calls whose workspace (sps_workspace_bytes(cfg, B,
 * K + 1, T_cap)) exceeds 64 MiB return SPS_E_CAPACITY and touch nothing
 * (the 70B shape at B = 1, K = 4 fits caches of up to 24k positions, B = 4
 * at 2k). Every
 * call on a device shares that device's array: calls that overlap on one
 * device (on concurrent streams, or from several threads) race, and must
 * be serialised by the caller. Same arguments, outputs and errors as
 * sps_verify_step otherwise; no contents of the array carry over between
 * calls. */
sps_status sps_verify_step_noalloc(sps_model_t target, sps_kv_t kv, const int32_t* tokens, int32_t B,
                                   int32_t K, sps_sampling sampling, float* logits_out, float* q_out,
                                   const sps_accept_io* acc, void* stream);

/* Modified rejection sampling on given distributions (Algorithm 2, accept
 * loop and final draw; Theorem 1). For each sequence, left to right, draft
 * x~_t = draft_tokens[b][t-1] is accepted iff r_t * p_t(x~_t) < q_t(x~_t),
 * evaluated exactly in fp64 (this is r < min(1, q/p) without a division).
 * At the first rejection (a = t-1 accepted) the next token is drawn from
 * (q_t - p_t)_+ (falling back to q_t if its fixed-point weights sum to 0);
 * if all K are accepted the bonus token is drawn from q_{K+1}. Draws use the
 * integer inverse CDF on weights floor(x * 2^32): the smallest index whose
 * prefix sum exceeds floor(floor(u * 2^24) * W / 2^24). Outputs are a pure
 * function of the inputs (bit-exact against the reference definition).
 * p_draft [B][K][V], q_target [B][K+1][V] fp32; draft_tokens [B][K];
 * uniforms [B][K+1] or NULL (then Philox: r_t purpose ACCEPT j=t-1, u purpose
 * RESAMPLE j=0). */
sps_status sps_accept_resample(const float* p_draft, const float* q_target,
                               const int32_t* draft_tokens, const float* uniforms,
                               sps_philox rng, int32_t B, int32_t K, int32_t V,
                               int32_t* out_tokens, int32_t* n_accepted, void* stream);

/* K auto-regressive draft samples (Algorithm 2, draft loop). ctx[b] =
 * (token at position lengths[b]-1, token at position lengths[b]) -- the
 * last committed token and the newest, not yet scored one. Step 1 runs the
 * draft over both (re-writing position lengths[b]-1 in the draft cache is
 * harmless and keeps every step one shape); step t >= 2 runs it over x~_{t-1}.
 * Each step forms p_t = the modified softmax(logits / T) of `sampling`,
 * writes it to p_out[b][t-1][:],
 * and draws x~_t with Philox purpose DRAFT, j = t-1. Writes the verify input
 * tokens[b] = (ctx[b][1], x~_1..x~_K) ([B][K+1]). Requires lengths[b] >= 1.
 * p_out is [B][K][V] fp32 with V the draft's vocabulary: a draft whose p rows
 * feed a target's verify step must have the target's vocabulary (the accept
 * ratio compares the two distributions over one token space). The
 * workspace must hold sps_workspace_bytes(cfg, B, 2, T_cap) bytes. */
sps_status sps_draft_step(sps_model_t draft, sps_kv_t kv, const int32_t* ctx, int32_t B,
                          int32_t K, sps_sampling sampling, sps_philox rng, int32_t* tokens,
                          float* p_out, void* workspace, size_t ws_bytes, void* stream);

/* End of an SpS loop (Algorithm 2: after the accept loop the sequence grows
 * by the a accepted drafts plus the resampled or bonus token, so n advances
 * by a + 1), on the device (no host synchronisation): for each
 * sequence with a = n_accepted[b], lengths[b] += a + 1, ctx[b] =
 * (tokens[b][a], out_tokens[b][a]); the a + 1 emitted tokens are appended to
 * seq_out[b][*] (capacity `cap` per sequence, int32 [B][cap]) at n_out[b].
 * A sequence whose n_out has reached `cap` is frozen (nothing changes).
 * seq_out / n_out may be NULL (then nothing is appended or frozen). */
sps_status sps_commit(sps_kv_t kv, const int32_t* tokens, const int32_t* out_tokens,
                      const int32_t* n_accepted, int32_t B, int32_t K, int32_t* ctx,
                      int32_t* seq_out, int32_t* n_out, int32_t cap, void* stream);

/* out[b][j] = Philox uniform for (rng.seed, rng.loop, purpose, b, j), [B][n]. */
sps_status sps_philox_uniforms(sps_philox rng, int32_t purpose, int32_t B, int32_t n,
                               float* out, void* stream);

/* probs[r][:] = the modified softmax(logits[r][:] / T) of `sampling` for
 * `rows` rows of V fp32 values, the same arithmetic as the q the verify step
 * feeds to acceptance. */
sps_status sps_softmax(const float* logits, int32_t rows, int32_t V, sps_sampling sampling,
                       float* probs, void* stream);

/* Measurement helpers. Between begin and end, every weight-streaming GEMM
 * launch (the linear layers: QKV, attention output, FFN, unembedding) is
 * issued `repeats` (1..64) times back to back between two HIP events on its
 * stream (the repeats amortise the event and dispatch latency so the
 * per-launch time is the kernel's own; they redo the launch's work, so a
 * residual epilogue adds its output once per repeat and a profiled forward
 * is for timing only). end
 * synchronises the events and returns the summed per-launch kernel time
 * (ms, divided by repeats), the number of distinct launches and their
 * algorithmic bytes (weights + input activations + outputs, once each).
 * Host-global state: not thread safe. */
sps_status sps_profile_gemm_begin(int32_t repeats);
sps_status sps_profile_gemm_end(float* total_ms /*host*/, int32_t* launches /*host*/,
                                double* bytes /*host*/);

/* Measurement helper: read `bytes` (a multiple of 16) of device memory at
 * `src` (16-byte aligned) once, with the same nontemporal 16-byte loads the
 * GEMMs stream their weights with, on `stream`. Nothing is written except,
 * in practice never, one word of `sink` (a device uint32). Timing this call
 * with events gives the attainable HBM read rate the verify step's kernels
 * are compared with. SPS_E_INVALID on null pointers, a misaligned `src` or
 * a size that is zero or not a multiple of 16. */
sps_status sps_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream);

/* Decode n (a multiple of 16) OCP FP8 E4M3 codes at `codes` (16-byte
 * aligned) into fp32 values `out`, with the conversion the FP8-weight GEMM
 * applies to its weight codes. SPS_E_INVALID on null pointers, misalignment
 * or a bad n. */
sps_status sps_fp8_decode(const uint8_t* codes, int32_t n, float* out, void* stream);

/* Synchronise `stream`, return the current device's sticky error bits in
 * *flags (host) and clear them if `clear` != 0. */
sps_status sps_device_error(void* stream, int32_t clear, int32_t* flags /*host*/);

#ifdef __cplusplus
}
#endif
#endif /* SPS_H */
