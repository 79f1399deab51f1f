// Host-side launchers of the libsps kernels (internal; not part of the ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"

namespace sps {

enum Epilogue { kEpiStore = 0, kEpiGelu = 1, kEpiSwiglu = 2, kEpiResid = 3, kEpiQkv = 4 };

// Y = X W^T for a packed weight W (see gemm.hip). dtype: 0 fp32, 1 bf16,
// 2 FP8 (E4M3) weight codes with per-row fp32 scales `wscale` and bf16
// activations: Y[m][n] = wscale[n] * sum_k X[m][k] value(W[n][k]).
// X, act and u are in the activation format (common.h: fp32, or bf16 hi/lo
// planes `*plane` elements apart). Rows are global rows m0 .. m0+M-1 of a
// forward over Mtot rows.
//
// Input normalisation: if ss_in != NULL, Y[m][:] *= rs[m] with
// rs[m] = 1 / sqrt(sum_g ss_in[g * Mtot + m] / d + eps) over g < ng_in.
// Since RMSNorm(h) W^T = rs * (h * gain) W^T, a normed matmul takes
// u = h * gain as its input and the scale in its epilogue.
//
//   kEpiStore : out[m][n] = Y (fp32)
//   kEpiGelu  : act[m][n] = gelu_tanh(Y[m][n])
//   kEpiSwiglu: act[m][c] = silu(Y[m][gate c]) * Y[m][up c]
//   kEpiResid : h[m][n] += Y; u[m][n] = h[m][n] * gain[n];
//               ss_out[group * Mtot + m] = sum over the group's columns of h^2
//   kEpiQkv   : rotate q, k (packed rope pairs), write q and append k, v to
//               the KV cache at the row's position
struct GemmParams {
  const void* X; int ldx; size_t xplane;
  int M, m0, Mtot;
  const void* W; int NT, KT, n_valid;
  const float* wscale;     // FP8 weights: scale of every packed row (else NULL)
  const float* ss_in; int ng_in; float inv_d, eps;
  float* out; int ldo;
  void* act; int lda; size_t aplane;
  float* h; const float* gain; void* u; int ldu; size_t uplane; float* ss_out;
  const int32_t* lengths; int pos_offset, Mps, H, DH; int T_cap;
  const float2* rope;  // (cos, sin) of the rotary angle of row gm, frequency f: rope[gm DH / 2 + f]
  void* q; void* kc; void* vc; int* err;
  float* part;             // split-K partials (wide GEMM)
  int epi;
};
hipError_t launch_gemm(int dtype, const GemmParams& p, hipStream_t st);

// Wide GEMM (bf16 activations, bf16 or FP8 weights, more than 8 rows;
// gemm_wide.hip) with the launch plan of plan.h.
hipError_t launch_gemm_wide(const GemmParams& p, const WidePlan& w, hipStream_t st);

// Pack canonical rows src[n][k] (n < n_src, k < Kd) into tile order. Row n goes
// to packed row map(n): kind 0: row_off + n; kind 1: (n/8)*16 + row_off*8 + n%8
// (SwiGLU gate: row_off 0, up: row_off 1); kind 2: rotary pairs of heads of
// `dh` dims side by side, row_off + head*dh + pi(f) (see gemm.hip). Rows
// [zero_from, zero_to) are cleared.
hipError_t launch_pack(int dtype, const void* src, int n_src, int Kd, void* dst, int KT, int kind,
                       int row_off, int dh, int zero_from, int zero_to, hipStream_t st);
// The same for an FP8 projection: bf16 rows src are quantised per row (scale
// = max |row| / 448, code = nearest E4M3 of w / scale, ties to even, clamped
// to +-448) into 16 x 64 code tiles (see gemm.hip); the scale of packed row
// map(n) goes to scales[map(n)]. Padding rows get code 0 and scale 1.
hipError_t launch_pack_fp8(const void* src, int n_src, int Kd, void* dst, float* scales, int KT, int kind,
                           int row_off, int dh, int zero_from, int zero_to, hipStream_t st);
// E4M3 codes -> fp32 values with the GEMM's conversion (n % 16 == 0).
hipError_t launch_fp8_decode(const void* codes, int n, float* out, hipStream_t st);

// Activations (x, attention output o, FFN hidden) are in the activation
// format of common.h; `xplane` is the element distance of the lo plane.
// h[m] = E[token]; u[m] = h[m] * gain; ss[m] = sum h[m]^2 (one group).
// Also fills the rotary table of the step: rope[row DH / 2 + f] = (cos,
// sin) of angle pos * base^(-2 f / DH), pos = lengths[b] + pos_offset + j.
hipError_t launch_embed(int dtype, const int32_t* tokens, int tok_stride, int Mps, int M, const void* E,
                        int V, int d, const float* gain, float* h, void* u, size_t uplane, float* ss,
                        const int32_t* lengths, int pos_offset, int DH, float rope_base, float2* rope,
                        int* err, hipStream_t st);
hipError_t launch_attention(int dtype, const void* q, const void* kc, const void* vc,
                            const int32_t* lengths, int pos_offset, int B, int Mps, int H, int DH,
                            int T_cap, float* part, void* o, size_t oplane, hipStream_t st);
hipError_t launch_kv_copy(int dtype, int to_cache, void* kc, void* vc, int H, int DH, int T_cap,
                          int pos0, int n, void* k, void* v, hipStream_t st);

// Sampling.
// Row statistics (stats, row_stat_bytes() each, may be NULL) and, if probs
// != NULL, the probabilities after temperature and the top-k / nucleus
// modifiers (top_k <= 0 or >= V: off; top_p >= 1: off). With stats and cut
// (rows x cut_row_bytes(V) bytes of scratch) given, rows with a modifier are
// cut over several CUs; otherwise one work-group per row does everything.
hipError_t launch_row_softmax(const float* logits, int rows, int V, float temperature, int top_k, float top_p,
                              void* stats, float* probs, char* cut, int* err, hipStream_t st);
hipError_t launch_accept_probs(const float* p, const float* q, const int32_t* drafts,
                               const float* unif, uint64_t seed, uint64_t loop, int B, int K,
                               int V, int32_t* out, int32_t* n_acc, int* err, hipStream_t st);
// The verify step's fused accept / resample (q from the logits and their
// row statistics). cut (B x cut_row_bytes(V) bytes of scratch), if given,
// takes the final draw over several CUs (V up to the cut-off's largest
// row); otherwise one work-group per sequence does all.
hipError_t launch_accept_logits(const float* p, const float* logits, const void* stats,
                                float temperature, const int32_t* tokens, const float* unif,
                                uint64_t seed, uint64_t loop, int B, int K, int V, int32_t* out,
                                int32_t* n_acc, char* cut, int* err, hipStream_t st);
// Draft step t: p_t of each sequence's last row into p_out and x~_{t+1}
// drawn from it. stats (B rows) and cut (B x cut_row_bytes(V)), if given,
// are scratch for the statistics, the cut (when a modifier is on), the
// export and the draw over several CUs at temperature > 0 and V up to the
// cut-off's largest row; otherwise one work-group per sequence does all.
hipError_t launch_draft_sample(const float* logits, int Mps, int B, int V, float temperature,
                               int top_k, float top_p, float* p_out, int K, int t, int32_t* tokens,
                               const int32_t* ctx, uint64_t seed, uint64_t loop, void* stats, char* cut, int* err,
                               hipStream_t st);
hipError_t launch_commit(int32_t* lengths, const int32_t* tokens, const int32_t* out,
                         const int32_t* n_acc, int B, int K, int32_t* ctx, int32_t* seq_out,
                         int32_t* n_out, int cap, hipStream_t st);
hipError_t launch_ctx_tokens(const int32_t* ctx, int B, int K, int32_t* tokens, hipStream_t st);
hipError_t launch_stream_read(const void* src, size_t n16, uint32_t* sink, hipStream_t st);
hipError_t launch_philox(uint64_t seed, uint64_t loop, int purpose, int B, int n, float* out,
                         hipStream_t st);

}  // namespace sps
