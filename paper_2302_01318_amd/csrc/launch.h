// Host-side launchers of the libsps kernels (internal; not part of the ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sps {

enum Epilogue { kEpiStore = 0, kEpiGelu = 1, kEpiSwiglu = 2 };

// Y = X W^T for a packed weight W (see gemm.hip). dtype: 0 fp32, 1 bf16.
//   kEpiStore : out[s][m][n] (fp32, row stride ldo) for split s of S
//   kEpiGelu  : act[m][n] = gelu_tanh(Y[m][n])            (S must be 1)
//   kEpiSwiglu: act[m][c] = silu(Y[m][gate c]) * Y[m][up c] (S must be 1)
// X and act are in the activation format (common.h: fp32, or bf16 hi/lo
// planes `xplane` / `aplane` elements apart); W is fp32 or bf16; split s of
// the output lives at out + s * oplane.
struct GemmArgs {
  const void* X; int ldx; size_t xplane; int M;
  const void* W; int N; int KT;   // N: packed rows (16-padded as stored), KT = K / 32
  int n_valid;                    // logical output columns written (<= N; SwiGLU: F)
  int S;
  float* out; int ldo; size_t oplane;
  void* act; int lda; size_t aplane;
  int epi;
};
hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t st);
int gemm_max_rows(int dtype);   // rows one launch handles (larger M: several launches)
int gemm_splits(int dtype, int NT, int KT, int M, int epi);

// Pack canonical rows src[n][k] (n < n_src, k < Kd) into tile order. Row n goes
// to packed row map(n): kind 0: row_off + n; kind 1: (n/8)*16 + row_off*8 + n%8
// (SwiGLU gate: row_off 0, up: row_off 1). Rows [zero_from, zero_to) are
// cleared.
hipError_t launch_pack(int dtype, const void* src, int n_src, int Kd, void* dst, int KT, int kind,
                       int row_off, int zero_from, int zero_to, hipStream_t st);

// Activations (x, attention output o, FFN hidden) are in the activation
// format of common.h; `xplane` is the element distance of the lo plane.
hipError_t launch_embed_norm(int dtype, const int32_t* tokens, int tok_stride, int Mps, int M,
                             const void* E, int V, int d, const float* gain, float eps, float* h,
                             void* x, size_t xplane, int* err, hipStream_t st);
hipError_t launch_add_norm(int dtype, float* h, const float* part, int S, int M, int d,
                           const float* gain, float eps, void* x, size_t xplane, hipStream_t st);
hipError_t launch_rope_kv(int dtype, const float* qkvp, int S, int M, int H, int DH, int Mps,
                          const int32_t* lengths, int pos_offset, float rope_base, void* qout,
                          void* kc, void* vc, int T_cap, int* err, hipStream_t st);
hipError_t launch_attention(int dtype, const void* q, const void* kc, const void* vc,
                            const int32_t* lengths, int pos_offset, int B, int Mps, int H, int DH,
                            int T_cap, float* part, void* o, size_t oplane, hipStream_t st);
int attn_partials(int T_cap);
hipError_t launch_kv_copy(int dtype, int to_cache, void* kc, void* vc, int H, int DH, int T_cap,
                          int pos0, int n, void* k, void* v, hipStream_t st);

// Sampling.
hipError_t launch_row_softmax(const float* logits, int rows, int V, float temperature,
                              float* stats, float* probs, hipStream_t st);
hipError_t launch_accept_probs(const float* p, const float* q, const int32_t* drafts,
                               const float* unif, uint64_t seed, uint64_t loop, int B, int K,
                               int V, int32_t* out, int32_t* n_acc, int* err, hipStream_t st);
hipError_t launch_accept_logits(const float* p, const float* logits, const float* stats,
                                float temperature, const int32_t* tokens, const float* unif,
                                uint64_t seed, uint64_t loop, int B, int K, int V, int32_t* out,
                                int32_t* n_acc, int* err, hipStream_t st);
hipError_t launch_draft_sample(const float* logits, int Mps, int B, int V, float temperature,
                               float* p_out, int K, int t, int32_t* tokens, const int32_t* ctx,
                               uint64_t seed, uint64_t loop, int* err, hipStream_t st);
hipError_t launch_commit(int32_t* lengths, const int32_t* tokens, const int32_t* out,
                         const int32_t* n_acc, int B, int K, int32_t* ctx, int32_t* seq_out,
                         int32_t* n_out, int cap, hipStream_t st);
hipError_t launch_ctx_tokens(const int32_t* ctx, int B, int K, int32_t* tokens, hipStream_t st);
hipError_t launch_philox(uint64_t seed, uint64_t loop, int purpose, int B, int n, float* out,
                         hipStream_t st);

}  // namespace sps
