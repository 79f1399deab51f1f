// Softmax with temperature, the fused accept / resample kernel of modified
// rejection sampling, draft-token sampling, the end-of-loop commit, and
// Philox uniforms.
//
// Categorical draws use an integer inverse CDF so that a parallel scan gives
// exactly the result of a serial loop: weights w_i = floor(x_i 2^32) for
// probabilities x_i (0 for x_i <= 0 or NaN, 2^32 for x_i >= 1), total W,
// threshold t = floor(m W / 2^24) for the grid index m = floor(u 2^24) of the
// uniform, result = smallest i whose inclusive prefix sum exceeds t. Each
// thread owns a contiguous chunk of the vocabulary; one block-wide uint64
// scan gives every chunk its exclusive prefix, and the one chunk containing
// the threshold is walked serially.
#include "common.h"
#include "launch.h"
#include "philox.h"

namespace sps {

constexpr int kSampleThreads = 1024;

__device__ __forceinline__ uint64_t fixed_weight(float x) {
  if (!(x > 0.f)) return 0;
  if (x >= 1.f) return 1ull << 32;
  return static_cast<uint64_t>(static_cast<double>(x) * 4294967296.0);
}

__device__ __forceinline__ uint64_t grid_threshold(float u, uint64_t W) {
  uint64_t m;
  if (!(u > 0.f)) m = 0;
  else if (u >= 1.f) m = (1u << 24) - 1;
  else m = static_cast<uint64_t>(u * 16777216.0f);
  return m * (W >> 24) + ((m * (W & 0xFFFFFFull)) >> 24);
}

// Row statistics of softmax(z / T): (max of z/T, sum of exp(z/T - max)); for
// T == 0 (greedy) (index of the first maximum, -1).
struct RowStat { float a, b; };

// Probability of entry i of a row. The same expression (no contraction) is
// used wherever q or p is materialised, so exported probabilities and the
// values the accept test sees are identical bit for bit.
__device__ __forceinline__ float prob_of(float z, RowStat st, float inv_t, int i) {
  if (st.b < 0.f) return i == static_cast<int>(st.a) ? 1.f : 0.f;
  const float t = __fsub_rn(__fmul_rn(z, inv_t), st.a);
  return __fdiv_rn(expf(t), st.b);
}

__device__ RowStat row_stat(const float* __restrict__ z, int V, float temperature, float* red, int* ired) {
  RowStat st;
  if (temperature == 0.f) {
    float best = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = threadIdx.x; i < V; i += blockDim.x) {
      const float v = z[i];
      if (v > best || (bi == 0x7fffffff)) { best = v; bi = i; }
    }
    // arg-max with the lowest index on ties
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o);
      const int oi = __shfl_xor(bi, o);
      if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) { red[threadIdx.x >> 6] = best; ired[threadIdx.x >> 6] = bi; }
    __syncthreads();
    best = red[0]; bi = ired[0];
    for (int w = 1; w < static_cast<int>(blockDim.x >> 6); ++w)
      if (red[w] > best || (red[w] == best && ired[w] < bi)) { best = red[w]; bi = ired[w]; }
    st.a = static_cast<float>(bi);
    st.b = -1.f;
    return st;
  }
  const float inv_t = 1.0f / temperature;
  float mx = -INFINITY;
  for (int i = threadIdx.x; i < V; i += blockDim.x) mx = fmaxf(mx, __fmul_rn(z[i], inv_t));
  mx = block_max(mx, red);
  float s = 0.f;
  for (int i = threadIdx.x; i < V; i += blockDim.x) s += expf(__fsub_rn(__fmul_rn(z[i], inv_t), mx));
  s = block_sum(s, red);
  st.a = mx;
  st.b = s;
  return st;
}

__global__ __launch_bounds__(kSampleThreads) void row_softmax_kernel(const float* __restrict__ logits, int V,
                                                                     float temperature, RowStat* __restrict__ stats,
                                                                     float* __restrict__ probs) {
  __shared__ float red[16];
  __shared__ int ired[16];
  const int row = blockIdx.x;
  const float* z = logits + static_cast<size_t>(row) * V;
  const RowStat st = row_stat(z, V, temperature, red, ired);
  if (threadIdx.x == 0 && stats) stats[row] = st;
  if (probs) {
    const float inv_t = temperature == 0.f ? 0.f : 1.0f / temperature;
    float* pr = probs + static_cast<size_t>(row) * V;
    for (int i = threadIdx.x; i < V; i += blockDim.x) pr[i] = prob_of(z[i], st, inv_t, i);
  }
}

// Target probabilities given as a [rows][V] array.
struct QProbs {
  const float* q;
  int V;
  __device__ float operator()(int row, int i) const { return q[static_cast<size_t>(row) * V + i]; }
};
// Target probabilities formed on the fly from logits and row statistics.
struct QLogits {
  const float* z;
  const RowStat* st;
  float inv_t;
  int V;
  __device__ float operator()(int row, int i) const {
    return prob_of(z[static_cast<size_t>(row) * V + i], st[row], inv_t, i);
  }
};

// One block per sequence. drafts[b * dstride + doff + t] is x~_{t+1}.
template <class QS>
__global__ __launch_bounds__(kSampleThreads) void accept_kernel(QS qs, const float* __restrict__ p,
                                                                const int32_t* __restrict__ drafts, int dstride,
                                                                int doff, const float* __restrict__ unif,
                                                                uint64_t seed, uint64_t loop, int K, int V,
                                                                int32_t* __restrict__ out,
                                                                int32_t* __restrict__ n_acc, int* err) {
  __shared__ int s_a, s_y;
  __shared__ uint64_t wsum[17];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int32_t* dr = drafts + static_cast<size_t>(b) * dstride + doff;

  // 1. left-to-right accept tests r_t * p_t(x~_t) < q_t(x~_t), exact in fp64
  if (tid < 64) {
    bool rejected = false, bad = false;
    if (tid < K) {
      const int x = dr[tid];
      if (x < 0 || x >= V) {
        bad = true;
        rejected = true;
      } else {
        const float rho = qs(b * (K + 1) + tid, x);
        const float pi = p[(static_cast<size_t>(b) * K + tid) * V + x];
        const float r = unif ? unif[b * (K + 1) + tid] : philox_uniform(seed, loop, 1, b, tid);
        rejected = !(static_cast<double>(r) * static_cast<double>(pi) < static_cast<double>(rho));
      }
    }
    const uint64_t rej = __ballot(rejected);
    const int a = rej ? __ffsll(static_cast<long long>(rej)) - 1 : K;
    if (tid == a && bad) atomicOr(err, kErrBadToken);
    if (tid == 0) { s_a = a; s_y = 0; }
  }
  __syncthreads();
  const int a = s_a;
  const int row = b * (K + 1) + a;
  const bool resid = a < K;
  const float* prow = p + (static_cast<size_t>(b) * K + (resid ? a : 0)) * V;

  // 2. weights of (q - p)_+ (or q for the bonus / the zero-residual fallback)
  const int C = (V + blockDim.x - 1) / blockDim.x;
  const int i0 = min(V, tid * C), i1 = min(V, i0 + C);
  auto weight = [&](int i, bool use_resid) -> uint64_t {
    const uint64_t wq = fixed_weight(qs(row, i));
    if (!use_resid) return wq;
    const uint64_t wp = fixed_weight(prow[i]);
    return wq > wp ? wq - wp : 0;
  };
  bool use_resid = resid;
  uint64_t loc = 0;
  for (int i = i0; i < i1; ++i) loc += weight(i, use_resid);
  uint64_t W;
  uint64_t ex = block_exscan_u64(loc, wsum, &W);
  if (use_resid && W == 0) {
    use_resid = false;
    loc = 0;
    for (int i = i0; i < i1; ++i) loc += weight(i, false);
    ex = block_exscan_u64(loc, wsum, &W);
  }

  // 3. inverse CDF draw
  if (W > 0) {
    const float u = unif ? unif[b * (K + 1) + K] : philox_uniform(seed, loop, 2, b, 0);
    const uint64_t thr = grid_threshold(u, W);
    if (ex <= thr && thr < ex + loc) {
      uint64_t acc = ex;
      for (int i = i0; i < i1; ++i) {
        acc += weight(i, use_resid);
        if (acc > thr) { s_y = i; break; }
      }
    }
  } else if (tid == 0) {
    atomicOr(err, kErrEmpty);
  }
  __syncthreads();
  if (tid <= K) out[static_cast<size_t>(b) * (K + 1) + tid] = tid < a ? dr[tid] : (tid == a ? s_y : -1);
  if (tid == 0) n_acc[b] = a;
}

// Draft step t: p_t = softmax(logits of the last row of each sequence / T),
// written to p_out[b][t][:], and x~_{t+1} drawn from it into tokens[b][t+1].
__global__ __launch_bounds__(kSampleThreads) void draft_sample_kernel(
    const float* __restrict__ logits, int Mps, int V, float temperature, float* __restrict__ p_out, int K, int t,
    int32_t* __restrict__ tokens, const int32_t* __restrict__ ctx, uint64_t seed, uint64_t loop, int* err) {
  __shared__ float red[16];
  __shared__ int ired[16];
  __shared__ uint64_t wsum[17];
  __shared__ int s_y;
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* z = logits + (static_cast<size_t>(b) * Mps + Mps - 1) * V;
  const RowStat st = row_stat(z, V, temperature, red, ired);
  const float inv_t = temperature == 0.f ? 0.f : 1.0f / temperature;
  float* pr = p_out + (static_cast<size_t>(b) * K + t) * V;
  for (int i = tid; i < V; i += blockDim.x) pr[i] = prob_of(z[i], st, inv_t, i);
  const int C = (V + blockDim.x - 1) / blockDim.x;
  const int i0 = min(V, tid * C), i1 = min(V, i0 + C);
  uint64_t loc = 0;
  for (int i = i0; i < i1; ++i) loc += fixed_weight(prob_of(z[i], st, inv_t, i));
  uint64_t W;
  const uint64_t ex = block_exscan_u64(loc, wsum, &W);
  if (tid == 0) s_y = 0;
  __syncthreads();
  if (W > 0) {
    const uint64_t thr = grid_threshold(philox_uniform(seed, loop, 0, b, t), W);
    if (ex <= thr && thr < ex + loc) {
      uint64_t acc = ex;
      for (int i = i0; i < i1; ++i) {
        acc += fixed_weight(prob_of(z[i], st, inv_t, i));
        if (acc > thr) { s_y = i; break; }
      }
    }
  } else if (tid == 0) {
    atomicOr(err, kErrEmpty);
  }
  __syncthreads();
  if (tid == 0) {
    tokens[static_cast<size_t>(b) * (K + 1) + t + 1] = s_y;
    if (t == 0) tokens[static_cast<size_t>(b) * (K + 1)] = ctx[2 * b + 1];
  }
}

__global__ void commit_kernel(int32_t* __restrict__ lengths, const int32_t* __restrict__ tokens,
                              const int32_t* __restrict__ out, const int32_t* __restrict__ n_acc, int B, int K,
                              int32_t* __restrict__ ctx, int32_t* __restrict__ seq_out, int32_t* __restrict__ n_out,
                              int cap) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int a = n_acc[b];
  a = a < 0 ? 0 : (a > K ? K : a);
  if (n_out) {
    const int n = n_out[b];
    if (n >= cap) return;
    int w = n;
    for (int i = 0; i <= a && w < cap; ++i, ++w) seq_out[static_cast<size_t>(b) * cap + w] = out[b * (K + 1) + i];
    n_out[b] = w;
  }
  lengths[b] += a + 1;
  ctx[2 * b] = tokens[b * (K + 1) + a];
  ctx[2 * b + 1] = out[b * (K + 1) + a];
}

__global__ void philox_kernel(uint64_t seed, uint64_t loop, int purpose, int B, int n, float* __restrict__ out) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(B) * n) return;
  out[i] = philox_uniform(seed, loop, static_cast<uint32_t>(purpose), static_cast<uint32_t>(i / n),
                          static_cast<uint32_t>(i % n));
}

hipError_t launch_row_softmax(const float* logits, int rows, int V, float temperature, float* stats, float* probs,
                              hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(row_softmax_kernel, dim3(rows), dim3(kSampleThreads), 0, st, logits, V, temperature,
                     reinterpret_cast<RowStat*>(stats), probs);
  return hipGetLastError();
}

hipError_t launch_accept_probs(const float* p, const float* q, const int32_t* drafts, const float* unif,
                               uint64_t seed, uint64_t loop, int B, int K, int V, int32_t* out, int32_t* n_acc,
                               int* err, hipStream_t st) {
  hipLaunchKernelGGL(accept_kernel<QProbs>, dim3(B), dim3(kSampleThreads), 0, st, QProbs{q, V}, p, drafts, K, 0,
                     unif, seed, loop, K, V, out, n_acc, err);
  return hipGetLastError();
}

hipError_t launch_accept_logits(const float* p, const float* logits, const float* stats, float temperature,
                                const int32_t* tokens, const float* unif, uint64_t seed, uint64_t loop, int B,
                                int K, int V, int32_t* out, int32_t* n_acc, int* err, hipStream_t st) {
  const float inv_t = temperature == 0.f ? 0.f : 1.0f / temperature;
  const QLogits qs{logits, reinterpret_cast<const RowStat*>(stats), inv_t, V};
  hipLaunchKernelGGL(accept_kernel<QLogits>, dim3(B), dim3(kSampleThreads), 0, st, qs, p, tokens, K + 1, 1, unif,
                     seed, loop, K, V, out, n_acc, err);
  return hipGetLastError();
}

hipError_t launch_draft_sample(const float* logits, int Mps, int B, int V, float temperature, float* p_out, int K,
                               int t, int32_t* tokens, const int32_t* ctx, uint64_t seed, uint64_t loop, int* err,
                               hipStream_t st) {
  hipLaunchKernelGGL(draft_sample_kernel, dim3(B), dim3(kSampleThreads), 0, st, logits, Mps, V, temperature, p_out,
                     K, t, tokens, ctx, seed, loop, err);
  return hipGetLastError();
}

hipError_t launch_commit(int32_t* lengths, const int32_t* tokens, const int32_t* out, const int32_t* n_acc, int B,
                         int K, int32_t* ctx, int32_t* seq_out, int32_t* n_out, int cap, hipStream_t st) {
  hipLaunchKernelGGL(commit_kernel, dim3((B + 255) / 256), dim3(256), 0, st, lengths, tokens, out, n_acc, B, K, ctx,
                     seq_out, n_out, cap);
  return hipGetLastError();
}

__global__ void ctx_tokens_kernel(const int32_t* __restrict__ ctx, int B, int K, int32_t* __restrict__ tokens) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) tokens[static_cast<size_t>(b) * (K + 1)] = ctx[2 * b + 1];
}

hipError_t launch_ctx_tokens(const int32_t* ctx, int B, int K, int32_t* tokens, hipStream_t st) {
  hipLaunchKernelGGL(ctx_tokens_kernel, dim3((B + 255) / 256), dim3(256), 0, st, ctx, B, K, tokens);
  return hipGetLastError();
}

hipError_t launch_philox(uint64_t seed, uint64_t loop, int purpose, int B, int n, float* out, hipStream_t st) {
  const long work = static_cast<long>(B) * n;
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(philox_kernel, dim3(static_cast<unsigned>((work + 255) / 256)), dim3(256), 0, st, seed, loop,
                     purpose, B, n, out);
  return hipGetLastError();
}

}  // namespace sps
