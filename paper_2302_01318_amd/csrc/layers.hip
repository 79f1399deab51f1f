// The embedding gather that starts a forward, and KV copies between
// canonical buffers and the cache's tile layout (k_offset / v_offset in
// common.h). RMSNorm, the residual adds, rotary encoding and the KV append
// run in the GEMM epilogues (gemm.hip).
#include "common.h"
#include "launch.h"

namespace sps {

// The embedding kernel uses 1024 threads per row; each thread owns up to
// kEmbedChunks groups of four consecutive elements, all loaded at once.
constexpr int kEmbedThreads = 1024;
constexpr int kEmbedChunks = 4;   // d_model <= 4 * 4 * 1024 = 16384

__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4(const bf16* p) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  return make_float4(static_cast<float>(v[0]), static_cast<float>(v[1]), static_cast<float>(v[2]),
                     static_cast<float>(v[3]));
}

// h[r] = E[token]; u[r] = h[r] * gain; ss[r] = sum h[r]^2: the first RMSNorm's
// input in the form the QKV GEMM consumes (one column group). One block per row.
template <typename T>
__global__ __launch_bounds__(kEmbedThreads) void embed_kernel(const int32_t* __restrict__ tokens, int tok_stride,
                                                              int Mps, const T* __restrict__ E, int V, int d,
                                                              const float* __restrict__ gain, float* __restrict__ h,
                                                              T* __restrict__ u, size_t uplane,
                                                              float* __restrict__ ss,
                                                              const int32_t* __restrict__ lengths, int pos_offset,
                                                              int DH, float rope_base, float2* __restrict__ rope,
                                                              int* err) {
  __shared__ float red[16];
  const int row = blockIdx.x;
  const int b = row / Mps, j = row % Mps;
  // Rotary table of this row (position lengths[b] + pos_offset + j), used by
  // the QKV epilogue of every layer: the angle and its cosine and sine in
  // double precision, rounded once to fp32.
  if (static_cast<int>(threadIdx.x) < DH / 2) {
    const int f = threadIdx.x;
    const int pos = lengths[b] + pos_offset + j;
    const double inv = exp2(-2.0 * f / DH * log2(static_cast<double>(rope_base)));
    double sn, cs;
    sincos(static_cast<double>(pos) * inv, &sn, &cs);
    rope[static_cast<size_t>(row) * (DH / 2) + f] = make_float2(static_cast<float>(cs), static_cast<float>(sn));
  }
  int tok = tokens[static_cast<size_t>(b) * tok_stride + j];
  const bool ok = tok >= 0 && tok < V;
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(err, kErrBadToken);
    tok = 0;
  }
  const T* e = E + static_cast<size_t>(tok) * d;
  float4 v[kEmbedChunks];
#pragma unroll
  for (int c = 0; c < kEmbedChunks; ++c) {
    const int i = (c * kEmbedThreads + threadIdx.x) * 4;
    v[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < d && ok) v[c] = load4(e + i);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kEmbedChunks; ++c) {
    const int i = (c * kEmbedThreads + threadIdx.x) * 4;
    if (i < d) {
      const size_t o = static_cast<size_t>(row) * d + i;
      *reinterpret_cast<float4*>(h + o) = v[c];
      const float4 g = load4(gain + i);
      store_act(u, uplane, o, v[c].x * g.x);
      store_act(u, uplane, o + 1, v[c].y * g.y);
      store_act(u, uplane, o + 2, v[c].z * g.z);
      store_act(u, uplane, o + 3, v[c].w * g.w);
      s += v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
    }
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) ss[row] = s;
}

// Canonical [H][n][DH] <-> cache tiles of one (layer, sequence).
template <typename T>
__global__ void kv_copy_kernel(int to_cache, T* __restrict__ kc, T* __restrict__ vc, int H, int DH, int T_cap,
                               int pos0, int n, T* __restrict__ k, T* __restrict__ v) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(H) * n * DH) return;
  const int hh = static_cast<int>(i / (static_cast<long>(n) * DH));
  const int p = static_cast<int>((i / DH) % n), d = static_cast<int>(i % DH);
  T* kr = kc + static_cast<size_t>(hh) * T_cap * DH;
  T* vr = vc + static_cast<size_t>(hh) * T_cap * DH;
  const size_t ko = k_offset(pos0 + p, d, DH), vo = v_offset(pos0 + p, d, DH);
  if (to_cache) { kr[ko] = k[i]; vr[vo] = v[i]; }
  else { k[i] = kr[ko]; v[i] = vr[vo]; }
}

hipError_t launch_embed(int dtype, const int32_t* tokens, int tok_stride, int Mps, int M, const void* E, int V,
                        int d, const float* gain, float* h, void* u, size_t uplane, float* ss,
                        const int32_t* lengths, int pos_offset, int DH, float rope_base, float2* rope, int* err,
                        hipStream_t st) {
  if (DH / 2 > kEmbedThreads) return hipErrorInvalidValue;
  if (dtype == 1)
    hipLaunchKernelGGL(embed_kernel<bf16>, dim3(M), dim3(kEmbedThreads), 0, st, tokens, tok_stride, Mps,
                       static_cast<const bf16*>(E), V, d, gain, h, static_cast<bf16*>(u), uplane, ss, lengths,
                       pos_offset, DH, rope_base, rope, err);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(kEmbedThreads), 0, st, tokens, tok_stride, Mps,
                       static_cast<const float*>(E), V, d, gain, h, static_cast<float*>(u), uplane, ss, lengths,
                       pos_offset, DH, rope_base, rope, err);
  return hipGetLastError();
}

hipError_t launch_kv_copy(int dtype, int to_cache, void* kc, void* vc, int H, int DH, int T_cap, int pos0, int n,
                          void* k, void* v, hipStream_t st) {
  const long work = static_cast<long>(H) * n * DH;
  if (work <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((work + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(kv_copy_kernel<bf16>, grid, dim3(256), 0, st, to_cache, static_cast<bf16*>(kc),
                       static_cast<bf16*>(vc), H, DH, T_cap, pos0, n, static_cast<bf16*>(k),
                       static_cast<bf16*>(v));
  else
    hipLaunchKernelGGL(kv_copy_kernel<float>, grid, dim3(256), 0, st, to_cache, static_cast<float*>(kc),
                       static_cast<float*>(vc), H, DH, T_cap, pos0, n, static_cast<float*>(k),
                       static_cast<float*>(v));
  return hipGetLastError();
}

}  // namespace sps

namespace sps {

// Streaming read of `n16` 16-byte words with the weight stream's nontemporal
// loads: the device's attainable HBM read rate, against which the verify
// step's kernels are measured. Each work-group reads one contiguous region,
// four 16-byte loads in flight per thread (the best of a sweep over grid,
// block, loads in flight and grid-stride vs contiguous regions: 512 x 256,
// regions, 4 loads). The folded words are stored only on a value the data
// cannot produce by chance in practice, which keeps every load live without
// writing back.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ src, size_t n16,
                                                          uint32_t key, uint32_t* __restrict__ sink) {
  constexpr int U = 4;
  const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const size_t begin = static_cast<size_t>(blockIdx.x) * per;
  const size_t end = begin + per < n16 ? begin + per : n16;
  const size_t step = blockDim.x;
  size_t i = begin + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (U - 1) * step < end; i += U * step) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i + u * step);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < end; i += step) {
    const u32x4 v = __builtin_nontemporal_load(src + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == key) sink[0] = acc;
}

hipError_t launch_stream_read(const void* src, size_t n16, uint32_t* sink, hipStream_t st) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(512), dim3(256), 0, st, static_cast<const u32x4*>(src), n16,
                     0x9e3779b9u, sink);
  return hipGetLastError();
}

}  // namespace sps
