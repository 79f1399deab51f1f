// Per-token kernels of the decoder forward: embedding + RMSNorm, residual
// add + RMSNorm, rotary position encoding with the KV-cache append, and KV
// copies between canonical buffers and the cache's tile layout.
//
// KV cache layout, per (layer, sequence, head), each of K and V holding
// T_cap positions x DH dims in the model dtype:
//   keys   : 16-position x 32-dim tiles, tile (p/16, d/32) in MFMA A-operand
//            order -- element (p, d) in lane (p%16) + 16 ((d%32)/8), slot d%8.
//   values : 32-position x 16-dim tiles, tile (p/32, d/16), element (p, d)
//            in lane (d%16) + 16 g, slot e, where position p%32 = 4 g + e for
//            p%32 < 16 and 16 + 4 g + (e-4) otherwise. This is the A operand
//            of the P V product whose B operand is the softmax tile exactly
//            as the score MFMA leaves it in registers (see attention.hip).
#include "common.h"
#include "launch.h"

namespace sps {

__device__ __forceinline__ size_t k_offset(int p, int d, int DH) {
  return ((static_cast<size_t>(p >> 4) * (DH >> 5) + (d >> 5)) * 64 + (p & 15) + 16 * ((d & 31) >> 3)) * 8 +
         (d & 7);
}
__device__ __forceinline__ size_t v_offset(int p, int d, int DH) {
  const int pp = p & 31;
  const int g = pp < 16 ? (pp >> 2) : ((pp - 16) >> 2);
  const int e = pp < 16 ? (pp & 3) : 4 + ((pp - 16) & 3);
  return ((static_cast<size_t>(p >> 5) * (DH >> 4) + (d >> 4)) * 64 + (d & 15) + 16 * g) * 8 + e;
}

// Row-wise kernels use 1024 threads and keep the row in registers: each
// thread owns up to kNormChunks groups of four consecutive elements, all of
// whose loads are issued before the reduction, so a row costs one memory
// round trip instead of one per loop iteration.
constexpr int kNormThreads = 1024;
constexpr int kNormChunks = 4;   // d_model <= 4 * 4 * 1024 = 16384
constexpr int kNormSplitGroup = 4;

template <typename T>
__device__ __forceinline__ void store4(T* dst, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* dst, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* dst, float a, float b, float c, float d) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 v;
  v[0] = static_cast<bf16>(a); v[1] = static_cast<bf16>(b); v[2] = static_cast<bf16>(c); v[3] = static_cast<bf16>(d);
  *reinterpret_cast<bf16x4*>(dst) = v;
}
__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4(const bf16* p) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  return make_float4(static_cast<float>(v[0]), static_cast<float>(v[1]), static_cast<float>(v[2]),
                     static_cast<float>(v[3]));
}

// x = h * rsqrt(mean(h^2) + eps) * gain for a row held as float4 chunks,
// stored in the activation format (fp32, or bf16 hi / lo planes).
__device__ __forceinline__ void store_act4(float* xr, size_t, float a, float b, float c, float d) {
  store4<float>(xr, a, b, c, d);
}
__device__ __forceinline__ void store_act4(bf16* xr, size_t plane, float a, float b, float c, float d) {
  const bf16 ha = static_cast<bf16>(a), hb = static_cast<bf16>(b), hc = static_cast<bf16>(c),
             hd = static_cast<bf16>(d);
  store4<bf16>(xr, a, b, c, d);
  store4<bf16>(xr + plane, a - static_cast<float>(ha), b - static_cast<float>(hb), c - static_cast<float>(hc),
               d - static_cast<float>(hd));
}

template <typename T>
__device__ __forceinline__ void norm_store(const float4* v, int d, float ss, const float* __restrict__ gain,
                                           float eps, T* __restrict__ xr, size_t plane) {
  const float rs = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int i = (c * kNormThreads + threadIdx.x) * 4;
    if (i < d) {
      const float4 g = load4(gain + i);
      store_act4(xr + i, plane, v[c].x * rs * g.x, v[c].y * rs * g.y, v[c].z * rs * g.z, v[c].w * rs * g.w);
    }
  }
}

// h[r] = E[token]; x[r] = rms(h[r]) * gain. One block per row.
template <typename T>
__global__ __launch_bounds__(kNormThreads) void embed_norm_kernel(const int32_t* __restrict__ tokens,
                                                                  int tok_stride, int Mps, const T* __restrict__ E,
                                                                  int V, int d, const float* __restrict__ gain,
                                                                  float eps, float* __restrict__ h,
                                                                  T* __restrict__ x, size_t xplane, int* err) {
  __shared__ float red[16];
  const int row = blockIdx.x;
  const int b = row / Mps, j = row % Mps;
  int tok = tokens[static_cast<size_t>(b) * tok_stride + j];
  const bool ok = tok >= 0 && tok < V;
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(err, kErrBadToken);
    tok = 0;
  }
  const T* e = E + static_cast<size_t>(tok) * d;
  float* hr = h + static_cast<size_t>(row) * d;
  float4 v[kNormChunks];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int i = (c * kNormThreads + threadIdx.x) * 4;
    v[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < d && ok) v[c] = load4(e + i);
  }
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int i = (c * kNormThreads + threadIdx.x) * 4;
    if (i < d) {
      *reinterpret_cast<float4*>(hr + i) = v[c];
      ss += v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
    }
  }
  ss = block_sum(ss, red);
  norm_store<T>(v, d, ss, gain, eps, x + static_cast<size_t>(row) * d, xplane);
}

// h[r] += sum_s part[s][r]; x[r] = rms(h[r]) * gain. One block per row.
template <typename T>
__global__ __launch_bounds__(kNormThreads) void add_norm_kernel(float* __restrict__ h, const float* __restrict__ part,
                                                                int S, int M, int d, const float* __restrict__ gain,
                                                                float eps, T* __restrict__ x, size_t xplane) {
  __shared__ float red[16];
  const int row = blockIdx.x;
  float* hr = h + static_cast<size_t>(row) * d;
  float4 v[kNormChunks];
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int i = (c * kNormThreads + threadIdx.x) * 4;
    v[c] = i < d ? load4(hr + i) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  // Split-K partial planes, four at a time: every load of a group is in
  // flight before the adds.
  for (int s0 = 0; s0 < S; s0 += kNormSplitGroup) {
    float4 t[kNormSplitGroup][kNormChunks];
#pragma unroll
    for (int u = 0; u < kNormSplitGroup; ++u) {
      const float* pr = part + (static_cast<size_t>(s0 + u) * M + row) * d;
#pragma unroll
      for (int c = 0; c < kNormChunks; ++c) {
        const int i = (c * kNormThreads + threadIdx.x) * 4;
        t[u][c] = (s0 + u < S && i < d) ? load4(pr + i) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < kNormSplitGroup; ++u)
#pragma unroll
      for (int c = 0; c < kNormChunks; ++c) {
        v[c].x += t[u][c].x; v[c].y += t[u][c].y; v[c].z += t[u][c].z; v[c].w += t[u][c].w;
      }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int i = (c * kNormThreads + threadIdx.x) * 4;
    if (i < d) {
      *reinterpret_cast<float4*>(hr + i) = v[c];
      ss += v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
    }
  }
  ss = block_sum(ss, red);
  norm_store<T>(v, d, ss, gain, eps, x + static_cast<size_t>(row) * d, xplane);
}

// Sum the QKV split partials, rotate q and k (rotate-half pairing: dims f and
// f + DH/2 turn by pos * base^(-2f/DH)), store q for attention and append k, v
// to the cache at the row's position. Grid: (row, group of 256 dim pairs);
// each thread owns one (head, f) pair, so it forms one angle (in fp64) and
// moves two q, two k and two v values.
template <typename T>
__global__ __launch_bounds__(256) void rope_kv_kernel(const float* __restrict__ qkvp, int S, int M, int H, int DH,
                                                      int Mps, const int32_t* __restrict__ lengths,
                                                      int pos_offset, float rope_base, T* __restrict__ qout,
                                                      T* __restrict__ kc, T* __restrict__ vc, int T_cap,
                                                      int* err) {
  const int row = blockIdx.x;
  const int b = row / Mps, j = row % Mps;
  const int HD = H * DH, half = DH / 2;
  const int pos = lengths[b] + pos_offset + j;
  const bool ok = pos >= 0 && pos < T_cap;
  if (!ok && threadIdx.x == 0 && blockIdx.y == 0) atomicOr(err, kErrCapacity);
  const int i = blockIdx.y * blockDim.x + threadIdx.x;
  if (i >= H * half) return;
  const int hh = i / half, f = i % half;
  const size_t ld = 3 * static_cast<size_t>(HD);
  const float* src = qkvp + static_cast<size_t>(row) * ld;
  const size_t plane = static_cast<size_t>(M) * ld;
  const int c1 = hh * DH + f, c2 = c1 + half;
  float q1 = 0.f, q2 = 0.f, k1 = 0.f, k2 = 0.f, v1 = 0.f, v2 = 0.f;
  for (int sp = 0; sp < S; ++sp) {
    const float* p = src + sp * plane;
    q1 += p[c1]; q2 += p[c2]; k1 += p[HD + c1]; k2 += p[HD + c2]; v1 += p[2 * HD + c1]; v2 += p[2 * HD + c2];
  }
  const double inv = exp2(-2.0 * f / DH * log2(static_cast<double>(rope_base)));
  double sn, cs;
  sincos(static_cast<double>(pos) * inv, &sn, &cs);
  const float c = static_cast<float>(cs), s = static_cast<float>(sn);
  T* qr = qout + static_cast<size_t>(row) * HD;
  qr[c1] = from_f32<T>(q1 * c - q2 * s);
  qr[c2] = from_f32<T>(q2 * c + q1 * s);
  if (ok) {
    const size_t region = (static_cast<size_t>(b) * H + hh) * T_cap * DH;
    kc[region + k_offset(pos, f, DH)] = from_f32<T>(k1 * c - k2 * s);
    kc[region + k_offset(pos, f + half, DH)] = from_f32<T>(k2 * c + k1 * s);
    vc[region + v_offset(pos, f, DH)] = from_f32<T>(v1);
    vc[region + v_offset(pos, f + half, DH)] = from_f32<T>(v2);
  }
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

hipError_t launch_embed_norm(int dtype, const int32_t* tokens, int tok_stride, int Mps, int M, const void* E,
                             int V, int d, const float* gain, float eps, float* h, void* x, size_t xplane, int* err,
                             hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(embed_norm_kernel<bf16>, dim3(M), dim3(kNormThreads), 0, st, tokens, tok_stride, Mps,
                       static_cast<const bf16*>(E), V, d, gain, eps, h, static_cast<bf16*>(x), xplane, err);
  else
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(M), dim3(kNormThreads), 0, st, tokens, tok_stride, Mps,
                       static_cast<const float*>(E), V, d, gain, eps, h, static_cast<float*>(x), xplane, err);
  return hipGetLastError();
}

hipError_t launch_add_norm(int dtype, float* h, const float* part, int S, int M, int d, const float* gain,
                           float eps, void* x, size_t xplane, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(add_norm_kernel<bf16>, dim3(M), dim3(kNormThreads), 0, st, h, part, S, M, d, gain, eps,
                       static_cast<bf16*>(x), xplane);
  else
    hipLaunchKernelGGL(add_norm_kernel<float>, dim3(M), dim3(kNormThreads), 0, st, h, part, S, M, d, gain, eps,
                       static_cast<float*>(x), xplane);
  return hipGetLastError();
}

hipError_t launch_rope_kv(int dtype, const float* qkvp, int S, int M, int H, int DH, int Mps,
                          const int32_t* lengths, int pos_offset, float rope_base, void* qout, void* kc, void* vc,
                          int T_cap, int* err, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(rope_kv_kernel<bf16>, dim3(M, (H * DH / 2 + 255) / 256), dim3(256), 0, st, qkvp, S, M, H, DH, Mps, lengths,
                       pos_offset, rope_base, static_cast<bf16*>(qout), static_cast<bf16*>(kc),
                       static_cast<bf16*>(vc), T_cap, err);
  else
    hipLaunchKernelGGL(rope_kv_kernel<float>, dim3(M, (H * DH / 2 + 255) / 256), dim3(256), 0, st, qkvp, S, M, H, DH, Mps, lengths,
                       pos_offset, rope_base, static_cast<float*>(qout), static_cast<float*>(kc),
                       static_cast<float*>(vc), T_cap, err);
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
