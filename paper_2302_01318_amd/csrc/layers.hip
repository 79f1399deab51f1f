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

// h[r] = E[token]; x[r] = rms(h[r]) * gain. One block per row.
template <typename T>
__global__ __launch_bounds__(256) void embed_norm_kernel(const int32_t* __restrict__ tokens, int tok_stride,
                                                         int Mps, const T* __restrict__ E, int V, int d,
                                                         const float* __restrict__ gain, float eps,
                                                         float* __restrict__ h, T* __restrict__ x, int* err) {
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
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    const float v = ok ? to_f32(e[i]) : 0.f;
    hr[i] = v;
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float rs = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
  T* xr = x + static_cast<size_t>(row) * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) xr[i] = from_f32<T>(hr[i] * rs * gain[i]);
}

// h[r] += sum_s part[s][r]; x[r] = rms(h[r]) * gain. One block per row.
template <typename T>
__global__ __launch_bounds__(256) void add_norm_kernel(float* __restrict__ h, const float* __restrict__ part, int S,
                                                       int M, int d, const float* __restrict__ gain, float eps,
                                                       T* __restrict__ x) {
  __shared__ float red[16];
  const int row = blockIdx.x;
  float* hr = h + static_cast<size_t>(row) * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    float v = hr[i];
    for (int s = 0; s < S; ++s) v += part[(static_cast<size_t>(s) * M + row) * d + i];
    hr[i] = v;
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float rs = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
  T* xr = x + static_cast<size_t>(row) * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) xr[i] = from_f32<T>(hr[i] * rs * gain[i]);
}

// Sum the QKV split partials, rotate q and k (rotate-half pairing: dims f and
// f + DH/2 turn by pos * base^(-2f/DH)), store q for attention and append k, v
// to the cache at the row's position. Angles are formed in fp64.
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
  if (!ok && threadIdx.x == 0) atomicOr(err, kErrCapacity);
  const size_t ld = 3 * static_cast<size_t>(HD);
  const float* src = qkvp + static_cast<size_t>(row) * ld;
  const size_t plane = static_cast<size_t>(M) * ld;
  for (int i = threadIdx.x; i < H * half; i += blockDim.x) {
    const int hh = i / half, f = i % half;
    const double inv = pow(static_cast<double>(rope_base), -2.0 * f / DH);
    double sn, cs;
    sincos(static_cast<double>(pos) * inv, &sn, &cs);
    const float c = static_cast<float>(cs), s = static_cast<float>(sn);
    const int c1 = hh * DH + f, c2 = c1 + half;
    float q1 = 0.f, q2 = 0.f, k1 = 0.f, k2 = 0.f;
    for (int sp = 0; sp < S; ++sp) {
      const float* p = src + sp * plane;
      q1 += p[c1]; q2 += p[c2]; k1 += p[HD + c1]; k2 += p[HD + c2];
    }
    T* qr = qout + static_cast<size_t>(row) * HD;
    qr[c1] = from_f32<T>(q1 * c - q2 * s);
    qr[c2] = from_f32<T>(q2 * c + q1 * s);
    if (ok) {
      T* kr = kc + (static_cast<size_t>(b) * H + hh) * T_cap * DH;
      kr[k_offset(pos, f, DH)] = from_f32<T>(k1 * c - k2 * s);
      kr[k_offset(pos, f + half, DH)] = from_f32<T>(k2 * c + k1 * s);
    }
  }
  if (ok) {
    for (int i = threadIdx.x; i < HD; i += blockDim.x) {
      float v = 0.f;
      for (int sp = 0; sp < S; ++sp) v += src[sp * plane + 2 * HD + i];
      const int hh = i / DH, dd = i % DH;
      T* vr = vc + (static_cast<size_t>(b) * H + hh) * T_cap * DH;
      vr[v_offset(pos, dd, DH)] = from_f32<T>(v);
    }
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
                             int V, int d, const float* gain, float eps, float* h, void* x, int* err,
                             hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(embed_norm_kernel<bf16>, dim3(M), dim3(256), 0, st, tokens, tok_stride, Mps,
                       static_cast<const bf16*>(E), V, d, gain, eps, h, static_cast<bf16*>(x), err);
  else
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(M), dim3(256), 0, st, tokens, tok_stride, Mps,
                       static_cast<const float*>(E), V, d, gain, eps, h, static_cast<float*>(x), err);
  return hipGetLastError();
}

hipError_t launch_add_norm(int dtype, float* h, const float* part, int S, int M, int d, const float* gain,
                           float eps, void* x, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(add_norm_kernel<bf16>, dim3(M), dim3(256), 0, st, h, part, S, M, d, gain, eps,
                       static_cast<bf16*>(x));
  else
    hipLaunchKernelGGL(add_norm_kernel<float>, dim3(M), dim3(256), 0, st, h, part, S, M, d, gain, eps,
                       static_cast<float*>(x));
  return hipGetLastError();
}

hipError_t launch_rope_kv(int dtype, const float* qkvp, int S, int M, int H, int DH, int Mps,
                          const int32_t* lengths, int pos_offset, float rope_base, void* qout, void* kc, void* vc,
                          int T_cap, int* err, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(rope_kv_kernel<bf16>, dim3(M), dim3(256), 0, st, qkvp, S, M, H, DH, Mps, lengths,
                       pos_offset, rope_base, static_cast<bf16*>(qout), static_cast<bf16*>(kc),
                       static_cast<bf16*>(vc), T_cap, err);
  else
    hipLaunchKernelGGL(rope_kv_kernel<float>, dim3(M), dim3(256), 0, st, qkvp, S, M, H, DH, Mps, lengths,
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
