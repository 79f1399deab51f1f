// Device-side building blocks shared by the libsps kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sps {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

// Device error bits (mirrors SPS_DEV_* in sps.h).
constexpr int kErrBadToken = 1;
constexpr int kErrEmpty = 2;
constexpr int kErrCapacity = 4;
constexpr int kErrNonFinite = 8;

// ---------------------------------------------------------------------------
// Eight-element operand fragments.
//
// Every matrix product in the library is built from 16x16 output tiles with a
// contraction depth of 32 per step. Lane l of a wave owns operand row
// (l % 16) and the eight consecutive contraction indices 8*(l/16) .. +7, which
// is the register layout of v_mfma_f32_16x16x32_bf16 for both the A and the B
// operand. For fp32 the same 32-deep step is eight v_mfma_f32_16x16x4_f32
// instructions, the s-th consuming element s of every lane's fragment, so the
// two element types share every tile layout. The 16x16 result C[i][j] is held
// by lane 16*(i/4) + j, component i % 4.
// ---------------------------------------------------------------------------
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  bf16x8 v;
  __device__ static Frag zero() { Frag f; f.v = bf16x8{}; return f; }
};
template <> struct Frag<float> {
  f32x8 v;
  __device__ static Frag zero() { Frag f; f.v = f32x8{}; return f; }
};

template <typename T> __device__ __forceinline__ Frag<T> load_frag(const T* p);
template <> __device__ __forceinline__ Frag<bf16> load_frag<bf16>(const bf16* p) {
  Frag<bf16> f; f.v = *reinterpret_cast<const bf16x8*>(p); return f;
}
template <> __device__ __forceinline__ Frag<float> load_frag<float>(const float* p) {
  Frag<float> f; f.v = *reinterpret_cast<const f32x8*>(p); return f;
}

// Streaming variant for data that is read exactly once (weights).
template <typename T> __device__ __forceinline__ Frag<T> load_frag_stream(const T* p);
template <> __device__ __forceinline__ Frag<bf16> load_frag_stream<bf16>(const bf16* p) {
  Frag<bf16> f; f.v = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(p)); return f;
}
template <> __device__ __forceinline__ Frag<float> load_frag_stream<float>(const float* p) {
  Frag<float> f; f.v = __builtin_nontemporal_load(reinterpret_cast<const f32x8*>(p)); return f;
}

__device__ __forceinline__ f32x4 mma8(f32x4 acc, const Frag<bf16>& a, const Frag<bf16>& b) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma8(f32x4 acc, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
  for (int s = 0; s < 8; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[s], b.v[s], acc, 0, 0, 0);
  return acc;
}

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }

// Activation format. fp32 models keep activations as fp32 [rows][ld]. bf16
// models keep each activation x as two bf16 planes, hi = bf16(x) at element
// i and lo = bf16(x - hi) at element plane + i, so that a bf16 MFMA can
// consume x at ~2^-16 relative precision (see gemm.hip).
__device__ __forceinline__ void store_act(float* act, size_t, size_t i, float v) { act[i] = v; }
__device__ __forceinline__ void store_act(bf16* act, size_t plane, size_t i, float v) {
  const bf16 h = static_cast<bf16>(v);
  act[i] = h;
  act[plane + i] = static_cast<bf16>(v - static_cast<float>(h));
}

// KV cache layout, per (layer, sequence, head), each of K and V holding
// T_cap positions x DH dims in the model dtype:
//   keys   : 16-position x 32-dim tiles, tile (p/16, d/32) in MFMA A-operand
//            order -- element (p, d) in lane (p%16) + 16 ((d%32)/8), slot d%8.
//   values : 32-position x 16-dim tiles, tile (p/32, d/16), element (p, d)
//            in lane (d%16) + 16 g, slot e, where position p%32 = 4 g + e for
//            p%32 < 16 and 16 + 4 g + (e-4) otherwise. This is the A operand
//            of the P V product whose B operand is the softmax tile exactly
//            as the score MFMA leaves it in registers (see attention.hip).
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

// ---------------------------------------------------------------------------
// Reductions (deterministic: fixed butterfly order, then waves in order).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Block-wide sum / max for blockDim.x a multiple of 64 (<= 1024). `red` is
// a __shared__ float[16]. Every thread receives the result.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = red[0];
  for (int i = 1; i < nw; ++i) s = fmaxf(s, red[i]);
  return s;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int d) {
  uint32_t lo = static_cast<uint32_t>(v), hi = static_cast<uint32_t>(v >> 32);
  lo = __shfl_up(lo, d);
  hi = __shfl_up(hi, d);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Exclusive prefix sum of one uint64 per thread over the block (blockDim.x a
// multiple of 64, <= 1024). `wsum` is __shared__ uint64_t[17]. Returns the
// exclusive prefix; *total receives the block total.
__device__ __forceinline__ uint64_t block_exscan_u64(uint64_t v, uint64_t* wsum, uint64_t* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  uint64_t inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint64_t o = shfl_up_u64(inc, d);
    if (lane >= d) inc += o;
  }
  __syncthreads();
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t acc = 0;
    for (int i = 0; i < nw; ++i) { uint64_t t = wsum[i]; wsum[i] = acc; acc += t; }
    wsum[16] = acc;
  }
  __syncthreads();
  *total = wsum[16];
  return wsum[w] + inc - v;
}

}  // namespace sps
