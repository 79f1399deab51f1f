// Weight-streaming skinny GEMM for the verify / draft forward (the linear
// layers of the Conditional Scoring section: QKV, attention output, FFN,
// unembedding). At M = B (K+1) <= 160 rows every weight byte is used for at
// most M multiply-adds, far below the MI355X ridge point, so the kernel is an
// HBM stream: its job is to keep enough bytes in flight.
//
// Packed weight layout: W [N][K] (nn.Linear orientation) is stored as 16 x 32
// tiles, tile (nt, kt) holding rows 16 nt .. +15 and columns 32 kt .. +31 in
// MFMA B-operand register order: lane l owns row 16 nt + l % 16, columns
// 32 kt + 8 (l / 16) .. +7. Tiles are ordered [nt][kt], so one wave-wide 16 B
// (bf16) per lane load is one contiguous KiB and a work-group streams one
// contiguous region per output tile.
//
// Grid: one work-group per (16-column output tile, K split). Its waves walk
// the split's k-tiles in chunks of U, round robin, each accumulating a
// 16 x 16 (per 16-row M tile) fp32 partial with MFMA; the waves' partials are
// summed in LDS and the epilogue applies GELU / SwiGLU or stores fp32 split
// partials (summed by the consumer kernel, so results do not depend on
// atomics).
#include "common.h"
#include "launch.h"

namespace sps {

__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f, k1 = 0.044715f;
  return 0.5f * x * (1.0f + tanhf(k0 * (x + k1 * x * x * x)));
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

template <typename T, int MT, int WAVES, int U, int EPI>
__global__ __launch_bounds__(WAVES * 64) void gemm_kernel(
    const T* __restrict__ X, int ldx, int M, const T* __restrict__ W, int KT, int S, int n_valid,
    float* __restrict__ out, int ldo, T* __restrict__ act, int lda) {
  constexpr int kTile = 512;  // elements per 16 x 32 tile
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nt = blockIdx.x, s = blockIdx.y;
  const int kt0 = static_cast<int>((static_cast<long>(KT) * s) / S);
  const int kt1 = static_cast<int>((static_cast<long>(KT) * (s + 1)) / S);
  const int r16 = lane & 15, grp = lane >> 4;

  const T* wp = W + static_cast<size_t>(nt) * KT * kTile + lane * 8;
  const T* xp[MT];
  bool xv[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + r16;
    xv[mt] = m < M;
    xp[mt] = X + static_cast<size_t>(xv[mt] ? m : 0) * ldx + grp * 8;
  }
  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  int kb = kt0 + wave * U;
  for (; kb + U <= kt1; kb += WAVES * U) {
    Frag<T> b[U];
    Frag<T> a[MT][U];
#pragma unroll
    for (int u = 0; u < U; ++u) b[u] = load_frag_stream(wp + static_cast<size_t>(kb + u) * kTile);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int u = 0; u < U; ++u)
        a[mt][u] = xv[mt] ? load_frag(xp[mt] + (kb + u) * 32) : Frag<T>::zero();
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = mma8(acc[mt], a[mt][u], b[u]);
  }
  if (kb < kt1) {  // ragged last chunk of this wave
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kt = kb + u;
      if (kt < kt1) {
        const Frag<T> bb = load_frag_stream(wp + static_cast<size_t>(kt) * kTile);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const Frag<T> aa = xv[mt] ? load_frag(xp[mt] + kt * 32) : Frag<T>::zero();
          acc[mt] = mma8(acc[mt], aa, bb);
        }
      }
    }
  }

  // Sum the waves' partials in LDS, then the epilogue.
  __shared__ float red[WAVES][MT][4][64];
  __shared__ float tot[MT][4][64];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][mt][r][lane] = acc[mt][r];
  __syncthreads();
  for (int e = threadIdx.x; e < MT * 256; e += WAVES * 64) {
    const int mt = e >> 8, r = (e >> 6) & 3, ln = e & 63;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) v += red[w][mt][r][ln];
    tot[mt][r][ln] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < MT * 256; e += WAVES * 64) {
    const int mt = e >> 8, r = (e >> 6) & 3, ln = e & 63;
    const int m = mt * 16 + (ln >> 4) * 4 + r;
    const int col = ln & 15;
    if (m >= M) continue;
    const float v = tot[mt][r][ln];
    if (EPI == kEpiStore) {
      const int n = nt * 16 + col;
      if (n < n_valid) out[(static_cast<size_t>(s) * M + m) * ldo + n] = v;
    } else if (EPI == kEpiGelu) {
      const int n = nt * 16 + col;
      if (n < n_valid) act[static_cast<size_t>(m) * lda + n] = from_f32<T>(gelu_tanh(v));
    } else {  // SwiGLU: packed rows 0..7 are gate columns, 8..15 the matching up columns
      if (col < 8) {
        const int c = nt * 8 + col;
        const float up = tot[mt][r][ln + 8];
        if (c < n_valid) act[static_cast<size_t>(m) * lda + c] = from_f32<T>(silu(v) * up);
      }
    }
  }
}

template <typename T, int MT, int WAVES, int U>
static hipError_t gemm_dispatch_epi(const GemmArgs& a, hipStream_t st) {
  const dim3 grid(a.N / 16, a.S), block(WAVES * 64);
  const T* X = static_cast<const T*>(a.X);
  const T* W = static_cast<const T*>(a.W);
  T* act = static_cast<T*>(a.act);
  switch (a.epi) {
    case kEpiStore:
      hipLaunchKernelGGL((gemm_kernel<T, MT, WAVES, U, kEpiStore>), grid, block, 0, st, X, a.ldx, a.M, W,
                         a.KT, a.S, a.n_valid, a.out, a.ldo, act, a.lda);
      break;
    case kEpiGelu:
      hipLaunchKernelGGL((gemm_kernel<T, MT, WAVES, U, kEpiGelu>), grid, block, 0, st, X, a.ldx, a.M, W,
                         a.KT, a.S, a.n_valid, a.out, a.ldo, act, a.lda);
      break;
    default:
      hipLaunchKernelGGL((gemm_kernel<T, MT, WAVES, U, kEpiSwiglu>), grid, block, 0, st, X, a.ldx, a.M, W,
                         a.KT, a.S, a.n_valid, a.out, a.ldo, act, a.lda);
      break;
  }
  return hipGetLastError();
}

// Waves per work-group and k-tiles per chunk for each row-tile count.
template <typename T>
static hipError_t gemm_dispatch(const GemmArgs& a, hipStream_t st) {
  constexpr bool kB = sizeof(T) == 2;
  const int MT = (a.M + 15) / 16;
  switch (MT) {
    case 1: return gemm_dispatch_epi<T, 1, 8, kB ? 8 : 4>(a, st);
    case 2: return gemm_dispatch_epi<T, 2, 8, kB ? 8 : 4>(a, st);
    case 3: return gemm_dispatch_epi<T, 3, 4, kB ? 8 : 4>(a, st);
    case 4: return gemm_dispatch_epi<T, 4, 4, kB ? 8 : 4>(a, st);
    case 5:
    case 6: return gemm_dispatch_epi<T, 6, 4, 4>(a, st);
    case 7:
    case 8: return gemm_dispatch_epi<T, 8, 4, 4>(a, st);
    default: return gemm_dispatch_epi<T, 10, 4, 4>(a, st);
  }
}

hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t st) {
  return dtype == 1 ? gemm_dispatch<bf16>(a, st) : gemm_dispatch<float>(a, st);
}

int gemm_splits(int dtype, int NT, int KT, int M, int epi) {
  if (epi != kEpiStore) return 1;
  const int MT = (M + 15) / 16;
  const int waves = MT <= 2 ? 8 : 4;
  const int U = (dtype == 1 && MT <= 4) ? 8 : 4;
  const int per_round = waves * U;
  int S = 2048 / (NT > 0 ? NT : 1);
  if (S > 8) S = 8;
  const int cap = KT / per_round;
  if (S > cap) S = cap;
  return S < 1 ? 1 : S;
}

// ---------------------------------------------------------------------------
// Packing canonical [n][k] rows into tile order.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void pack_kernel(const T* __restrict__ src, int n_src, int Kd, T* __restrict__ dst, int KT,
                            int kind, int row_off) {
  const int groups = Kd / 8;
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(n_src) * groups) return;
  const int n = static_cast<int>(i / groups), k = static_cast<int>(i % groups) * 8;
  const int nf = kind == 0 ? row_off + n : (n / 8) * 16 + row_off * 8 + (n % 8);
  const int nt = nf / 16, rr = nf % 16, kt = k / 32, grp = (k % 32) / 8;
  const size_t o = ((static_cast<size_t>(nt) * KT + kt) * 64 + rr + 16 * grp) * 8;
  const T* s = src + static_cast<size_t>(n) * Kd + k;
#pragma unroll
  for (int e = 0; e < 8; ++e) dst[o + e] = s[e];
}

template <typename T>
__global__ void pack_zero_kernel(T* __restrict__ dst, int KT, int zero_from, int zero_to) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int groups = KT * 4;
  if (i >= static_cast<long>(zero_to - zero_from) * groups) return;
  const int nf = zero_from + static_cast<int>(i / groups), k = static_cast<int>(i % groups) * 8;
  const int nt = nf / 16, rr = nf % 16, kt = k / 32, grp = (k % 32) / 8;
  const size_t o = ((static_cast<size_t>(nt) * KT + kt) * 64 + rr + 16 * grp) * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) dst[o + e] = from_f32<T>(0.f);
}

template <typename T>
static hipError_t pack_t(const void* src, int n_src, int Kd, void* dst, int KT, int kind, int row_off,
                         int zero_from, int zero_to, hipStream_t st) {
  const long work = static_cast<long>(n_src) * (Kd / 8);
  if (work > 0)
    hipLaunchKernelGGL(pack_kernel<T>, dim3(static_cast<unsigned>((work + 255) / 256)), dim3(256), 0, st,
                       static_cast<const T*>(src), n_src, Kd, static_cast<T*>(dst), KT, kind, row_off);
  const long zwork = static_cast<long>(zero_to - zero_from) * KT * 4;
  if (zwork > 0)
    hipLaunchKernelGGL(pack_zero_kernel<T>, dim3(static_cast<unsigned>((zwork + 255) / 256)), dim3(256), 0,
                       st, static_cast<T*>(dst), KT, zero_from, zero_to);
  return hipGetLastError();
}

hipError_t launch_pack(int dtype, const void* src, int n_src, int Kd, void* dst, int KT, int kind,
                       int row_off, int zero_from, int zero_to, hipStream_t st) {
  return dtype == 1 ? pack_t<bf16>(src, n_src, Kd, dst, KT, kind, row_off, zero_from, zero_to, st)
                    : pack_t<float>(src, n_src, Kd, dst, KT, kind, row_off, zero_from, zero_to, st);
}

}  // namespace sps
