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
// Activation operand. fp32 models: X is fp32 [M][K] and an M tile is 16 rows.
// bf16 models: X holds every activation x as a pair of bf16 planes hi and lo
// (x = hi + lo to ~2^-16 relative), and an M tile is 8 rows: MFMA rows 0-7
// read the hi plane and rows 8-15 the lo plane of the same 8 activation
// rows, so one bf16 MFMA produces both halves and the epilogue adds output
// row i + 8 to row i. The product equals an fp32-activation x bf16-weight
// product up to fp32 accumulation at the cost of no extra instruction (at
// M <= 8 the lo half uses rows that would otherwise multiply zeros).
//
// Grid: one work-group per (16-column output tile, K split). Its waves walk
// the split's k-tiles in chunks of U, round robin, each accumulating one
// 16 x 16 fp32 tile per M tile with MFMA; the waves' partials are summed in
// LDS and the epilogue applies GELU / SwiGLU or stores fp32 split partials
// (summed by the consumer kernel, so results do not depend on atomics).
#include <cstdlib>

#include "common.h"
#include "launch.h"

namespace sps {

__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f, k1 = 0.044715f;
  return 0.5f * x * (1.0f + tanhf(k0 * (x + k1 * x * x * x)));
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

template <typename T> struct ActRows;
template <> struct ActRows<bf16> { static constexpr int kRows = 8; };
template <> struct ActRows<float> { static constexpr int kRows = 16; };

template <typename T, int MT, int NTW, int WAVES, int U, int EPI, int MINW>
__global__ __launch_bounds__(WAVES * 64) __attribute__((amdgpu_waves_per_eu(MINW, 8))) void gemm_kernel(
    const T* __restrict__ X, int ldx, size_t xplane, int M, const T* __restrict__ W, int NT, int KT, int S,
    int n_valid, float* __restrict__ out, int ldo, size_t oplane, T* __restrict__ act, int lda, size_t aplane) {
  constexpr int kTile = 512;  // elements per 16 x 32 tile
  constexpr int kRows = ActRows<T>::kRows;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nt0 = blockIdx.x * NTW, s = blockIdx.y;
  const int kt0 = static_cast<int>((static_cast<long>(KT) * s) / S);
  const int kt1 = static_cast<int>((static_cast<long>(KT) * (s + 1)) / S);
  const int r16 = lane & 15, grp = lane >> 4;

  const T* wp[NTW];
  bool wv[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    wv[j] = nt0 + j < NT;
    wp[j] = W + static_cast<size_t>(wv[j] ? nt0 + j : 0) * KT * kTile + lane * 8;
  }
  const T* xp[MT];
  bool xv[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * kRows + (kRows == 8 ? (r16 & 7) : r16);
    const size_t plane = kRows == 8 ? (r16 >> 3) * xplane : 0;
    xv[mt] = m < M;
    xp[mt] = X + plane + static_cast<size_t>(xv[mt] ? m : 0) * ldx + grp * 8;
  }
  f32x4 acc[NTW][MT];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  int kb = kt0 + wave * U;
  for (; kb + U <= kt1; kb += WAVES * U) {
    Frag<T> b[NTW][U];
    Frag<T> a[MT][U];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
      for (int u = 0; u < U; ++u)
        b[j][u] = wv[j] ? load_frag_stream(wp[j] + static_cast<size_t>(kb + u) * kTile) : Frag<T>::zero();
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int u = 0; u < U; ++u) a[mt][u] = xv[mt] ? load_frag(xp[mt] + (kb + u) * 32) : Frag<T>::zero();
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[j][mt] = mma8(acc[j][mt], a[mt][u], b[j][u]);
  }
  if (kb < kt1) {  // ragged last chunk of this wave
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kt = kb + u;
      if (kt < kt1) {
        Frag<T> aa[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) aa[mt] = xv[mt] ? load_frag(xp[mt] + kt * 32) : Frag<T>::zero();
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          const Frag<T> bb = wv[j] ? load_frag_stream(wp[j] + static_cast<size_t>(kt) * kTile) : Frag<T>::zero();
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[j][mt] = mma8(acc[j][mt], aa[mt], bb);
        }
      }
    }
  }

  // Sum the waves' partials in LDS, then the epilogue.
  __shared__ float red[WAVES][NTW][MT][4][64];
  __shared__ float tot[NTW][MT][4][64];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][j][mt][r][lane] = acc[j][mt][r];
  __syncthreads();
  for (int e = threadIdx.x; e < NTW * MT * 256; e += WAVES * 64) {
    const int j = e / (MT * 256), mt = (e >> 8) % MT, r = (e >> 6) & 3, ln = e & 63;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) v += red[w][j][mt][r][ln];
    tot[j][mt][r][ln] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < NTW * MT * 256; e += WAVES * 64) {
    const int j = e / (MT * 256), mt = (e >> 8) % MT, r = (e >> 6) & 3, ln = e & 63;
    const int nt = nt0 + j;
    if (nt >= NT) continue;
    const int i = (ln >> 4) * 4 + r;          // MFMA output row
    if (kRows == 8 && i >= 8) continue;       // lo rows are folded into their hi row
    const int m = mt * kRows + i;
    const int col = ln & 15;
    if (m >= M) continue;
    const float v = kRows == 8 ? tot[j][mt][r][ln] + tot[j][mt][r][ln + 32] : tot[j][mt][r][ln];
    if (EPI == kEpiStore) {
      const int n = nt * 16 + col;
      if (n < n_valid) out[s * oplane + static_cast<size_t>(m) * ldo + n] = v;
    } else if (EPI == kEpiGelu) {
      const int n = nt * 16 + col;
      if (n < n_valid) store_act(act, aplane, static_cast<size_t>(m) * lda + n, gelu_tanh(v));
    } else {  // SwiGLU: packed rows 0..7 are gate columns, 8..15 the matching up columns
      if (col < 8) {
        const int c = nt * 8 + col;
        const float up = kRows == 8 ? tot[j][mt][r][ln + 8] + tot[j][mt][r][ln + 40] : tot[j][mt][r][ln + 8];
        if (c < n_valid) store_act(act, aplane, static_cast<size_t>(m) * lda + c, silu(v) * up);
      }
    }
  }
}

template <typename T, int MT, int NTW, int WAVES, int U, int MINW = 1>
static hipError_t gemm_dispatch_epi(const GemmArgs& a, hipStream_t st) {
  const int NT = a.N / 16;
  const dim3 grid((NT + NTW - 1) / NTW, a.S), block(WAVES * 64);
  const T* X = static_cast<const T*>(a.X);
  const T* W = static_cast<const T*>(a.W);
  T* act = static_cast<T*>(a.act);
  switch (a.epi) {
    case kEpiStore:
      hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiStore, MINW>), grid, block, 0, st, X, a.ldx, a.xplane,
                         a.M, W, NT, a.KT, a.S, a.n_valid, a.out, a.ldo, a.oplane, act, a.lda, a.aplane);
      break;
    case kEpiGelu:
      hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiGelu, MINW>), grid, block, 0, st, X, a.ldx, a.xplane,
                         a.M, W, NT, a.KT, a.S, a.n_valid, a.out, a.ldo, a.oplane, act, a.lda, a.aplane);
      break;
    default:
      hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiSwiglu, MINW>), grid, block, 0, st, X, a.ldx, a.xplane,
                         a.M, W, NT, a.KT, a.S, a.n_valid, a.out, a.ldo, a.oplane, act, a.lda, a.aplane);
      break;
  }
  return hipGetLastError();
}

// Launch shape of the single-M-tile case (every verify and draft step):
// n-tiles per wave, waves per work-group, k-tiles per chunk. Overridable with
// SPS_GEMM_SHAPE=<index> for tuning sweeps.
struct GemmShape { int ntw, waves, u; };
constexpr GemmShape kShapes[] = {{1, 8, 8}, {2, 8, 8}, {2, 4, 8}, {4, 4, 4}, {1, 4, 16}, {2, 8, 4},
                                 {2, 8, 2}, {1, 8, 4}, {2, 4, 4}, {4, 4, 2}};
constexpr int kDefaultShape = 5;

int gemm_shape_index() {
  static int idx = -1;
  if (idx < 0) {
    const char* e = getenv("SPS_GEMM_SHAPE");
    int v = e ? atoi(e) : kDefaultShape;
    if (v < 0 || v >= static_cast<int>(sizeof(kShapes) / sizeof(kShapes[0]))) v = kDefaultShape;
    idx = v;
  }
  return idx;
}

template <typename T>
static hipError_t gemm_dispatch(const GemmArgs& a, hipStream_t st) {
  constexpr bool kB = sizeof(T) == 2;
  const int MT = (a.M + ActRows<T>::kRows - 1) / ActRows<T>::kRows;
  if constexpr (kB) {
    if (MT == 1) switch (gemm_shape_index()) {
      case 1: return gemm_dispatch_epi<T, 1, 2, 8, 8>(a, st);
      case 2: return gemm_dispatch_epi<T, 1, 2, 4, 8>(a, st);
      case 3: return gemm_dispatch_epi<T, 1, 4, 4, 4>(a, st);
      case 4: return gemm_dispatch_epi<T, 1, 1, 4, 16>(a, st);
      case 5: return gemm_dispatch_epi<T, 1, 2, 8, 4>(a, st);
      case 6: return gemm_dispatch_epi<T, 1, 2, 8, 2, 8>(a, st);
      case 7: return gemm_dispatch_epi<T, 1, 1, 8, 4, 8>(a, st);
      case 8: return gemm_dispatch_epi<T, 1, 2, 4, 4, 6>(a, st);
      case 9: return gemm_dispatch_epi<T, 1, 4, 4, 2, 8>(a, st);
      default: return gemm_dispatch_epi<T, 1, 1, 8, 8>(a, st);
    }
  }
  switch (MT) {
    case 1: return gemm_dispatch_epi<T, 1, 1, 8, kB ? 8 : 4>(a, st);
    case 2: return gemm_dispatch_epi<T, 2, 1, 8, kB ? 8 : 4>(a, st);
    case 3: return gemm_dispatch_epi<T, 3, 1, 4, kB ? 8 : 4>(a, st);
    case 4: return gemm_dispatch_epi<T, 4, 1, 4, kB ? 8 : 4>(a, st);
    case 5:
    case 6: return gemm_dispatch_epi<T, 6, 1, 4, 4>(a, st);
    case 7:
    case 8: return gemm_dispatch_epi<T, 8, 1, 4, 4>(a, st);
    default: return gemm_dispatch_epi<T, 10, 1, 4, 2>(a, st);
  }
}

int gemm_max_rows(int dtype) { return 10 * (dtype == 1 ? ActRows<bf16>::kRows : ActRows<float>::kRows); }

hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t st) {
  return dtype == 1 ? gemm_dispatch<bf16>(a, st) : gemm_dispatch<float>(a, st);
}

int gemm_splits(int dtype, int NT, int KT, int M, int epi) {
  if (epi != kEpiStore) return 1;
  const int MT = (M + (dtype == 1 ? 7 : 15)) / (dtype == 1 ? 8 : 16);
  int ntw = 1, waves = MT <= 2 ? 8 : 4;
  int U = MT >= 9 ? 2 : ((dtype == 1 && MT <= 4) ? 8 : 4);
  if (MT == 1 && dtype == 1) {
    const GemmShape g = kShapes[gemm_shape_index()];
    ntw = g.ntw; waves = g.waves; U = g.u;
  }
  const int groups = (NT + ntw - 1) / ntw;
  const int per_round = waves * U;
  int S = 2048 / (groups > 0 ? groups : 1);
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
