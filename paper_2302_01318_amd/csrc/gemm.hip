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
// Grid: one work-group per group of NTW 16-column output tiles; every
// work-group owns its output columns over the whole K, so epilogues can
// finish them without atomics. Its waves walk the k-tiles in chunks of U,
// round robin, each accumulating one 16 x 16 fp32 tile per (n-tile, M tile)
// with MFMA; the waves' partials are summed in LDS in a fixed order.
//
// FP8 weights (weight-only FP8 models): codes are stored in 16 x 64 tiles,
// one per pair of 32-deep k-tiles, ordered [nt][k-tile pair]. Lane l holds 16
// bytes: row 16 nt + l % 16, columns 8 (l / 16) .. +7 of the pair's first
// k-tile, then the same columns of its second, so one wave-wide 16 B load is
// still one contiguous KiB and yields two B fragments after an exact
// conversion to bf16 (fp8.h). The row scale multiplies the output in the
// epilogue: Y[m][n] = scale[n] * sum_k X[m][k] value(code[n][k]).
//
// Epilogues fuse the per-token work around each matmul:
//  * input RMSNorm: the producer of a normed activation writes u = h * gain
//    and per-column-group sums of squares; the consumer multiplies its
//    output row m by rs[m] = 1/sqrt(mean h^2 + eps) (RMSNorm is linear in h
//    once rs is known), so no separate norm kernel runs;
//  * residual (W_O, W_2): h += Y, then u = h * gain of the next norm and the
//    group's sums of squares;
//  * QKV: rotary encoding of q and k (rotate-half pairs are packed side by
//    side in one 16-row tile) and the KV-cache append;
//  * FFN: GELU or SwiGLU.
#include "common.h"
#include "fp8.h"
#include "gemm_epi.h"
#include "launch.h"

namespace sps {

template <typename T, int MT, int NTW, int WAVES, int U, int EPI, bool W8>
__global__ __launch_bounds__(WAVES * 64) void gemm_kernel(const GemmParams p) {
  static_assert(!W8 || (sizeof(T) == 2 && U % 2 == 0), "FP8 weights: bf16 activations, whole k-tile pairs");
  constexpr int kTile = 512;  // elements per 16 x 32 tile
  constexpr int kRows = ActRows<T>::kRows;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nt0 = blockIdx.x * NTW;
  const int KT = p.KT, M = p.M;
  const int r16 = lane & 15, grp = lane >> 4;
  const T* X = static_cast<const T*>(p.X);
  const T* W = static_cast<const T*>(p.W);

  const T* wp[NTW];
  bool wv[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    wv[j] = nt0 + j < p.NT;
    wp[j] = W + static_cast<size_t>(wv[j] ? nt0 + j : 0) * KT * kTile + lane * 8;
  }
  const T* xp[MT];
  bool xv[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * kRows + (kRows == 8 ? (r16 & 7) : r16);
    const size_t plane = kRows == 8 ? (r16 >> 3) * p.xplane : 0;
    xv[mt] = m < M;
    xp[mt] = X + plane + static_cast<size_t>(p.m0 + (xv[mt] ? m : 0)) * p.ldx + grp * 8;
  }
  f32x4 acc[NTW][MT];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One M tile with at most one output element per thread: the epilogue's
  // memory inputs (the input norm's group sums of squares, the old residual
  // and gain or the rotary table and length, FP8 row scales) are loaded
  // before the weight stream, so that the tail after the last weight load
  // waits on no memory round but its own stores.
  constexpr int kMaxRows = MT * kRows;
  constexpr bool kPre = MT == 1 && NTW * 256 <= WAVES * 64;
  constexpr int kPreRows = kPre ? (kMaxRows + WAVES - 1) / WAVES : 1;
  NormPre pre_norm[kPreRows];
  EpiIn pre_in{0.f, 0.f, 0};
  float pre_sc = 1.f, pre_sc2 = 1.f;
  if constexpr (kPre) {
#pragma unroll
    for (int i = 0; i < kPreRows; ++i) pre_norm[i] = norm_prefetch(p, wave + i * WAVES, lane);
    const int e = threadIdx.x;
    if (e < NTW * 256) {
      const int j = e >> 8, r = (e >> 6) & 3, ln = e & 63;
      const int nt = nt0 + j, i = (ln >> 4) * 4 + r, col = ln & 15;
      if (!(kRows == 8 && i >= 8) && nt < p.NT && i < M) {
        pre_in = epilogue_inputs<EPI>(p, p.m0 + i, nt, col);
        if (W8) {
          pre_sc = p.wscale[nt * 16 + col];
          if ((EPI == kEpiSwiglu || EPI == kEpiQkv) && col < 8) pre_sc2 = p.wscale[nt * 16 + col + 8];
        }
      }
    }
  }

  if constexpr (W8) {
    // Code tile pair kp of n-tile j: 64 lanes x 16 B at wq[j] + 64 kp.
    const u32x4* wq[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
      wq[j] = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(p.W) +
                                             static_cast<size_t>(wv[j] ? nt0 + j : 0) * KT * kTile) + lane;
    // One pair: two activation fragments, one code load per n-tile.
    auto pair = [&](int kt, const u32x4 (&raw)[NTW], const Frag<T> (&a0)[MT], const Frag<T> (&a1)[MT]) {
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        Frag<T> b0, b1;
        e4m3x16_to_frags(raw[j], b0, b1);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          acc[j][mt] = mma8(acc[j][mt], a0[mt], b0);
          acc[j][mt] = mma8(acc[j][mt], a1[mt], b1);
        }
      }
    };
    int kb = wave * U;
    for (; kb + U <= KT; kb += WAVES * U) {
      u32x4 raw[U / 2][NTW];
      Frag<T> a[U][MT];
#pragma unroll
      for (int u = 0; u < U / 2; ++u)
#pragma unroll
        for (int j = 0; j < NTW; ++j)
          raw[u][j] = wv[j] ? __builtin_nontemporal_load(wq[j] + static_cast<size_t>(kb / 2 + u) * 64)
                            : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) a[u][mt] = xv[mt] ? load_frag(xp[mt] + (kb + u) * 32) : Frag<T>::zero();
#pragma unroll
      for (int u = 0; u < U / 2; ++u) pair(kb + 2 * u, raw[u], a[2 * u], a[2 * u + 1]);
    }
    // Ragged last chunk: KT is even, so pairs stay whole.
    for (int kt = kb; kt < KT && kt < kb + U; kt += 2) {
      u32x4 raw[NTW];
      Frag<T> a0[MT], a1[MT];
#pragma unroll
      for (int j = 0; j < NTW; ++j)
        raw[j] = wv[j] ? __builtin_nontemporal_load(wq[j] + static_cast<size_t>(kt / 2) * 64) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        a0[mt] = xv[mt] ? load_frag(xp[mt] + kt * 32) : Frag<T>::zero();
        a1[mt] = xv[mt] ? load_frag(xp[mt] + (kt + 1) * 32) : Frag<T>::zero();
      }
      pair(kt, raw, a0, a1);
    }
  } else {
  int kb = wave * U;
  for (; kb + U <= KT; kb += WAVES * U) {
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
  if (kb < KT) {  // ragged last chunk of this wave
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kt = kb + u;
      if (kt < KT) {
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
  }

  // Sum the waves' partials in LDS (fixed order), then the epilogue.
  __shared__ float red[WAVES][NTW][MT][4][64];
  __shared__ float tot[NTW][MT][4][64];
  __shared__ float s_rs[kMaxRows];
  // Squares of the residual outputs reuse the wave-partial buffer, which is
  // dead once `tot` holds the sums.
  constexpr int kSqLd = NTW * 16 + 1;
  static_assert(kMaxRows * kSqLd <= WAVES * NTW * MT * 256, "square buffer must fit the partial buffer");
  float (*s_sq)[kSqLd] = reinterpret_cast<float (*)[kSqLd]>(&red[0][0][0][0][0]);
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][j][mt][r][lane] = acc[j][mt][r];
  // Row scales of the input RMSNorm.
  if constexpr (kPre) {
#pragma unroll
    for (int i = 0; i < kPreRows; ++i) {
      const int m = wave + i * WAVES;
      if (m < kMaxRows) {
        const float v = norm_from_pre(p, m, lane, pre_norm[i]);
        if (lane == 0) s_rs[m] = v;
      }
    }
  } else {
    for (int m = wave; m < kMaxRows; m += WAVES) {
      const float v = norm_scale(p, m, lane);
      if (lane == 0) s_rs[m] = v;
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < NTW * MT * 256; e += WAVES * 64) {
    const int j = e / (MT * 256), mt = (e >> 8) % MT, r = (e >> 6) & 3, ln = e & 63;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) v += red[w][j][mt][r][ln];
    tot[j][mt][r][ln] = v;
  }
  __syncthreads();

  // Value of output (row i of M tile mt, column ln & 15 of n-tile j) with the
  // lo-plane rows of a bf16 tile folded in.
  auto out_value = [&](int j, int mt, int r, int ln) -> float {
    return kRows == 8 ? tot[j][mt][r][ln] + tot[j][mt][r][ln + 32] : tot[j][mt][r][ln];
  };
  for (int e = threadIdx.x; e < NTW * MT * 256; e += WAVES * 64) {
    const int j = e / (MT * 256), mt = (e >> 8) % MT, r = (e >> 6) & 3, ln = e & 63;
    const int nt = nt0 + j;
    const int i = (ln >> 4) * 4 + r;          // MFMA output row
    const int col = ln & 15;
    const int m = mt * kRows + i;
    if (kRows == 8 && i >= 8) continue;       // lo rows are folded into their hi row
    if (EPI == kEpiResid) s_sq[m < kMaxRows ? m : 0][j * 16 + col] = 0.f;
    if (nt >= p.NT || m >= M) continue;
    const int gm = p.m0 + m;
    const float rs = s_rs[m];
    const float sc = !W8 ? 1.f : kPre ? pre_sc : p.wscale[nt * 16 + col];
    const float v = out_value(j, mt, r, ln) * rs * sc;
    const float v2 = (EPI == kEpiSwiglu || EPI == kEpiQkv) && col < 8
                         ? out_value(j, mt, r, ln + 8) * rs * (!W8 ? 1.f : kPre ? pre_sc2 : p.wscale[nt * 16 + col + 8])
                         : 0.f;
    const float sq = epilogue_apply<T, EPI>(p, gm, nt, col, v, v2, kPre ? pre_in : epilogue_inputs<EPI>(p, gm, nt, col));
    if (EPI == kEpiResid && nt * 16 + col < p.n_valid) s_sq[m][j * 16 + col] = sq;
  }
  if (EPI == kEpiResid) {
    // Sums of squares of this group's columns, per row, in a fixed order.
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += WAVES * 64) {
      float s = 0.f;
      for (int c = 0; c < NTW * 16; ++c) s += s_sq[m][c];
      p.ss_out[static_cast<size_t>(blockIdx.x) * p.Mtot + p.m0 + m] = s;
    }
  }
}

// Launch shape for one launch: n-tiles per wave, waves per work-group, k-tiles
// per chunk. A single M tile (every verify and draft step) streams two n-tiles
// per wave with 8-wave work-groups on large matrices (single_tile_ntw), else
// one n-tile per wave with 16-wave work-groups.
template <typename T, int MT, int NTW, int WAVES, int U, bool W8 = false>
static hipError_t gemm_launch(const GemmParams& p, hipStream_t st) {
  const dim3 grid((p.NT + NTW - 1) / NTW), block(WAVES * 64);
  switch (p.epi) {
    case kEpiStore: hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiStore, W8>), grid, block, 0, st, p); break;
    case kEpiGelu: hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiGelu, W8>), grid, block, 0, st, p); break;
    case kEpiSwiglu: hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiSwiglu, W8>), grid, block, 0, st, p); break;
    case kEpiResid: hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiResid, W8>), grid, block, 0, st, p); break;
    default: hipLaunchKernelGGL((gemm_kernel<T, MT, NTW, WAVES, U, kEpiQkv, W8>), grid, block, 0, st, p); break;
  }
  return hipGetLastError();
}

// fp32 models (16-row M tiles) at any row count, bf16 models at <= 8 rows.
// bf16 launches over more rows go to the wide kernel (gemm_wide.hip).
static hipError_t gemm_dispatch_f32(const GemmParams& p, hipStream_t st) {
  using T = float;
  const int MT = (p.M + ActRows<T>::kRows - 1) / ActRows<T>::kRows;
  if (MT == 1) {
    if (p.Mtot <= ActRows<T>::kRows && single_tile_ntw(p.NT, p.KT) == 2) return gemm_launch<T, 1, 2, 8, 4>(p, st);
    return gemm_launch<T, 1, 1, 16, 4>(p, st);
  }
  switch (MT) {
    case 2: return gemm_launch<T, 2, 1, 8, 4>(p, st);
    case 3: return gemm_launch<T, 3, 1, 4, 4>(p, st);
    case 4: return gemm_launch<T, 4, 1, 4, 4>(p, st);
    case 5:
    case 6: return gemm_launch<T, 6, 1, 4, 4>(p, st);
    case 7:
    case 8: return gemm_launch<T, 8, 1, 4, 4>(p, st);
    default: return gemm_launch<T, 10, 1, 4, 2>(p, st);
  }
}

static hipError_t gemm_dispatch_bf16(const GemmParams& p, hipStream_t st) {
  using T = bf16;
  if (gemm_is_wide(1, p.Mtot)) return launch_gemm_wide(p, wide_plan(p.NT, p.KT, p.M, false), st);
  if (p.M > ActRows<T>::kRows) return hipErrorInvalidValue;
  if (single_tile_ntw(p.NT, p.KT) == 2) return gemm_launch<T, 1, 2, 8, 4>(p, st);
  // Narrow outputs over a long contraction (the 7B W_2 and the draft's W_2:
  // 256 or fewer n-tiles, >= 256 k-tiles) stream faster from 8-wave groups.
  if (p.KT >= 256) return gemm_launch<T, 1, 1, 8, 4>(p, st);
  // Wide, shallow matrices (>= 512 n-tiles over <= 128 k-tiles: the draft's
  // QKV and W_1, the 7B QKV) from 4-wave groups of 2-k-tile chunks: each
  // wave streams 24-32 k-tiles instead of 6-8, and the group's reduction
  // sums 4 partials instead of 16 (a sweep over 4 / 8 / 16 waves and 2 / 4 /
  // 8 k-tiles per chunk at 1, 2 and 5 rows: draft W_1 15.3 -> 14.0 us, 7B QKV
  // 20.5 -> 19.5 us).
  if (p.NT >= 512 && p.KT <= 128) return gemm_launch<T, 1, 1, 4, 2>(p, st);
  return gemm_launch<T, 1, 1, 16, 4>(p, st);
}

static hipError_t gemm_dispatch_fp8(const GemmParams& p, hipStream_t st) {
  using T = bf16;
  if (!p.wscale || p.KT % 2) return hipErrorInvalidValue;
  if (gemm_is_wide(2, p.Mtot)) return launch_gemm_wide(p, wide_plan(p.NT, p.KT, p.M, true), st);
  if (p.M > ActRows<T>::kRows) return hipErrorInvalidValue;
  if (fp8_ntw(p.NT, p.KT) == 2) return gemm_launch<T, 1, 2, 8, 4, true>(p, st);
  return gemm_launch<T, 1, 1, 16, 8, true>(p, st);
}


hipError_t launch_gemm(int dtype, const GemmParams& p, hipStream_t st) {
  return dtype == 2 ? gemm_dispatch_fp8(p, st) : dtype == 1 ? gemm_dispatch_bf16(p, st) : gemm_dispatch_f32(p, st);
}

// ---------------------------------------------------------------------------
// Packing canonical [n][k] rows into tile order.
// ---------------------------------------------------------------------------
// Packed row of canonical row n: kind 0 row_off + n; kind 1 SwiGLU gate /
// up interleaving; kind 2 rotary partners side by side.
__device__ __forceinline__ int packed_row(int n, int kind, int row_off, int dh) {
  return kind == 0   ? row_off + n
         : kind == 1 ? (n / 8) * 16 + row_off * 8 + (n % 8)
                     : row_off + (n / dh) * dh + rope_pack_index(n % dh, dh);
}

template <typename T>
__global__ void pack_kernel(const T* __restrict__ src, int n_src, int Kd, T* __restrict__ dst, int KT,
                            int kind, int row_off, int dh) {
  const int groups = Kd / 8;
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(n_src) * groups) return;
  const int n = static_cast<int>(i / groups), k = static_cast<int>(i % groups) * 8;
  const int nf = packed_row(n, kind, row_off, dh);
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
static hipError_t pack_t(const void* src, int n_src, int Kd, void* dst, int KT, int kind, int row_off, int dh,
                         int zero_from, int zero_to, hipStream_t st) {
  const long work = static_cast<long>(n_src) * (Kd / 8);
  if (work > 0)
    hipLaunchKernelGGL(pack_kernel<T>, dim3(static_cast<unsigned>((work + 255) / 256)), dim3(256), 0, st,
                       static_cast<const T*>(src), n_src, Kd, static_cast<T*>(dst), KT, kind, row_off, dh);
  const long zwork = static_cast<long>(zero_to - zero_from) * KT * 4;
  if (zwork > 0)
    hipLaunchKernelGGL(pack_zero_kernel<T>, dim3(static_cast<unsigned>((zwork + 255) / 256)), dim3(256), 0,
                       st, static_cast<T*>(dst), KT, zero_from, zero_to);
  return hipGetLastError();
}

// Byte offset of code (packed row nf, column k) in an FP8 projection of KT
// k-tiles (16 x 64 tiles of k-tile pairs, see the header comment).
__device__ __forceinline__ size_t fp8_offset(int nf, int k, int KT) {
  const int nt = nf / 16, rr = nf % 16, kp = k / 64, half = (k % 64) / 32, grp = (k % 32) / 8;
  return ((static_cast<size_t>(nt) * (KT / 2) + kp) * 64 + rr + 16 * grp) * 16 + half * 8 + (k % 8);
}

// One work-group per canonical row: the row's largest |w| (exact in fp32),
// its scale, then every code.
__global__ __launch_bounds__(256) void pack_fp8_kernel(const bf16* __restrict__ src, int Kd,
                                                       uint8_t* __restrict__ dst, float* __restrict__ scales,
                                                       int KT, int kind, int row_off, int dh) {
  __shared__ float red[16];
  const int n = blockIdx.x;
  const bf16* s = src + static_cast<size_t>(n) * Kd;
  float amax = 0.f;
  for (int k = threadIdx.x; k < Kd; k += blockDim.x) amax = fmaxf(amax, fabsf(static_cast<float>(s[k])));
  amax = block_max(amax, red);
  const float sc = amax > 0.f ? __fdiv_rn(amax, 448.0f) : 1.0f;
  const int nf = packed_row(n, kind, row_off, dh);
  if (threadIdx.x == 0) scales[nf] = sc;
  for (int k = threadIdx.x; k < Kd; k += blockDim.x)
    dst[fp8_offset(nf, k, KT)] = static_cast<uint8_t>(e4m3_encode(__fdiv_rn(static_cast<float>(s[k]), sc)));
}

// Padding rows [zero_from, zero_to): code 0, scale 1.
__global__ void pack_zero_fp8_kernel(uint8_t* __restrict__ dst, float* __restrict__ scales, int KT, int zero_from,
                                     int zero_to) {
  const int Kd = KT * 32;
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(zero_to - zero_from) * Kd) return;
  const int nf = zero_from + static_cast<int>(i / Kd), k = static_cast<int>(i % Kd);
  dst[fp8_offset(nf, k, KT)] = 0;
  if (k == 0) scales[nf] = 1.0f;
}

hipError_t launch_pack_fp8(const void* src, int n_src, int Kd, void* dst, float* scales, int KT, int kind,
                           int row_off, int dh, int zero_from, int zero_to, hipStream_t st) {
  if (KT % 2 || Kd != KT * 32) return hipErrorInvalidValue;
  if (n_src > 0)
    hipLaunchKernelGGL(pack_fp8_kernel, dim3(n_src), dim3(256), 0, st, static_cast<const bf16*>(src), Kd,
                       static_cast<uint8_t*>(dst), scales, KT, kind, row_off, dh);
  const long zwork = static_cast<long>(zero_to - zero_from) * Kd;
  if (zwork > 0)
    hipLaunchKernelGGL(pack_zero_fp8_kernel, dim3(static_cast<unsigned>((zwork + 255) / 256)), dim3(256), 0, st,
                       static_cast<uint8_t*>(dst), scales, KT, zero_from, zero_to);
  return hipGetLastError();
}

// E4M3 codes to fp32 with the GEMM's conversion: 16 codes per thread.
__global__ void fp8_decode_kernel(const u32x4* __restrict__ codes, int n16, float* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n16) return;
  Frag<bf16> lo, hi;
  e4m3x16_to_frags(codes[i], lo, hi);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    out[static_cast<size_t>(i) * 16 + e] = static_cast<float>(lo.v[e]);
    out[static_cast<size_t>(i) * 16 + 8 + e] = static_cast<float>(hi.v[e]);
  }
}

hipError_t launch_fp8_decode(const void* codes, int n, float* out, hipStream_t st) {
  if (n % 16) return hipErrorInvalidValue;
  const int n16 = n / 16;
  if (n16 > 0)
    hipLaunchKernelGGL(fp8_decode_kernel, dim3((n16 + 255) / 256), dim3(256), 0, st,
                       static_cast<const u32x4*>(codes), n16, out);
  return hipGetLastError();
}

hipError_t launch_pack(int dtype, const void* src, int n_src, int Kd, void* dst, int KT, int kind,
                       int row_off, int dh, int zero_from, int zero_to, hipStream_t st) {
  return dtype == 1 ? pack_t<bf16>(src, n_src, Kd, dst, KT, kind, row_off, dh, zero_from, zero_to, st)
                    : pack_t<float>(src, n_src, Kd, dst, KT, kind, row_off, dh, zero_from, zero_to, st);
}

}  // namespace sps
