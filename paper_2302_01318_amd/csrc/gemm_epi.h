// Per-element GEMM epilogues shared by the single-tile and the wide GEMM
// kernels (gemm.hip, gemm_wide.hip). See launch.h for what each computes.
#pragma once
#include "common.h"
#include "launch.h"

namespace sps {

__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f, k1 = 0.044715f;
  return 0.5f * x * (1.0f + tanhf(k0 * (x + k1 * x * x * x)));
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// Activation rows per 16-row MFMA tile: bf16 tiles carry 8 rows as hi and lo
// planes, fp32 tiles 16 rows.
template <typename T> struct ActRows;
template <> struct ActRows<bf16> { static constexpr int kRows = kActRowsBf16; };
template <> struct ActRows<float> { static constexpr int kRows = kActRowsF32; };

// Packed position of dim f of a head in a QKV tile: the rotate-half partners
// f and f + DH/2 sit in rows r and r + 8 of the same 16-row tile.
__host__ __device__ __forceinline__ int rope_pack_index(int f, int DH) {
  const int half = DH / 2;
  return f < half ? (f / 8) * 16 + f % 8 : ((f - half) / 8) * 16 + 8 + (f - half) % 8;
}

// Row scale of the input RMSNorm for local row m (1 when the GEMM has no
// normed input): rs = 1 / sqrt(sum_g ss_in[g][m] / d + eps). One wave sums
// the groups, lane l those of index l, l + 64, ... in that order; every lane
// returns the result. norm_first loads a lane's first group and norm_finish
// adds the rest and reduces, so that callers can issue the first loads of
// several rows together.
__device__ __forceinline__ float norm_first(const GemmParams& p, int m, int lane) {
  return p.ss_in && m < p.M && lane < p.ng_in ? p.ss_in[static_cast<size_t>(lane) * p.Mtot + p.m0 + m] : 0.f;
}
__device__ __forceinline__ float norm_finish(const GemmParams& p, int m, int lane, float s) {
  if (!p.ss_in || m >= p.M) return 1.f;
  for (int g = lane + 64; g < p.ng_in; g += 64) s += p.ss_in[static_cast<size_t>(g) * p.Mtot + p.m0 + m];
  s = wave_sum(s);
  return 1.0f / sqrtf(s * p.inv_d + p.eps);
}
__device__ __forceinline__ float norm_scale(const GemmParams& p, int m, int lane) {
  return norm_finish(p, m, lane, norm_first(p, m, lane));
}

// The same row scale with a lane's first kNormPre groups loaded ahead (by
// norm_prefetch, e.g. before a GEMM's main loop, so that the loads' latency
// hides under the weight stream); norm_from_pre adds them and any further
// groups in the order norm_scale does, so the result is the same bits.
constexpr int kNormPre = 4;
struct NormPre {
  float v[kNormPre];
};
__device__ __forceinline__ NormPre norm_prefetch(const GemmParams& p, int m, int lane) {
  NormPre r;
  const bool on = p.ss_in && m < p.M;
#pragma unroll
  for (int q = 0; q < kNormPre; ++q) {
    const int g = lane + 64 * q;
    r.v[q] = on && g < p.ng_in ? p.ss_in[static_cast<size_t>(g) * p.Mtot + p.m0 + m] : 0.f;
  }
  return r;
}
__device__ __forceinline__ float norm_from_pre(const GemmParams& p, int m, int lane, const NormPre& r) {
  if (!p.ss_in || m >= p.M) return 1.f;
  float s = r.v[0];
#pragma unroll
  for (int q = 1; q < kNormPre; ++q)
    if (lane + 64 * q < p.ng_in) s += r.v[q];
  for (int g = lane + 64 * kNormPre; g < p.ng_in; g += 64) s += p.ss_in[static_cast<size_t>(g) * p.Mtot + p.m0 + m];
  s = wave_sum(s);
  return 1.0f / sqrtf(s * p.inv_d + p.eps);
}

// Inputs of an element's epilogue that live in memory: the old residual
// value and the norm gain (kEpiResid), the sequence's length and the rotary
// (cos, sin) of a q / k pair (kEpiQkv). Loading them for several elements
// before any of their stores lets a thread's loads overlap: in a loop of
// whole elements the compiler keeps each load behind the previous element's
// stores, which may alias it.
struct EpiIn {
  float a, b;
  int len;
};
template <int EPI>
__device__ __forceinline__ EpiIn epilogue_inputs(const GemmParams& p, int gm, int nt, int col) {
  EpiIn in{0.f, 0.f, 0};
  const int n = nt * 16 + col;
  if (EPI == kEpiResid) {
    if (n < p.n_valid) {
      in.a = p.h[static_cast<size_t>(gm) * p.n_valid + n];
      in.b = p.gain[n];
    }
  } else if (EPI == kEpiQkv) {
    in.len = p.lengths[gm / p.Mps];
    if (n < 2 * p.H * p.DH && col < 8) {
      const int f = ((n % p.DH) / 16) * 8 + col;
      const float2 cs = p.rope[static_cast<size_t>(gm) * (p.DH / 2) + f];   // cos, sin (embed_kernel)
      in.a = cs.x;
      in.b = cs.y;
    }
  }
  return in;
}

// Epilogue of output element (global row gm, packed column 16 nt + col) with
// value v (already scaled by the row's norm scale) and its memory inputs in.
// v2 is the value of column 16 nt + col + 8 when col < 8: the SwiGLU up
// projection of a gate column, or the rotate-half partner of a q / k dim.
// Returns h^2 of the new residual value for kEpiResid (0 for columns past
// n_valid), else 0.
template <typename T, int EPI>
__device__ __forceinline__ float epilogue_apply(const GemmParams& p, int gm, int nt, int col, float v, float v2,
                                                const EpiIn& in) {
  if (EPI == kEpiStore) {
    const int n = nt * 16 + col;
    if (n < p.n_valid) p.out[static_cast<size_t>(gm) * p.ldo + n] = v;
  } else if (EPI == kEpiGelu) {
    const int n = nt * 16 + col;
    if (n < p.n_valid) store_act(static_cast<T*>(p.act), p.aplane, static_cast<size_t>(gm) * p.lda + n, gelu_tanh(v));
  } else if (EPI == kEpiSwiglu) {  // packed rows 0..7 gate columns, 8..15 the matching up columns
    if (col < 8) {
      const int c = nt * 8 + col;
      if (c < p.n_valid) store_act(static_cast<T*>(p.act), p.aplane, static_cast<size_t>(gm) * p.lda + c, silu(v) * v2);
    }
  } else if (EPI == kEpiResid) {
    const int n = nt * 16 + col;
    if (n < p.n_valid) {
      const float hn = in.a + v;
      p.h[static_cast<size_t>(gm) * p.n_valid + n] = hn;
      store_act(static_cast<T*>(p.u), p.uplane, static_cast<size_t>(gm) * p.ldu + n, hn * in.b);
      return hn * hn;
    }
  } else {  // kEpiQkv
    const int n = nt * 16 + col;
    const int HD = p.H * p.DH;
    const int b = gm / p.Mps, jr = gm % p.Mps;
    const int pos = in.len + p.pos_offset + jr;
    const bool ok = pos >= 0 && pos < p.T_cap;
    if (!ok && n == 0) atomicOr(p.err, kErrCapacity);
    if (n < 2 * HD) {                        // q or k: rotate the pair held by columns col, col + 8
      if (col < 8) {
        const int hh = (n % HD) / p.DH, pi = n % p.DH;
        const int f = (pi / 16) * 8 + col;
        const float c = in.a, s = in.b;
        const float y1 = v * c - v2 * s, y2 = v2 * c + v * s;
        const int half = p.DH / 2;
        if (n < HD) {
          T* q = static_cast<T*>(p.q) + static_cast<size_t>(gm) * HD + hh * p.DH;
          q[f] = from_f32<T>(y1);
          q[f + half] = from_f32<T>(y2);
        } else if (ok) {
          T* kr = static_cast<T*>(p.kc) + (static_cast<size_t>(b) * p.H + hh) * p.T_cap * p.DH;
          kr[k_offset(pos, f, p.DH)] = from_f32<T>(y1);
          kr[k_offset(pos, f + half, p.DH)] = from_f32<T>(y2);
        }
      }
    } else if (ok && n < 3 * HD) {           // v: straight into the cache
      const int hh = (n - 2 * HD) / p.DH, dd = (n - 2 * HD) % p.DH;
      T* vr = static_cast<T*>(p.vc) + (static_cast<size_t>(b) * p.H + hh) * p.T_cap * p.DH;
      vr[v_offset(pos, dd, p.DH)] = from_f32<T>(v);
    }
  }
  return 0.f;
}

}  // namespace sps
