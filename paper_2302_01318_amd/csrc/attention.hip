// Decode attention of the verify / draft forward: the M_s new queries of each
// sequence (K+1 in a verify step) against its whole KV cache, which includes
// the keys and values of the new tokens themselves (query j at position
// P + j sees positions <= P + j). The paper notes this part is bound by the
// KV-cache reads and is nearly independent of K (Conditional Scoring section).
//
// Split-KV: each wave owns 128 consecutive positions (four 32-position blocks)
// of one (sequence, head) and up to 16 queries per query tile. Per block it
// computes S^T = K Q^T with MFMA (A = key tile, B = Q^T), runs the online
// softmax on the S^T registers, and accumulates O^T = V^T P^T (A = value
// tile, B = the softmax tile as the score MFMA left it in registers, thanks
// to the value tile layout). Each wave writes its (O, running max, running
// sum) partial; a second kernel merges the partials of a (sequence, head,
// query) and normalises.
#include "common.h"
#include "launch.h"

namespace sps {

constexpr int kPosPerWave = 128;

template <typename T, int DH, int QT>
__global__ __launch_bounds__(256) void attn_partial_kernel(const T* __restrict__ q, const T* __restrict__ kc,
                                                           const T* __restrict__ vc,
                                                           const int32_t* __restrict__ lengths, int pos_offset,
                                                           int Mps, int H, int T_cap, int NP, float c_log2,
                                                           float* __restrict__ part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int b = blockIdx.z, h = blockIdx.y;
  const int pw = blockIdx.x * 4 + wave;
  if (pw >= NP) return;
  const int r16 = lane & 15, grp = lane >> 4;
  const int len = lengths[b] + pos_offset;        // position of query 0
  int nkv = len + Mps;
  if (nkv > T_cap) nkv = T_cap;
  const int p0 = pw * kPosPerWave;
  const int HD = H * DH;
  const size_t region = (static_cast<size_t>(b) * H + h) * static_cast<size_t>(T_cap) * DH;
  const T* kr = kc + region;
  const T* vr = vc + region;

  Frag<T> qf[QT][DH / 32];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qi = qt * 16 + r16;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
      qf[qt][dt] = qi < Mps ? load_frag(q + (static_cast<size_t>(b) * Mps + qi) * HD + h * DH + dt * 32 + grp * 8)
                            : Frag<T>::zero();
  }
  float m_run[QT], l_run[QT];
  f32x4 o[QT][DH / 16];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_run[qt] = -INFINITY;
    l_run[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  int nblk = nkv > p0 ? (nkv - p0 + 31) / 32 : 0;
  if (nblk > kPosPerWave / 32) nblk = kPosPerWave / 32;
  for (int blk = 0; blk < nblk; ++blk) {
    const int pb = p0 / 32 + blk;
    Frag<T> kf[2][DH / 32];
    Frag<T> vf[DH / 16];
#pragma unroll
    for (int pt = 0; pt < 2; ++pt)
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt)
        kf[pt][dt] = load_frag(kr + ((static_cast<size_t>(pb * 2 + pt) * (DH / 32) + dt) * 64 + lane) * 8);
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt)
      vf[dt] = load_frag(vr + ((static_cast<size_t>(pb) * (DH / 16) + dt) * 64 + lane) * 8);
    if (pb * 32 + 32 > nkv) {
      // Positions past the last written one hold whatever the buffer held;
      // their softmax weight is 0, but 0 * NaN is not, so clear them.
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int pos = pb * 32 + (e < 4 ? grp * 4 + e : 16 + grp * 4 + e - 4);
        if (pos >= nkv) {
#pragma unroll
          for (int dt = 0; dt < DH / 16; ++dt) vf[dt].v[e] = from_f32<T>(0.f);
        }
      }
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      f32x4 s[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int pt = 0; pt < 2; ++pt)
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) s[pt] = mma8(s[pt], kf[pt][dt], qf[qt][dt]);
      const int qi = qt * 16 + r16;
      const int qpos = len + qi;
      float mx = -INFINITY;
#pragma unroll
      for (int pt = 0; pt < 2; ++pt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pos = pb * 32 + pt * 16 + grp * 4 + r;
          const bool valid = qi < Mps && pos <= qpos && pos < nkv;
          s[pt][r] = valid ? s[pt][r] : -INFINITY;
          mx = fmaxf(mx, s[pt][r]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[qt], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f((m_run[qt] - m_use) * c_log2);
      Frag<T> pf;
      float ps = 0.f;
#pragma unroll
      for (int pt = 0; pt < 2; ++pt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const T pv = from_f32<T>(exp2f((s[pt][r] - m_use) * c_log2));
          pf.v[pt * 4 + r] = pv;
          ps += to_f32(pv);
        }
      l_run[qt] = l_run[qt] * alpha + ps;
      m_run[qt] = m_new;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
        o[qt][dt] *= alpha;
        o[qt][dt] = mma8(o[qt][dt], vf[dt], pf);
      }
    }
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float l = l_run[qt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int qi = qt * 16 + r16;
    if (qi < Mps) {
      float* dst = part + (((static_cast<size_t>(b) * H + h) * NP + pw) * Mps + qi) * (DH + 2);
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[dt * 16 + grp * 4 + r] = o[qt][dt][r];
      if (grp == 0) {
        dst[DH] = m_run[qt];
        dst[DH + 1] = l;
      }
    }
  }
}

// Merge the per-wave partials of one (sequence, query) for all heads and
// normalise: o = sum_w 2^{(m_w - M) c} O_w / sum_w 2^{(m_w - M) c} l_w.
template <typename T, int DH>
__global__ __launch_bounds__(DH) void attn_combine_kernel(const float* __restrict__ part, const int32_t* __restrict__ lengths,
                                                          int pos_offset, int Mps, int H, int T_cap, int NP,
                                                          float c_log2, T* __restrict__ o) {
  const int row = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
  const int b = row / Mps, qi = row % Mps;
  int nkv = lengths[b] + pos_offset + Mps;
  if (nkv > T_cap) nkv = T_cap;
  int np = (nkv + kPosPerWave - 1) / kPosPerWave;
  if (np > NP) np = NP;
  if (np < 0) np = 0;
  const float* base = part + ((static_cast<size_t>(b) * H + h) * NP * Mps + qi) * (DH + 2);
  const size_t stride = static_cast<size_t>(Mps) * (DH + 2);
  float M = -INFINITY;
  for (int p = 0; p < np; ++p) M = fmaxf(M, base[p * stride + DH]);
  float L = 0.f, acc = 0.f;
  if (M != -INFINITY) {
    for (int p = 0; p < np; ++p) {
      const float* pp = base + p * stride;
      const float mp = pp[DH];
      if (mp == -INFINITY) continue;
      const float w = exp2f((mp - M) * c_log2);
      L += w * pp[DH + 1];
      acc += w * pp[d];
    }
  }
  o[static_cast<size_t>(row) * H * DH + h * DH + d] = from_f32<T>(L > 0.f ? acc / L : 0.f);
}

int attn_partials(int T_cap) { return (T_cap + kPosPerWave - 1) / kPosPerWave; }

template <typename T, int DH>
static hipError_t attn_t(const void* q, const void* kc, const void* vc, const int32_t* lengths, int pos_offset,
                         int B, int Mps, int H, int T_cap, float* part, void* o, hipStream_t st) {
  const int NP = attn_partials(T_cap);
  const float c_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(DH));
  const dim3 grid((NP + 3) / 4, H, B);
  const T* qq = static_cast<const T*>(q);
  const T* kk = static_cast<const T*>(kc);
  const T* vv = static_cast<const T*>(vc);
  if (Mps <= 16)
    hipLaunchKernelGGL((attn_partial_kernel<T, DH, 1>), grid, dim3(256), 0, st, qq, kk, vv, lengths, pos_offset,
                       Mps, H, T_cap, NP, c_log2, part);
  else if (Mps <= 32)
    hipLaunchKernelGGL((attn_partial_kernel<T, DH, 2>), grid, dim3(256), 0, st, qq, kk, vv, lengths, pos_offset,
                       Mps, H, T_cap, NP, c_log2, part);
  else
    hipLaunchKernelGGL((attn_partial_kernel<T, DH, 4>), grid, dim3(256), 0, st, qq, kk, vv, lengths, pos_offset,
                       Mps, H, T_cap, NP, c_log2, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), dim3(B * Mps, H), dim3(DH), 0, st, part, lengths, pos_offset,
                     Mps, H, T_cap, NP, c_log2, static_cast<T*>(o));
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const void* q, const void* kc, const void* vc, const int32_t* lengths,
                            int pos_offset, int B, int Mps, int H, int DH, int T_cap, float* part, void* o,
                            hipStream_t st) {
  if (dtype == 1)
    return DH == 128 ? attn_t<bf16, 128>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, st)
                     : attn_t<bf16, 64>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, st);
  return DH == 128 ? attn_t<float, 128>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, st)
                   : attn_t<float, 64>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, st);
}

}  // namespace sps
