// Decode attention of the verify / draft forward: the M_s new queries of each
// sequence (K+1 in a verify step) against its whole KV cache, which includes
// the keys and values of the new tokens themselves (query j at position
// P + j sees positions <= P + j). The paper notes this part is bound by the
// KV-cache reads and is nearly independent of K (Conditional Scoring section).
//
// Split-KV: each wave owns 64 consecutive positions (two 32-position blocks)
// of one (sequence, head) and up to 16 queries per query tile. Per block it
// computes S^T = K Q^T with MFMA (A = key tile, B = Q^T), runs the online
// softmax on the S^T registers, and accumulates O^T = V^T P^T (A = value
// tile, B = the softmax tile as the score MFMA left it in registers, thanks
// to the value tile layout). The (O, running max, running sum) partials are
// merged per work-group in LDS when possible; a second kernel merges the
// partials of a (sequence, head, query) and normalises.
#include "common.h"
#include "launch.h"

namespace sps {

constexpr int kWavePos = kAttnWavePos;   // positions per wave (prefill chunks): two 32-position blocks

// One 32-position block for one query tile: scores, masked online softmax,
// and accumulation of O^T. For bf16 the softmax weights enter the P V MFMA
// as a hi + lo pair of bf16 values (p = hi + lo to ~2^-16 relative), so the
// product is as accurate as an fp32 P at the cost of one more MFMA.
template <typename T, int DH>
__device__ __forceinline__ void attn_block(const Frag<T> (&kf)[2][DH / 32], const Frag<T> (&vf)[DH / 16],
                                           const Frag<T> (&qf)[DH / 32], int pb, int qi, int qpos, bool qvalid,
                                           int nkv, int grp, float c_log2, float& m_run, float& l_run,
                                           f32x4 (&o)[DH / 16]) {
  f32x4 s[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int pt = 0; pt < 2; ++pt)
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt) s[pt] = mma8(s[pt], kf[pt][dt], qf[dt]);
  float mx = -INFINITY;
#pragma unroll
  for (int pt = 0; pt < 2; ++pt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int pos = pb * 32 + pt * 16 + grp * 4 + r;
      const bool valid = qvalid && pos <= qpos && pos < nkv;
      s[pt][r] = valid ? s[pt][r] : -INFINITY;
      mx = fmaxf(mx, s[pt][r]);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(m_run, mx);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = exp2f((m_run - m_use) * c_log2);
  Frag<T> hi, lo;
  float ps = 0.f;
#pragma unroll
  for (int pt = 0; pt < 2; ++pt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float pv = exp2f((s[pt][r] - m_use) * c_log2);
      const T h = from_f32<T>(pv);
      hi.v[pt * 4 + r] = h;
      lo.v[pt * 4 + r] = from_f32<T>(pv - to_f32(h));
      ps += pv;
    }
  l_run = l_run * alpha + ps;
  m_run = m_new;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    o[dt] *= alpha;
    o[dt] = mma8(o[dt], vf[dt], hi);
    if (sizeof(T) == 2) o[dt] = mma8(o[dt], vf[dt], lo);
  }
}

// NTL: nontemporal (streaming) loads of the key and value tiles.
template <typename T, int DH, bool NTL>
__device__ __forceinline__ void load_block(const T* __restrict__ kr, const T* __restrict__ vr, int pb, int lane,
                                           int grp, int nkv, Frag<T> (&kf)[2][DH / 32], Frag<T> (&vf)[DH / 16]) {
  auto ld = [](const T* p) { return NTL ? load_frag_stream(p) : load_frag(p); };
#pragma unroll
  for (int pt = 0; pt < 2; ++pt)
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
      kf[pt][dt] = ld(kr + ((static_cast<size_t>(pb * 2 + pt) * (DH / 32) + dt) * 64 + lane) * 8);
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
    vf[dt] = ld(vr + ((static_cast<size_t>(pb) * (DH / 16) + dt) * 64 + lane) * 8);
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
}

// Work-group of the grid (G, H, B) with dispatch-order index L (x fastest):
// every (sequence b, head h) has G position groups. With short_first, the
// first H B work-groups take the last group of each (sequence, head), partly
// filled or empty, and the rest groups 0 .. G - 2 of each (sequence, head) in
// turn, neighbouring regions of its cache; otherwise work-group L takes
// group L % G of (sequence, head) L / G.
__device__ __forceinline__ void attn_group(bool short_first, int* h, int* b, int* g) {
  if (!short_first) {
    *g = static_cast<int>(blockIdx.x);
    *h = static_cast<int>(blockIdx.y);
    *b = static_cast<int>(blockIdx.z);
    return;
  }
  const long G = gridDim.x, H = gridDim.y;
  const long L = blockIdx.x + G * (blockIdx.y + H * static_cast<long>(blockIdx.z));
  const long nlast = H * gridDim.z;
  long hb;
  if (L < nlast) {
    hb = L;
    *g = static_cast<int>(G - 1);
  } else {
    hb = (L - nlast) / (G - 1);              // G > 1 here: L < G H B
    *g = static_cast<int>((L - nlast) % (G - 1));
  }
  *h = static_cast<int>(hb % H);
  *b = static_cast<int>(hb / H);
}

// Grid (G, H, B), G = ceil(T_cap / (4 WP)), 4 waves. Wave w of position
// group g covers positions 4 WP g + WP w .. + WP - 1 (WP = 32 or 64: one or
// two blocks),
// issuing the loads of KP blocks together. With one query tile (QT == 1: up
// to 16 new tokens per sequence, every verify and draft step) the four
// waves' partials are merged in LDS and the work-group writes one partial
// per 4 WP positions; with more query tiles (prefill chunks) every wave
// writes its own. With short_first (set by short_first_order) the short
// last groups run first and finish while the full groups start, instead of
// landing as a third work-group beside two full ones on some CUs.
template <typename T, int DH, int QT, int WP, int KP = 1, bool NTL = false>
__global__ __launch_bounds__(256) void attn_partial_kernel(const T* __restrict__ q, const T* __restrict__ kc,
                                                           const T* __restrict__ vc,
                                                           const int32_t* __restrict__ lengths, int pos_offset,
                                                           int Mps, int H, int T_cap, int NP, bool short_first,
                                                           float c_log2,
                                                           float* __restrict__ part) {
  constexpr bool kMerge = QT == 1;
  constexpr int kPre = KP;   // blocks whose loads are issued together
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int h, b, g;
  attn_group(short_first, &h, &b, &g);
  const int r16 = lane & 15, grp = lane >> 4;
  const int len = lengths[b] + pos_offset;        // position of query 0
  int nkv = len + Mps;
  if (nkv > T_cap) nkv = T_cap;
  static_assert(WP == 32 || WP == 64, "one or two 32-position blocks per wave");
  const int p0 = g * 4 * WP + wave * WP;
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
  if (nblk > WP / 32) nblk = WP / 32;
  for (int b0 = 0; b0 < nblk; b0 += kPre) {
    Frag<T> kf[kPre][2][DH / 32];
    Frag<T> vf[kPre][DH / 16];
#pragma unroll
    for (int u = 0; u < kPre; ++u)
      if (b0 + u < nblk) load_block<T, DH, NTL>(kr, vr, p0 / 32 + b0 + u, lane, grp, nkv, kf[u], vf[u]);
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
      if (b0 + u < nblk) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          const int qi = qt * 16 + r16;
          attn_block<T, DH>(kf[u], vf[u], qf[qt], p0 / 32 + b0 + u, qi, len + qi, qi < Mps, nkv, grp, c_log2,
                            m_run[qt], l_run[qt], o[qt]);
        }
      }
    }
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    l_run[qt] += __shfl_xor(l_run[qt], 16);
    l_run[qt] += __shfl_xor(l_run[qt], 32);
  }
  if (kMerge) {
    __shared__ float sm[4][16], sl[4][16];
    __shared__ float so[4][16][DH + 1];
    if (grp == 0) {
      sm[wave][r16] = m_run[0];
      sl[wave][r16] = l_run[0];
    }
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) so[wave][r16][dt * 16 + grp * 4 + r] = o[0][dt][r];
    __syncthreads();
    float* dst = part + ((static_cast<size_t>(b) * H + h) * NP + g) * Mps * (DH + 2);
    for (int e = threadIdx.x; e < 16 * DH; e += blockDim.x) {
      const int qi = e / DH, d = e % DH;
      if (qi >= Mps) continue;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) M = fmaxf(M, sm[w][qi]);
      float L = 0.f, acc = 0.f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float a = sm[w][qi] == -INFINITY ? 0.f : exp2f((sm[w][qi] - M) * c_log2);
          L += a * sl[w][qi];
          acc += a * so[w][qi][d];
        }
      }
      dst[qi * (DH + 2) + d] = acc;
      if (d == 0) {
        dst[qi * (DH + 2) + DH] = M;
        dst[qi * (DH + 2) + DH + 1] = L;
      }
    }
  } else {
    const int pidx = g * 4 + wave;
    if (pidx < NP) {
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const int qi = qt * 16 + r16;
        if (qi < Mps) {
          float* dst = part + (((static_cast<size_t>(b) * H + h) * NP + pidx) * Mps + qi) * (DH + 2);
#pragma unroll
          for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[dt * 16 + grp * 4 + r] = o[qt][dt][r];
          if (grp == 0) {
            dst[DH] = m_run[qt];
            dst[DH + 1] = l_run[qt];
          }
        }
      }
    }
  }
}

// Merge the partials of one (sequence, query) for every head and normalise:
// o = sum_p 2^{(m_p - M) c} O_p / sum_p 2^{(m_p - M) c} l_p. Each partial
// covers `pp` positions.
template <typename T, int DH>
__global__ __launch_bounds__(DH) void attn_combine_kernel(const float* __restrict__ part, const int32_t* __restrict__ lengths,
                                                          int pos_offset, int Mps, int H, int T_cap, int NP, int pp,
                                                          float c_log2, T* __restrict__ o, size_t oplane) {
  const int row = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
  const int b = row / Mps, qi = row % Mps;
  int nkv = lengths[b] + pos_offset + Mps;
  if (nkv > T_cap) nkv = T_cap;
  int np = (nkv + pp - 1) / pp;
  if (np > NP) np = NP;
  if (np < 0) np = 0;
  const float* base = part + ((static_cast<size_t>(b) * H + h) * NP * Mps + qi) * (DH + 2);
  const size_t stride = static_cast<size_t>(Mps) * (DH + 2);
  float M = -INFINITY;
#pragma unroll 8
  for (int p = 0; p < np; ++p) M = fmaxf(M, base[p * stride + DH]);
  float L = 0.f, acc = 0.f;
  if (M != -INFINITY) {
#pragma unroll 8
    for (int p = 0; p < np; ++p) {
      const float* pr = base + p * stride;
      const float mp = pr[DH];
      const float w = mp == -INFINITY ? 0.f : exp2f((mp - M) * c_log2);
      L += w * pr[DH + 1];
      acc += w * pr[d];
    }
  }
  // L == 0: no visible position (nothing to average). A NaN among the
  // scores or values makes L or acc NaN, and the NaN is passed on.
  store_act(o, oplane, static_cast<size_t>(row) * H * DH + h * DH + d, L == 0.f ? 0.f : acc / L);
}


// Whether the partial kernel runs every (sequence, head)'s last position
// group first: where every CU gets one or two full groups. Per kernel trace:
// 7B at ctx 2048 (256 full groups) 11.5 -> 10.3 us, 70B at ctx 2048 (512)
// 16.1 -> 15.7 us; the 3072-wide draft (192 full groups, fewer than the
// CUs) 8.0 -> 8.4 us, and with 2048 (70B at B = 4 or ctx 8192) no gain.
static bool short_first_order(int groups, int H, int B) {
  const long full = static_cast<long>(groups - 1) * H * B;
  return full >= kCUs && full <= 2L * kCUs;
}

// Decode launches (up to 16 new tokens per sequence): WP positions per wave,
// partials merged per work-group of 4 WP positions.
template <typename T, int DH, int WP, int KP = 1, bool NTL = false>
static hipError_t attn_decode_t(const void* q, const void* kc, const void* vc, const int32_t* lengths,
                                int pos_offset, int B, int Mps, int H, int T_cap, float* part, void* o,
                                size_t oplane, hipStream_t st) {
  const float c_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(DH));
  const int groups = (T_cap + 4 * WP - 1) / (4 * WP);
  hipLaunchKernelGGL((attn_partial_kernel<T, DH, 1, WP, KP, NTL>), dim3(groups, H, B), dim3(256), 0, st,
                     static_cast<const T*>(q), static_cast<const T*>(kc), static_cast<const T*>(vc), lengths,
                     pos_offset, Mps, H, T_cap, groups, short_first_order(groups, H, B), c_log2, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), dim3(B * Mps, H), dim3(DH), 0, st, part, lengths, pos_offset,
                     Mps, H, T_cap, groups, 4 * WP, c_log2, static_cast<T*>(o), oplane);
  return hipGetLastError();
}

template <typename T, int DH>
static hipError_t attn_t(const void* q, const void* kc, const void* vc, const int32_t* lengths, int pos_offset,
                         int B, int Mps, int H, int T_cap, float* part, void* o, size_t oplane, hipStream_t st) {
  if (Mps <= 16) {
    // From a sweep over 24-64 heads, contexts 2048-8192 and 1-4 sequences:
    // with >= 512 work-groups (two per CU) both blocks' loads in flight and
    // nontemporal K/V loads (70B at ctx 2048: 19.3 vs 20.6 us, at ctx 8192:
    // 56.9 vs 66.1 us); below, one block at a time with regular loads.
    const long wgs = static_cast<long>((T_cap + 255) / 256) * H * B;
    if (wgs >= 512)
      return attn_decode_t<T, DH, 64, 2, true>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, oplane, st);
    return attn_decode_t<T, DH, 64>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, oplane, st);
  }
  // Prefill chunks: 2 or 4 query tiles, every wave writes its own partial.
  const float c_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(DH));
  const int groups = (T_cap + 4 * kWavePos - 1) / (4 * kWavePos);
  const dim3 grid(groups, H, B);
  const T* qq = static_cast<const T*>(q);
  const T* kk = static_cast<const T*>(kc);
  const T* vv = static_cast<const T*>(vc);
  const int NP = attn_partials(T_cap);
  if (Mps <= 32)
    hipLaunchKernelGGL((attn_partial_kernel<T, DH, 2, kWavePos>), grid, dim3(256), 0, st, qq, kk, vv, lengths,
                       pos_offset, Mps, H, T_cap, NP, short_first_order(groups, H, B), c_log2, part);
  else
    hipLaunchKernelGGL((attn_partial_kernel<T, DH, 4, kWavePos>), grid, dim3(256), 0, st, qq, kk, vv, lengths,
                       pos_offset, Mps, H, T_cap, NP, short_first_order(groups, H, B), c_log2, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), dim3(B * Mps, H), dim3(DH), 0, st, part, lengths, pos_offset,
                     Mps, H, T_cap, NP, kWavePos, c_log2, static_cast<T*>(o), oplane);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const void* q, const void* kc, const void* vc, const int32_t* lengths,
                            int pos_offset, int B, int Mps, int H, int DH, int T_cap, float* part, void* o,
                            size_t oplane, hipStream_t st) {
  if (dtype == 1)
    return DH == 128 ? attn_t<bf16, 128>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, oplane, st)
                     : attn_t<bf16, 64>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, oplane, st);
  return DH == 128 ? attn_t<float, 128>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, oplane, st)
                   : attn_t<float, 64>(q, kc, vc, lengths, pos_offset, B, Mps, H, T_cap, part, o, oplane, st);
}

}  // namespace sps
