// Softmax with temperature, the fused accept / resample kernel of modified
// rejection sampling, draft-token sampling, the end-of-loop commit, and
// Philox uniforms.
//
// Categorical draws use an integer inverse CDF so that a parallel scan gives
// exactly the result of a serial loop: weights w_i = floor(x_i 2^32) for
// probabilities x_i (0 for x_i <= 0 or NaN, 2^32 for x_i >= 1), total W,
// threshold t = floor(m W / 2^24) for the grid index m = floor(u 2^24) of the
// uniform, result = smallest i whose inclusive prefix sum exceeds t. Wave w
// of the work-group owns one contiguous segment of the vocabulary and reads
// it 64 consecutive entries at a time; the 16 segment totals give every
// segment its exclusive prefix, and only the wave whose segment holds the
// threshold scans it again to find the index.
#include <algorithm>

#include "common.h"
#include "launch.h"
#include "philox.h"

namespace sps {

constexpr int kTotalBatch = 8;          // entries per lane read together (segment totals)
constexpr int kScanPerLane = 16;        // entries per lane of the threshold search (registers)

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), o);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), o);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl(static_cast<uint32_t>(v), src);
  const uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), src);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += shfl_xor_u64(v, o);
  return v;
}
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t o = shfl_up_u64(v, d);
    if (lane >= d) v += o;
  }
  return v;
}

// Branch-free (selects only), so that loops over a row keep their loads in
// flight together: floor(x 2^32) for x in (0, 1), 2^32 for x >= 1, 0 for
// x <= 0 or NaN. In double precision, where x 2^32 is exact and the
// conversion truncates. (Shifting the fp32 significand gives the same
// integers but made the draft draw ~40 % slower: 45 against 32 us.)
__device__ __forceinline__ uint64_t fixed_weight(float x) {
  const double d = x > 0.f ? fmin(static_cast<double>(x), 1.0) : 0.0;
  const double f = fmin(d * 4294967296.0, 4294967295.0);        // d = 1 adds the missing unit below
  return static_cast<uint64_t>(static_cast<uint32_t>(f)) + (d >= 1.0 ? 1u : 0u);
}

__device__ __forceinline__ uint64_t grid_threshold(float u, uint64_t W) {
  uint64_t m;
  if (!(u > 0.f)) m = 0;
  else if (u >= 1.f) m = (1u << 24) - 1;
  else m = static_cast<uint64_t>(u * 16777216.0f);
  return m * (W >> 24) + ((m * (W & 0xFFFFFFull)) >> 24);
}

// Row statistics of softmax(z / T): (a, b) = (max of z/T, sum of
// exp(z/T - max)), for T == 0 (greedy) (index of the first maximum, -1).
// With a top-k / nucleus modifier, s > 0 is the renormaliser and tau the
// smallest kept ranking key (see row_cutoff); s == 0 means unmodified.
// A row with a NaN or +Inf logit (or z/T overflowing to +Inf) has no
// distribution: it is marked non-finite and defined as one-hot at index 0
// (a = 0, b = -1, like a greedy row), and whoever uses it raises the device
// flag.
struct RowStat {
  float a, b, s;
  uint32_t nonfinite;
  uint64_t tau;
};
static_assert(sizeof(RowStat) == kRowStatBytes, "workspace row statistics");

// Probability of entry i of a row. The same expression (no contraction) is
// used wherever q or p is materialised, so exported probabilities and the
// values the accept test sees are identical bit for bit.
__device__ __forceinline__ float prob_of(float z, RowStat st, float inv_t, int i) {
  const float t = __fsub_rn(__fmul_rn(z, inv_t), st.a);
  const float v = __fdiv_rn(expf(t), st.b);
  const float g = i == __float2int_rz(st.a) ? 1.f : 0.f;        // greedy row: one-hot at the arg-max
  return st.b < 0.f ? g : v;
}

// Ranking key of the top-k / nucleus modifiers: the draw weight above the
// complement of the index, so larger keys rank first, equal weights rank
// by lower index, and every entry's key is distinct and >= 1 (V < 2^24).
__device__ __forceinline__ uint64_t rank_key(uint64_t w, int i) {
  return (w << 24) | static_cast<uint64_t>(0xFFFFFF - i);
}

// The probability the sampling stages use: prob_of, then (MOD: the row has
// a top-k / nucleus cut, st.s > 0) the cut and the renormalisation x / s.
// Branch-free; callers pick MOD once per row (a uniform branch outside
// their loops).
template <bool MOD>
__device__ __forceinline__ float prob_final(float z, const RowStat& st, float inv_t, int i) {
  const float x = prob_of(z, st, inv_t, i);
  if (!MOD) return x;
  const bool keep = rank_key(fixed_weight(x), i) >= st.tau;
  return keep ? __fdiv_rn(x, st.s) : 0.f;
}
__device__ __forceinline__ bool row_modified(const RowStat& st) { return st.s > 0.f; }

// Softmax partials of row_stat (rows of up to kPerLane nt entries): thread
// t of nt takes entries t + k nt, k < kPerLane, all loads in flight
// together, and returns the max of x = z / T and the sum of exp(x - max)
// over them (in k order) and whether one is NaN or +Inf; wave_soft_merge
// combines a wave's partials by butterfly, soft_merge one partial into
// another. row_stat and the cut-off's partial kernel both use these, so a
// row's statistics are the same bits in either.
struct SoftPart {
  float m, s;
  bool bad;
};
__device__ __forceinline__ SoftPart thread_soft_part(const float* __restrict__ z, int V, float inv_t, unsigned t,
                                                     unsigned nt) {
  SoftPart p{-INFINITY, 0.f, false};
  float x[kPerLane];
#pragma unroll
  for (int k = 0; k < kPerLane; ++k)   // all loads first (clamped: none behind a branch)
    x[k] = z[min(t + k * nt, static_cast<unsigned>(V - 1))];
#pragma unroll
  for (int k = 0; k < kPerLane; ++k) {
    x[k] = t + k * nt < static_cast<unsigned>(V) ? __fmul_rn(x[k], inv_t) : -INFINITY;
    p.bad |= !(x[k] < INFINITY);
    p.m = fmaxf(p.m, x[k]);
  }
  if (p.m > -INFINITY) {
#pragma unroll
    for (int k = 0; k < kPerLane; ++k) p.s += expf(x[k] - p.m);
  }
  return p;
}
// (Explicit roundings: a contracted multiply-add could be formed differently
// where the merge is inlined, and the partials' consumers must reproduce
// row_stat's bits.)
__device__ __forceinline__ void soft_merge(float& m, float& s2, float om, float os) {
  const float nm = fmaxf(m, om);
  if (nm == -INFINITY) return;
  s2 = __fadd_rn(__fmul_rn(s2, expf(m - nm)), __fmul_rn(os, expf(om - nm)));
  m = nm;
}
__device__ __forceinline__ void wave_soft_merge(float& m, float& s2) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o), os = __shfl_xor(s2, o);
    soft_merge(m, s2, om, os);
  }
}

// red: __shared__ float[32], ired: __shared__ int[16].
__device__ __forceinline__ RowStat row_stat(const float* __restrict__ z, int V, float temperature, float* red,
                                          int* ired) {
  RowStat st;
  st.s = 0.f;
  st.nonfinite = 0;
  st.tau = 0;
  if (temperature == 0.f) {
    float best = -INFINITY;
    int bi = 0x7fffffff;
    bool bad = false;
    for (int i = threadIdx.x; i < V; i += blockDim.x) {
      const float v = z[i];
      bad |= !(v < INFINITY);                       // NaN or +Inf
      if (v > best || (bi == 0x7fffffff)) { best = v; bi = i; }
    }
    // arg-max with the lowest index on ties
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o);
      const int oi = __shfl_xor(bi, o);
      if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) { red[threadIdx.x >> 6] = best; ired[threadIdx.x >> 6] = bi; }
    __syncthreads();
    best = red[0]; bi = ired[0];
    for (int w = 1; w < static_cast<int>(blockDim.x >> 6); ++w)
      if (red[w] > best || (red[w] == best && ired[w] < bi)) { best = red[w]; bi = ired[w]; }
    st.nonfinite = __syncthreads_or(bad) ? 1u : 0u;
    st.a = st.nonfinite ? 0.f : static_cast<float>(bi);
    st.b = -1.f;
    return st;
  }
  // Rows of up to kPerLane * blockDim entries are read once into registers
  // (all loads in flight together), then max and sum of exp(x - max) come
  // from the registers; longer rows keep a running (max, sum) per thread.
  const float inv_t = 1.0f / temperature;
  float mx = -INFINITY, sm = 0.f;
  bool bad = false;
  if (V <= kPerLane * static_cast<int>(blockDim.x)) {
    const SoftPart p = thread_soft_part(z, V, inv_t, threadIdx.x, blockDim.x);
    mx = p.m;
    sm = p.s;
    bad = p.bad;
  } else {
    for (int i = threadIdx.x; i < V; i += blockDim.x) {
      const float x = __fmul_rn(z[i], inv_t);
      bad |= !(x < INFINITY);
      if (x > mx) {
        sm = sm * expf(mx - x) + 1.f;
        mx = x;
      } else if (x > -INFINITY) {
        sm += expf(x - mx);
      }
    }
  }
  wave_soft_merge(mx, sm);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) { red[threadIdx.x >> 6] = mx; red[16 + (threadIdx.x >> 6)] = sm; }
  __syncthreads();
  mx = red[0];
  sm = red[16];
  for (int w = 1; w < static_cast<int>(blockDim.x >> 6); ++w) soft_merge(mx, sm, red[w], red[16 + w]);
  st.a = mx;
  st.b = sm;
  if (__syncthreads_or(bad)) {
    st.nonfinite = 1;
    st.a = 0.f;
    st.b = -1.f;
  }
  return st;
}

// Scratch of row_cutoff (LDS).
// Buckets of the cut-off's first pass: weight 0, then for w >= 1 the
// position e (0..32) of its leading one bit and the next 4 bits. The bucket
// is monotone in w, so the buckets split the ranking into contiguous key
// ranges (~6 % of a weight wide).
constexpr int kCutCand = 1024;            // keys of one bucket resolved exactly (kCutBuckets: plan.h)

__device__ __forceinline__ int cut_bucket(uint64_t w) {
  if (w == 0) return 0;
  const int e = 63 - __clzll(static_cast<long long>(w));
  const int m = e >= 4 ? static_cast<int>((w >> (e - 4)) & 15) : static_cast<int>((w << (4 - e)) & 15);
  return 1 + e * 16 + m;
}

struct CutScratch {
  uint64_t hist[256];
  uint64_t prefix, need;
  uint64_t wsum[16];
  uint64_t bins[kCutBuckets];       // per bucket: count of keys
  uint64_t wbins[kCutBuckets];      // per bucket: their weight
  uint64_t cand[kCutCand];
  uint64_t above, above_w;
  int nb, ncand, weighted;
};

// The row's draw weights for the cut-off, in LDS (dynamic shared memory of
// cutoff_lds_bytes(V)): the low 32 bits of every weight and a bitmask of the
// weights equal to 2^32 (x >= 1).
struct RowKeys {
  uint32_t* wl;    // [V]
  uint32_t* big;   // [ceil(V / 32)]
  int V;
  __device__ __forceinline__ uint64_t weight(int i) const {
    return static_cast<uint64_t>(wl[i]) | (static_cast<uint64_t>((big[i >> 5] >> (i & 31)) & 1u) << 32);
  }
  __device__ __forceinline__ uint64_t key(int i) const { return rank_key(weight(i), i); }
};

// Sum of the weights of keys >= lo, over the block.
__device__ __forceinline__ uint64_t kept_weight(const RowKeys& rk, uint64_t lo, CutScratch& sc) {
  uint64_t v = 0;
#pragma unroll 4
  for (int i = threadIdx.x; i < rk.V; i += blockDim.x) v += rk.key(i) >= lo ? rk.weight(i) : 0;
  v = wave_sum_u64(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sc.wsum[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t t = 0;
  for (int w = 0; w < static_cast<int>(blockDim.x >> 6); ++w) t += sc.wsum[w];
  return t;
}

// Radix select over the row's keys: the key tau such that the count
// (WEIGHTED: the weight) of keys >= max(tau, lo) reaches `need` (>= 1) while
// that of keys > tau does not. Eight passes of 8-bit digits from the top;
// per pass a 256-bin LDS histogram of the keys that match the digits chosen
// so far. Digit 0 (the leading zeros of the many small weights) is summed
// per thread and added once per wave.
template <bool WEIGHTED>
__device__ __forceinline__ uint64_t radix_select(const RowKeys& rk, uint64_t lo, uint64_t need, CutScratch& sc) {
  const int tid = threadIdx.x;
  uint64_t P = 0;
  for (int sh = 56; sh >= 0; sh -= 8) {
    for (int b = tid; b < 256; b += blockDim.x) sc.hist[b] = 0;
    __syncthreads();
    const uint64_t hm = sh + 8 >= 64 ? 0 : ~((1ull << (sh + 8)) - 1);
    uint64_t zero = 0;
#pragma unroll 4
    for (int i = tid; i < rk.V; i += blockDim.x) {
      const uint64_t key = rk.key(i);
      const bool in = key >= lo && (key & hm) == (P & hm);
      const uint32_t d = static_cast<uint32_t>(key >> sh) & 255u;
      const uint64_t v = WEIGHTED ? rk.weight(i) : 1;
      if (in && d == 0) zero += v;
      else if (in && v) atomicAdd(reinterpret_cast<unsigned long long*>(&sc.hist[d]), v);
    }
    zero = wave_sum_u64(zero);
    if ((tid & 63) == 0 && zero) atomicAdd(reinterpret_cast<unsigned long long*>(&sc.hist[0]), zero);
    __syncthreads();
    if (tid < 64) {
      // Bins from the top: lane l owns bins 255 - 4l .. 252 - 4l. The first
      // lane whose inclusive total reaches `need` walks its four bins.
      uint64_t h[4], tot = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        h[j] = sc.hist[255 - 4 * tid - j];
        tot += h[j];
      }
      const uint64_t inc = wave_incl_scan_u64(tot);
      const uint64_t hit = __ballot(inc >= need);
      if (tid == __ffsll(static_cast<long long>(hit)) - 1) {
        uint64_t c = inc - tot;
        int b = 255 - 4 * tid - 3;
#pragma unroll
        for (int j = 0; j < 3; ++j) {
          if (c + h[j] >= need) {
            b = 255 - 4 * tid - j;
            break;
          }
          c += h[j];
        }
        sc.prefix = P | (static_cast<uint64_t>(b) << sh);
        sc.need = need - c;
      }
    }
    __syncthreads();
    P = sc.prefix;
    need = sc.need;
  }
  return P;
}

// The select in two passes where it can. One pass histograms the keys >= lo
// over kCutBuckets weight buckets, counting them and summing their weights.
// The target is `need` keys counted from the top, or (NUCLEUS) a weight:
// floor(floor(top_p 2^24) W / 2^24) of the histogram's total W, the nucleus
// threshold on what keys >= lo hold (when that is 0, the one top key). One
// wave finds the bucket where the total from the top reaches the target and
// what the buckets above it hold; the keys of that bucket are gathered (at
// most kCutCand) and every candidate counts (sums) the candidates above it,
// so exactly one sees the total reach the target at itself: that key is tau.
// *kept = the weight of the keys >= tau. Returns false, leaving the answer to
// the radix passes, when the bucket holds more than kCutCand keys (a flat or
// nearly flat run of weights).
template <bool NUCLEUS>
__device__ __forceinline__ bool bucket_select(const RowKeys& rk, uint64_t lo, uint64_t need, float top_p,
                                              CutScratch& sc, uint64_t* tau, uint64_t* kept) {
  const int tid = threadIdx.x, bd = blockDim.x;
  for (int b = tid; b < kCutBuckets; b += bd) {
    sc.bins[b] = 0;
    sc.wbins[b] = 0;
  }
  if (tid == 0) sc.ncand = 0;
  __syncthreads();
  // Consecutive entries of a thread that fall in one bucket add once (a flat
  // row: two atomics per thread instead of two per entry).
  int cur = -1;
  uint64_t rc = 0, rw = 0;
  for (int i = tid; i < rk.V; i += bd) {
    const uint64_t key = rk.key(i);
    if (key < lo) continue;
    const uint64_t w = key >> 24;
    const int b = cut_bucket(w);
    if (b != cur) {
      if (rc) atomicAdd(reinterpret_cast<unsigned long long*>(&sc.bins[cur]), rc);
      if (rw) atomicAdd(reinterpret_cast<unsigned long long*>(&sc.wbins[cur]), rw);
      cur = b;
      rc = rw = 0;
    }
    rc += 1;
    rw += w;
  }
  if (rc) atomicAdd(reinterpret_cast<unsigned long long*>(&sc.bins[cur]), rc);
  if (rw) atomicAdd(reinterpret_cast<unsigned long long*>(&sc.wbins[cur]), rw);
  __syncthreads();
  bool weighted = false;
  if (tid < 64) {
    // Lane l owns kPer buckets from the top; the first lane whose inclusive
    // total reaches the target walks its buckets.
    constexpr int kPer = (kCutBuckets + 63) / 64;
    uint64_t hc[kPer], hw[kPer], tc = 0, tw = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int b = kCutBuckets - 1 - (tid * kPer + j);
      hc[j] = b >= 0 ? sc.bins[b] : 0;
      hw[j] = b >= 0 ? sc.wbins[b] : 0;
      tc += hc[j];
      tw += hw[j];
    }
    const uint64_t ic = wave_incl_scan_u64(tc), iw = wave_incl_scan_u64(tw);
    if (NUCLEUS) {
      const uint64_t W = shfl_u64(iw, 63);
      const uint64_t target = grid_threshold(top_p, W);
      weighted = target != 0;
      need = weighted ? target : 1;
    }
    const uint64_t inc = weighted ? iw : ic;
    const uint64_t hit = __ballot(inc >= need);
    if (tid == __ffsll(static_cast<long long>(hit)) - 1) {
      uint64_t c = inc - (weighted ? tw : tc), cw = iw - tw;
      int jb = kPer - 1;
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const uint64_t h = weighted ? hw[j] : hc[j];
        if (c + h >= need) {
          jb = j;
          break;
        }
        c += h;
        cw += hw[j];
      }
      sc.nb = kCutBuckets - 1 - (tid * kPer + jb);
      sc.above = c;
      sc.above_w = cw;
      sc.need = need;
      sc.weighted = weighted;                  // which total the candidates count
    }
  }
  __syncthreads();
  const int nb = sc.nb;
  const uint64_t above = sc.above;
  need = sc.need;
  weighted = sc.weighted != 0;
  for (int i = tid; i < rk.V; i += bd) {
    const uint64_t key = rk.key(i);
    if (key >= lo && cut_bucket(key >> 24) == nb) {
      const int slot = atomicAdd(&sc.ncand, 1);
      if (slot < kCutCand) sc.cand[slot] = key;
    }
  }
  __syncthreads();
  const int n = sc.ncand;
  if (n > kCutCand) return false;          // uniform over the block
  for (int t = tid; t < n; t += bd) {
    const uint64_t k = sc.cand[t];
    uint64_t sum = 0;
    for (int u = 0; u < n; ++u) {
      const uint64_t ku = sc.cand[u];
      sum += ku > k ? (weighted ? ku >> 24 : 1) : 0;
    }
    const uint64_t v = weighted ? k >> 24 : 1;
    if (above + sum < need && above + sum + v >= need) sc.prefix = k;   // exactly one candidate
  }
  __syncthreads();
  const uint64_t t_key = sc.prefix;
  uint64_t w = 0;
  for (int t = tid; t < n; t += bd) w += sc.cand[t] >= t_key ? sc.cand[t] >> 24 : 0;
  w = wave_sum_u64(w);
  if ((tid & 63) == 0) sc.wsum[tid >> 6] = w;
  __syncthreads();
  uint64_t s = sc.above_w;
  for (int v = 0; v < static_cast<int>(bd >> 6); ++v) s += sc.wsum[v];
  *tau = t_key;
  *kept = s;
  __syncthreads();                         // sc reusable by the next select
  return true;
}

// LDS bytes row_cutoff needs for a row of V entries.
__host__ __device__ __forceinline__ size_t cutoff_lds_bytes(int V) {
  return (static_cast<size_t>(V) + (V + 31) / 32) * sizeof(uint32_t);
}

// Top-k / nucleus cut-off of one row whose probabilities are pf(i), i < V,
// applied in that order: top-k keeps the top_k highest keys (1 <= top_k <
// V), nucleus then keeps the shortest prefix of the ranking among those
// whose weight total reaches floor(floor(top_p 2^24) W_k / 2^24) (top_p <
// 1), at least one entry. Sets st.tau to the smallest kept key and
// st.s = fp32(S) 2^-32 for the kept weight total S (0, i.e. unmodified, if
// S == 0). Block-wide; lds holds cutoff_lds_bytes(V) bytes.
template <class PF>
__device__ __forceinline__ void row_cutoff(PF pf, int V, int top_k, float top_p, RowStat& st, CutScratch& sc,
                                           uint32_t* lds) {
  RowKeys rk{lds, lds + V, V};
  for (int j = threadIdx.x; j < (V + 31) / 32; j += blockDim.x) rk.big[j] = 0;
  __syncthreads();
  const int bd = blockDim.x;
  for (int base = 0; base < V; base += 8 * bd) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = pf(min(base + k * bd + static_cast<int>(threadIdx.x), V - 1));
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = base + k * bd + threadIdx.x;
      const uint64_t w = fixed_weight(x[k]);
      if (i < V) {
        rk.wl[i] = static_cast<uint32_t>(w);
        if (w >> 32) atomicOr(&rk.big[i >> 5], 1u << (i & 31));
      }
    }
  }
  __syncthreads();
  // Top-k, then nucleus among what top-k kept; each select also gives the
  // weight kept at its key (the radix fallback sums it in one more pass).
  uint64_t tau = 1, S = 0;
  bool have_s = false;
  if (top_k >= 1 && top_k < V) {
    have_s = bucket_select<false>(rk, 1, static_cast<uint64_t>(top_k), 1.f, sc, &tau, &S);
    if (!have_s) tau = radix_select<false>(rk, 1, static_cast<uint64_t>(top_k), sc);
  }
  if (top_p < 1.f) {
    uint64_t tp;
    have_s = bucket_select<true>(rk, tau, 0, top_p, sc, &tp, &S);
    if (!have_s) {
      const uint64_t target = grid_threshold(top_p, kept_weight(rk, tau, sc));
      tp = target == 0 ? radix_select<false>(rk, tau, 1, sc) : radix_select<true>(rk, tau, target, sc);
    }
    tau = tp > tau ? tp : tau;
  }
  if (!have_s) S = kept_weight(rk, tau, sc);
  st.tau = tau;
  st.s = S == 0 ? 0.f : __ull2float_rn(S) * 2.3283064365386963e-10f;   // * 2^-32, exact
}

// Whether the modifiers change a row (greedy rows are never modified).
__host__ __device__ __forceinline__ bool modifiers_active(float temperature, int top_k, float top_p, int V) {
  return temperature > 0.f && ((top_k >= 1 && top_k < V) || top_p < 1.f);
}

// Row statistics with the top-k / nucleus cut-off applied (block-wide). A
// non-finite row stays one-hot at index 0 (never cut) and raises the flag.
__device__ __forceinline__ RowStat row_stat_final(const float* __restrict__ z, int V, float temperature, int top_k,
                                                  float top_p, float* red, int* ired, CutScratch& sc,
                                                  uint32_t* lds, int* err) {
  RowStat st = row_stat(z, V, temperature, red, ired);
  if (st.nonfinite) {
    if (threadIdx.x == 0) atomicOr(err, kErrNonFinite);
  } else if (modifiers_active(temperature, top_k, top_p, V)) {
    const float inv_t = 1.0f / temperature;
    const RowStat base = st;
    row_cutoff([&](int i) { return prob_of(z[i], base, inv_t, i); }, V, top_k, top_p, st, sc, lds);
  }
  return st;
}

// pr[i] = prob_final(z[i]) for the whole row, 8 loads per thread in flight.
template <bool MOD>
__device__ __forceinline__ void write_probs_t(const float* __restrict__ z, int V, const RowStat& st, float inv_t,
                                              float* __restrict__ pr) {
  const int bd = blockDim.x;
  for (int base = 0; base < V; base += 8 * bd) {
    float zz[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) zz[k] = z[min(base + k * bd + static_cast<int>(threadIdx.x), V - 1)];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = base + k * bd + threadIdx.x;
      if (i < V) pr[i] = prob_final<MOD>(zz[k], st, inv_t, i);
    }
  }
}
__device__ __forceinline__ void write_probs(const float* __restrict__ z, int V, const RowStat& st, float inv_t,
                                            float* __restrict__ pr) {
  if (row_modified(st)) write_probs_t<true>(z, V, st, inv_t, pr);
  else write_probs_t<false>(z, V, st, inv_t, pr);
}

__global__ __launch_bounds__(kSampleThreads) void row_softmax_kernel(const float* __restrict__ logits, int V,
                                                                     float temperature, int top_k, float top_p,
                                                                     RowStat* __restrict__ stats,
                                                                     float* __restrict__ probs, int* err) {
  __shared__ float red[32];
  __shared__ int ired[16];
  __shared__ CutScratch sc;
  extern __shared__ uint32_t s_rowkeys[];
  const int row = blockIdx.x;
  const float* z = logits + static_cast<size_t>(row) * V;
  const RowStat st = row_stat_final(z, V, temperature, top_k, top_p, red, ired, sc, s_rowkeys, err);
  const float inv_t = temperature == 0.f ? 0.f : 1.0f / temperature;
  if (threadIdx.x == 0 && stats) stats[row] = st;
  if (probs) write_probs(z, V, st, inv_t, probs + static_cast<size_t>(row) * V);
}

// ---------------------------------------------------------------------------
// The top-k / nucleus cut-off of the rows of a verify or draft step over
// several CUs (one work-group per row is instruction-bound at ~290 VALU
// instructions per vocabulary entry). cut_part_kernel's work-groups are the
// waves of row_stat, each writing that wave's softmax partial (every
// consumer merges them in row_stat's order, so the row's probabilities are
// those of the unmodified row bit for bit), and clear the row's bucket
// histogram; cut_hist_kernel's work-groups each take one segment of a row: the draw
// weights, each entry's bucket, and the segment's bucket counts and weights
// added to the row's histogram (integer atomics: the totals do not depend on
// the order); cut_select_kernel finds the bucket holding each cut from the
// histogram, gathers that bucket's keys alone (their weights recomputed) and
// resolves the cut as bucket_select does, else (more than kCutCand keys in
// the bucket, a flat run of weights) it runs row_cutoff over the whole row.
// Row r of a launch is logits row r rstride + roff.
// ---------------------------------------------------------------------------

// Per-row scratch (cut_row_bytes(V) bytes): bucket counts, bucket weights,
// the softmax partials of the row_stat waves, then a 16-bit bucket id per
// entry.
struct CutPart {
  float m, s;
  uint32_t bad, pad;
};
constexpr int kStatWaves = kSampleThreads / 64;     // waves of row_stat
static_assert(kStatWaves * sizeof(CutPart) <= 256, "partials fit their scratch slot");
struct CutRowScratch {
  uint64_t* n;
  uint64_t* w;
  CutPart* part;
  uint16_t* bid;
};
__device__ __forceinline__ CutRowScratch cut_row(char* base, size_t row_bytes, int r) {
  constexpr size_t kHist = (static_cast<size_t>(kCutBuckets) * 2 * sizeof(uint64_t) + 255) & ~static_cast<size_t>(255);
  char* p = base + static_cast<size_t>(r) * row_bytes;
  return CutRowScratch{reinterpret_cast<uint64_t*>(p), reinterpret_cast<uint64_t*>(p) + kCutBuckets,
                       reinterpret_cast<CutPart*>(p + kHist), reinterpret_cast<uint16_t*>(p + kHist + 256)};
}

// Row statistics from the wave partials, merged in wave order as row_stat
// merges them (the same bits).
__device__ __forceinline__ RowStat stat_of_parts(const CutPart* __restrict__ part) {
  float mx = part[0].m, sm = part[0].s;
  bool bad = part[0].bad != 0;
  for (int w = 1; w < kStatWaves; ++w) {
    soft_merge(mx, sm, part[w].m, part[w].s);
    bad |= part[w].bad != 0;
  }
  RowStat st;
  st.s = 0.f;
  st.tau = 0;
  st.nonfinite = bad ? 1u : 0u;
  st.a = bad ? 0.f : mx;
  st.b = bad ? -1.f : sm;
  return st;
}

__device__ __forceinline__ const float* cut_logits(const float* logits, int r, int rstride, int roff, int V) {
  return logits + (static_cast<size_t>(r) * rstride + roff) * V;
}

// Grid (kStatWaves, rows), one wave each: wave w of row_stat's work-group,
// its partial into the row's scratch; wave 0 also clears the histogram.
__global__ __launch_bounds__(64) void cut_part_kernel(const float* __restrict__ logits, int V, int rstride, int roff,
                                                     float temperature, char* __restrict__ cut, size_t cut_bytes) {
  const int r = blockIdx.y, w = blockIdx.x;
  SoftPart p = thread_soft_part(cut_logits(logits, r, rstride, roff, V), V, 1.0f / temperature,
                                w * 64 + threadIdx.x, kSampleThreads);
  wave_soft_merge(p.m, p.s);
  const bool bad = __ballot(p.bad) != 0;
  const CutRowScratch cs = cut_row(cut, cut_bytes, r);
  if (threadIdx.x == 0) cs.part[w] = CutPart{p.m, p.s, bad ? 1u : 0u, 0u};
  if (w == 0)
    for (int b = threadIdx.x; b < kCutBuckets; b += 64) {
      cs.n[b] = 0;
      cs.w[b] = 0;
    }
}

constexpr int kCutSegThreads = 256;

// Grid (segments, rows): segment s of a row is entries [s seg, (s + 1) seg).
__global__ __launch_bounds__(kCutSegThreads) void cut_hist_kernel(const float* __restrict__ logits, int V, int rstride,
                                                                  int roff, float temperature,
                                                                  RowStat* __restrict__ stats, char* __restrict__ cut,
                                                                  size_t cut_bytes, int seg) {
  __shared__ uint64_t hn[kCutBuckets], hw[kCutBuckets];
  const int r = blockIdx.y, s = blockIdx.x;
  const CutRowScratch cs = cut_row(cut, cut_bytes, r);
  const RowStat st = stat_of_parts(cs.part);
  // The row's statistics as merged here go to stats[r]: the select reads these
  // bits rather than merging again, so its keys are the ones bucketed here.
  if (s == 0 && threadIdx.x == 0) stats[r] = st;
  if (st.nonfinite) return;                        // uniform over the block
  for (int b = threadIdx.x; b < kCutBuckets; b += blockDim.x) {
    hn[b] = 0;
    hw[b] = 0;
  }
  __syncthreads();
  const float* z = cut_logits(logits, r, rstride, roff, V);
  const float inv_t = 1.0f / temperature;
  const int i0 = s * seg, i1 = min(V, i0 + seg);
  for (int i = i0 + static_cast<int>(threadIdx.x); i < i1; i += kCutSegThreads) {
    const uint64_t w = fixed_weight(prob_of(z[i], st, inv_t, i));
    const int b = cut_bucket(w);
    cs.bid[i] = static_cast<uint16_t>(b);
    atomicAdd(reinterpret_cast<unsigned long long*>(&hn[b]), 1ull);
    if (w) atomicAdd(reinterpret_cast<unsigned long long*>(&hw[b]), static_cast<unsigned long long>(w));
  }
  __syncthreads();
  for (int b = threadIdx.x; b < kCutBuckets; b += blockDim.x) {
    if (hn[b]) atomicAdd(reinterpret_cast<unsigned long long*>(&cs.n[b]), static_cast<unsigned long long>(hn[b]));
    if (hw[b]) atomicAdd(reinterpret_cast<unsigned long long*>(&cs.w[b]), static_cast<unsigned long long>(hw[b]));
  }
}

// A row's bucket ids held in registers: thread t owns the 8 ids of vector
// t + j kSampleThreads (entries 8 (t + j kSampleThreads) .. + 7), j < kIdVecs,
// loaded together (V <= 8 kIdVecs kSampleThreads).
constexpr int kIdVecs = 4;
typedef uint32_t id8 __attribute__((ext_vector_type(4)));   // eight 16-bit bucket ids
static_assert(8 * kIdVecs * kSampleThreads >= kPerLane * kSampleThreads, "bucket ids of the largest cut row");
struct RowIds {
  id8 v[kIdVecs];
  __device__ __forceinline__ int id(int j, int e) const {
    const uint32_t w = v[j][e >> 1];
    return static_cast<int>(e & 1 ? w >> 16 : w & 0xFFFFu);
  }
};
__device__ __forceinline__ RowIds load_ids(const uint16_t* __restrict__ bid, int V) {
  RowIds ids;
  const id8* src = reinterpret_cast<const id8*>(bid);
  const int nv = (V + 7) / 8;                      // vectors holding entries (the scratch pads to 256 bytes)
#pragma unroll
  for (int j = 0; j < kIdVecs; ++j) ids.v[j] = src[min(static_cast<int>(threadIdx.x) + j * kSampleThreads, nv - 1)];
  return ids;
}

// The keys of bucket nb (every one of them: nb lies above the previous
// cut's bucket) into sc.cand; false (uniform) when there are more than
// kCutCand.
template <class PF>
__device__ __forceinline__ bool gather_bucket(PF pf, const RowIds& ids, int V, int nb, CutScratch& sc) {
  const int tid = threadIdx.x;
  if (tid == 0) sc.ncand = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kIdVecs; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = 8 * (tid + j * kSampleThreads) + e;
      if (i < V && ids.id(j, e) == nb) {
        const int slot = atomicAdd(&sc.ncand, 1);
        if (slot < kCutCand) sc.cand[slot] = rank_key(fixed_weight(pf(i)), i);
      }
    }
  __syncthreads();
  return sc.ncand <= kCutCand;
}

// One select over the keys >= lo, as bucket_select, from the bucket totals
// in sc.bins / sc.wbins (all keys of every bucket) instead of a pass over
// the row. lob is the bucket of lo (-1: lo admits every key); its keys are
// sc.cand[0 .. nlo), gathered by the previous select, of which only those >=
// lo count. Sets *tau, *kept (weight of the keys >= tau) and the bucket and
// candidates now in sc.cand; false (uniform) where the bucket of the cut
// holds more than kCutCand keys.
template <bool NUCLEUS, class PF>
__device__ bool hist_select(PF pf, const RowIds& ids, int V, uint64_t lo, int lob, int nlo,
                            uint64_t need, float top_p, CutScratch& sc, uint64_t* sub_n, uint64_t* sub_w,
                            uint64_t* tau, uint64_t* kept, int* nb_out, int* n_out) {
  const int tid = threadIdx.x, bd = blockDim.x;
  if (lob >= 0) {
    // Bucket lob: only its candidates >= lo; the buckets under it: nothing.
    uint64_t c = 0, w = 0;
    for (int t = tid; t < nlo; t += bd) {
      const uint64_t k = sc.cand[t];
      c += k >= lo ? 1 : 0;
      w += k >= lo ? k >> 24 : 0;
    }
    c = wave_sum_u64(c);
    w = wave_sum_u64(w);
    __syncthreads();
    if ((tid & 63) == 0) {
      sc.wsum[tid >> 6] = c;
      sc.hist[tid >> 6] = w;
    }
    __syncthreads();
    if (tid == 0) {
      uint64_t cc = 0, ww = 0;
      for (int v = 0; v < bd / 64; ++v) {
        cc += sc.wsum[v];
        ww += sc.hist[v];
      }
      sc.bins[lob] = cc;
      sc.wbins[lob] = ww;
    }
    for (int b = tid; b < lob; b += bd) {
      sc.bins[b] = 0;
      sc.wbins[b] = 0;
    }
  }
  if (tid == 0) sc.nb = -2;
  __syncthreads();
  if (tid < 64) {
    // Lane l owns kPer buckets from the top; the first lane whose inclusive
    // total reaches the target walks its buckets.
    constexpr int kPer = (kCutBuckets + 63) / 64;
    uint64_t hc[kPer], hw[kPer], tc = 0, tw = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int b = kCutBuckets - 1 - (tid * kPer + j);
      hc[j] = b >= 0 ? sc.bins[b] : 0;
      hw[j] = b >= 0 ? sc.wbins[b] : 0;
      tc += hc[j];
      tw += hw[j];
    }
    const uint64_t ic = wave_incl_scan_u64(tc), iw = wave_incl_scan_u64(tw);
    bool weighted = false;
    if (NUCLEUS) {
      const uint64_t W = shfl_u64(iw, 63);
      const uint64_t target = grid_threshold(top_p, W);
      weighted = target != 0;
      need = weighted ? target : 1;
    }
    const uint64_t inc = weighted ? iw : ic;
    const uint64_t hit = __ballot(inc >= need);
    if (hit && tid == __ffsll(static_cast<long long>(hit)) - 1) {
      uint64_t c = inc - (weighted ? tw : tc), cw = iw - tw;
      int jb = kPer - 1;
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const uint64_t h = weighted ? hw[j] : hc[j];
        if (c + h >= need) {
          jb = j;
          break;
        }
        c += h;
        cw += hw[j];
      }
      sc.nb = kCutBuckets - 1 - (tid * kPer + jb);
      sc.above = c;
      sc.above_w = cw;
      sc.need = need;
      sc.weighted = weighted;
    }
  }
  __syncthreads();
  const int nb = sc.nb;
  if (nb < 0 || nb < lob) return false;            // (no bucket reaches the target: not for a valid row)
  const uint64_t above = sc.above;                 // count / weight above bucket nb; sc.above_w its weight
  need = sc.need;
  const bool weighted = sc.weighted != 0;
  int n = nlo;
  if (nb != lob) {
    if (!gather_bucket(pf, ids, V, nb, sc)) return false;
    n = sc.ncand;
  }
  // Second level: the candidates' key range (keys >= lo) in 256 sub-ranges
  // of 2^sh keys (sub-range (k - kmin) >> sh, monotone in k); one wave finds
  // the sub-range where the total from the top reaches the target, and only
  // its candidates, gathered into sc.hist, are compared pairwise (all n of
  // them where it holds more than 256).
  uint64_t kmin = ~0ull, kmax = 0;
  for (int t = tid; t < n; t += bd) {
    const uint64_t k = sc.cand[t];
    kmin = k >= lo && k < kmin ? k : kmin;
    kmax = k >= lo && k > kmax ? k : kmax;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t a = shfl_xor_u64(kmin, o), b = shfl_xor_u64(kmax, o);
    kmin = a < kmin ? a : kmin;
    kmax = b > kmax ? b : kmax;
  }
  if ((tid & 63) == 0) {
    sc.wsum[tid >> 6] = kmin;
    sc.hist[tid >> 6] = kmax;
  }
  for (int b = tid; b < 256; b += bd) {
    sub_n[b] = 0;
    sub_w[b] = 0;
  }
  __syncthreads();
  kmin = ~0ull;
  kmax = 0;
  for (int v = 0; v < bd / 64; ++v) {
    kmin = sc.wsum[v] < kmin ? sc.wsum[v] : kmin;
    kmax = sc.hist[v] > kmax ? sc.hist[v] : kmax;
  }
  if (kmax < kmin) return false;                   // no candidate >= lo (uniform; not for a valid row)
  const uint64_t span = kmax - kmin;
  const int sh = span >> 8 ? 64 - __clzll(static_cast<long long>(span >> 8)) : 0;   // span >> sh < 256
  for (int t = tid; t < n; t += bd) {
    const uint64_t k = sc.cand[t];
    if (k >= lo) {
      const int sb = static_cast<int>((k - kmin) >> sh);
      atomicAdd(reinterpret_cast<unsigned long long*>(&sub_n[sb]), 1ull);
      atomicAdd(reinterpret_cast<unsigned long long*>(&sub_w[sb]), static_cast<unsigned long long>(k >> 24));
    }
  }
  if (tid == 0) {
    sc.prefix = 0;
    sc.nb = -1;
  }
  __syncthreads();
  if (tid < 64) {
    // Lane l owns sub-ranges 255 - 4l .. 252 - 4l; the first lane whose
    // inclusive total (above the bucket's included) reaches the target walks them.
    uint64_t hc[4], hw[4], tc = 0, tw = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      hc[j] = sub_n[255 - 4 * tid - j];
      hw[j] = sub_w[255 - 4 * tid - j];
      tc += hc[j];
      tw += hw[j];
    }
    const uint64_t ic = wave_incl_scan_u64(tc), iw = wave_incl_scan_u64(tw);
    const uint64_t inc = above + (weighted ? iw : ic);
    const uint64_t hit = __ballot(inc >= need);
    if (hit && tid == __ffsll(static_cast<long long>(hit)) - 1) {
      uint64_t c = inc - (weighted ? tw : tc), cw = sc.above_w + iw - tw;
      int jb = 3;
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        const uint64_t h = weighted ? hw[j] : hc[j];
        if (c + h >= need) {
          jb = j;
          break;
        }
        c += h;
        cw += hw[j];
      }
      sc.nb = 255 - 4 * tid - jb;                  // the sub-range
      sc.above = c;                                // count / weight above it
      sc.above_w = cw;                             // weight above it
      sc.ncand = 0;
    }
  }
  __syncthreads();
  const int sbt = sc.nb;
  if (sbt < 0) return false;
  const uint64_t above2 = sc.above;
  for (int t = tid; t < n; t += bd) {
    const uint64_t k = sc.cand[t];
    if (k >= lo && static_cast<int>((k - kmin) >> sh) == sbt) {
      const int slot = atomicAdd(&sc.ncand, 1);
      if (slot < 256) sc.hist[slot] = k;
    }
  }
  __syncthreads();
  const int m = sc.ncand;
  const bool small = m <= 256;
  const uint64_t* list = small ? sc.hist : sc.cand;
  const int nl = small ? m : n;
  for (int t = tid; t < nl; t += bd) {
    const uint64_t k = list[t];
    if (k < lo || static_cast<int>((k - kmin) >> sh) != sbt) continue;
    uint64_t sum = 0;
    for (int u = 0; u < nl; ++u) {
      const uint64_t ku = list[u];
      sum += ku > k && static_cast<int>((ku - kmin) >> sh) == sbt ? (weighted ? ku >> 24 : 1) : 0;
    }
    const uint64_t v = weighted ? k >> 24 : 1;
    if (above2 + sum < need && above2 + sum + v >= need) sc.prefix = k;   // exactly one candidate
  }
  __syncthreads();
  const uint64_t t_key = sc.prefix;
  if (t_key == 0) return false;
  uint64_t w = 0;
  for (int t = tid; t < nl; t += bd) {
    const uint64_t k = list[t];
    w += k >= t_key && static_cast<int>((k - kmin) >> sh) == sbt ? k >> 24 : 0;
  }
  w = wave_sum_u64(w);
  if ((tid & 63) == 0) sc.wsum[tid >> 6] = w;
  __syncthreads();
  uint64_t total = sc.above_w;                     // weight above the sub-range
  for (int v = 0; v < bd / 64; ++v) total += sc.wsum[v];
  *tau = t_key;
  *kept = total;
  *nb_out = nb;
  *n_out = n;
  __syncthreads();                                 // sc reusable by the next select
  return true;
}

// grid (rows), kSampleThreads threads, dynamic LDS cutoff_lds_bytes(V) (for
// the fallback).
__global__ __launch_bounds__(kSampleThreads) void cut_select_kernel(const float* __restrict__ logits, int V,
                                                                    int rstride, int roff, float temperature,
                                                                    int top_k, float top_p,
                                                                    RowStat* __restrict__ stats,
                                                                    char* __restrict__ cut, size_t cut_bytes, int* err) {
  __shared__ CutScratch sc;
  __shared__ uint64_t sub_n[256], sub_w[256];
  extern __shared__ uint32_t s_rowkeys[];
  const int r = blockIdx.x;
  const CutRowScratch cs = cut_row(cut, cut_bytes, r);
  const RowIds ids = load_ids(cs.bid, V);          // in flight with the histogram's and the partials' loads
  for (int b = threadIdx.x; b < kCutBuckets; b += blockDim.x) {
    sc.bins[b] = cs.n[b];
    sc.wbins[b] = cs.w[b];
  }
  const RowStat base = stats[r];                   // merged by cut_hist_kernel
  if (base.nonfinite) {                            // uniform: one-hot at index 0, never cut (as row_stat_final)
    if (threadIdx.x == 0) atomicOr(err, kErrNonFinite);
    return;
  }
  __syncthreads();
  const float* z = cut_logits(logits, r, rstride, roff, V);
  const float inv_t = 1.0f / temperature;
  auto pf = [&](int i) { return prob_of(z[i], base, inv_t, i); };
  // Top-k, then nucleus among what top-k kept (row_cutoff's order).
  uint64_t tau = 1, S = 0;
  int lob = -1, nk = 0;
  bool ok = true;
  if (top_k >= 1 && top_k < V)
    ok = hist_select<false>(pf, ids, V, 1, -1, 0, static_cast<uint64_t>(top_k), 1.f, sc, sub_n, sub_w, &tau, &S, &lob,
                            &nk);
  if (ok && top_p < 1.f) {
    uint64_t tp = 0, Sp = 0;
    int lp = -1, np = 0;
    ok = hist_select<true>(pf, ids, V, tau, lob, nk, 0, top_p, sc, sub_n, sub_w, &tp, &Sp, &lp, &np);
    tau = tp > tau ? tp : tau;
    S = Sp;
  }
  RowStat st = base;
  if (ok) {
    st.tau = tau;
    st.s = S == 0 ? 0.f : __ull2float_rn(S) * 2.3283064365386963e-10f;   // * 2^-32, exact
  } else {
    row_cutoff(pf, V, top_k, top_p, st, sc, s_rowkeys);
  }
  if (threadIdx.x == 0) stats[r] = st;
}

// Probabilities of rows (with their cut) into probs[row][V], one segment per
// work-group: grid (segments, rows).
__global__ __launch_bounds__(kCutSegThreads) void cut_export_kernel(const float* __restrict__ logits, int V,
                                                                    float temperature,
                                                                    const RowStat* __restrict__ stats,
                                                                    float* __restrict__ probs, int seg) {
  const int r = blockIdx.y, s = blockIdx.x;
  const RowStat st = stats[r];
  const float* z = logits + static_cast<size_t>(r) * V;
  float* pr = probs + static_cast<size_t>(r) * V;
  const float inv_t = 1.0f / temperature;
  const int i0 = s * seg, i1 = min(V, i0 + seg);
  if (row_modified(st)) {
    for (int i = i0 + static_cast<int>(threadIdx.x); i < i1; i += kCutSegThreads) pr[i] = prob_final<true>(z[i], st, inv_t, i);
  } else {
    for (int i = i0 + static_cast<int>(threadIdx.x); i < i1; i += kCutSegThreads) pr[i] = prob_final<false>(z[i], st, inv_t, i);
  }
}

// ---------------------------------------------------------------------------
// The draft step's softmax export and draw over several CUs (temperature >
// 0): draft_p_kernel's work-groups take one segment of a sequence's row
// each -- the row statistics (stored by the cut-off kernels, or merged from
// cut_part_kernel's wave partials, the same bits as row_stat), p_t written
// for the segment and the total of its draw weights; draft_draw_kernel then
// finds the segment holding the threshold from the totals and scans only
// that segment. The draw is the one of draft_sample_kernel (integer inverse
// CDF over the stored probabilities, in index order).
// ---------------------------------------------------------------------------
template <bool MOD>
__device__ __forceinline__ uint64_t segment_probs(const float* __restrict__ z, const RowStat& st, float inv_t, int i0,
                                                  int i1, float* __restrict__ pr) {
  uint64_t w = 0;
  for (int i = i0 + static_cast<int>(threadIdx.x); i < i1; i += kCutSegThreads) {
    const float x = prob_final<MOD>(z[i], st, inv_t, i);
    pr[i] = x;
    w += fixed_weight(x);
  }
  return w;
}

__global__ __launch_bounds__(kCutSegThreads) void draft_p_kernel(const float* __restrict__ logits, int Mps, int V,
                                                                 float temperature, const RowStat* __restrict__ pre,
                                                                 char* __restrict__ cut, size_t cut_bytes, int seg,
                                                                 float* __restrict__ p_out, int K, int t, int* err) {
  __shared__ uint64_t s_w[kCutSegThreads / 64];
  const int b = blockIdx.y, s = blockIdx.x;
  const CutRowScratch cs = cut_row(cut, cut_bytes, b);
  const RowStat st = pre ? pre[b] : stat_of_parts(cs.part);
  if (!pre && st.nonfinite && s == 0 && threadIdx.x == 0) atomicOr(err, kErrNonFinite);   // one-hot at token 0
  const float* z = logits + (static_cast<size_t>(b) * Mps + Mps - 1) * V;
  float* pr = p_out + (static_cast<size_t>(b) * K + t) * V;
  const float inv_t = 1.0f / temperature;
  const int i0 = s * seg, i1 = min(V, i0 + seg);
  uint64_t w = row_modified(st) ? segment_probs<true>(z, st, inv_t, i0, i1, pr)
                                : segment_probs<false>(z, st, inv_t, i0, i1, pr);
  w = wave_sum_u64(w);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = w;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t tot = 0;
    for (int v = 0; v < kCutSegThreads / 64; ++v) tot += s_w[v];
    cs.n[s] = tot;                                 // the histogram's slots: free once the cut is taken
  }
}

constexpr int kDrawPer = 8;                        // entries per thread of the segment scan

// One work-group per sequence. Threshold t of the row's total W (as
// block_draw); the segment whose range of the cumulative weights holds it is
// scanned with thread r owning kDrawPer consecutive entries per round.
__global__ __launch_bounds__(kCutSegThreads) void draft_draw_kernel(const char* __restrict__ cut, size_t cut_bytes,
                                                                    int nseg, int seg, int V,
                                                                    const float* __restrict__ p_out, int K, int t,
                                                                    int32_t* __restrict__ tokens,
                                                                    const int32_t* __restrict__ ctx, uint64_t seed,
                                                                    uint64_t loop, int* err) {
  __shared__ uint64_t wsum[17];
  __shared__ uint64_t s_thr, s_off;
  __shared__ int s_seg, s_y;
  const int b = blockIdx.x, tid = threadIdx.x;
  const CutRowScratch cs = cut_row(const_cast<char*>(cut), cut_bytes, b);
  const size_t tok = static_cast<size_t>(b) * (K + 1);
  static_assert(kMaxRowSegments <= 64, "one wave holds the segment totals");
  // Wave 0: the segment totals in order (nseg <= kMaxRowSegments), the threshold and the
  // segment whose range of the cumulative weight holds it, for every wave.
  if (tid < 64) {
    const float u = philox_uniform(seed, loop, 0, b, t);
    const uint64_t tot = tid < nseg ? cs.n[tid] : 0;
    uint64_t inc = tot;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t o = shfl_up_u64(inc, d);
      if (tid >= d) inc += o;
    }
    const uint64_t W = shfl_u64(inc, 63);
    const uint64_t thr = grid_threshold(u, W);
    const uint64_t hit = W ? __ballot(tid < nseg && inc > thr) : 0;
    const int sstar = hit ? __ffsll(static_cast<long long>(hit)) - 1 : -1;
    const uint64_t off = shfl_u64(inc - tot, sstar < 0 ? 0 : sstar);   // weight before segment sstar
    if (tid == 0) {
      s_thr = thr;
      s_off = off;
      s_seg = sstar;
      s_y = -1;
    }
  }
  __syncthreads();
  const int sstar = s_seg;
  const uint64_t thr = s_thr;
  if (sstar >= 0) {                                // uniform
    const float* pr = p_out + (static_cast<size_t>(b) * K + t) * V;
    const int i0 = sstar * seg, i1 = min(V, i0 + seg);
    uint64_t run = s_off;
    for (int base = i0; base < i1; base += kCutSegThreads * kDrawPer) {
      uint64_t w[kDrawPer], lt = 0;
      const int c0 = base + kDrawPer * tid;
#pragma unroll
      for (int k = 0; k < kDrawPer; ++k) {
        const uint64_t x = fixed_weight(pr[min(c0 + k, i1 - 1)]);
        w[k] = c0 + k < i1 ? x : 0;
        lt += w[k];
      }
      uint64_t total;
      const uint64_t ex = run + block_exscan_u64(lt, wsum, &total);
      if (ex <= thr && thr < ex + lt) {            // exactly one thread
        uint64_t acc = ex;
        int hitk = -1;
#pragma unroll
        for (int k = 0; k < kDrawPer; ++k) {
          acc += w[k];
          if (hitk < 0 && acc > thr) hitk = k;
        }
        s_y = c0 + hitk;
      }
      __syncthreads();
      if (s_y >= 0) break;                         // uniform
      run += total;
    }
  }
  if (tid == 0) {
    int y = s_y;
    if (y < 0) {                                   // every weight zero
      y = 0;
      atomicOr(err, kErrEmpty);
    }
    tokens[tok + t + 1] = y;
    if (t == 0) tokens[tok] = ctx[2 * b + 1];
  }
}

// Segment [b0, b1) of the vocabulary owned by this wave: a multiple of 64
// entries, the waves' segments in order.
struct Segment { int b0, b1; };
__device__ __forceinline__ Segment wave_segment(int V) {
  const int nw = blockDim.x >> 6, w = threadIdx.x >> 6;
  const int S = ((V + nw - 1) / nw + 63) & ~63;
  const int b0 = min(V, w * S);
  return Segment{b0, min(V, b0 + S)};
}

// Total of the weights wf(i) over this wave's segment (every lane gets it).
// Lane l reads entries base + 64 k + l: every load instruction is coalesced.
template <class WF>
__device__ __forceinline__ uint64_t segment_total(WF wf, Segment sg) {
  const int lane = threadIdx.x & 63;
  uint64_t loc = 0;
  for (int base = sg.b0; base < sg.b1; base += 64 * kTotalBatch) {
    // Indexes past the segment read its last entry and are masked after
    // the load, so that no load sits behind a branch and a batch is in
    // flight together.
#pragma unroll
    for (int k = 0; k < kTotalBatch; ++k) {
      const int i = base + 64 * k + lane;
      const uint64_t x = wf(min(i, sg.b1 - 1));
      loc += i < sg.b1 ? x : 0;
    }
  }
  return wave_sum_u64(loc);
}

// Block-wide integer inverse-CDF draw with weights wf(i), i < V, given every
// wave's segment total `tot` (from segment_total). s_tot is __shared__
// uint64_t[16 + 1], s_res a __shared__ int. Returns the drawn index to every
// thread, or -1 when all weights are zero (W == 0). The wave whose segment
// holds the threshold reads it again (now cache-resident) with lane l owning
// kScanPerLane consecutive entries of a super-chunk, scans the lane totals and
// lets the one lane whose range holds the threshold walk its registers.
template <class WF>
__device__ int block_draw(WF wf, Segment sg, uint64_t tot, float u, uint64_t* s_tot, int* s_res) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();                         // s_tot / s_res free from any previous draw
  if (lane == 0) s_tot[wave] = tot;
  if (threadIdx.x == 0) *s_res = -1;
  __syncthreads();
  uint64_t off = 0, W = 0;
  for (int w = 0; w < nw; ++w) {
    const uint64_t t = s_tot[w];
    off += w < wave ? t : 0;
    W += t;
  }
  if (W == 0) return -1;                   // uniform over the block
  const uint64_t thr = grid_threshold(u, W);
  if (off <= thr && thr < off + tot) {     // the crossing lies in this wave's segment
    uint64_t run = off;
    for (int base = sg.b0; base < sg.b1; base += 64 * kScanPerLane) {
      uint64_t w[kScanPerLane];
      uint64_t lt = 0;
      const int c0 = base + kScanPerLane * lane;
#pragma unroll
      for (int k = 0; k < kScanPerLane; ++k) {
        const uint64_t x = wf(min(c0 + k, sg.b1 - 1));
        w[k] = c0 + k < sg.b1 ? x : 0;
        lt += w[k];
      }
      const uint64_t inc = wave_incl_scan_u64(lt);
      const uint64_t all = (static_cast<uint64_t>(__shfl(static_cast<uint32_t>(inc >> 32), 63)) << 32) |
                           __shfl(static_cast<uint32_t>(inc), 63);
      if (run + all > thr) {               // wave-uniform
        const uint64_t ex = run + inc - lt;
        if (ex <= thr && thr < ex + lt) {  // exactly one lane
          uint64_t acc = ex;
          int hit = -1;                    // first entry whose inclusive prefix exceeds thr
#pragma unroll
          for (int k = 0; k < kScanPerLane; ++k) {
            acc += w[k];
            if (hit < 0 && acc > thr) hit = k;
          }
          *s_res = c0 + hit;
        }
        break;
      }
      run += all;
    }
  }
  __syncthreads();
  return *s_res;
}

// Target probabilities given as a [rows][V] array; row(r)(i) = q_r(i).
struct QProbs {
  const float* q;
  int V;
  struct Row {
    const float* q;
    __device__ bool modified() const { return false; }
    __device__ bool nonfinite() const { return false; }   // given values: checked where read
    template <bool MOD> __device__ float get(int i) const { return q[i]; }
    __device__ float operator()(int i) const { return q[i]; }
  };
  __device__ Row row(int r) const { return Row{q + static_cast<size_t>(r) * V}; }
};
// Target probabilities formed on the fly from logits and row statistics.
struct QLogits {
  const float* z;
  const RowStat* st;
  float inv_t;
  int V;
  struct Row {
    const float* z;
    RowStat st;
    float inv_t;
    __device__ bool modified() const { return row_modified(st); }
    __device__ bool nonfinite() const { return st.nonfinite != 0; }
    template <bool MOD> __device__ float get(int i) const { return prob_final<MOD>(z[i], st, inv_t, i); }
    __device__ float operator()(int i) const {
      return modified() ? get<true>(i) : get<false>(i);
    }
  };
  __device__ Row row(int r) const { return Row{z + static_cast<size_t>(r) * V, st[r], inv_t}; }
};

__device__ __forceinline__ bool not_finite(float x) { return !(fabsf(x) < INFINITY); }

// The final draw of one sequence: from (q - p)_+ if resid (falling back to
// q when its weights sum to 0), else from q. -1 if q's weights are all 0,
// -2 if a value of a row it read is NaN or infinite.
template <bool MOD, class Row>
__device__ __forceinline__ int accept_draw(const Row& qr, const float* __restrict__ prow, bool resid, int V,
                                           float u, uint64_t* wsum, int* s_y) {
  const Segment sg = wave_segment(V);
  bool nf = false;
  auto wq = [&](int i) -> uint64_t {
    const float x = qr.template get<MOD>(i);
    nf |= not_finite(x);
    return fixed_weight(x);
  };
  auto wr = [&](int i) -> uint64_t {
    const float xq = qr.template get<MOD>(i), xp = prow[i];
    nf |= not_finite(xq) | not_finite(xp);
    const uint64_t x = fixed_weight(xq), y = fixed_weight(xp);
    return x > y ? x - y : 0;
  };
  int y = -1;
  if (resid) y = block_draw(wr, sg, segment_total(wr, sg), u, wsum, s_y);
  if (y < 0) y = block_draw(wq, sg, segment_total(wq, sg), u, wsum, s_y);
  return __syncthreads_or(nf) ? -2 : y;
}

// The accept tests of sequence b, left to right, r_t p_t(x~_t) < q_t(x~_t)
// exact in fp64 (wave 0 of the work-group; lane t tests draft t): a = the
// first rejected draft (K if none), bad = x~_a is out of range, nf = a value
// the tests read or a target row of the sequence is non-finite. Every lane
// of the wave returns the same values. drafts[t] is x~_{t+1}.
template <class QS>
__device__ __forceinline__ void accept_tests(const QS& qs, const float* __restrict__ p,
                                             const int32_t* __restrict__ dr, const float* __restrict__ unif,
                                             uint64_t seed, uint64_t loop, int K, int V, int b, int* a_out,
                                             bool* bad_out, bool* nf_out) {
  const int tid = threadIdx.x;
  bool rejected = false, bad = false, nf = false;
  if (tid < K) {
    const int x = dr[tid];
    if (x < 0 || x >= V) {
      bad = true;
      rejected = true;
    } else {
      const float rho = qs.row(b * (K + 1) + tid)(x);
      const float pi = p[(static_cast<size_t>(b) * K + tid) * V + x];
      const float r = unif ? unif[b * (K + 1) + tid] : philox_uniform(seed, loop, 1, b, tid);
      nf = not_finite(rho) | not_finite(pi);
      rejected = !(static_cast<double>(r) * static_cast<double>(pi) < static_cast<double>(rho));
    }
  }
  if (tid <= K) nf |= qs.row(b * (K + 1) + tid).nonfinite();
  const uint64_t rej = __ballot(rejected);
  const uint64_t badm = __ballot(bad);
  *nf_out = __ballot(nf) != 0;                     // wave-wide, outside any branch
  const int a = rej ? __ffsll(static_cast<long long>(rej)) - 1 : K;
  *a_out = a;
  *bad_out = a < K && ((badm >> a) & 1ull) != 0;
}

// The outcome of sequence b from a and the draw y (-2: a non-finite value
// was read, -1: every weight zero): out[b][0 .. K] = the accepted drafts, the
// drawn token, then -1; n_acc[b] = a. A sequence whose inputs hold a
// non-finite value -- a target row with a NaN / +Inf logit, a NaN or
// infinite gathered probability, or one in a row of the final draw -- has
// no defined outcome: it is given a = 0 and token 0, and the device flag is
// raised.
__device__ __forceinline__ void accept_finish(int b, int a, int y, const int32_t* __restrict__ dr, int K,
                                              int32_t* __restrict__ out, int32_t* __restrict__ n_acc, int* err) {
  const int tid = threadIdx.x;
  if (y == -2) {
    a = 0;
    y = 0;
    if (tid == 0) atomicOr(err, kErrNonFinite);
  } else if (y < 0) {
    y = 0;
    if (tid == 0) atomicOr(err, kErrEmpty);
  }
  if (tid <= K) out[static_cast<size_t>(b) * (K + 1) + tid] = tid < a ? dr[tid] : (tid == a ? y : -1);
  if (tid == 0) n_acc[b] = a;
}

// One block per sequence. drafts[b * dstride + doff + t] is x~_{t+1}.
template <class QS>
__global__ __launch_bounds__(kSampleThreads) void accept_kernel(QS qs, const float* __restrict__ p,
                                                                const int32_t* __restrict__ drafts, int dstride,
                                                                int doff, const float* __restrict__ unif,
                                                                uint64_t seed, uint64_t loop, int K, int V,
                                                                int32_t* __restrict__ out,
                                                                int32_t* __restrict__ n_acc, int* err) {
  __shared__ int s_a, s_y, s_nf;
  __shared__ uint64_t wsum[17];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int32_t* dr = drafts + static_cast<size_t>(b) * dstride + doff;

  // 1. left-to-right accept tests
  if (tid < 64) {
    int a;
    bool bad, nf;
    accept_tests(qs, p, dr, unif, seed, loop, K, V, b, &a, &bad, &nf);
    if (tid == 0) {
      if (bad) atomicOr(err, kErrBadToken);
      s_a = a;
      s_y = 0;
      s_nf = nf;
    }
  }
  __syncthreads();
  const int a = s_a;
  const bool nf_in = s_nf != 0;
  const int row = b * (K + 1) + a;
  const bool resid = a < K;
  const float* prow = p + (static_cast<size_t>(b) * K + (resid ? a : 0)) * V;

  // 2. draw from (q - p)_+ (or q for the bonus / the zero-residual fallback)
  int y = -2;
  if (!nf_in) {                            // uniform over the block
    const typename QS::Row qr = qs.row(row);
    const float u = unif ? unif[b * (K + 1) + K] : philox_uniform(seed, loop, 2, b, 0);
    y = qr.modified() ? accept_draw<true>(qr, prow, resid, V, u, wsum, &s_y)
                      : accept_draw<false>(qr, prow, resid, V, u, wsum, &s_y);
  }
  accept_finish(b, a, y, dr, K, out, n_acc, err);
}

// ---------------------------------------------------------------------------
// The verify step's accept / resample over several CUs (the same outcome as
// accept_kernel). accept_part_kernel's work-groups take one segment of the
// final draw's row each: every one runs the accept tests (K gathers) to find
// that row, then adds its segment's residual weights (q - p)_+ and q
// weights (the zero-residual fallback and the bonus draw) and flags a
// non-finite value among them; accept_draw_kernel finds the segment that
// holds the draw's threshold from the totals and scans only it. Integer sums
// do not depend on their order, so the token is accept_kernel's.
// Row scratch: cs.n[s] residual and cs.w[s] q totals of segment s,
// cs.n[kAccNf + s] its non-finite flag, cs.n[kAccHead ..] a, the tests'
// non-finite flag and the bad-token flag.
// ---------------------------------------------------------------------------
constexpr int kAccNf = 64, kAccHead = 128;
static_assert(kAccNf >= kMaxRowSegments && kAccHead >= kAccNf + kMaxRowSegments && kAccHead + 3 <= kCutBuckets,
              "accept totals fit the row scratch");

template <bool MOD, class Row>
__device__ __forceinline__ void segment_accept_weights(const Row& qr, const float* __restrict__ prow, bool resid,
                                                       int i0, int i1, uint64_t* wr, uint64_t* wq, bool* nf) {
  for (int i = i0 + static_cast<int>(threadIdx.x); i < i1; i += kCutSegThreads) {
    const float xq = qr.template get<MOD>(i);
    *nf |= not_finite(xq);
    const uint64_t x = fixed_weight(xq);
    *wq += x;
    if (resid) {
      const float xp = prow[i];
      *nf |= not_finite(xp);
      const uint64_t y = fixed_weight(xp);
      *wr += x > y ? x - y : 0;
    }
  }
}

// Grid (segments, B), kCutSegThreads threads.
template <class QS>
__global__ __launch_bounds__(kCutSegThreads) void accept_part_kernel(QS qs, const float* __restrict__ p,
                                                                     const int32_t* __restrict__ drafts, int dstride,
                                                                     int doff, const float* __restrict__ unif,
                                                                     uint64_t seed, uint64_t loop, int K, int V,
                                                                     char* __restrict__ cut, size_t cut_bytes,
                                                                     int seg) {
  __shared__ int s_a, s_nf;
  __shared__ uint64_t s_r[kCutSegThreads / 64], s_q[kCutSegThreads / 64];   // per wave: residual, q totals
  __shared__ int s_wnf[kCutSegThreads / 64];                                  // per wave: a non-finite value
  const int b = blockIdx.y, s = blockIdx.x, tid = threadIdx.x;
  const int32_t* dr = drafts + static_cast<size_t>(b) * dstride + doff;
  const CutRowScratch cs = cut_row(cut, cut_bytes, b);
  if (tid < 64) {
    int a;
    bool bad, nf;
    accept_tests(qs, p, dr, unif, seed, loop, K, V, b, &a, &bad, &nf);
    if (tid == 0) {
      s_a = a;
      s_nf = nf;
      if (s == 0) {
        cs.n[kAccHead] = static_cast<uint64_t>(a);
        cs.n[kAccHead + 1] = nf ? 1u : 0u;
        cs.n[kAccHead + 2] = bad ? 1u : 0u;
      }
    }
  }
  __syncthreads();
  const int a = s_a;
  uint64_t wr = 0, wq = 0;
  bool nf = false;
  if (!s_nf) {                                     // uniform: the tests' inputs were finite
    const bool resid = a < K;
    const typename QS::Row qr = qs.row(b * (K + 1) + a);
    const float* prow = p + (static_cast<size_t>(b) * K + (resid ? a : 0)) * V;
    const int i0 = s * seg, i1 = min(V, i0 + seg);
    if (qr.modified())
      segment_accept_weights<true>(qr, prow, resid, i0, i1, &wr, &wq, &nf);
    else
      segment_accept_weights<false>(qr, prow, resid, i0, i1, &wr, &wq, &nf);
  }
  wr = wave_sum_u64(wr);
  wq = wave_sum_u64(wq);
  const bool wnf = __ballot(nf) != 0;
  if ((tid & 63) == 0) {
    s_r[tid >> 6] = wr;
    s_q[tid >> 6] = wq;
    s_wnf[tid >> 6] = wnf ? 1 : 0;
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t tr = 0, tq = 0;
    int f = 0;
    for (int v = 0; v < kCutSegThreads / 64; ++v) {
      tr += s_r[v];
      tq += s_q[v];
      f |= s_wnf[v];
    }
    cs.n[s] = tr;
    cs.w[s] = tq;
    cs.n[kAccNf + s] = static_cast<uint64_t>(f);
  }
}

// One work-group (kCutSegThreads threads) per sequence.
template <class QS>
__global__ __launch_bounds__(kCutSegThreads) void accept_draw_kernel(QS qs, const float* __restrict__ p,
                                                                     const int32_t* __restrict__ drafts, int dstride,
                                                                     int doff, const float* __restrict__ unif,
                                                                     uint64_t seed, uint64_t loop, int K, int V,
                                                                     const char* __restrict__ cut, size_t cut_bytes,
                                                                     int nseg, int seg, int32_t* __restrict__ out,
                                                                     int32_t* __restrict__ n_acc, int* err) {
  static_assert(kMaxRowSegments <= 64, "one wave holds the segment totals");
  __shared__ uint64_t wsum[17];
  __shared__ uint64_t s_thr, s_off;
  __shared__ int s_seg, s_y, s_mode;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int32_t* dr = drafts + static_cast<size_t>(b) * dstride + doff;
  const CutRowScratch cs = cut_row(const_cast<char*>(cut), cut_bytes, b);
  const int a = static_cast<int>(cs.n[kAccHead]);
  const bool nf_in = cs.n[kAccHead + 1] != 0;
  if (tid == 0 && cs.n[kAccHead + 2] != 0) atomicOr(err, kErrBadToken);
  const bool resid = a < K;
  // Wave 0: the segments' flags and totals; the weights drawn from (the
  // residual, or q for the bonus and when the residual sums to 0); the
  // threshold and the segment holding it.
  if (tid < 64) {
    const bool in = tid < nseg;
    const bool nf = __ballot(in && cs.n[kAccNf + tid] != 0) != 0;
    const uint64_t tr = in ? cs.n[tid] : 0, tq = in ? cs.w[tid] : 0;
    uint64_t ir = tr, iq = tq;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t o1 = shfl_up_u64(ir, d), o2 = shfl_up_u64(iq, d);
      if (tid >= d) {
        ir += o1;
        iq += o2;
      }
    }
    const uint64_t Wr = shfl_u64(ir, 63), Wq = shfl_u64(iq, 63);
    const bool use_r = resid && Wr != 0;
    const uint64_t W = use_r ? Wr : Wq, inc = use_r ? ir : iq, tot = use_r ? tr : tq;
    const float u = unif ? unif[b * (K + 1) + K] : philox_uniform(seed, loop, 2, b, 0);
    const uint64_t thr = grid_threshold(u, W);
    const uint64_t hit = W ? __ballot(in && inc > thr) : 0;
    const int sstar = hit ? __ffsll(static_cast<long long>(hit)) - 1 : -1;
    const uint64_t off = shfl_u64(inc - tot, sstar < 0 ? 0 : sstar);
    if (tid == 0) {
      s_thr = thr;
      s_off = off;
      s_seg = sstar;
      s_mode = nf_in || nf ? -2 : use_r ? 1 : 0;   // -2: a non-finite value was read
      s_y = -1;
    }
  }
  __syncthreads();
  const int mode = s_mode, sstar = s_seg;
  if (mode != -2 && sstar >= 0) {                 // uniform
    const typename QS::Row qr = qs.row(b * (K + 1) + a);
    const float* prow = p + (static_cast<size_t>(b) * K + (resid ? a : 0)) * V;
    const bool mod = qr.modified();
    auto wt = [&](int i) -> uint64_t {
      const uint64_t x = fixed_weight(mod ? qr.template get<true>(i) : qr.template get<false>(i));
      if (mode == 0) return x;
      const uint64_t y = fixed_weight(prow[i]);
      return x > y ? x - y : 0;
    };
    const uint64_t thr = s_thr;
    const int i0 = sstar * seg, i1 = min(V, i0 + seg);
    uint64_t run = s_off;
    for (int base = i0; base < i1; base += kCutSegThreads * kDrawPer) {
      uint64_t w[kDrawPer], lt = 0;
      const int c0 = base + kDrawPer * tid;
#pragma unroll
      for (int k = 0; k < kDrawPer; ++k) {
        w[k] = c0 + k < i1 ? wt(c0 + k) : 0;
        lt += w[k];
      }
      uint64_t total;
      const uint64_t ex = run + block_exscan_u64(lt, wsum, &total);
      if (ex <= thr && thr < ex + lt) {            // exactly one thread
        uint64_t acc = ex;
        int hitk = -1;
#pragma unroll
        for (int k = 0; k < kDrawPer; ++k) {
          acc += w[k];
          if (hitk < 0 && acc > thr) hitk = k;
        }
        s_y = c0 + hitk;
      }
      __syncthreads();
      if (s_y >= 0) break;                         // uniform
      run += total;
    }
  }
  __syncthreads();
  accept_finish(b, a, mode == -2 ? -2 : s_y, dr, K, out, n_acc, err);
}

// Draft step t: p_t = softmax(logits of the last row of each sequence / T),
// written to p_out[b][t][:], and x~_{t+1} drawn from it into tokens[b][t+1].
__global__ __launch_bounds__(kSampleThreads) void draft_sample_kernel(
    const float* __restrict__ logits, int Mps, int V, float temperature, int top_k, float top_p,
    const RowStat* __restrict__ pre, float* __restrict__ p_out, int K, int t, int32_t* __restrict__ tokens,
    const int32_t* __restrict__ ctx, uint64_t seed, uint64_t loop, int* err) {
  __shared__ float red[32];
  __shared__ int ired[16];
  __shared__ uint64_t wsum[17];
  __shared__ int s_y;
  __shared__ CutScratch sc;
  extern __shared__ uint32_t s_rowkeys[];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* z = logits + (static_cast<size_t>(b) * Mps + Mps - 1) * V;
  // (A row with a NaN / +Inf logit becomes p_t = one-hot at token 0, a valid
  // draft distribution, so the draw gives token 0 and the flag is raised.)
  // (pre: the statistics, with the cut, of the row of sequence b, taken by
  // the cut-off kernels, which also raised the flag for a non-finite row.)
  const RowStat st = pre ? pre[b] : row_stat_final(z, V, temperature, top_k, top_p, red, ired, sc, s_rowkeys, err);
  const float inv_t = temperature == 0.f ? 0.f : 1.0f / temperature;
  // p_t once into p_out, then the draw from the stored values (visible to
  // the whole block after the barrier).
  float* pr = p_out + (static_cast<size_t>(b) * K + t) * V;
  write_probs(z, V, st, inv_t, pr);
  __syncthreads();
  const Segment sg = wave_segment(V);
  auto wp = [&](int i) -> uint64_t { return fixed_weight(pr[i]); };
  int y = block_draw(wp, sg, segment_total(wp, sg), philox_uniform(seed, loop, 0, b, t), wsum, &s_y);
  if (y < 0) {
    y = 0;
    if (tid == 0) atomicOr(err, kErrEmpty);
  }
  if (tid == 0) {
    tokens[static_cast<size_t>(b) * (K + 1) + t + 1] = y;
    if (t == 0) tokens[static_cast<size_t>(b) * (K + 1)] = ctx[2 * b + 1];
  }
}

__global__ void commit_kernel(int32_t* __restrict__ lengths, const int32_t* __restrict__ tokens,
                              const int32_t* __restrict__ out, const int32_t* __restrict__ n_acc, int B, int K,
                              int32_t* __restrict__ ctx, int32_t* __restrict__ seq_out, int32_t* __restrict__ n_out,
                              int cap) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int a = n_acc[b];
  a = a < 0 ? 0 : (a > K ? K : a);
  if (n_out) {
    const int n = n_out[b];
    if (n >= cap) return;
    int w = n;
    for (int i = 0; i <= a && w < cap; ++i, ++w) seq_out[static_cast<size_t>(b) * cap + w] = out[b * (K + 1) + i];
    n_out[b] = w;
  }
  lengths[b] += a + 1;
  ctx[2 * b] = tokens[b * (K + 1) + a];
  ctx[2 * b + 1] = out[b * (K + 1) + a];
}

__global__ void philox_kernel(uint64_t seed, uint64_t loop, int purpose, int B, int n, float* __restrict__ out) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(B) * n) return;
  out[i] = philox_uniform(seed, loop, static_cast<uint32_t>(purpose), static_cast<uint32_t>(i / n),
                          static_cast<uint32_t>(i % n));
}

// Dynamic LDS of a sampling launch: the cut-off's row weights when a
// modifier is on (above the default 64 KiB limit the kernel is opted in
// once per process to the CU's full LDS).
static hipError_t cutoff_lds(const void* kernel, float temperature, int top_k, float top_p, int V, size_t* bytes) {
  const bool on = temperature > 0.f && ((top_k >= 1 && top_k < V) || top_p < 1.f);
  *bytes = on ? (cutoff_lds_bytes(V) + 15) / 16 * 16 : 0;
  if (*bytes > 65536) {
    static bool opted[3] = {false, false, false};
    const int which = kernel == reinterpret_cast<const void*>(&row_softmax_kernel)  ? 0
                      : kernel == reinterpret_cast<const void*>(&cut_select_kernel) ? 2
                                                                                     : 1;
    if (!opted[which]) {
      // The largest row the cut-off handles (the kernels' static LDS and this
      // fit the CU's 160 KiB).
      const int most = static_cast<int>((cutoff_lds_bytes(modifier_max_vocab()) + 15) / 16 * 16);
      const hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, most);
      if (e != hipSuccess) return e;
      opted[which] = true;
    }
  }
  return hipSuccess;
}

// The cut-off over several CUs for `rows` rows (logits row r rstride +
// roff), their statistics into stats[0 .. rows).
static hipError_t cut_rows(const float* logits, int rows, int rstride, int roff, int V, float temperature, int top_k,
                           float top_p, RowStat* stats, char* cut, int* err, int* seg_out, int* nseg_out,
                           hipStream_t st) {
  const size_t cut_bytes = cut_row_bytes(V);
  int seg = 0, nseg = 0;
  cut_segments(rows, V, &seg, &nseg);
  size_t lds = 0;
  hipError_t e = cutoff_lds(reinterpret_cast<const void*>(&cut_select_kernel), temperature, top_k, top_p, V, &lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cut_part_kernel, dim3(kStatWaves, rows), dim3(64), 0, st, logits, V, rstride, roff, temperature,
                     cut, cut_bytes);
  hipLaunchKernelGGL(cut_hist_kernel, dim3(nseg, rows), dim3(kCutSegThreads), 0, st, logits, V, rstride,
                     roff, temperature, stats, cut, cut_bytes, seg);
  hipLaunchKernelGGL(cut_select_kernel, dim3(rows), dim3(kSampleThreads), lds, st, logits, V, rstride, roff,
                     temperature, top_k, top_p, stats, cut, cut_bytes, err);
  *seg_out = seg;
  *nseg_out = nseg;
  return hipGetLastError();
}

hipError_t launch_row_softmax(const float* logits, int rows, int V, float temperature, int top_k, float top_p,
                              void* stats, float* probs, char* cut, int* err, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (cut && stats && modifiers_active(temperature, top_k, top_p, V) && V <= modifier_max_vocab()) {
    int seg = 0, nseg = 0;
    RowStat* rs = reinterpret_cast<RowStat*>(stats);
    const hipError_t e = cut_rows(logits, rows, 1, 0, V, temperature, top_k, top_p, rs, cut, err, &seg, &nseg, st);
    if (e != hipSuccess || !probs) return e;
    hipLaunchKernelGGL(cut_export_kernel, dim3(nseg, rows), dim3(kCutSegThreads), 0, st, logits, V, temperature, rs,
                       probs, seg);
    return hipGetLastError();
  }
  size_t lds = 0;
  const hipError_t e = cutoff_lds(reinterpret_cast<const void*>(&row_softmax_kernel), temperature, top_k, top_p, V,
                                  &lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(row_softmax_kernel, dim3(rows), dim3(kSampleThreads), lds, st, logits, V, temperature, top_k,
                     top_p, reinterpret_cast<RowStat*>(stats), probs, err);
  return hipGetLastError();
}

hipError_t launch_accept_probs(const float* p, const float* q, const int32_t* drafts, const float* unif,
                               uint64_t seed, uint64_t loop, int B, int K, int V, int32_t* out, int32_t* n_acc,
                               int* err, hipStream_t st) {
  hipLaunchKernelGGL(accept_kernel<QProbs>, dim3(B), dim3(kSampleThreads), 0, st, QProbs{q, V}, p, drafts, K, 0,
                     unif, seed, loop, K, V, out, n_acc, err);
  return hipGetLastError();
}

hipError_t launch_accept_logits(const float* p, const float* logits, const void* stats, float temperature,
                                const int32_t* tokens, const float* unif, uint64_t seed, uint64_t loop, int B,
                                int K, int V, int32_t* out, int32_t* n_acc, char* cut, int* err, hipStream_t st) {
  const float inv_t = temperature == 0.f ? 0.f : 1.0f / temperature;
  const QLogits qs{logits, reinterpret_cast<const RowStat*>(stats), inv_t, V};
  if (cut && V <= modifier_max_vocab()) {
    int seg = 0, nseg = 0;
    cut_segments(B, V, &seg, &nseg);
    const size_t cut_bytes = cut_row_bytes(V);
    hipLaunchKernelGGL(accept_part_kernel<QLogits>, dim3(nseg, B), dim3(kCutSegThreads), 0, st, qs, p, tokens, K + 1,
                       1, unif, seed, loop, K, V, cut, cut_bytes, seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(accept_draw_kernel<QLogits>, dim3(B), dim3(kCutSegThreads), 0, st, qs, p, tokens, K + 1, 1,
                       unif, seed, loop, K, V, static_cast<const char*>(cut), cut_bytes, nseg, seg, out, n_acc,
                       err);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(accept_kernel<QLogits>, dim3(B), dim3(kSampleThreads), 0, st, qs, p, tokens, K + 1, 1, unif,
                     seed, loop, K, V, out, n_acc, err);
  return hipGetLastError();
}

hipError_t launch_draft_sample(const float* logits, int Mps, int B, int V, float temperature, int top_k,
                               float top_p, float* p_out, int K, int t, int32_t* tokens, const int32_t* ctx,
                               uint64_t seed, uint64_t loop, void* stats, char* cut, int* err, hipStream_t st) {
  if (cut && stats && temperature > 0.f && V <= modifier_max_vocab()) {
    // Statistics (and the cut) over several CUs, then p_t and the draw.
    const size_t cut_bytes = cut_row_bytes(V);
    RowStat* rs = reinterpret_cast<RowStat*>(stats);
    const bool mod = modifiers_active(temperature, top_k, top_p, V);
    int seg = 0, nseg = 0;
    hipError_t e = hipSuccess;
    if (mod) {
      e = cut_rows(logits, B, Mps, Mps - 1, V, temperature, top_k, top_p, rs, cut, err, &seg, &nseg, st);
    } else {
      cut_segments(B, V, &seg, &nseg);
      hipLaunchKernelGGL(cut_part_kernel, dim3(kStatWaves, B), dim3(64), 0, st, logits, V, Mps, Mps - 1, temperature,
                         cut, cut_bytes);
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(draft_p_kernel, dim3(nseg, B), dim3(kCutSegThreads), 0, st, logits, Mps, V, temperature,
                       mod ? static_cast<const RowStat*>(rs) : static_cast<const RowStat*>(nullptr), cut, cut_bytes, seg,
                       p_out, K, t, err);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(draft_draw_kernel, dim3(B), dim3(kCutSegThreads), 0, st, cut, cut_bytes, nseg, seg, V, p_out, K,
                       t, tokens, ctx, seed, loop, err);
    return hipGetLastError();
  }
  size_t lds = 0;
  const hipError_t e = cutoff_lds(reinterpret_cast<const void*>(&draft_sample_kernel), temperature, top_k, top_p, V,
                                  &lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(draft_sample_kernel, dim3(B), dim3(kSampleThreads), lds, st, logits, Mps, V, temperature, top_k,
                     top_p, static_cast<const RowStat*>(nullptr), p_out, K, t, tokens, ctx, seed, loop, err);
  return hipGetLastError();
}

hipError_t launch_commit(int32_t* lengths, const int32_t* tokens, const int32_t* out, const int32_t* n_acc, int B,
                         int K, int32_t* ctx, int32_t* seq_out, int32_t* n_out, int cap, hipStream_t st) {
  hipLaunchKernelGGL(commit_kernel, dim3((B + 255) / 256), dim3(256), 0, st, lengths, tokens, out, n_acc, B, K, ctx,
                     seq_out, n_out, cap);
  return hipGetLastError();
}

__global__ void ctx_tokens_kernel(const int32_t* __restrict__ ctx, int B, int K, int32_t* __restrict__ tokens) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) tokens[static_cast<size_t>(b) * (K + 1)] = ctx[2 * b + 1];
}

hipError_t launch_ctx_tokens(const int32_t* ctx, int B, int K, int32_t* tokens, hipStream_t st) {
  hipLaunchKernelGGL(ctx_tokens_kernel, dim3((B + 255) / 256), dim3(256), 0, st, ctx, B, K, tokens);
  return hipGetLastError();
}

hipError_t launch_philox(uint64_t seed, uint64_t loop, int purpose, int B, int n, float* out, hipStream_t st) {
  const long work = static_cast<long>(B) * n;
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(philox_kernel, dim3(static_cast<unsigned>((work + 255) / 256)), dim3(256), 0, st, seed, loop,
                     purpose, B, n, out);
  return hipGetLastError();
}

}  // namespace sps
