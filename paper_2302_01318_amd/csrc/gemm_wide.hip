// Wide skinny GEMM for bf16 models at 9..160 rows (batched verify steps:
// M = B (K+1) with several sequences). Same packed weights, activation format
// and epilogues as gemm.hip; what changes is who shares what.
//
// The single-tile kernel lets every wave load its own copy of the activation
// fragments it multiplies. At MT M tiles that is MT activation bytes per
// weight byte through the vector caches, and above MT = 1 that traffic, not
// HBM, sets the speed. Here:
//
//  * a work-group of WV waves (4, or 8 where bf16 weights are staged
//    through LDS) owns WV NTW consecutive n-tiles (NTW = 2) and one
//    contiguous range of the k-tiles; wave w multiplies n-tiles
//    NTW w .. NTW w + NTW - 1 by all MT M tiles;
//  * per chunk of KC k-tiles the work-group copies the chunk's activations
//    once into LDS with global_load_lds (16 B per lane, whole 128-byte
//    lines per instruction: act_piece_src), so all the waves share them,
//    and every wave streams its own weight fragments from HBM into
//    registers (from 14 M tiles, 8 with FP8 codes, through LDS as well:
//    the staged loop);
//  * where N is too small to give every CU a work-group (the d_model-wide
//    outputs), the k range is split S ways (split-K): each split writes its
//    fp32 partial tile to the workspace and a second kernel sums the splits
//    in split order and runs the epilogue, one work-group per norm group
//    (8 n-tiles, 128 columns: the unit of the residual epilogue's sums of
//    squares whatever NTW is) and M tile. (A last-arriving-split fixup
//    inside one kernel would need device-scope fences, which on this GPU
//    write back and invalidate the L2 and cost more than the launch.)
//
// FP8 weights (W8): the weight fragments come from the 16 x 64 code tiles of
// gemm.hip, one 16-byte load per lane and n-tile for each pair of k-tiles of
// a chunk (KC even), converted exactly to two bf16 B fragments before their
// MFMAs; the row scale is applied in the epilogue.
#include <algorithm>

#include "common.h"
#include "fp8.h"
#include "gemm_epi.h"
#include "launch.h"

namespace sps {

// s_waitcnt operand that waits until at most n vector memory operations of
// this wave are outstanding, ignoring the export and LDS/scalar counters
// (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) & 3) << 14 | 7 << 4 | 15 << 8; }

// Partial tile of one wave: NTW x MT fragments of 32 lanes x 4 floats (the
// hi rows after folding the lo rows in), in register order.
template <int MT, int NTW> constexpr int wide_part_floats() { return NTW * MT * 128; }

template <int MT, bool W8> constexpr int wide_waves_per_simd() { return waves_per_simd(MT, W8); }

// Weight registers of one chunk: bf16 fragments, or the raw FP8 code loads
// (one per k-tile pair) that become fragments right before their MFMAs.
template <bool W8, int NTW, int KC> struct WideB;
template <int NTW, int KC> struct WideB<false, NTW, KC> { Frag<bf16> f[NTW][KC]; };
template <int NTW, int KC> struct WideB<true, NTW, KC> { u32x4 r[NTW][KC / 2]; };

// One global_load_lds copy (16 bytes per lane, lane l to LDS address
// lds + 16 l), written as inline assembly so that the compiler's wait-count
// insertion does not track it: for a tracked copy it makes every later LDS
// read wait for all copies in flight, whatever buffer they fill. The caller
// waits for the copies itself (s_waitcnt vmcnt) before reading what they
// wrote; the kernel has no other vector memory operations in flight then.
__device__ __forceinline__ void lds_copy16_untracked(const void* src, uint32_t lds) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(lds) : "memory");
}

// One activation fragment of zeros: the source of activation pieces past
// KT (zero activations times finite weights add exact zeros).
__device__ const bf16x8 kZeroFrag[64] = {};

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));   // low half of the flat address
}

// Activation blocks. A chunk's activations go to LDS as blocks of 1 KiB, one
// per (M tile mt, k-tile pair, half h): rows 4 h .. 4 h + 3 of the M tile in
// both planes, each row's 128 bytes (the two k-tiles of the pair) whole, so
// every copy instruction reads 8 complete 128-byte lines where a copy in
// MFMA fragment order would read 16 half lines. Lane 8 rho + q of a block
// copies the 16-byte piece q ^ r ^ pl of row r = 4 h + rho % 4 of plane
// pl = rho / 4; the XOR swizzle makes the MFMA-order reads conflict-free
// (every 8 and every 16 consecutive lanes of a ds_read_b128 hit distinct
// 16-byte bank groups).
//
// Source of this lane's piece of block (mt, h) of the pair starting at
// k-tile kb; pieces of k-tiles past KT read zeros.
__device__ __forceinline__ const void* act_piece_src(const GemmParams& p, int lane, int mt, int h, int kb) {
  const int rho = lane >> 3, pl = rho >> 2;
  const int r = h * 4 + (rho & 3);
  const int piece = (lane & 7) ^ r ^ pl;            // k-tile kb + piece / 4, k-group piece % 4
  const int m = mt * 8 + r;
  if (kb + (piece >> 2) >= p.KT) return &kZeroFrag[lane];
  return static_cast<const bf16*>(p.X) + pl * p.xplane + static_cast<size_t>(p.m0 + (m < p.M ? m : 0)) * p.ldx +
         kb * 32 + piece * 8;
}

// Where the MFMA A operand of a pair's k-tile u (0 or 1) sits for this
// lane (row l % 8 of plane (l / 8) % 2, k-group l / 16): block half
// act_half(lane), slot act_slot(lane, u).
__device__ __forceinline__ int act_half(int lane) { return (lane & 7) >> 2; }
__device__ __forceinline__ int act_slot(int lane, int u) {
  const int r = lane & 7, pl = (lane >> 3) & 1, g = lane >> 4;
  return (pl * 4 + (r & 3)) * 8 + ((u * 4 + g) ^ r ^ pl);
}

// The lo-plane rows of an accumulator tile (lanes 32-63) added into their
// hi rows (lanes 0-31), which then hold the output rows.
__device__ __forceinline__ void fold_lo(f32x4& a) {
#pragma unroll
  for (int r = 0; r < 4; ++r) a[r] += __shfl_xor(a[r], 32);
}

// Accumulate chunks [c0, c1) of column group g into acc (the caller folds
// the lo-plane rows into the hi rows with fold_lo). Double
// buffered: while a chunk's MFMAs run, the next chunk's activation
// fragments are already on their way into the other LDS buffer (s_a holds
// 2 * MT * KC fragments) and its weight fragments into the other register
// set; one barrier per chunk.
template <int MT, int KC, int NTW, int WV, bool W8>
__device__ __forceinline__ void wide_mainloop(const GemmParams& p, int g, int c0, int c1, bf16x8 (*s_a)[64],
                                              f32x4 (&acc)[NTW][MT]) {
  static_assert(KC % 2 == 0, "chunks hold whole k-tile pairs (activation blocks, FP8 codes)");
  using B = WideB<W8, NTW, KC>;
  using T = bf16;
  constexpr int kTile = 512;                       // elements per 16 x 32 tile
  constexpr int kBuf = MT * KC;                    // fragments per LDS buffer
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ntw = g * WV * NTW + wave * NTW;          // first n-tile of this wave
  const int KT = p.KT;
  const T* W = static_cast<const T*>(p.W);

  const T* wp[NTW];
  const u32x4* wq[NTW];                            // FP8: pair kp of n-tile j at wq[j] + 64 kp
  bool wv[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    wv[j] = ntw + j < p.NT;
    wp[j] = W + static_cast<size_t>(wv[j] ? ntw + j : 0) * KT * kTile + lane * 8;
    wq[j] = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(p.W) +
                                           static_cast<size_t>(wv[j] ? ntw + j : 0) * KT * kTile) + lane;
  }
  const int a_half = act_half(lane), a_slot0 = act_slot(lane, 0), a_slot1 = act_slot(lane, 1);

#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Activation blocks of chunk c into LDS buffer bb: block f = 2 (mt KC / 2
  // + pair) + h; pairs wholly past KT are skipped (their MFMAs are).
  auto issue_a = [&](int c, int bb) {
    const int kb = c * KC;
    for (int f = wave; f < kBuf; f += WV) {
      const int h = f & 1, pr = (f >> 1) % (KC / 2), mt = (f >> 1) / (KC / 2);
      if (kb + 2 * pr < KT)
        __builtin_amdgcn_global_load_lds(act_piece_src(p, lane, mt, h, kb + 2 * pr),
                                         reinterpret_cast<void*>(&s_a[bb * kBuf + f][0]), 16, 0, 0);
    }
  };
  // A operand of k-tile u of the chunk, M tile mt, from buffer bb.
  auto frag_a = [&](int bb, int mt, int u) {
    return s_a[bb * kBuf + (mt * (KC / 2) + u / 2) * 2 + a_half][u % 2 ? a_slot1 : a_slot0];
  };
  auto load_b = [&](int c, B& b) {
    const int kb = c * KC;
    if constexpr (W8) {
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int u = 0; u < KC / 2; ++u)     // KT is even: a pair is whole or absent
          b.r[j][u] = wv[j] && kb + 2 * u < KT ? __builtin_nontemporal_load(wq[j] + static_cast<size_t>(kb / 2 + u) * 64)
                                               : u32x4{0u, 0u, 0u, 0u};
    } else {
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int u = 0; u < KC; ++u)
          b.f[j][u] = wv[j] && kb + u < KT ? load_frag_stream(wp[j] + static_cast<size_t>(kb + u) * kTile)
                                           : Frag<T>::zero();
    }
  };
  auto compute = [&](int c, int bb, const B& b) {
    const int kb = c * KC;
    if constexpr (W8) {
#pragma unroll
      for (int u = 0; u < KC / 2; ++u) {
        if (kb + 2 * u < KT) {
          Frag<T> b0[NTW], b1[NTW];
#pragma unroll
          for (int j = 0; j < NTW; ++j) e4m3x16_to_frags(b.r[j][u], b0[j], b1[j]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            Frag<T> a0, a1;
            a0.v = frag_a(bb, mt, 2 * u);
            a1.v = frag_a(bb, mt, 2 * u + 1);
#pragma unroll
            for (int j = 0; j < NTW; ++j) {
              acc[j][mt] = mma8(acc[j][mt], a0, b0[j]);
              acc[j][mt] = mma8(acc[j][mt], a1, b1[j]);
            }
          }
        }
      }
    } else {
      // Fragment f = u MT + mt. LDS reads run kLook fragments ahead of the
      // MFMAs that consume them, so their latency hides behind the MFMAs of
      // the fragments before (at large MT one wave per SIMD leaves nothing
      // else to hide it).
      constexpr int kNF = KC * MT;
      constexpr int kLook = 4;
      const int nu = KT - kb < KC ? KT - kb : KC;  // k-tiles of this chunk that exist
      auto frag_at = [&](int f) { return frag_a(bb, f % MT, f / MT); };
      Frag<T> ring[kLook];
#pragma unroll
      for (int f = 0; f < kLook && f < kNF; ++f) ring[f].v = frag_at(f);
#pragma unroll
      for (int f = 0; f < kNF; ++f) {
        const int u = f / MT, mt = f % MT;
        const Frag<T> a = ring[f % kLook];
        if (f + kLook < kNF) ring[f % kLook].v = frag_at(f + kLook);
        if (u < nu) {
#pragma unroll
          for (int j = 0; j < NTW; ++j) acc[j][mt] = mma8(acc[j][mt], a, b.f[j][u]);
        }
      }
    }
  };
  // One chunk: wait for its loads (the only ones outstanding), start the
  // next chunk's, then multiply. Buffer bb ^ 1 is free: every wave passed
  // this barrier only after finishing the previous chunk, which used it.
  auto step = [&](int c, int bb, const B& bcur, B& bnext) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (c + 1 < c1) {
      issue_a(c + 1, bb ^ 1);
      load_b(c + 1, bnext);
    }
    compute(c, bb, bcur);
  };

  B b0, b1;
  if (c0 < c1) {
    issue_a(c0, 0);
    load_b(c0, b0);
  }
  for (int c = c0; c < c1; c += 2) {
    step(c, 0, b0, b1);
    if (c + 1 < c1) step(c + 1, 1, b1, b0);
  }
  __syncthreads();                                 // LDS free for the caller (epilogue tile)
}

// The main loop with the weights, too, copied into LDS: activation chunks
// double-buffered as in wide_mainloop, weight chunks in a ring of
// kS = wide_stages(MT, W8) buffers filled kS - 2 chunks ahead of the chunk
// whose activations are copied. Step c copies the activations of chunk c + 1
// and then the weights of chunk c + kS - 1 (each only if that chunk is one of
// this work-group's), so when step c starts, the copies issued after chunk
// c's activations are at most the weights of chunk c + kS - 2:
// waiting until only those are outstanding (vmcnt), then a barrier, makes
// chunk c's activations and weights visible to every wave while later
// weights stay in flight. With two stages (kS = 2) the weights of chunk c
// follow its activations and the wait drains every copy. A buffer is
// refilled only after the barrier that follows the last reads of the chunk
// it held.
template <int MT, int KC, int NTW, int WV, bool W8>
__device__ __forceinline__ void wide_mainloop_staged(const GemmParams& p, int g, int c0, int c1,
                                                     bf16x8 (*s_a)[64], bf16x8 (*s_w)[64],
                                                     f32x4 (&acc)[NTW][MT]) {
  using T = bf16;
  constexpr int kS = wide_stages(MT, W8);
  constexpr int kBuf = MT * KC;                              // activation fragments per chunk
  constexpr int kWF = W8 ? KC / 2 : KC;                      // weight fragments per n-tile and chunk
  constexpr int kWSlots = WV * NTW * kWF;                    // weight fragments per stage
  constexpr int kALoads = (kBuf + WV - 1) / WV;
  constexpr int kWLoads = NTW * kWF;
  constexpr uint32_t kFragBytes = 64 * 16;
  static_assert(KC == 2, "activation blocks hold the two k-tiles of a chunk");
  static_assert(kS >= 2 && kALoads + (kS - 1) * kWLoads <= 63, "copies in flight fit the vmcnt counter");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ntw = g * WV * NTW + wave * NTW;                // first n-tile of this wave
  const int KT = p.KT;
  // This lane's 16 bytes of weight fragment (n-tile j, unit k) at
  // wbase[j] + 1 KiB k, a unit being a k-tile (bf16) or a k-tile pair (FP8
  // codes). n-tiles past NT read n-tile 0; their outputs are never stored.
  const char* wbase[NTW];
#pragma unroll
  for (int j = 0; j < NTW; ++j)
    wbase[j] = static_cast<const char*>(p.W) +
               static_cast<size_t>(ntw + j < p.NT ? ntw + j : 0) * KT * 512 * (W8 ? 1 : 2) + lane * 16;
  const int kUnits = W8 ? KT / 2 : KT;
  const uint32_t a_lds = lds_address(&s_a[0][0]), w_lds = lds_address(&s_w[0][0]);

#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Activation chunk c (one k-tile pair) into buffer bb as 2 MT blocks:
  // block 2 mt + h. Pieces of k-tiles past KT read zeros, so every chunk
  // runs all its MFMAs.
  auto issue_a = [&](int c, int bb) {
#pragma unroll
    for (int i = 0; i < kALoads; ++i) {
      const int f = wave + i * WV;
      if (kBuf % WV && f >= kBuf) break;               // uneven split: this wave's count is one lower
      lds_copy16_untracked(act_piece_src(p, lane, f >> 1, f & 1, c * KC), a_lds + (bb * kBuf + f) * kFragBytes);
    }
  };
  const int a_half = act_half(lane), a_slot0 = act_slot(lane, 0), a_slot1 = act_slot(lane, 1);
  // Weight fragments of chunk c into stage st: slot (wave NTW + j) kWF + u;
  // units past the last re-read it (finite weights, times zero activations).
  auto issue_w = [&](int c, int st) {
    const int ub = c * kWF;
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
      for (int u = 0; u < kWF; ++u) {
        const int k = ub + u < kUnits ? ub + u : kUnits - 1;
        lds_copy16_untracked(wbase[j] + static_cast<size_t>(k) * kFragBytes,
                             w_lds + (st * kWSlots + (wave * NTW + j) * kWF + u) * kFragBytes);
      }
  };
  // MFMAs of a chunk (activation buffer bb, weight stage st), k-tile-major:
  // activation fragment f = u MT + mt times the B fragments of k-tile u
  // (FP8: converted from their pair's codes first). LDS reads run kLook
  // fragments ahead of their MFMAs; the scheduling barriers keep the compiler
  // from sinking each read back to just before its use, where with one wave
  // per SIMD nothing hides its latency.
  auto compute = [&](int bb, int st) {
    const bf16x8* wst = &s_w[st * kWSlots + wave * NTW * kWF][0];
    Frag<T> b[NTW][KC];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
      for (int u = 0; u < kWF; ++u) {
        const bf16x8 raw = wst[(j * kWF + u) * 64 + lane];
        if constexpr (W8)
          e4m3x16_to_frags(__builtin_bit_cast(u32x4, raw), b[j][2 * u], b[j][2 * u + 1]);
        else
          b[j][u].v = raw;
      }
    constexpr int kNF = KC * MT;
    constexpr int kLook = 4;
    auto frag_at = [&](int f) {
      return s_a[bb * kBuf + (f % MT) * 2 + a_half][f / MT ? a_slot1 : a_slot0];
    };
    Frag<T> ring[kLook];
#pragma unroll
    for (int f = 0; f < kLook && f < kNF; ++f) ring[f].v = frag_at(f);
#pragma unroll
    for (int f = 0; f < kNF; ++f) {
      const int u = f / MT, mt = f % MT;
      const Frag<T> a = ring[f % kLook];
      if (f + kLook < kNF) ring[f % kLook].v = frag_at(f + kLook);
#pragma unroll
      for (int j = 0; j < NTW; ++j) acc[j][mt] = mma8(acc[j][mt], a, b[j][u]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if (c0 < c1) {
#pragma unroll
    for (int i = 0; i < kS - 2; ++i)
      if (c0 + i < c1) issue_w(c0 + i, i);
    issue_a(c0, 0);
    if (c0 + kS - 2 < c1) issue_w(c0 + kS - 2, kS - 2);
    for (int c = c0; c < c1; ++c) {
      const int bb = (c - c0) & 1, st = (c - c0) % kS;
      if (kS >= 3 && c + kS - 2 < c1)
        __builtin_amdgcn_s_waitcnt(vmcnt_only(kWLoads));   // chunk c + kS - 2's weights may stay in flight
      else
        __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
      // A bare barrier: __syncthreads() would also wait for every copy in
      // flight. The clobber keeps the compiler from moving LDS accesses across.
      asm volatile("s_barrier" ::: "memory");
      if (c + 1 < c1) issue_a(c + 1, bb ^ 1);
      if (c + kS - 1 < c1) issue_w(c + kS - 1, (c + kS - 1 - c0) % kS);
      compute(bb, st);
    }
  }
  __syncthreads();                                 // LDS free for the caller (epilogue tile)
}

// Row scales of the input RMSNorm for rows mt0 * 8 .. (mt0 + NMT) * 8 - 1
// into s_rs (the caller synchronises before use); NW waves, wave w takes
// rows w, w + NW, ..., their first loads issued together.
template <int NMT, int NW>
__device__ __forceinline__ void wide_row_scales(const GemmParams& p, int mt0, float* s_rs) {
  constexpr int kR = (NMT * 8 + NW - 1) / NW;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float v[kR];
#pragma unroll
  for (int k = 0; k < kR; ++k) v[k] = norm_first(p, mt0 * 8 + wave + k * NW, lane);
#pragma unroll
  for (int k = 0; k < kR; ++k) {
    const int i = wave + k * NW;
    if (i < NMT * 8) {
      const float r = norm_finish(p, mt0 * 8 + i, lane, v[k]);
      if (lane == 0) s_rs[i] = r;
    }
  }
}

// Epilogue of norm group gs (n-tiles 8 gs .. 8 gs + 7) for M tiles mt0 ..
// mt0 + NMT - 1. ep holds their output tile in LDS as [8 n-tiles][NMT][8
// rows][16 columns] and s_rs their row scales, both visible to every thread.
template <int NMT, int EPI>
__device__ __forceinline__ void wide_epilogue_group(const GemmParams& p, int gs, int mt0, float* ep,
                                                    const float* s_rs) {
  using T = bf16;
  constexpr int kN = kNormTiles * NMT * 128;       // elements of the group
  constexpr int kB = 4;                            // elements per thread whose inputs load together
  const int M = p.M, r0 = mt0 * 8, bd = blockDim.x;
  if (gs * kNormTiles >= p.NT) return;             // whole group past the last n-tile
  for (int e0 = threadIdx.x; e0 < kN; e0 += kB * bd) {
    // Loads only (every product waits for its operands, so the arithmetic
    // follows below), then each element's arithmetic and stores.
    float x[kB], x2[kB], sc[kB], sc2[kB];
    EpiIn in[kB];
    bool ok[kB];
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      const int e = e0 + b * bd;
      const int jj = e / (NMT * 128), mtl = (e >> 7) % NMT, i = (e >> 4) & 7, col = e & 15;
      const int m = r0 + mtl * 8 + i, nt = gs * kNormTiles + jj;
      ok[b] = e < kN && m < M && nt < p.NT;
      x[b] = x2[b] = 0.f;
      sc[b] = sc2[b] = 1.f;
      in[b] = EpiIn{0.f, 0.f, 0};
      if (ok[b]) {
        const bool pair = (EPI == kEpiSwiglu || EPI == kEpiQkv) && col < 8;
        x[b] = ep[e];
        if (pair) x2[b] = ep[e + 8];
        if (p.wscale) {                            // FP8 row scales (NULL for bf16 weights)
          sc[b] = p.wscale[nt * 16 + col];
          if (pair) sc2[b] = p.wscale[nt * 16 + col + 8];
        }
        in[b] = epilogue_inputs<EPI>(p, p.m0 + m, nt, col);
      }
    }
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      const int e = e0 + b * bd;
      if (e >= kN) continue;
      if (!ok[b]) {
        if (EPI == kEpiResid) ep[e] = 0.f;
        continue;
      }
      const int jj = e / (NMT * 128), mtl = (e >> 7) % NMT, i = (e >> 4) & 7, col = e & 15;
      const float rs = s_rs[mtl * 8 + i];
      const float v = x[b] * rs * sc[b];
      const float v2 = (EPI == kEpiSwiglu || EPI == kEpiQkv) && col < 8 ? x2[b] * rs * sc2[b] : 0.f;
      const float sq = epilogue_apply<T, EPI>(p, p.m0 + r0 + mtl * 8 + i, gs * kNormTiles + jj, col, v, v2, in[b]);
      if (EPI == kEpiResid) ep[e] = sq;            // only this thread reads element e here
    }
  }
  if (EPI == kEpiResid) {
    // Sums of squares of the group's 128 columns per row, in a fixed order.
    __syncthreads();
    for (int r = threadIdx.x; r < NMT * 8; r += blockDim.x) {
      const int m = r0 + r;
      if (m >= M) continue;
      const int mtl = r >> 3, i = r & 7;
      float sum = 0.f;
      for (int jj = 0; jj < kNormTiles; ++jj)
        for (int c = 0; c < 16; ++c) sum += ep[((jj * NMT + mtl) * 8 + i) * 16 + c];
      p.ss_out[static_cast<size_t>(gs) * p.Mtot + p.m0 + m] = sum;
    }
  }
}

// One work-group per column group (WV NTW n-tiles) over the whole k range,
// epilogue fused: the folded tile goes to LDS one norm group at a time.
template <int MT, int KC, int NTW, int WV, int EPI, bool W8>
__global__ __launch_bounds__(WV * 64) __attribute__((amdgpu_waves_per_eu(wide_waves_per_simd<MT, W8>())))
void gemm_wide_kernel(const GemmParams p, int chunks) {
  __shared__ bf16x8 s_a[2 * MT * KC][64];          // two chunks of activation fragments
  __shared__ bf16x8 s_w[wide_staged(MT, W8) ? wide_stages(MT, W8) * WV * NTW * (W8 ? KC / 2 : KC) : 1][64];
  // One norm group's output tile reuses the chunk buffers, dead after the
  // loop, and so do the row scales where they fit behind it.
  constexpr int kTile = kNormTiles * MT * 128;     // floats
  static_assert(kTile * sizeof(float) <= sizeof(s_a), "epilogue tile must fit the chunk buffers");
  constexpr bool kRsInA = (kTile + MT * 8) * sizeof(float) <= sizeof(s_a);
  __shared__ float s_rs_own[kRsInA ? 1 : MT * 8];
  constexpr int kGroups = WV * NTW / kNormTiles;   // norm groups per work-group
  constexpr int kWavesPerGroup = WV / kGroups;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  f32x4 acc[NTW][MT];
  if constexpr (wide_staged(MT, W8))
    wide_mainloop_staged<MT, KC, NTW, WV, W8>(p, blockIdx.x, 0, chunks, s_a, s_w, acc);
  else
    wide_mainloop<MT, KC, NTW, WV, W8>(p, blockIdx.x, 0, chunks, s_a, acc);
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) fold_lo(acc[j][mt]);
  float* ep = reinterpret_cast<float*>(&s_a[0][0]);
  float* s_rs = kRsInA ? ep + kTile : s_rs_own;
#pragma unroll
  for (int h = 0; h < kGroups; ++h) {
    if (wave / kWavesPerGroup == h && lane < 32) {
      const int jw = (wave % kWavesPerGroup) * NTW;
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            ep[(((jw + j) * MT + mt) * 8 + (lane >> 4) * 4 + r) * 16 + (lane & 15)] = acc[j][mt][r];
    }
    if (h == 0) wide_row_scales<MT, WV>(p, 0, s_rs);   // after the first dump: fewer live registers
    __syncthreads();
    wide_epilogue_group<MT, EPI>(p, blockIdx.x * kGroups + h, 0, ep, s_rs);
    if (h + 1 < kGroups) __syncthreads();          // ep is rewritten for the next group
  }
}

// Split s of column group g (work-group s + g S): chunks [s C / S, (s+1) C / S)
// into the partial buffer. Work-group b runs on XCD b % 8, so with the split
// index fastest every XCD streams the activations of one split (S dividing 8;
// two or three splits for S = 3, 6) and its L2 holds that slice for all the
// column groups it runs, instead of every split's slice.
template <int MT, int KC, int NTW, int WV, bool W8>
__global__ __launch_bounds__(WV * 64) __attribute__((amdgpu_waves_per_eu(wide_waves_per_simd<MT, W8>())))
void gemm_wide_split_kernel(const GemmParams p, int S, int chunks) {
  __shared__ bf16x8 s_a[2 * MT * KC][64];
  __shared__ bf16x8 s_w[wide_staged(MT, W8) ? wide_stages(MT, W8) * WV * NTW * (W8 ? KC / 2 : KC) : 1][64];
  const int G = (p.NT + WV * NTW - 1) / (WV * NTW);
  const int s = blockIdx.x % S, g = blockIdx.x / S;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c0 = static_cast<int>(static_cast<long>(s) * chunks / S);
  const int c1 = static_cast<int>(static_cast<long>(s + 1) * chunks / S);
  f32x4 acc[NTW][MT];
  if constexpr (wide_staged(MT, W8))
    wide_mainloop_staged<MT, KC, NTW, WV, W8>(p, g, c0, c1, s_a, s_w, acc);
  else
    wide_mainloop<MT, KC, NTW, WV, W8>(p, g, c0, c1, s_a, acc);
  // Fold and store one tile at a time (folding every tile first would keep
  // all the shuffled copies live at once).
  float* mine = p.part + ((static_cast<size_t>(s) * G + g) * WV + wave) * wide_part_floats<MT, NTW>() + lane * 4;
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      fold_lo(acc[j][mt]);
      if (lane < 32) *reinterpret_cast<f32x4*>(mine + (j * MT + mt) * 128) = acc[j][mt];
      __builtin_amdgcn_sched_barrier(0);
    }
}

// Sum of the S partials of norm group gs = blockIdx.x, M tile mt =
// blockIdx.y, in split order, then the epilogue of that tile. Thread t sums
// lane t % 32 of n-tile 8 gs + t / 32, which column group (8 gs + t / 32) /
// (WV NTW) of the split kernel holds in wave ((8 gs + t / 32) % (WV NTW)) / NTW:
// one coalesced 16 B load per split.
template <int MT, int NTW, int WV, int EPI>
__global__ __launch_bounds__(kNormTiles * 32) void gemm_wide_reduce_kernel(const GemmParams p, int S) {
  __shared__ float ep[kNormTiles * 128];
  __shared__ float s_rs[8];
  constexpr int kNg = WV * NTW;
  const int G = (p.NT + kNg - 1) / kNg;
  const int gs = blockIdx.x, mt = blockIdx.y;
  const int t = threadIdx.x, jj = t >> 5, ln = t & 31;
  const int nt = gs * kNormTiles + jj, g = nt / kNg, wave = (nt % kNg) / NTW, j = nt % NTW;
  const float* src = p.part + (static_cast<size_t>(g) * WV + wave) * wide_part_floats<MT, NTW>() +
                     ((j * MT + mt) * 32 + ln) * 4;
  const size_t split = static_cast<size_t>(G) * WV * wide_part_floats<MT, NTW>();
  // Every split's load in flight at once (a loop over S would wait for each),
  // and the row scales' loads beside them; the sum stays in split order.
  // (Splits past S re-read the last one's slot, an L1 hit, so no load sits
  // behind a branch.)
  f32x4 part[kMaxSplits];
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s) part[s] = *reinterpret_cast<const f32x4*>(src + min(s, S - 1) * split);
  wide_row_scales<1, kNormTiles * 32 / 64>(p, mt, s_rs);   // the block's waves
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s)
    if (s < S) acc += part[s];
#pragma unroll
  for (int r = 0; r < 4; ++r) ep[(jj * 8 + (ln >> 4) * 4 + r) * 16 + (ln & 15)] = acc[r];
  __syncthreads();
  wide_epilogue_group<1, EPI>(p, gs, mt, ep, s_rs);
}

// ---------------------------------------------------------------------------
// Launch planning.
// ---------------------------------------------------------------------------
template <int MT, bool W8, int KC = wide_kc(MT, W8), int NTW = wide_ntw(MT, W8), int WV = wide_waves(MT, W8)>
static hipError_t wide_launch(const GemmParams& p, const WidePlan& w, hipStream_t st) {
  const dim3 block(WV * 64), rblock(kNormTiles * 32);
  if (w.NTW != NTW || w.KC != KC || w.WV != WV || w.w8 != W8) return hipErrorInvalidValue;
  if (w.S > 1) {
    hipLaunchKernelGGL((gemm_wide_split_kernel<MT, KC, NTW, WV, W8>), dim3(w.G * w.S), block, 0, st, p, w.S, w.chunks);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 rgrid(wide_groups(p.NT), MT);
    switch (p.epi) {
      case kEpiStore: hipLaunchKernelGGL((gemm_wide_reduce_kernel<MT, NTW, WV, kEpiStore>), rgrid, rblock, 0, st, p, w.S); break;
      case kEpiGelu: hipLaunchKernelGGL((gemm_wide_reduce_kernel<MT, NTW, WV, kEpiGelu>), rgrid, rblock, 0, st, p, w.S); break;
      case kEpiSwiglu: hipLaunchKernelGGL((gemm_wide_reduce_kernel<MT, NTW, WV, kEpiSwiglu>), rgrid, rblock, 0, st, p, w.S); break;
      case kEpiResid: hipLaunchKernelGGL((gemm_wide_reduce_kernel<MT, NTW, WV, kEpiResid>), rgrid, rblock, 0, st, p, w.S); break;
      default: hipLaunchKernelGGL((gemm_wide_reduce_kernel<MT, NTW, WV, kEpiQkv>), rgrid, rblock, 0, st, p, w.S); break;
    }
    return hipGetLastError();
  }
  const dim3 grid(w.G);
  switch (p.epi) {
    case kEpiStore: hipLaunchKernelGGL((gemm_wide_kernel<MT, KC, NTW, WV, kEpiStore, W8>), grid, block, 0, st, p, w.chunks); break;
    case kEpiGelu: hipLaunchKernelGGL((gemm_wide_kernel<MT, KC, NTW, WV, kEpiGelu, W8>), grid, block, 0, st, p, w.chunks); break;
    case kEpiSwiglu: hipLaunchKernelGGL((gemm_wide_kernel<MT, KC, NTW, WV, kEpiSwiglu, W8>), grid, block, 0, st, p, w.chunks); break;
    case kEpiResid: hipLaunchKernelGGL((gemm_wide_kernel<MT, KC, NTW, WV, kEpiResid, W8>), grid, block, 0, st, p, w.chunks); break;
    default: hipLaunchKernelGGL((gemm_wide_kernel<MT, KC, NTW, WV, kEpiQkv, W8>), grid, block, 0, st, p, w.chunks); break;
  }
  return hipGetLastError();
}

template <bool W8>
static hipError_t wide_dispatch(const GemmParams& p, const WidePlan& w, hipStream_t st) {
  switch (w.MT) {
    case 2: return wide_launch<2, W8>(p, w, st);
    case 3: return wide_launch<3, W8>(p, w, st);
    case 4: return wide_launch<4, W8>(p, w, st);
    case 5: return wide_launch<5, W8>(p, w, st);
    case 6: return wide_launch<6, W8>(p, w, st);
    case 8: return wide_launch<8, W8>(p, w, st);
    case 10: return wide_launch<10, W8>(p, w, st);
    case 12: return wide_launch<12, W8>(p, w, st);
    case 14: return wide_launch<14, W8>(p, w, st);
    case 16: return wide_launch<16, W8>(p, w, st);
    case 18: return wide_launch<18, W8>(p, w, st);
    default: return wide_launch<20, W8>(p, w, st);
  }
}

hipError_t launch_gemm_wide(const GemmParams& p, const WidePlan& w, hipStream_t st) {
  if ((w.S > 1 && !p.part) || w.S > kMaxSplits) return hipErrorInvalidValue;
  if (w.w8 != (p.wscale != nullptr) || (w.w8 && p.KT % 2)) return hipErrorInvalidValue;
  return w.w8 ? wide_dispatch<true>(p, w, st) : wide_dispatch<false>(p, w, st);
}

}  // namespace sps
