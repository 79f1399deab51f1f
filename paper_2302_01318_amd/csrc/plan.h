// Host-side planning of libsps (internal; not part of the ABI): the launch
// geometry constants the kernels are compiled with, the packed-weight and
// workspace layouts, and the launch plans of the GEMMs and attention. Plain
// C++ with no HIP dependency, so that the same code is built into the
// library and into a host-only checker that runs under AddressSanitizer and
// UndefinedBehaviorSanitizer.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include "../../include/sps.h"

namespace sps {

// ---- limits of one call ------------------------------------------------
constexpr int kMaxTokensPerSeq = 64;   // new tokens per sequence in one forward
constexpr int kMaxRows = 160;          // B * tokens per sequence in one forward
constexpr int kMaxK = 63;              // lookahead
constexpr int kMaxTCap = 1 << 22;      // KV capacity (positions): keeps grid extents and partial counts far inside their ranges

// ---- GPU and kernel geometry -------------------------------------------
constexpr int kCUs = 256;              // compute units of the MI355X
constexpr long kLdsBytes = 160 * 1024; // LDS per CU

// Activation rows per 16-row MFMA tile: bf16 tiles carry 8 rows as hi and
// lo planes, fp32 tiles 16 rows.
constexpr int kActRowsBf16 = 8;
constexpr int kActRowsF32 = 16;

// Wide GEMM (bf16 activations, more than 8 rows; gemm_wide.hip).
constexpr int kNormTiles = 8;          // n-tiles per norm group (128 columns)
constexpr int kWideMT[] = {2, 3, 4, 5, 6, 8, 10, 12, 14, 16, 18, 20};   // compiled M-tile counts
constexpr int kMaxSplits = 8;          // largest k split of a wide launch (the reduction holds one load per split)

// n-tiles per wave. (With register-held weights, 4 at 14 M tiles ran the
// 70B W_1 and W_2 22-24 % faster than 2; the staged loop beats both.)
constexpr int wide_ntw(int, bool) { return 2; }

// Where the weights go through LDS too (wide_mainloop_staged): from 14 M
// tiles for bf16 weights, where one wave per SIMD with register-held weights
// has one chunk in flight, and from 8 for FP8 codes, whose register path
// keeps only 4 KiB per wave in flight. Below, the register path with two to
// three work-groups per CU is faster.
constexpr bool wide_staged(int MT, bool w8) { return MT >= (w8 ? 8 : 14); }

// Waves per work-group: 4, and 8 (two per SIMD, 16 n-tiles per group)
// from 8 M tiles with bf16 weights and wherever FP8 codes go through LDS:
// the activation copies per weight byte halve, which with the weights
// share each CU's outstanding L2 requests, and each SIMD has a second wave
// to issue while one waits. 70B steps at B = 16 against 4-wave groups: bf16
// K = 3 / 4 / 5 44.1 / 48.8 / 52.1 -> 43.4 / 48.1 / 50.3 ms, K = 6 53.9 ->
// 52.6 ms, K = 8 66.0 -> 59.6 ms; FP8 K = 6 / 8 50.9 / 58.0 -> 46.7 /
// 53.7 ms. Below 8 M tiles, where three 4-wave groups share a CU, 8-wave
// groups measured 2-12 % slower (bf16 and FP8, B = 4 and B = 16 at K <= 2).
// (4 n-tiles per wave in 4 waves instead spills its 288 accumulators from
// 18 M tiles.)
constexpr int wide_waves(int MT, bool w8) { return (w8 ? wide_staged(MT, w8) : MT >= 8) ? 8 : 4; }

// LDS weight stages of the staged loop: 4 (3 and 5 measured the same with
// 4-wave groups: the wait for a chunk's activations also waits for every
// copy issued before them, so each chunk's weights get two steps to land
// however deep the ring). The 32 KiB bf16 stages of 8-wave groups leave
// room beside the activation buffers for 3 at 14 M tiles (weights two
// steps ahead, 1.7 % faster than 2) and 2 above (the weights then land
// with the activations); 8-wave FP8 stages are 16 KiB, so 4.
constexpr int wide_stages(int MT, bool w8) {
  return w8 || wide_waves(MT, w8) == 4 ? 4 : MT == 14 ? 3 : 2;
}

// Waves per SIMD the register allocation must allow (the compiler would
// otherwise hoist every LDS fragment read of a chunk into registers): two
// for 8-wave work-groups (one group per CU), else 3 up to 6 M tiles (three
// 4-wave groups per CU) and 1 from 14 (FP8 codes below 8 M tiles are the
// only 4-wave groups past 6).
constexpr int waves_per_simd(int MT, bool w8) {
  return wide_waves(MT, w8) == 8 ? 2 : MT > 12 ? 1 : MT <= 6 ? 3 : 2;
}

// k-tiles per chunk, whole pairs (activation blocks, FP8 codes): the two
// chunk buffers (2 MT KC KiB of LDS) leave room for the work-groups a CU
// holds (three 4-wave groups up to 6 M tiles, one 8-wave group from 8;
// the staged loop also needs LDS for its weight ring) and hold a norm
// group's output tile (4 MT KiB).
constexpr int wide_kc(int MT, bool w8) { return wide_staged(MT, w8) ? 2 : MT <= 10 ? 4 : 2; }

// Decode attention: positions per wave (two 32-position blocks).
constexpr int kAttnWavePos = 64;

// Sampling kernels: threads per work-group and row entries per thread held
// in registers (the largest row the top-k / nucleus cut-off handles).
constexpr int kSampleThreads = 1024;
constexpr int kPerLane = 32;
constexpr size_t kRowStatBytes = 24;   // sizeof(RowStat), sampling.hip
constexpr int kCutBuckets = 1 + 33 * 16;   // weight buckets of the top-k / nucleus cut-off (sampling.hip)

// ---- launch plans ------------------------------------------------------
// Wide GEMM: M tiles, k-tiles per chunk, n-tiles per wave, waves per
// work-group, column groups (WV NTW n-tiles each), k splits and chunks of
// one launch.
struct WidePlan { int MT, KC, NTW, WV, G, S, chunks; bool w8; };
WidePlan wide_plan(int NT, int KT, int M, bool w8);   // w8: FP8 weight codes
size_t wide_part_bytes(const WidePlan& w);           // workspace for the split-K partials
int wide_groups(int NT);                             // norm groups (8 n-tiles each)

int single_tile_ntw(int NT, int KT);          // n-tiles per wave, bf16 / fp32 single-tile kernel
int fp8_ntw(int NT, int KT);                  // n-tiles per wave, FP8 single-tile kernel
int gemm_max_rows(int dtype);                 // rows one launch handles
bool gemm_is_wide(int dtype, int Mtot);       // bf16 / FP8 launches past one M tile
int gemm_groups(int dtype, int NT, int KT, int Mtot);   // column groups (ss_out groups) of a GEMM
int attn_partials(int T_cap);                 // attention partials per (sequence, head)
int modifier_max_vocab();                     // largest vocabulary the cut-off handles

// ---- buffer layouts ----------------------------------------------------
bool valid_config(const sps_config* c);

// Element type of the activations, the embedding and the KV cache: 0 fp32
// for fp32 models, 1 bf16 for bf16 and FP8-weight models.
inline int act_dtype(const sps_config& c) { return c.dtype == SPS_DTYPE_F32 ? 0 : 1; }

// Byte offsets of every tensor in the packed weight buffer. For FP8 models
// each projection's codes are followed by its fp32 row scales (`*_sc`).
struct Layout {
  int es, wes, d, L, H, DH, HD, F, V, NU, N1;   // es: activation / KV element bytes; wes: weight
  bool swiglu, fp8;
  size_t embed, final_norm, unembed, unembed_sc, layer0, layer_stride;
  size_t l_attn_norm, l_ffn_norm, l_qkv, l_o, l_w1, l_w2, l_qkv_sc, l_o_sc, l_w1_sc, l_w2_sc;
  size_t total;
};
Layout make_layout(const sps_config* c);   // c must be valid

// Offsets of the forward's scratch buffers within the workspace.
struct WsLayout {
  size_t h, x, o, q, rope, apart, act, ss_a, ss_b, logits, stats, cut, gpart, total;
};

// The workspace of a call that runs forwards of B sequences with any number
// of new tokens per sequence from 1 to Mps (a draft step runs 2, then 1; a
// verify step K + 1): every buffer is sized for B * Mps rows, and the
// split-K partials for the largest any of those forwards' launches writes.
WsLayout make_ws(const Layout& L, int B, int Mps, int T_cap);

// sps_workspace_bytes: 0 for an invalid request (see sps.h).
size_t workspace_bytes(const sps_config* cfg, int B, int max_tokens_per_seq, int T_cap);

// Per-row scratch of the top-k / nucleus cut-off over several CUs: the
// row's bucket histogram (counts, weights) and a bucket id per entry; 0
// where the vocabulary is past what the cut-off handles.
size_t cut_row_bytes(int V);

// Segments of a row for the sampling kernels that take one segment per
// work-group (the cut-off's histogram, the draft export): about 512
// work-groups per launch, at most kMaxRowSegments per row (the draft draw
// scans the segment totals with one wave), every segment non-empty:
// *nseg = ceil(V / *seg). rows >= 1, V >= 1.
constexpr int kMaxRowSegments = 32;
void cut_segments(int rows, int V, int* seg, int* nseg);

// Bytes of split-K partials the launches of one forward over M rows write.
size_t forward_part_bytes(const Layout& L, int M);

// Host-side check of the sampling parameters for a vocabulary of V.
sps_status check_sampling(const sps_sampling& sp, int V);

}  // namespace sps
