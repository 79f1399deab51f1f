// Host-side planning of libsps: packed-weight and workspace layouts and the
// launch plans of the GEMMs (see plan.h). No HIP dependency.
#include "plan.h"

#include <algorithm>
#include <cstring>

namespace sps {

namespace {
size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }
}  // namespace

// ---- launch plans ------------------------------------------------------

WidePlan wide_plan(int NT, int KT, int M, bool w8) {
  WidePlan w{};
  const int mt = (M + kActRowsBf16 - 1) / kActRowsBf16;
  w.MT = kWideMT[sizeof(kWideMT) / sizeof(kWideMT[0]) - 1];
  for (int v : kWideMT)
    if (v >= mt) { w.MT = v; break; }
  w.w8 = w8;
  w.KC = wide_kc(w.MT, w8);
  w.NTW = wide_ntw(w.MT, w8);
  w.WV = wide_waves(w.MT, w8);
  w.G = (NT + w.WV * w.NTW - 1) / (w.WV * w.NTW);
  w.chunks = (KT + w.KC - 1) / w.KC;
  // Split count: the work-groups a CU holds at once (LDS of the split
  // kernel, waves per SIMD the registers allow) give the launch's slots; a
  // launch of G S work-groups runs in ceil(G S / slots) rounds of ~chunks / S
  // chunks plus a fixed cost per work-group (~8 chunks). Minimising that over
  // the measured split counts picks full last rounds: 4 splits for 192
  // column groups at one work-group per CU (768 = 3 x 256; 2 splits leave a
  // half-empty second round, 16 % slower), 2 for 250 at two per CU.
  const bool staged = wide_staged(w.MT, w8);
  const long lds = 2L * w.MT * w.KC * 1024 +
                   (staged ? static_cast<long>(wide_stages(w.MT, w8)) * w.WV * w.NTW * (w8 ? w.KC / 2 : w.KC) * 1024 : 0);
  const int by_regs = 4 * waves_per_simd(w.MT, w8) / w.WV;   // work-groups per CU the registers allow
  const int occ = std::max(1, std::min(static_cast<int>(kLdsBytes / lds), by_regs));
  const long slots = static_cast<long>(kCUs) * occ;
  long best = -1;
  w.S = 1;
  for (int S : {1, 2, 3, 4, 6, kMaxSplits}) {
    if (S > 1 && S > w.chunks / 2) break;
    const long rounds = (static_cast<long>(w.G) * S + slots - 1) / slots;
    const long cost = rounds * ((w.chunks + S - 1) / S + 8);
    if (best < 0 || cost < best) { best = cost; w.S = S; }
  }
  return w;
}

size_t wide_part_bytes(const WidePlan& w) {
  return w.S > 1 ? static_cast<size_t>(w.S) * w.G * w.WV * w.NTW * w.MT * 128 * sizeof(float) : 0;
}

int wide_groups(int NT) { return (NT + kNormTiles - 1) / kNormTiles; }

// Two output tiles per wave (half the activation loads per weight byte, 8
// waves per work-group) once the matrix is large enough (>= 512 tiles wide,
// >= ~120 MB of bf16 weights) for 256+ work-groups to stream long enough;
// smaller matrices keep one tile per wave and 16 waves.
int single_tile_ntw(int NT, int KT) {
  return (NT % 2 == 0 && NT >= 512 && static_cast<long>(NT) * KT >= 120000) ? 2 : 1;
}

// FP8 weights, one M tile (8 rows; more rows take the wide kernel). From a
// launch-shape sweep over the 70B, 7B and draft matrices at 0, 1 and 5 rows:
// from 512 n-tiles, two n-tiles per wave (each activation fragment feeds two
// MFMA pairs), 8-wave work-groups and 4 k-tiles (2 code loads of 16 B per
// lane and n-tile) per chunk; below, one n-tile, 16 waves and 8 k-tiles
// (enough work-groups for the 3072- and 4096-wide outputs). At 5 rows the
// activation fragments, read by every wave from L2, cost ~10 % of the 70B
// launches against the same launch with no activation rows.
int fp8_ntw(int NT, int) { return NT % 2 == 0 && NT >= 512 ? 2 : 1; }

// One launch covers up to 160 rows (20 M tiles of 8 bf16 rows, 10 of 16
// fp32); bf16 and FP8 weights take the wide kernel above 8 rows.
int gemm_max_rows(int dtype) { return dtype == SPS_DTYPE_F32 ? 10 * kActRowsF32 : 20 * kActRowsBf16; }

bool gemm_is_wide(int dtype, int Mtot) { return dtype != SPS_DTYPE_F32 && Mtot > kActRowsBf16; }

int gemm_groups(int dtype, int NT, int KT, int Mtot) {
  if (gemm_is_wide(dtype, Mtot)) return wide_groups(NT);
  if (dtype == SPS_DTYPE_FP8) {
    const int ntw = fp8_ntw(NT, KT);
    return (NT + ntw - 1) / ntw;
  }
  const int rows = dtype == SPS_DTYPE_BF16 ? kActRowsBf16 : kActRowsF32;
  const int ntw = (Mtot <= rows) ? single_tile_ntw(NT, KT) : 1;
  return (NT + ntw - 1) / ntw;
}

// Upper bound of partials per (sequence, head): one per wave (prefill).
int attn_partials(int T_cap) {
  return static_cast<int>((static_cast<long>(T_cap) + kAttnWavePos - 1) / kAttnWavePos);
}

int modifier_max_vocab() { return kPerLane * kSampleThreads; }

void cut_segments(int rows, int V, int* seg, int* nseg) {
  const int n = std::max(1, std::min(kMaxRowSegments, (512 + rows - 1) / rows));
  *seg = (V + n - 1) / n;
  *nseg = (V + *seg - 1) / *seg;
}

// ---- buffer layouts ----------------------------------------------------

bool valid_config(const sps_config* c) {
  if (!c) return false;
  if (c->d_model < 32 || c->d_model % 32 || c->d_model > 16384) return false;
  if (c->n_layers < 1 || c->n_layers > 4096 || c->n_heads < 1 || c->n_heads > 1024) return false;
  if (c->head_dim != 64 && c->head_dim != 128) return false;
  if ((c->n_heads * c->head_dim) % 32) return false;
  if (c->d_ff < 32 || c->d_ff % 32 || c->d_ff > (1 << 20)) return false;
  if (c->vocab < 2 || c->vocab >= (1 << 24)) return false;
  if (c->ffn_kind != SPS_FFN_GELU && c->ffn_kind != SPS_FFN_SWIGLU) return false;
  if (c->dtype != SPS_DTYPE_F32 && c->dtype != SPS_DTYPE_BF16 && c->dtype != SPS_DTYPE_FP8) return false;
  // FP8 codes are packed in 64-deep k-tile pairs: every contraction depth of
  // the forward (d_model, n_heads * head_dim, d_ff) must be a multiple of 64.
  if (c->dtype == SPS_DTYPE_FP8 && (c->d_model % 64 || (c->n_heads * c->head_dim) % 64 || c->d_ff % 64))
    return false;
  if (!(c->rms_eps > 0.f) || !(c->rope_base > 1.f)) return false;
  return true;
}

Layout make_layout(const sps_config* c) {
  Layout L{};
  L.es = c->dtype == SPS_DTYPE_F32 ? 4 : 2;
  L.fp8 = c->dtype == SPS_DTYPE_FP8;
  L.wes = L.fp8 ? 1 : L.es;
  L.d = c->d_model; L.L = c->n_layers; L.H = c->n_heads; L.DH = c->head_dim;
  L.HD = L.H * L.DH; L.F = c->d_ff; L.V = c->vocab;
  L.NU = (L.V + 15) / 16 * 16;
  L.swiglu = c->ffn_kind == SPS_FFN_SWIGLU;
  L.N1 = L.swiglu ? 2 * L.F : L.F;
  const size_t es = L.es, wes = L.wes;
  // Row scales of a projection with n packed rows (FP8 models only).
  auto scales = [&](size_t n) { return L.fp8 ? align256(n * 4) : 0; };
  size_t o = 0;
  L.embed = o; o = align256(o + static_cast<size_t>(L.V) * L.d * es);
  L.final_norm = o; o = align256(o + static_cast<size_t>(L.d) * 4);
  L.unembed = o; o = align256(o + static_cast<size_t>(L.NU) * L.d * wes);
  L.unembed_sc = o; o += scales(L.NU);
  L.layer0 = o;
  size_t lo = 0;
  L.l_attn_norm = lo; lo = align256(lo + static_cast<size_t>(L.d) * 4);
  L.l_ffn_norm = lo; lo = align256(lo + static_cast<size_t>(L.d) * 4);
  L.l_qkv = lo; lo = align256(lo + static_cast<size_t>(3) * L.HD * L.d * wes);
  L.l_qkv_sc = lo; lo += scales(static_cast<size_t>(3) * L.HD);
  L.l_o = lo; lo = align256(lo + static_cast<size_t>(L.d) * L.HD * wes);
  L.l_o_sc = lo; lo += scales(L.d);
  L.l_w1 = lo; lo = align256(lo + static_cast<size_t>(L.N1) * L.d * wes);
  L.l_w1_sc = lo; lo += scales(L.N1);
  L.l_w2 = lo; lo = align256(lo + static_cast<size_t>(L.d) * L.F * wes);
  L.l_w2_sc = lo; lo += scales(L.d);
  L.layer_stride = lo;
  L.total = L.layer0 + L.layer_stride * L.L;
  return L;
}

// The GEMMs of one forward as (n-tiles, k-tiles): QKV, W_O, W_1 (gate and
// up for SwiGLU), W_2, unembedding.
static void forward_gemms(const Layout& L, int out[5][2]) {
  const int shapes[5][2] = {{3 * L.HD / 16, L.d / 32}, {L.d / 16, L.HD / 32}, {L.N1 / 16, L.d / 32},
                            {L.d / 16, L.F / 32}, {L.NU / 16, L.d / 32}};
  std::memcpy(out, shapes, sizeof(shapes));
}

size_t forward_part_bytes(const Layout& L, int M) {
  const int dt = L.fp8 ? SPS_DTYPE_FP8 : L.es == 2 ? SPS_DTYPE_BF16 : SPS_DTYPE_F32;   // GEMM dtype
  if (M < 1 || !gemm_is_wide(dt, M)) return 0;
  int g[5][2];
  forward_gemms(L, g);
  // A GEMM over M rows runs as launches of gemm_max_rows rows and the
  // remainder (every launch of a forward past 8 rows is wide).
  const int cap = gemm_max_rows(dt);
  const int rows[2] = {std::min(M, cap), M % cap};
  size_t part = 0;
  for (int r : rows) {
    if (r <= 0) continue;
    for (int i = 0; i < 5; ++i) part = std::max(part, wide_part_bytes(wide_plan(g[i][0], g[i][1], r, L.fp8)));
  }
  return part;
}

size_t cut_row_bytes(int V) {
  if (V > modifier_max_vocab()) return 0;
  // histogram, 16 softmax partials (256 bytes), bucket ids
  return align256(static_cast<size_t>(kCutBuckets) * 2 * sizeof(uint64_t)) + 256 + align256(static_cast<size_t>(V) * 2);
}

WsLayout make_ws(const Layout& L, int B, int Mps, int T_cap) {
  WsLayout w{};
  const size_t M = static_cast<size_t>(B) * Mps;
  const size_t NP = static_cast<size_t>(attn_partials(T_cap));
  const size_t ng = (L.d + 15) / 16;   // column groups a residual GEMM can produce
  // Split-K partials: fewer rows can split more ways than more rows, so
  // the largest over every row count a call with up to Mps tokens per
  // sequence can run.
  size_t part = 0;
  for (int mps = 1; mps <= Mps; ++mps) part = std::max(part, forward_part_bytes(L, B * mps));
  size_t o = 0;
  w.h = o; o = align256(o + M * L.d * 4);                 // residual stream (fp32)
  w.x = o; o = align256(o + M * L.d * 4);                 // u = h * gain (activation format)
  w.o = o; o = align256(o + M * L.HD * 4);                // attention output (activation format)
  w.q = o; o = align256(o + M * L.HD * L.es);             // rotated queries (model dtype)
  w.rope = o; o = align256(o + M * (L.DH / 2) * 8);       // rotary (cos, sin) per row and frequency
  w.apart = o; o = align256(o + static_cast<size_t>(B) * L.H * NP * Mps * (L.DH + 2) * 4);
  w.act = o; o = align256(o + M * L.F * 4);               // FFN hidden (activation format)
  w.ss_a = o; o = align256(o + ng * M * 4);               // per-group sums of squares of h
  w.ss_b = o; o = align256(o + ng * M * 4);
  w.logits = o; o = align256(o + M * L.V * 4);
  w.stats = o; o = align256(o + M * kRowStatBytes);
  w.cut = o; o = align256(o + M * cut_row_bytes(L.V));   // top-k / nucleus scratch per row
  w.gpart = o; o = align256(o + part);
  w.total = o;
  return w;
}

size_t workspace_bytes(const sps_config* cfg, int B, int max_tokens_per_seq, int T_cap) {
  if (!valid_config(cfg) || B < 1 || max_tokens_per_seq < 1 || T_cap < 32 || T_cap > kMaxTCap) return 0;
  // No call runs more tokens per sequence or more rows than this.
  if (max_tokens_per_seq > kMaxTokensPerSeq || static_cast<long>(B) * max_tokens_per_seq > kMaxRows) return 0;
  return make_ws(make_layout(cfg), B, max_tokens_per_seq, T_cap).total;
}

sps_status check_sampling(const sps_sampling& sp, int V) {
  if (!(sp.temperature >= 0.f) || sp.temperature > 1e30f) return SPS_E_INVALID;
  if (sp.top_k < 0 || !(sp.top_p >= 0.f && sp.top_p <= 1.f)) return SPS_E_INVALID;
  const bool mod = sp.temperature > 0.f && ((sp.top_k >= 1 && sp.top_k < V) || sp.top_p < 1.f);
  if (mod && V > modifier_max_vocab()) return SPS_E_UNSUPPORTED;
  return SPS_OK;
}

}  // namespace sps
