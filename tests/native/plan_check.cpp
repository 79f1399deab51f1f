// Host-only checker of libsps's planning code (csrc/plan.cpp), built with g++
// under AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_plan_host.py. It walks the model shapes the library is used with
// and every batch / token count a call admits, and checks that every buffer a
// launch writes lies inside the workspace the call was given:
//  * the regions of a workspace layout are 256-byte aligned, ordered and end
//    at its total;
//  * the split-K partials of every launch a call can make (a draft step runs
//    forwards of 2 and then 1 token per sequence within one layout; a verify
//    step K + 1; a prefill chunk any count up to its maximum) fit the
//    layout's partial region;
//  * sps_workspace_bytes covers every layout a call with fewer tokens per
//    sequence uses, and is 0 for requests no call admits (quickly: no loop
//    over the requested count);
//  * wide-GEMM plans cover their matrix; attention partials fit their region;
//  * the sampling kernels' row segments tile every row, none empty, at most
//    kMaxRowSegments per row;
//  * config validation and the packed layout do no undefined arithmetic on
//    extreme field values.
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "../../paper_2302_01318_amd/csrc/plan.h"

using namespace sps;

static int failures = 0;
#define CHECK(cond, ...)                                    \
  do {                                                      \
    if (!(cond)) {                                          \
      if (failures < 20) {                                  \
        std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
        std::fprintf(stderr, __VA_ARGS__);                  \
        std::fprintf(stderr, "\n");                         \
      }                                                     \
      ++failures;                                           \
    }                                                       \
  } while (0)

static sps_config cfg(int d, int L, int H, int DH, int F, int V, int ffn, int dt) {
  sps_config c{};
  c.d_model = d; c.n_layers = L; c.n_heads = H; c.head_dim = DH; c.d_ff = F; c.vocab = V;
  c.ffn_kind = ffn; c.dtype = dt; c.rms_eps = 1e-5f; c.rope_base = 10000.f;
  return c;
}

static void check_layout(const WsLayout& w, const char* what) {
  const size_t r[] = {w.h, w.x, w.o, w.q, w.rope, w.apart, w.act, w.ss_a, w.ss_b, w.logits, w.stats, w.cut, w.gpart,
                      w.total};
  for (size_t i = 0; i + 1 < sizeof(r) / sizeof(r[0]); ++i) {
    CHECK(r[i] % 256 == 0, "%s: region %zu not aligned", what, i);
    CHECK(r[i] <= r[i + 1], "%s: region %zu out of order", what, i);
  }
}

// Every launch of a call that runs forwards of B sequences with `mps` tokens
// each, within the layout `w` built for up to `mps_layout` tokens.
static void check_call(const Layout& L, int B, int mps, const WsLayout& w, int T_cap, const char* what) {
  const size_t part = forward_part_bytes(L, B * mps);
  CHECK(w.gpart + part <= w.total, "%s: split-K partials of B %d x %d rows (%zu B) past the workspace end",
        what, B, mps, part);
  // Attention partials: decode launches (<= 16 tokens) write one per 256
  // positions and query, prefill launches one per 64.
  const size_t per = mps <= 16 ? static_cast<size_t>((T_cap + 255) / 256) : static_cast<size_t>(attn_partials(T_cap));
  const size_t need = static_cast<size_t>(B) * L.H * per * mps * (L.DH + 2) * 4;
  CHECK(w.apart + need <= w.act, "%s: attention partials of B %d x %d overflow", what, B, mps);
  const size_t M = static_cast<size_t>(B) * mps;
  CHECK(w.x - w.h >= M * L.d * 4 && w.o - w.x >= M * L.d * 4 && w.q - w.o >= M * L.HD * 4 &&
            w.rope - w.q >= M * L.HD * L.es && w.ss_a - w.act >= M * L.F * 4 && w.stats - w.logits >= M * L.V * 4 &&
            w.cut - w.stats >= M * kRowStatBytes && w.gpart - w.cut >= M * cut_row_bytes(L.V),
        "%s: activation regions too small for B %d x %d", what, B, mps);
}

static void check_shape(const sps_config& c, const char* name) {
  CHECK(valid_config(&c), "%s: config rejected", name);
  if (!valid_config(&c)) return;
  const Layout L = make_layout(&c);
  const int T_caps[] = {64, 2112, 8256};
  for (int T_cap : T_caps) {
    for (int B = 1; B <= kMaxRows; ++B) {
      const int max_mps = std::min(kMaxTokensPerSeq, kMaxRows / B);
      for (int mps = 1; mps <= max_mps; ++mps) {
        const WsLayout w = make_ws(L, B, mps, T_cap);
        check_layout(w, name);
        const size_t bytes = workspace_bytes(&c, B, mps, T_cap);
        CHECK(bytes >= w.total, "%s: workspace_bytes(B %d, %d) below its layout", name, B, mps);
        // A call with up to mps tokens per sequence: every count below runs
        // within this layout (draft step: 2 then 1; prefill: ragged chunks).
        for (int m = 1; m <= mps; ++m) {
          check_call(L, B, m, w, T_cap, name);
          CHECK(bytes >= make_ws(L, B, m, T_cap).total, "%s: workspace_bytes(B %d, %d) below the layout of %d",
                name, B, mps, m);
        }
      }
      CHECK(workspace_bytes(&c, B, max_mps + 1, T_cap) == 0 || max_mps == kMaxTokensPerSeq,
            "%s: B %d x %d rows admitted", name, B, max_mps + 1);
    }
  }
}

static void check_wide_plans() {
  for (int w8 = 0; w8 < 2; ++w8)
    for (int NT = 1; NT <= 4096; NT = NT < 64 ? NT + 1 : NT * 5 / 4)
      for (int KT = 2; KT <= 1024; KT = KT < 16 ? KT + 2 : KT * 3 / 2 / 2 * 2)
        for (int M = kActRowsBf16 + 1; M <= kMaxRows; ++M) {
          const WidePlan p = wide_plan(NT, KT, M, w8 != 0);
          CHECK(p.MT * kActRowsBf16 >= M, "wide plan NT %d KT %d M %d: %d M tiles", NT, KT, M, p.MT);
          CHECK((p.WV == 4 || p.WV == 8) && p.G * p.WV * p.NTW >= NT, "wide plan NT %d: %d groups", NT, p.G);
          CHECK(p.chunks * p.KC >= KT && p.S >= 1 && p.S <= kMaxSplits, "wide plan KT %d: chunks %d S %d", KT, p.chunks, p.S);
          CHECK(!w8 || p.KC % 2 == 0, "FP8 plan with odd chunk");
          const size_t pb = wide_part_bytes(p);
          CHECK(p.S == 1 ? pb == 0 : pb == static_cast<size_t>(p.S) * p.G * p.WV * p.NTW * p.MT * 512,
                "wide plan part bytes");
        }
}

// Row segments of the sampling kernels: between 1 and kMaxRowSegments per
// row, none empty, together covering the row; about 512 work-groups per
// launch at most.
static void check_segments() {
  const int Vs[] = {1, 2, 7, 31, 32, 33, 1000, 1024, 4095, 12289, 32000, 32768};
  for (int rows = 1; rows <= kMaxRows; ++rows)
    for (int V : Vs) {
      int seg = 0, nseg = 0;
      cut_segments(rows, V, &seg, &nseg);
      CHECK(nseg >= 1 && nseg <= kMaxRowSegments && seg >= 1, "segments of rows %d V %d: %d x %d", rows, V, nseg, seg);
      CHECK(static_cast<long>(nseg) * seg >= V && static_cast<long>(nseg - 1) * seg < V,
            "segments of rows %d V %d do not tile the row: %d x %d", rows, V, nseg, seg);
      CHECK(static_cast<long>(nseg) * rows <= 512 + rows, "rows %d V %d: %d segments per row", rows, V, nseg);
    }
}

static void check_extremes() {
  const int vals[] = {INT_MIN, -1, 0, 1, 2, 31, 32, 64, 128, 4096, 16384, 16416, 1 << 20, (1 << 24) - 1, 1 << 24,
                      INT_MAX};
  std::mt19937 g(7);
  for (int it = 0; it < 200000; ++it) {
    sps_config c{};
    auto pick = [&]() { return vals[g() % (sizeof(vals) / sizeof(vals[0]))]; };
    c.d_model = pick(); c.n_layers = pick(); c.n_heads = pick(); c.head_dim = g() % 2 ? 64 : pick();
    c.d_ff = pick(); c.vocab = pick(); c.ffn_kind = static_cast<int>(g() % 3) - 0; c.dtype = static_cast<int>(g() % 4);
    const float f[] = {NAN, -1.f, 0.f, 1e-5f, 1.f, 10000.f, INFINITY};
    c.rms_eps = f[g() % 7]; c.rope_base = f[g() % 7];
    if (!valid_config(&c)) continue;
    const Layout L = make_layout(&c);
    // The packed size in exact arithmetic: no wrap-around of size_t.
    const long double per_layer = (3.0L * L.HD * L.d + 1.0L * L.d * L.HD + 1.0L * L.N1 * L.d + 1.0L * L.d * L.F) * L.wes;
    const long double total = per_layer * L.L + 1.0L * L.V * L.d * L.es + 1.0L * L.NU * L.d * L.wes;
    CHECK(static_cast<long double>(L.total) >= total * 0.999L, "packed layout wrapped around");
    const int B = 1 + static_cast<int>(g() % kMaxRows);
    const int mps = 1 + static_cast<int>(g() % 64);
    const int T = pick();
    (void)workspace_bytes(&c, B, mps, T);
  }
  // Requests no call admits are refused at once.
  const sps_config c = cfg(8192, 80, 64, 128, 32768, 32000, SPS_FFN_GELU, SPS_DTYPE_BF16);
  CHECK(workspace_bytes(&c, 1, INT_MAX, 2112) == 0, "huge token count admitted");
  CHECK(workspace_bytes(&c, INT_MAX, 1, 2112) == 0, "huge batch admitted");
  CHECK(workspace_bytes(&c, 1, 65, 2112) == 0, "65 tokens per sequence admitted");
  CHECK(workspace_bytes(&c, 1, 64, kMaxTCap) > 0, "largest capacity refused");
  CHECK(workspace_bytes(&c, 1, 64, kMaxTCap + 32) == 0, "capacity past the largest admitted");
  CHECK(workspace_bytes(&c, 1, 64, INT_MAX) == 0, "INT_MAX capacity admitted");
  CHECK(workspace_bytes(&c, 1, 5, 31) == 0, "capacity below 32 admitted");
  sps_sampling s{1.f, 0, 1.f};
  CHECK(check_sampling(s, 32000) == SPS_OK, "plain sampling refused");
  s.top_p = NAN;
  CHECK(check_sampling(s, 32000) == SPS_E_INVALID, "NaN nucleus admitted");
  s = sps_sampling{NAN, 0, 1.f};
  CHECK(check_sampling(s, 32000) == SPS_E_INVALID, "NaN temperature admitted");
  s = sps_sampling{1.f, 5, 1.f};
  CHECK(check_sampling(s, modifier_max_vocab() + 1) == SPS_E_UNSUPPORTED, "cut-off past its vocabulary admitted");
}

int main() {
  const int V = 32000;
  struct { sps_config c; const char* name; } shapes[] = {
      {cfg(8192, 80, 64, 128, 32768, V, SPS_FFN_GELU, SPS_DTYPE_BF16), "70b bf16"},
      {cfg(8192, 80, 64, 128, 32768, V, SPS_FFN_GELU, SPS_DTYPE_FP8), "70b fp8"},
      {cfg(3072, 24, 24, 128, 12288, V, SPS_FFN_GELU, SPS_DTYPE_BF16), "70b draft bf16"},
      {cfg(3072, 24, 24, 128, 12288, V, SPS_FFN_GELU, SPS_DTYPE_FP8), "70b draft fp8"},
      {cfg(4096, 32, 32, 128, 11008, V, SPS_FFN_SWIGLU, SPS_DTYPE_BF16), "7b bf16"},
      {cfg(4096, 32, 32, 128, 11008, V, SPS_FFN_SWIGLU, SPS_DTYPE_FP8), "7b fp8"},
      {cfg(256, 4, 4, 64, 1024, 1024, SPS_FFN_GELU, SPS_DTYPE_F32), "tiny target f32"},
      {cfg(128, 2, 2, 64, 512, 1024, SPS_FFN_GELU, SPS_DTYPE_F32), "tiny draft f32"},
      {cfg(192, 2, 3, 64, 320, 1000, SPS_FFN_SWIGLU, SPS_DTYPE_BF16), "small bf16"},
      {cfg(160, 2, 3, 64, 288, 1000, SPS_FFN_SWIGLU, SPS_DTYPE_BF16), "odd depth bf16"},
  };
  for (const auto& s : shapes) check_shape(s.c, s.name);
  check_wide_plans();
  check_segments();
  check_extremes();
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("plan check ok\n");
  return 0;
}
