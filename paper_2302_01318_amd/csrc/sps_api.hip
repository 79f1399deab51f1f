// C ABI of libsps: argument validation, buffer layouts and launch sequencing.
// Every entry point validates on the host before touching HIP.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/sps.h"
#include "launch.h"

// Sticky device error bits (SPS_DEV_*), one copy per device.
__device__ int sps_dev_err;

// Workspace of sps_verify_step_noalloc: a file-scope device array, one copy
// per device, held until the process ends. Host code reaches it only through
// the device address hipGetSymbolAddress returns (the array's name in host
// code is a host-side stand-in, not a device address).
constexpr size_t kNoAllocScratchBytes = static_cast<size_t>(64) << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

using sps::GemmParams;
using sps::Layout;
using sps::WsLayout;
using sps::act_dtype;
using sps::check_sampling;
using sps::kMaxK;
using sps::kMaxRows;
using sps::kMaxTokensPerSeq;
using sps::make_layout;
using sps::make_ws;
using sps::valid_config;

int* device_error_ptr() {
  static int* ptrs[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  if (!ptrs[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(sps_dev_err)) != hipSuccess) return nullptr;
    ptrs[dev] = static_cast<int*>(p);
  }
  return ptrs[dev];
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Device address of this device's `scratch`, looked up once per device (with
// that device current) on its first use.
char* scratch_ptr() {
  static char* ptrs[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  if (!ptrs[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    ptrs[dev] = static_cast<char*>(p);
  }
  return ptrs[dev];
}

}  // namespace

struct sps_model_s {
  sps_config cfg;
  Layout L;
  char* base;
};

struct sps_kv_s {
  sps_config cfg;
  Layout L;
  int B, T_cap;
  char* buf;
  int32_t* lengths;
  size_t plane_bytes;  // one of K or V for one layer: B * H * T_cap * DH elements
};

namespace {

char* layer_ptr(const sps_model_s* m, int l, size_t off) {
  return m->base + m->L.layer0 + m->L.layer_stride * l + off;
}
// Row scales of a projection of layer l (FP8 models), else NULL.
const float* scale_ptr(const sps_model_s* m, int l, size_t off) {
  return m->L.fp8 ? reinterpret_cast<const float*>(layer_ptr(m, l, off)) : nullptr;
}
void* kv_k(const sps_kv_s* kv, int l) { return kv->buf + kv->plane_bytes * (2 * static_cast<size_t>(l)); }
void* kv_v(const sps_kv_s* kv, int l) { return kv->buf + kv->plane_bytes * (2 * static_cast<size_t>(l) + 1); }

#define SPS_HIP(expr)                                 \
  do {                                                \
    if ((expr) != hipSuccess) return SPS_E_HIP;       \
  } while (0)

// Optional timing of every GEMM launch with HIP events on the launch stream
// (sps_profile_gemm_begin / _end): the benchmark's live measurement of the
// weight-streaming kernel.
struct GemmProfile {
  bool on = false;
  int repeats = 1;              // back-to-back launches per bracket (amortises the event latency)
  std::vector<hipEvent_t> ev;   // start, stop pairs
  std::vector<double> bytes;    // algorithmic bytes per launch
  size_t used = 0;
};
GemmProfile g_prof;

// Y = X W^T over p.Mtot rows (several launches when they exceed one launch's
// rows). Fields M and m0 of p are set per launch.
sps_status gemm(int dtype, GemmParams p, hipStream_t st) {
  const int cap = sps::gemm_max_rows(dtype);
  for (int m0 = 0; m0 < p.Mtot; m0 += cap) {
    p.m0 = m0;
    p.M = std::min(cap, p.Mtot - m0);
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (g_prof.on) {
      if (g_prof.used + 2 > g_prof.ev.size()) {
        for (int i = 0; i < 2; ++i) {
          hipEvent_t e;
          SPS_HIP(hipEventCreate(&e));
          g_prof.ev.push_back(e);
        }
      }
      e0 = g_prof.ev[g_prof.used];
      e1 = g_prof.ev[g_prof.used + 1];
      g_prof.used += 2;
      const double wes = dtype == SPS_DTYPE_FP8 ? 1.0 : dtype == SPS_DTYPE_BF16 ? 2.0 : 4.0;
      const double rows_w = p.epi == sps::kEpiSwiglu ? 2.0 * p.n_valid : static_cast<double>(p.n_valid);
      const double scale_bytes = dtype == SPS_DTYPE_FP8 ? 4.0 * rows_w : 0.0;
      g_prof.bytes.push_back(rows_w * p.KT * 32 * wes + scale_bytes + 4.0 * p.M * p.KT * 32 + 4.0 * p.M * p.n_valid);
      SPS_HIP(hipEventRecord(e0, st));
    }
    // Repeats redo the launch's work (a residual epilogue adds its output
    // again), so a profiled forward is for timing only.
    const int reps = g_prof.on ? g_prof.repeats : 1;
    for (int r = 0; r < reps; ++r) SPS_HIP(sps::launch_gemm(dtype, p, st));
    if (e1) SPS_HIP(hipEventRecord(e1, st));
  }
  return SPS_OK;
}

// The decoder forward (Conditional Scoring section) over Mps new tokens per
// sequence at positions lengths[b] + pos_offset + j. Per layer: QKV GEMM
// (input RMSNorm scale, rotary encoding, KV append), attention, W_O GEMM
// (residual add, next norm's input), W_1 GEMM (norm scale, GELU / SwiGLU),
// W_2 GEMM (residual add, next norm's input).
sps_status forward_impl(const sps_model_s* m, const sps_kv_s* kv, const int32_t* tokens, int tok_stride, int B,
                        int Mps, int pos_offset, float* logits, char* ws_base, const WsLayout& ws, int* err,
                        hipStream_t st) {
  const Layout& L = m->L;
  const int dt = m->cfg.dtype;             // GEMM dtype (weight format)
  const int adt = act_dtype(m->cfg);       // activations, embedding, KV cache
  const int M = B * Mps;
  float* h = reinterpret_cast<float*>(ws_base + ws.h);
  void* x = ws_base + ws.x;
  void* o = ws_base + ws.o;
  void* q = ws_base + ws.q;
  float* apart = reinterpret_cast<float*>(ws_base + ws.apart);
  void* act = ws_base + ws.act;
  float* ss_cur = reinterpret_cast<float*>(ws_base + ws.ss_a);
  float* ss_nxt = reinterpret_cast<float*>(ws_base + ws.ss_b);
  const size_t uplane = static_cast<size_t>(M) * L.d;    // lo planes of the activation format
  const size_t oplane = static_cast<size_t>(M) * L.HD;
  const size_t aplane = static_cast<size_t>(M) * L.F;
  const int KTd = L.d / 32, KThd = L.HD / 32, KTf = L.F / 32;
  const float inv_d = 1.0f / static_cast<float>(L.d);

  GemmParams base{};
  base.Mtot = M;
  base.inv_d = inv_d;
  base.eps = m->cfg.rms_eps;
  base.part = reinterpret_cast<float*>(ws_base + ws.gpart);

  float2* rope = reinterpret_cast<float2*>(ws_base + ws.rope);
  SPS_HIP(sps::launch_embed(adt, tokens, tok_stride, Mps, M, m->base + L.embed, L.V, L.d,
                            reinterpret_cast<const float*>(layer_ptr(m, 0, L.l_attn_norm)), h, x, uplane, ss_cur,
                            kv->lengths, pos_offset, L.DH, m->cfg.rope_base, rope, err, st));
  int ng = 1;
  for (int l = 0; l < L.L; ++l) {
    GemmParams p = base;                     // QKV: norm scale, rotary encoding, KV append
    p.X = x; p.ldx = L.d; p.xplane = uplane;
    p.W = layer_ptr(m, l, L.l_qkv); p.NT = 3 * L.HD / 16; p.KT = KTd; p.n_valid = 3 * L.HD;
    p.wscale = scale_ptr(m, l, L.l_qkv_sc);
    p.ss_in = ss_cur; p.ng_in = ng;
    p.lengths = kv->lengths; p.pos_offset = pos_offset; p.Mps = Mps; p.H = L.H; p.DH = L.DH;
    p.T_cap = kv->T_cap; p.q = q; p.kc = kv_k(kv, l); p.vc = kv_v(kv, l);
    p.rope = rope;
    p.err = err; p.epi = sps::kEpiQkv;
    sps_status s = gemm(dt, p, st);
    if (s != SPS_OK) return s;

    SPS_HIP(sps::launch_attention(adt, q, kv_k(kv, l), kv_v(kv, l), kv->lengths, pos_offset, B, Mps, L.H, L.DH,
                                  kv->T_cap, apart, o, oplane, st));

    p = base;                                // W_O: residual add, input of the FFN norm
    p.X = o; p.ldx = L.HD; p.xplane = oplane;
    p.W = layer_ptr(m, l, L.l_o); p.NT = L.d / 16; p.KT = KThd; p.n_valid = L.d;
    p.wscale = scale_ptr(m, l, L.l_o_sc);
    p.h = h; p.gain = reinterpret_cast<const float*>(layer_ptr(m, l, L.l_ffn_norm));
    p.u = x; p.ldu = L.d; p.uplane = uplane; p.ss_out = ss_nxt; p.epi = sps::kEpiResid;
    s = gemm(dt, p, st);
    if (s != SPS_OK) return s;
    const int ng_o = sps::gemm_groups(dt, L.d / 16, KThd, M);

    p = base;                                // W_1: norm scale, GELU / SwiGLU
    p.X = x; p.ldx = L.d; p.xplane = uplane;
    p.W = layer_ptr(m, l, L.l_w1); p.NT = L.N1 / 16; p.KT = KTd; p.n_valid = L.F;
    p.wscale = scale_ptr(m, l, L.l_w1_sc);
    p.ss_in = ss_nxt; p.ng_in = ng_o;
    p.act = act; p.lda = L.F; p.aplane = aplane;
    p.epi = L.swiglu ? sps::kEpiSwiglu : sps::kEpiGelu;
    s = gemm(dt, p, st);
    if (s != SPS_OK) return s;

    p = base;                                // W_2: residual add, input of the next norm
    p.X = act; p.ldx = L.F; p.xplane = aplane;
    p.W = layer_ptr(m, l, L.l_w2); p.NT = L.d / 16; p.KT = KTf; p.n_valid = L.d;
    p.wscale = scale_ptr(m, l, L.l_w2_sc);
    p.h = h;
    p.gain = l + 1 < L.L ? reinterpret_cast<const float*>(layer_ptr(m, l + 1, L.l_attn_norm))
                         : reinterpret_cast<const float*>(m->base + L.final_norm);
    p.u = x; p.ldu = L.d; p.uplane = uplane; p.ss_out = ss_cur; p.epi = sps::kEpiResid;
    s = gemm(dt, p, st);
    if (s != SPS_OK) return s;
    ng = sps::gemm_groups(dt, L.d / 16, KTf, M);
  }
  if (logits) {
    GemmParams p = base;                     // final norm scale + unembedding
    p.X = x; p.ldx = L.d; p.xplane = uplane;
    p.W = m->base + L.unembed; p.NT = L.NU / 16; p.KT = KTd; p.n_valid = L.V;
    p.wscale = L.fp8 ? reinterpret_cast<const float*>(m->base + L.unembed_sc) : nullptr;
    p.ss_in = ss_cur; p.ng_in = ng;
    p.out = logits; p.ldo = L.V; p.epi = sps::kEpiStore;
    sps_status s = gemm(dt, p, st);
    if (s != SPS_OK) return s;
  }
  return SPS_OK;
}

sps_status check_forward_args(const sps_model_s* m, const sps_kv_s* kv, int B, int Mps, size_t ws_bytes,
                              const void* ws, WsLayout* out) {
  if (!m || !kv || !ws) return SPS_E_INVALID;
  if (B < 1 || Mps < 1) return SPS_E_INVALID;
  if (Mps > kMaxTokensPerSeq || B * Mps > kMaxRows) return SPS_E_SHAPE;
  if (B != kv->B) return SPS_E_SHAPE;
  const sps_config& a = m->cfg;
  const sps_config& b = kv->cfg;
  if (a.n_layers != b.n_layers || a.n_heads != b.n_heads || a.head_dim != b.head_dim ||
      act_dtype(a) != act_dtype(b))
    return SPS_E_SHAPE;
  *out = make_ws(m->L, B, Mps, kv->T_cap);
  if (ws_bytes < out->total) return SPS_E_CAPACITY;
  return SPS_OK;
}

}  // namespace

extern "C" {

const char* sps_status_string(int32_t status) {
  switch (status) {
    case SPS_OK: return "ok";
    case SPS_E_INVALID: return "invalid argument";
    case SPS_E_SHAPE: return "unsupported shape";
    case SPS_E_CAPACITY: return "buffer too small";
    case SPS_E_UNSUPPORTED: return "unsupported request";
    case SPS_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t sps_abi_version(void) { return 3; }

size_t sps_weight_bytes(const sps_config* cfg) { return valid_config(cfg) ? make_layout(cfg).total : 0; }

sps_status sps_pack_weight(const sps_config* cfg, int32_t tensor, int32_t layer, const void* src, void* packed,
                           void* stream) {
  if (!valid_config(cfg)) return SPS_E_SHAPE;
  if (!src || !packed) return SPS_E_INVALID;
  const Layout L = make_layout(cfg);
  const bool per_layer = tensor >= SPS_W_ATTN_NORM;
  if (tensor < SPS_W_EMBED || tensor > SPS_W_2) return SPS_E_INVALID;
  if (per_layer && (layer < 0 || layer >= L.L)) return SPS_E_INVALID;
  if (tensor == SPS_W_3 && !L.swiglu) return SPS_E_INVALID;
  char* base = static_cast<char*>(packed);
  char* lp = base + L.layer0 + L.layer_stride * (per_layer ? layer : 0);
  const hipStream_t st = as_stream(stream);
  const int dt = cfg->dtype;
  const size_t es = L.es;
  // One projection: canonical rows src [n_src][Kd] to packed rows (see
  // launch_pack); FP8 models quantise bf16 rows and write the row scales at
  // `sc`. Rows [zf, zt) are padding.
  auto pack = [&](int n_src, int Kd, char* dst, char* sc, int kind, int row_off, int dh, int zf, int zt) {
    return L.fp8 ? sps::launch_pack_fp8(src, n_src, Kd, dst, reinterpret_cast<float*>(sc), Kd / 32, kind, row_off,
                                        dh, zf, zt, st)
                 : sps::launch_pack(dt, src, n_src, Kd, dst, Kd / 32, kind, row_off, dh, zf, zt, st);
  };
  switch (tensor) {
    case SPS_W_EMBED:
      SPS_HIP(hipMemcpyAsync(base + L.embed, src, static_cast<size_t>(L.V) * L.d * es, hipMemcpyDeviceToDevice, st));
      return SPS_OK;
    case SPS_W_FINAL_NORM:
      SPS_HIP(hipMemcpyAsync(base + L.final_norm, src, static_cast<size_t>(L.d) * 4, hipMemcpyDeviceToDevice, st));
      return SPS_OK;
    case SPS_W_ATTN_NORM:
      SPS_HIP(hipMemcpyAsync(lp + L.l_attn_norm, src, static_cast<size_t>(L.d) * 4, hipMemcpyDeviceToDevice, st));
      return SPS_OK;
    case SPS_W_FFN_NORM:
      SPS_HIP(hipMemcpyAsync(lp + L.l_ffn_norm, src, static_cast<size_t>(L.d) * 4, hipMemcpyDeviceToDevice, st));
      return SPS_OK;
    case SPS_W_UNEMBED:
      SPS_HIP(pack(L.V, L.d, base + L.unembed, base + L.unembed_sc, 0, 0, 0, L.V, L.NU));
      return SPS_OK;
    case SPS_W_Q:   // rotary partners side by side (kind 2)
    case SPS_W_K:
      SPS_HIP(pack(L.HD, L.d, lp + L.l_qkv, lp + L.l_qkv_sc, 2, (tensor - SPS_W_Q) * L.HD, L.DH, 0, 0));
      return SPS_OK;
    case SPS_W_V:
      SPS_HIP(pack(L.HD, L.d, lp + L.l_qkv, lp + L.l_qkv_sc, 0, 2 * L.HD, 0, 0, 0));
      return SPS_OK;
    case SPS_W_O:
      SPS_HIP(pack(L.d, L.HD, lp + L.l_o, lp + L.l_o_sc, 0, 0, 0, 0, 0));
      return SPS_OK;
    case SPS_W_1:
      SPS_HIP(pack(L.F, L.d, lp + L.l_w1, lp + L.l_w1_sc, L.swiglu ? 1 : 0, 0, 0, 0, 0));
      return SPS_OK;
    case SPS_W_3:
      SPS_HIP(pack(L.F, L.d, lp + L.l_w1, lp + L.l_w1_sc, 1, 1, 0, 0, 0));
      return SPS_OK;
    case SPS_W_2:
      SPS_HIP(pack(L.d, L.F, lp + L.l_w2, lp + L.l_w2_sc, 0, 0, 0, 0, 0));
      return SPS_OK;
    default:
      return SPS_E_INVALID;
  }
}

sps_status sps_weight_slot(const sps_config* cfg, int32_t tensor, int32_t layer, size_t* offset, size_t* bytes,
                           size_t* scale_offset) {
  if (!offset || !bytes || !scale_offset) return SPS_E_INVALID;
  if (!valid_config(cfg)) return SPS_E_SHAPE;
  const Layout L = make_layout(cfg);
  const bool per_layer = tensor >= SPS_W_ATTN_NORM;
  if (tensor < SPS_W_EMBED || tensor > SPS_W_2) return SPS_E_INVALID;
  if (per_layer && (layer < 0 || layer >= L.L)) return SPS_E_INVALID;
  if (tensor == SPS_W_3 && !L.swiglu) return SPS_E_INVALID;
  const size_t lbase = L.layer0 + L.layer_stride * (per_layer ? layer : 0);
  const size_t wes = L.wes;
  size_t off = 0, n = 0, sc = 0;
  switch (tensor) {
    case SPS_W_EMBED: off = L.embed; n = static_cast<size_t>(L.V) * L.d * L.es; break;
    case SPS_W_FINAL_NORM: off = L.final_norm; n = static_cast<size_t>(L.d) * 4; break;
    case SPS_W_UNEMBED: off = L.unembed; n = static_cast<size_t>(L.NU) * L.d * wes; sc = L.unembed_sc; break;
    case SPS_W_ATTN_NORM: off = lbase + L.l_attn_norm; n = static_cast<size_t>(L.d) * 4; break;
    case SPS_W_FFN_NORM: off = lbase + L.l_ffn_norm; n = static_cast<size_t>(L.d) * 4; break;
    case SPS_W_Q:
    case SPS_W_K:
    case SPS_W_V:
      off = lbase + L.l_qkv; n = static_cast<size_t>(3) * L.HD * L.d * wes; sc = lbase + L.l_qkv_sc; break;
    case SPS_W_O: off = lbase + L.l_o; n = static_cast<size_t>(L.d) * L.HD * wes; sc = lbase + L.l_o_sc; break;
    case SPS_W_1:
    case SPS_W_3:
      off = lbase + L.l_w1; n = static_cast<size_t>(L.N1) * L.d * wes; sc = lbase + L.l_w1_sc; break;
    default: off = lbase + L.l_w2; n = static_cast<size_t>(L.d) * L.F * wes; sc = lbase + L.l_w2_sc; break;
  }
  *offset = off;
  *bytes = n;
  *scale_offset = L.fp8 ? sc : 0;
  return SPS_OK;
}

sps_status sps_model_create(const sps_config* cfg, void* packed, sps_model_t* out) {
  if (!out) return SPS_E_INVALID;
  *out = nullptr;
  if (!valid_config(cfg)) return SPS_E_SHAPE;
  if (!packed) return SPS_E_INVALID;
  sps_model_s* m = new (std::nothrow) sps_model_s;
  if (!m) return SPS_E_CAPACITY;
  m->cfg = *cfg;
  m->L = make_layout(cfg);
  m->base = static_cast<char*>(packed);
  *out = m;
  return SPS_OK;
}

void sps_model_destroy(sps_model_t model) { delete model; }

size_t sps_kv_bytes(const sps_config* cfg, int32_t B, int32_t T_cap) {
  if (!valid_config(cfg) || B < 1 || T_cap < 32 || T_cap % 32 || T_cap > sps::kMaxTCap) return 0;
  const Layout L = make_layout(cfg);
  return static_cast<size_t>(L.L) * 2 * B * L.H * static_cast<size_t>(T_cap) * L.DH * L.es;
}

sps_status sps_kv_create(const sps_config* cfg, int32_t B, int32_t T_cap, void* kv_buf, int32_t* lengths,
                         sps_kv_t* out) {
  if (!out) return SPS_E_INVALID;
  *out = nullptr;
  if (!valid_config(cfg)) return SPS_E_SHAPE;
  if (!kv_buf || !lengths || B < 1) return SPS_E_INVALID;
  if (T_cap < 32 || T_cap % 32 || T_cap > sps::kMaxTCap) return SPS_E_SHAPE;
  sps_kv_s* kv = new (std::nothrow) sps_kv_s;
  if (!kv) return SPS_E_CAPACITY;
  kv->cfg = *cfg;
  kv->L = make_layout(cfg);
  kv->B = B;
  kv->T_cap = T_cap;
  kv->buf = static_cast<char*>(kv_buf);
  kv->lengths = lengths;
  kv->plane_bytes = static_cast<size_t>(B) * kv->L.H * T_cap * kv->L.DH * kv->L.es;
  *out = kv;
  return SPS_OK;
}

void sps_kv_destroy(sps_kv_t kv) { delete kv; }

static sps_status kv_copy(sps_kv_t kv, int32_t layer, int32_t b, int32_t pos0, int32_t n, void* k, void* v,
                          int to_cache, void* stream) {
  if (!kv || !k || !v) return SPS_E_INVALID;
  if (layer < 0 || layer >= kv->L.L || b < 0 || b >= kv->B || pos0 < 0 || n < 0) return SPS_E_INVALID;
  if (pos0 + n > kv->T_cap) return SPS_E_CAPACITY;
  const size_t seq = static_cast<size_t>(b) * kv->L.H * kv->T_cap * kv->L.DH * kv->L.es;
  char* kc = static_cast<char*>(kv_k(kv, layer)) + seq;
  char* vc = static_cast<char*>(kv_v(kv, layer)) + seq;
  SPS_HIP(sps::launch_kv_copy(act_dtype(kv->cfg), to_cache, kc, vc, kv->L.H, kv->L.DH, kv->T_cap, pos0, n, k, v,
                              as_stream(stream)));
  return SPS_OK;
}

sps_status sps_kv_write(sps_kv_t kv, int32_t layer, int32_t b, int32_t pos0, int32_t n, const void* k_src,
                        const void* v_src, void* stream) {
  return kv_copy(kv, layer, b, pos0, n, const_cast<void*>(k_src), const_cast<void*>(v_src), 1, stream);
}

sps_status sps_kv_read(sps_kv_t kv, int32_t layer, int32_t b, int32_t pos0, int32_t n, void* k_dst, void* v_dst,
                       void* stream) {
  return kv_copy(kv, layer, b, pos0, n, k_dst, v_dst, 0, stream);
}

size_t sps_workspace_bytes(const sps_config* cfg, int32_t B, int32_t max_tokens_per_seq, int32_t T_cap) {
  return sps::workspace_bytes(cfg, B, max_tokens_per_seq, T_cap);
}

sps_status sps_forward(sps_model_t model, sps_kv_t kv, const int32_t* tokens, int32_t tok_stride, int32_t B,
                       int32_t M, int32_t pos_offset, float* logits_out, void* workspace, size_t ws_bytes,
                       void* stream) {
  WsLayout ws;
  sps_status s = check_forward_args(model, kv, B, M, ws_bytes, workspace, &ws);
  if (s != SPS_OK) return s;
  if (!tokens || tok_stride < M) return SPS_E_INVALID;
  int* err = device_error_ptr();
  if (!err) return SPS_E_HIP;
  return forward_impl(model, kv, tokens, tok_stride, B, M, pos_offset, logits_out, static_cast<char*>(workspace),
                      ws, err, as_stream(stream));
}

}  // extern "C"

namespace {

// The verify step on a workspace `base` of ws_bytes bytes (validated here).
sps_status verify_impl(sps_model_t target, sps_kv_t kv, const int32_t* tokens, int32_t B, int32_t K,
                       sps_sampling sampling, float* logits_out, float* q_out, const sps_accept_io* acc,
                       char* base, size_t ws_bytes, void* stream) {
  if (K < 0 || K > kMaxK) return SPS_E_INVALID;
  if (!target) return SPS_E_INVALID;
  sps_status s = check_sampling(sampling, target->cfg.vocab);
  if (s != SPS_OK) return s;
  WsLayout ws;
  s = check_forward_args(target, kv, B, K + 1, ws_bytes, base, &ws);
  if (s != SPS_OK) return s;
  if (!tokens) return SPS_E_INVALID;
  if (acc && (!acc->out_tokens || !acc->n_accepted || (K > 0 && !acc->p_draft))) return SPS_E_INVALID;
  int* err = device_error_ptr();
  if (!err) return SPS_E_HIP;
  float* logits = logits_out ? logits_out : reinterpret_cast<float*>(base + ws.logits);
  void* stats = base + ws.stats;
  const hipStream_t st = as_stream(stream);
  s = forward_impl(target, kv, tokens, K + 1, B, K + 1, 0, logits, base, ws, err, st);
  if (s != SPS_OK) return s;
  const int V = target->cfg.vocab;
  SPS_HIP(sps::launch_row_softmax(logits, B * (K + 1), V, sampling.temperature, sampling.top_k, sampling.top_p,
                                  stats, q_out, base + ws.cut, err, st));
  if (acc)
    SPS_HIP(sps::launch_accept_logits(acc->p_draft, logits, stats, sampling.temperature, tokens, acc->uniforms,
                                      acc->rng.seed, acc->rng.loop, B, K, V, acc->out_tokens, acc->n_accepted,
                                      base + ws.cut, err, st));
  return SPS_OK;
}

}  // namespace

extern "C" {

sps_status sps_verify_step(sps_model_t target, sps_kv_t kv, const int32_t* tokens, int32_t B, int32_t K,
                           sps_sampling sampling, float* logits_out, float* q_out, const sps_accept_io* acc,
                           void* workspace, size_t ws_bytes, void* stream) {
  return verify_impl(target, kv, tokens, B, K, sampling, logits_out, q_out, acc, static_cast<char*>(workspace),
                     ws_bytes, stream);
}

sps_status sps_verify_step_noalloc(sps_model_t target, sps_kv_t kv, const int32_t* tokens, int32_t B, int32_t K,
                                   sps_sampling sampling, float* logits_out, float* q_out, const sps_accept_io* acc,
                                   void* stream) {
  // The size check comes first, so a call past the limit touches nothing.
  if (!target || !kv || B < 1 || K < 0 || K > kMaxK) return SPS_E_INVALID;
  if (K + 1 > kMaxTokensPerSeq || B * (K + 1) > kMaxRows) return SPS_E_SHAPE;
  if (make_ws(target->L, B, K + 1, kv->T_cap).total > kNoAllocScratchBytes) return SPS_E_CAPACITY;
  char* base = scratch_ptr();
  if (!base) return SPS_E_HIP;
  return verify_impl(target, kv, tokens, B, K, sampling, logits_out, q_out, acc, base, kNoAllocScratchBytes,
                     stream);
}

sps_status sps_accept_resample(const float* p_draft, const float* q_target, const int32_t* draft_tokens,
                               const float* uniforms, sps_philox rng, int32_t B, int32_t K, int32_t V,
                               int32_t* out_tokens, int32_t* n_accepted, void* stream) {
  if (B < 1 || K < 0 || K > kMaxK || V < 2 || V >= (1 << 24)) return SPS_E_INVALID;
  if (!q_target || !out_tokens || !n_accepted) return SPS_E_INVALID;
  if (K > 0 && (!p_draft || !draft_tokens)) return SPS_E_INVALID;
  int* err = device_error_ptr();
  if (!err) return SPS_E_HIP;
  SPS_HIP(sps::launch_accept_probs(p_draft, q_target, draft_tokens, uniforms, rng.seed, rng.loop, B, K, V,
                                   out_tokens, n_accepted, err, as_stream(stream)));
  return SPS_OK;
}

sps_status sps_draft_step(sps_model_t draft, sps_kv_t kv, const int32_t* ctx, int32_t B, int32_t K,
                          sps_sampling sampling, sps_philox rng, int32_t* tokens, float* p_out, void* workspace,
                          size_t ws_bytes, void* stream) {
  if (K < 0 || K > kMaxK) return SPS_E_INVALID;
  if (!draft || !ctx || !tokens || (K > 0 && !p_out)) return SPS_E_INVALID;
  sps_status s = check_sampling(sampling, draft->cfg.vocab);
  if (s != SPS_OK) return s;
  WsLayout ws;
  s = check_forward_args(draft, kv, B, 2, ws_bytes, workspace, &ws);
  if (s != SPS_OK) return s;
  int* err = device_error_ptr();
  if (!err) return SPS_E_HIP;
  const hipStream_t st = as_stream(stream);
  if (K == 0) {
    SPS_HIP(sps::launch_ctx_tokens(ctx, B, K, tokens, st));
    return SPS_OK;
  }
  char* base = static_cast<char*>(workspace);
  float* logits = reinterpret_cast<float*>(base + ws.logits);
  const int V = draft->cfg.vocab;
  for (int t = 0; t < K; ++t) {
    if (t == 0)
      s = forward_impl(draft, kv, ctx, 2, B, 2, -1, logits, base, ws, err, st);
    else
      s = forward_impl(draft, kv, tokens + t, K + 1, B, 1, t, logits, base, ws, err, st);
    if (s != SPS_OK) return s;
    SPS_HIP(sps::launch_draft_sample(logits, t == 0 ? 2 : 1, B, V, sampling.temperature, sampling.top_k,
                                     sampling.top_p, p_out, K, t, tokens, ctx, rng.seed, rng.loop, base + ws.stats,
                                     base + ws.cut, err, st));
  }
  return SPS_OK;
}

sps_status sps_commit(sps_kv_t kv, const int32_t* tokens, const int32_t* out_tokens, const int32_t* n_accepted,
                      int32_t B, int32_t K, int32_t* ctx, int32_t* seq_out, int32_t* n_out, int32_t cap,
                      void* stream) {
  if (!kv || !tokens || !out_tokens || !n_accepted || !ctx) return SPS_E_INVALID;
  if (B != kv->B || K < 0 || K > kMaxK) return SPS_E_INVALID;
  if ((seq_out == nullptr) != (n_out == nullptr)) return SPS_E_INVALID;
  if (seq_out && cap < 1) return SPS_E_INVALID;
  SPS_HIP(sps::launch_commit(kv->lengths, tokens, out_tokens, n_accepted, B, K, ctx, seq_out, n_out, cap,
                             as_stream(stream)));
  return SPS_OK;
}

sps_status sps_philox_uniforms(sps_philox rng, int32_t purpose, int32_t B, int32_t n, float* out, void* stream) {
  if (!out || B < 0 || n < 0 || purpose < 0) return SPS_E_INVALID;
  SPS_HIP(sps::launch_philox(rng.seed, rng.loop, purpose, B, n, out, as_stream(stream)));
  return SPS_OK;
}

sps_status sps_softmax(const float* logits, int32_t rows, int32_t V, sps_sampling sampling, float* probs,
                       void* stream) {
  if (!logits || !probs || rows < 0 || V < 2 || V >= (1 << 24)) return SPS_E_INVALID;
  const sps_status s = check_sampling(sampling, V);
  if (s != SPS_OK) return s;
  int* err = device_error_ptr();
  if (!err) return SPS_E_HIP;
  SPS_HIP(sps::launch_row_softmax(logits, rows, V, sampling.temperature, sampling.top_k, sampling.top_p, nullptr,
                                  probs, nullptr, err, as_stream(stream)));
  return SPS_OK;
}

sps_status sps_profile_gemm_begin(int32_t repeats) {
  if (repeats < 1 || repeats > 64) return SPS_E_INVALID;
  g_prof.on = true;
  g_prof.repeats = repeats;
  g_prof.used = 0;
  g_prof.bytes.clear();
  return SPS_OK;
}

sps_status sps_profile_gemm_end(float* total_ms, int32_t* launches, double* bytes) {
  if (!total_ms || !launches || !bytes) return SPS_E_INVALID;
  g_prof.on = false;
  double ms = 0.0;
  for (size_t i = 0; i + 1 < g_prof.used; i += 2) {
    SPS_HIP(hipEventSynchronize(g_prof.ev[i + 1]));
    float t = 0.f;
    SPS_HIP(hipEventElapsedTime(&t, g_prof.ev[i], g_prof.ev[i + 1]));
    ms += t;
  }
  double b = 0.0;
  for (double x : g_prof.bytes) b += x;
  *total_ms = static_cast<float>(ms / g_prof.repeats);
  *launches = static_cast<int32_t>(g_prof.used / 2);
  *bytes = b;
  g_prof.used = 0;
  g_prof.bytes.clear();
  return SPS_OK;
}

sps_status sps_fp8_decode(const uint8_t* codes, int32_t n, float* out, void* stream) {
  if (!codes || !out || n < 0 || n % 16 != 0 || reinterpret_cast<uintptr_t>(codes) % 16 != 0) return SPS_E_INVALID;
  SPS_HIP(sps::launch_fp8_decode(codes, n, out, as_stream(stream)));
  return SPS_OK;
}

sps_status sps_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  if (!src || !sink || bytes == 0 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(src) % 16 != 0)
    return SPS_E_INVALID;
  SPS_HIP(sps::launch_stream_read(src, bytes / 16, sink, as_stream(stream)));
  return SPS_OK;
}

sps_status sps_device_error(void* stream, int32_t clear, int32_t* flags) {
  if (!flags) return SPS_E_INVALID;
  SPS_HIP(hipStreamSynchronize(as_stream(stream)));
  int v = 0;
  SPS_HIP(hipMemcpyFromSymbol(&v, HIP_SYMBOL(sps_dev_err), sizeof(int), 0, hipMemcpyDeviceToHost));
  *flags = v;
  if (clear) {
    const int zero = 0;
    SPS_HIP(hipMemcpyToSymbol(HIP_SYMBOL(sps_dev_err), &zero, sizeof(int), 0, hipMemcpyHostToDevice));
  }
  return SPS_OK;
}

}  // extern "C"
