// C ABI of librksc: argument validation, workspace layout and the layer loop of
// the verify pass (all kernels are launched on the caller's stream; nothing is
// allocated).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/rksc.h"
#include "../../include/rksc_testing.h"
#include "api_internal.h"
#include "kernels.h"
#include "status.h"

#define RKSC_EXPORT extern "C" __attribute__((visibility("default")))

namespace rksc {

std::string& last_error() {
  thread_local std::string text;
  return text;
}

rksc_status fail(rksc_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  last_error() = buf;
  return st;
}

rksc_status ok() {
  last_error().clear();
  return RKSC_OK;
}

}  // namespace rksc

namespace {

using rksc::fail;
using rksc::ok;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

using rksc::DType;
using rksc::GemmPlan;

struct Layout {
  size_t ctrl, x0, x1, act, ffn, q, kown, vown, pbig, pres, hn_a, hn_b, parts, rope, opart, mlpart, total;
  GemmPlan qkv, o, gu, down;
  int nparts;
  rksc::AttnPlan attn;
  int max_rows;
};

rksc_status check_config(const rksc_model_config* c) {
  if (!c) return fail(RKSC_ERR_INVALID_ARGUMENT, "model config is NULL");
  if (c->n_layers < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_layers must be >= 1 (got %d)", c->n_layers);
  if (c->d_model < 8 || c->d_model % 8)
    return fail(RKSC_ERR_UNSUPPORTED, "d_model must be a positive multiple of 8 (got %d)", c->d_model);
  if (c->d_model > 16384) return fail(RKSC_ERR_UNSUPPORTED, "d_model above 16384 (got %d)", c->d_model);
  if (c->n_heads < 1 || c->n_kv_heads < 1)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "head counts must be >= 1 (got %d, %d)", c->n_heads, c->n_kv_heads);
  if (c->n_heads % c->n_kv_heads)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "n_heads %% n_kv_heads != 0 (%d, %d)", c->n_heads, c->n_kv_heads);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(RKSC_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", c->head_dim);
  if (c->d_ff < 8 || c->d_ff % 8)
    return fail(RKSC_ERR_UNSUPPORTED, "d_ff must be a positive multiple of 8 (got %d)", c->d_ff);
  if (c->vocab < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "vocab must be >= 1 (got %d)", c->vocab);
  if (!(c->rms_eps >= 0.f) || !std::isfinite(c->rms_eps))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "rms_eps must be finite and >= 0");
  if (!(c->rope_base > 0.f) || !std::isfinite(c->rope_base))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "rope_base must be finite and > 0");
  if (c->dtype != RKSC_F32 && c->dtype != RKSC_BF16)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "unknown dtype %d", c->dtype);
  return RKSC_OK;
}

// Whether a model's gate|up weight has the tiled layout of rksc_tile_gate_up.
bool gate_up_tileable(const rksc_model_config* c) {
  return c->dtype == RKSC_BF16 && c->d_model % 64 == 0 && (2 * c->d_ff) % rksc::kTileRows == 0;
}

// The optional tiled gate|up copy of a layer: only where the layout exists, 16-byte aligned.
rksc_status check_tiled(const rksc_model_config* c, const rksc_layer_weights& lw, int l) {
  if (!lw.w_gate_up_tiled) return RKSC_OK;
  if (!gate_up_tileable(c))
    return fail(RKSC_ERR_UNSUPPORTED,
                "layer %d: w_gate_up_tiled is set, but this model has no tiled gate|up layout "
                "(bf16, d_model %% 64 == 0, 2 d_ff %% 256 == 0)", l);
  if (reinterpret_cast<uintptr_t>(lw.w_gate_up_tiled) % 16)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "layer %d: w_gate_up_tiled must be 16-byte aligned", l);
  return RKSC_OK;
}

// The caches of a prefix chain in position order (root first); empty caches are
// left out. Rejects more than kMaxPrefixSegs caches (which also ends a cycle).
struct Chain {
  int nseg = 0;
  long long n = 0;
  const rksc_prefix_kv* seg[rksc::kMaxPrefixSegs] = {};
};

rksc_status collect_chain(const rksc_prefix_kv* kv, Chain* ch) {
  const rksc_prefix_kv* rev[rksc::kMaxPrefixSegs];
  int cnt = 0;
  for (const rksc_prefix_kv* p = kv; p; p = p->parent) {
    if (cnt == rksc::kMaxPrefixSegs)
      return fail(RKSC_ERR_UNSUPPORTED, "a prefix chain of more than %d caches (or a cycle)", rksc::kMaxPrefixSegs);
    if (p->n_prefix < 0) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 0 (got %d)", p->n_prefix);
    if (p->n_prefix > 0 && (!p->k || !p->v))
      return fail(RKSC_ERR_INVALID_ARGUMENT, "prefix k/v are NULL with n_prefix = %d", p->n_prefix);
    rev[cnt++] = p;
  }
  *ch = Chain{};
  for (int i = cnt - 1; i >= 0; --i) {
    if (rev[i]->n_prefix == 0) continue;
    ch->seg[ch->nseg++] = rev[i];
    ch->n += rev[i]->n_prefix;
  }
  if (ch->n > (1LL << 30)) return fail(RKSC_ERR_UNSUPPORTED, "a prefix of more than 2^30 entries");
  return RKSC_OK;
}

// Layer l of the chain for the attention kernels (each cache is [L, Hkv, n_i, hd]).
rksc::PrefixView layer_view(const Chain& ch, int l, int Hkv, int hd, size_t T) {
  rksc::PrefixView v;
  v.n = (int)ch.n;
  v.nseg = ch.nseg;
  int start = 0;
  for (int i = 0; i < ch.nseg; ++i) {
    const rksc_prefix_kv* p = ch.seg[i];
    const size_t layer = (size_t)Hkv * p->n_prefix * hd * T;
    v.start[i] = start;
    v.len[i] = p->n_prefix;
    v.k[i] = static_cast<const char*>(p->k) + (size_t)l * layer;
    v.v[i] = static_cast<const char*>(p->v) + (size_t)l * layer;
    start += p->n_prefix;
  }
  return v;
}

rksc_status make_layout(const rksc_model_config* c, int B, int s, int n_prefix, Layout* lay) {
  rksc_status st = check_config(c);
  if (st != RKSC_OK) return st;
  if (B < 1 || B > RKSC_MAX_BRANCHES)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "n_branches must be in [1, %d] (got %d)", RKSC_MAX_BRANCHES, B);
  if (s < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "branch_len must be >= 1 (got %d)", s);
  if ((long long)B * s > (1 << 20))
    return fail(RKSC_ERR_UNSUPPORTED, "n_branches * branch_len above 2^20 (got %lld)", (long long)B * s);
  const DType dt = c->dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const int d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, hd = c->head_dim, F = c->d_ff;
  const int M = B * s;
  const int Nqkv = (H + 2 * Hkv) * hd;
  lay->max_rows = M;
  lay->qkv = rksc::plan_gemm(dt, M, Nqkv, d);
  lay->o = rksc::plan_gemm(dt, M, d, H * hd);
  lay->gu = rksc::plan_gemm(dt, M, 2 * F, d);
  lay->down = rksc::plan_gemm(dt, M, d, F);
  lay->nparts = rksc::entropy_parts(dt, c->vocab, B);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  const size_t Ms = (size_t)M;
  lay->ctrl = take(sizeof(rksc::Ctrl));
  lay->x0 = take(Ms * d * 4);
  lay->x1 = take(Ms * d * 4);
  // Activations are fp32 for every model dtype.
  lay->act = take(Ms * (size_t)(d > H * hd ? d : H * hd) * 4);
  lay->ffn = take(Ms * F * 4);
  lay->q = take(Ms * H * hd * 4);
  lay->kown = take((size_t)B * Hkv * s * hd * 4);
  lay->vown = take((size_t)B * Hkv * s * hd * 4);
  const size_t pq = (size_t)lay->qkv.splits * Ms * Nqkv, pg = (size_t)lay->gu.splits * Ms * 2 * F;
  lay->pbig = take((pq > pg ? pq : pg) * 4);
  const int sres = lay->o.splits > lay->down.splits ? lay->o.splits : lay->down.splits;
  lay->pres = take((size_t)sres * Ms * d * 4);
  lay->hn_a = take((size_t)RKSC_MAX_BRANCHES * d * (dt == DType::BF16 ? 2 : 4));
  lay->hn_b = take((size_t)RKSC_MAX_BRANCHES * d * 2);
  lay->parts = take((size_t)lay->nparts * 64 * 4 * 4);   // (m, s, t[, argmax]) per column
  lay->rope = take((size_t)s * (hd / 2) * 8);
  lay->attn = rksc::plan_attention(dt, B, n_prefix, s, H, Hkv);
  const size_t nch = (size_t)lay->attn.partials;
  lay->opart = take(nch * Ms * H * hd * 4);
  lay->mlpart = take(nch * Ms * H * 2 * 4);
  lay->total = off;
  return RKSC_OK;
}

// Exit window: the lm_head-entropy stream of the probe (one read of W_lm) is
// shared by `window` consecutive layers, whose rows become extra columns of the
// same stream; the exit rule still runs layer by layer at the window's end (a
// branch's layers after its exit inside the window are computed and discarded).
// The window is chosen by a cost model. A pass of L layers pays L / w streams of
// W_lm, and an exit, whose layer is not known in advance and is taken as placed
// uniformly within its window, wastes (w - 1) / 2 computed layers on average;
// w* = sqrt(2 L c_probe / c_layer) minimises the sum. c_probe is the stream of
// W_lm at 6 TB/s (measured on MI355X: its cost barely grows with the columns);
// c_layer is the layer's projections (the larger of their weight bytes at
// 3 TB/s and their hi/lo MFMA work at half the bf16 peak), its attention at
// 0.8 PFLOP/s, and about 30 us of row kernels. w is w* rounded to a power of two
// in [1, min(8, 64 / B)] (at most 64 stream columns).
constexpr int kMaxWindow = 8;
constexpr int kAutoWindow = 0;   // verify_impl's window argument: take exit_window's
int exit_window(const rksc_model_config* c, int B, int s, int n) {
  const double d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, hd = c->head_dim, F = c->d_ff;
  const double T = c->dtype == RKSC_BF16 ? 2.0 : 4.0;
  const double P = d * (H + 2 * Hkv) * hd + H * hd * d + 3 * d * F;
  const double M = (double)B * s;
  const double c_probe = (double)c->vocab * d * T / 6e12;
  const double t_gemm = std::max(P * T / 3e12, 4.0 * M * P / 1.25e15);
  const double t_attn = 8.0 * hd * H * B * ((double)s * n + 0.5 * (double)s * s) / 0.8e15;
  const double c_layer = t_gemm + t_attn + 30e-6;
  const double w_star = std::sqrt(2.0 * c->n_layers * c_probe / c_layer);
  int w = 1;
  while (w * 2 <= kMaxWindow && w * 2 * B <= 64 && w_star >= w * 1.4142135623730951) w *= 2;
  return w;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(RKSC_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

}  // namespace

RKSC_EXPORT int32_t rksc_abi_version(void) { return RKSC_ABI_VERSION; }

RKSC_EXPORT size_t rksc_gate_up_tiled_bytes(const rksc_model_config* cfg) {
  if (check_config(cfg) != RKSC_OK) return 0;
  if (!gate_up_tileable(cfg)) {
    fail(RKSC_ERR_UNSUPPORTED, "no tiled gate|up layout for this model (bf16, d_model %% 64 == 0, 2 d_ff %% 256 == 0)");
    return 0;
  }
  return (size_t)2 * cfg->d_ff * cfg->d_model * 2;
}

// The 256-row x 64-column blocks of the gate|up weight made contiguous, in the
// order the 128-row projection kernel streams them (a storage layout of the
// FFN's gate|up weight; rksc_layer_weights.w_gate_up_tiled).
RKSC_EXPORT rksc_status rksc_tile_gate_up(const rksc_model_config* cfg, const void* w_gate_up, void* out,
                                          size_t out_bytes, void* stream) {
  const rksc_status st = check_config(cfg);
  if (st != RKSC_OK) return st;
  if (!gate_up_tileable(cfg))
    return fail(RKSC_ERR_UNSUPPORTED,
                "no tiled gate|up layout for this model (bf16, d_model %% 64 == 0, 2 d_ff %% 256 == 0)");
  if (!w_gate_up || !out) return fail(RKSC_ERR_INVALID_ARGUMENT, "w_gate_up and out must not be NULL");
  const size_t bytes = (size_t)2 * cfg->d_ff * cfg->d_model * 2;
  if (out_bytes < bytes) return fail(RKSC_ERR_INVALID_ARGUMENT, "out has %zu bytes, needs %zu", out_bytes, bytes);
  const uintptr_t a = reinterpret_cast<uintptr_t>(w_gate_up), b = reinterpret_cast<uintptr_t>(out);
  if (a % 16 || b % 16) return fail(RKSC_ERR_INVALID_ARGUMENT, "w_gate_up and out must be 16-byte aligned");
  if (a < b + bytes && b < a + bytes) return fail(RKSC_ERR_INVALID_ARGUMENT, "w_gate_up and out overlap");
  const hipError_t e = rksc::launch_tile_rows(w_gate_up, out, 2 * cfg->d_ff, cfg->d_model,
                                              static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(RKSC_ERR_HIP, "tiling launch failed: %s", hipGetErrorString(e));
  return ok();
}

RKSC_EXPORT const char* rksc_status_string(rksc_status s) {
  switch (s) {
    case RKSC_OK: return "ok";
    case RKSC_ERR_INVALID_ARGUMENT: return "invalid argument";
    case RKSC_ERR_UNSUPPORTED: return "unsupported";
    case RKSC_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case RKSC_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

RKSC_EXPORT const char* rksc_last_error(void) { return rksc::last_error().c_str(); }

RKSC_EXPORT size_t rksc_verify_workspace_size(const rksc_model_config* cfg, int32_t n_branches,
                                              int32_t branch_len, int32_t n_prefix) {
  if (n_prefix < 0) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 0 (got %d)", n_prefix);
    return 0;
  }
  Layout lay;
  if (make_layout(cfg, n_branches, branch_len, n_prefix, &lay) != RKSC_OK) return 0;
  return lay.total;
}

namespace {

// Shared body of rksc_verify_forward and rksc_verify_forward_profiled. `events`
// (may be NULL) holds RKSC_PROFILE_EVENTS_PER_LAYER events per layer.
rksc_status verify_impl(const rksc_weights* w, const rksc_prefix_kv* kv, const int32_t* branch_tokens,
                        int32_t n_branches, int32_t branch_len, float tau, int32_t patience, float* entropy,
                        int32_t* exit_layer, float* hidden_last, void* workspace, size_t workspace_bytes,
                        void* stream, void* const* events, int32_t window, uint32_t drop = 0) {
  if (!w) return fail(RKSC_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!kv) return fail(RKSC_ERR_INVALID_ARGUMENT, "prefix_kv is NULL");
  if (!branch_tokens) return fail(RKSC_ERR_INVALID_ARGUMENT, "branch_tokens is NULL");
  if (!entropy) return fail(RKSC_ERR_INVALID_ARGUMENT, "entropy is NULL");
  if (!exit_layer) return fail(RKSC_ERR_INVALID_ARGUMENT, "exit_layer is NULL");
  if (!workspace) return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  if (std::isnan(tau) || tau < 0.f) return fail(RKSC_ERR_INVALID_ARGUMENT, "tau must be >= 0 and not NaN");
  if (patience < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "patience must be >= 1 (got %d)", patience);
  if (window != kAutoWindow && (window < 1 || window > kMaxWindow || (long long)window * n_branches > 64))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "window must be in [1, %d] with window * n_branches <= 64 (got %d, %d)",
                kMaxWindow, window, n_branches);
  const rksc_model_config* c = &w->cfg;
  Chain chain;
  rksc_status st = collect_chain(kv, &chain);
  if (st != RKSC_OK) return st;
  Layout lay;
  st = make_layout(c, n_branches, branch_len, (int)chain.n, &lay);
  if (st != RKSC_OK) return st;
  if (workspace_bytes < lay.total)
    return fail(RKSC_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, needs %zu", workspace_bytes, lay.total);
  if (!w->embed || !w->final_norm || !w->lm_head || !w->layers)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "embed, final_norm, lm_head and layers must not be NULL");
  for (int l = 0; l < c->n_layers; ++l) {
    const rksc_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.w_qkv || !lw.w_o || !lw.ffn_norm || !lw.w_gate_up || !lw.w_down)
      return fail(RKSC_ERR_INVALID_ARGUMENT, "layer %d has a NULL weight pointer", l);
    if (const rksc_status e = check_tiled(c, lw, l); e != RKSC_OK) return e;
  }
  const int win = window == kAutoWindow ? exit_window(c, n_branches, branch_len, (int)chain.n) : window;

  const DType dt = c->dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const size_t T = dt == DType::BF16 ? 2 : 4;
  const int L = c->n_layers, d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, hd = c->head_dim;
  const int F = c->d_ff, V = c->vocab, B = n_branches, s = branch_len, n = (int)chain.n;
  const int M = lay.max_rows;
  const int Nqkv = (H + 2 * Hkv) * hd;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  rksc::Ctrl* ctrl = reinterpret_cast<rksc::Ctrl*>(ws + lay.ctrl);
  float* x0 = reinterpret_cast<float*>(ws + lay.x0);
  float* x1 = reinterpret_cast<float*>(ws + lay.x1);
  float* act = reinterpret_cast<float*>(ws + lay.act);
  float* ffn = reinterpret_cast<float*>(ws + lay.ffn);
  float* qb = reinterpret_cast<float*>(ws + lay.q);
  float* kown = reinterpret_cast<float*>(ws + lay.kown);
  float* vown = reinterpret_cast<float*>(ws + lay.vown);
  float* pbig = reinterpret_cast<float*>(ws + lay.pbig);
  float* pres = reinterpret_cast<float*>(ws + lay.pres);
  void* hn_a = ws + lay.hn_a;
  void* hn_b = ws + lay.hn_b;
  float* parts = reinterpret_cast<float*>(ws + lay.parts);
  float2* rope = reinterpret_cast<float2*>(ws + lay.rope);
  float* opart = reinterpret_cast<float*>(ws + lay.opart);
  float* mlpart = reinterpret_cast<float*>(ws + lay.mlpart);
  const size_t res_stride = (size_t)M * d;
  // Start of the lo plane of a BF16-model projection input of `elems` elements per plane.
  auto plane_lo = [&](float* buf, size_t elems) -> const void* {
    return dt == DType::BF16 ? static_cast<const void*>(reinterpret_cast<const uint16_t*>(buf) + elems) : nullptr;
  };
  // Precision ablation (test hook only): zero the lo plane of a projection input of
  // `elems` elements per plane, so that the projection sees the bf16 hi part alone.
  if (drop && dt != DType::BF16) return fail(RKSC_ERR_UNSUPPORTED, "the precision ablation needs a bf16 model");
  auto drop_lo = [&](float* buf, size_t elems) -> hipError_t {
    return hipMemsetAsync(reinterpret_cast<uint16_t*>(buf) + elems, 0, elems * 2, strm);
  };

  HIP_TRY(rksc::launch_init(ctrl, B, L, entropy, exit_layer, hidden_last, (size_t)L * B * d, strm));
  HIP_TRY(rksc::launch_rope_table(rope, s, n, hd, (double)c->rope_base, strm));
  HIP_TRY(rksc::launch_embed(dt, w->embed, branch_tokens, V, x0, M, d, strm));

  auto event_at = [&](int l, int slot) -> hipEvent_t {
    return events ? static_cast<hipEvent_t>(events[(size_t)l * RKSC_PROFILE_EVENTS_PER_LAYER + slot]) : nullptr;
  };
  auto mark = [&](int l, int slot) -> hipError_t {
    hipEvent_t e = event_at(l, slot);
    return e ? hipEventRecord(e, strm) : hipSuccess;
  };
  for (int l = 0; l < L; ++l) {
    const rksc_layer_weights& lw = w->layers[l];
    float* x_prev = (l % 2 == 0) ? x0 : x1;
    float* x_cur = (l % 2 == 0) ? x1 : x0;
    // Residual stream of the live rows (gathered), plus the previous layer's FFN output.
    // The live set changes only at window ends: the survivors are gathered at a window's first layer.
    // Inside a window this kernel also taps the previous layer's last-token rows.
    rksc::TapArgs tap;
    if (l % win != 0) {
      tap.gamma = w->final_norm;
      tap.hidden_last = hidden_last;
      tap.layer0 = l - 1;
      tap.B = B;
      tap.jrow = (l - 1) % win;
      tap.hn_a = hn_a;
      tap.hn_b = hn_b;
    }
    HIP_TRY(rksc::launch_add_norm(dt, x_prev, pres, l == 0 ? 0 : lay.down.splits, res_stride, l % win == 0, ctrl,
                                  s, x_cur, act, lw.attn_norm, d, c->rms_eps, M, strm, tap));
    if (drop & RKSC_DROP_QKV_LO) HIP_TRY(drop_lo(act, (size_t)M * d));
    HIP_TRY(mark(l, 0));
    // Projection inputs: bf16 planes hi = act[0, M*K), lo = act[M*K, 2*M*K) for BF16 models.
    HIP_TRY(rksc::launch_gemm(dt, lay.qkv, act, plane_lo(act, (size_t)M * d), lw.w_qkv, pbig, (size_t)M * Nqkv, ctrl,
                              s, M, Nqkv, d, strm));
    HIP_TRY(mark(l, 1));
    HIP_TRY(rksc::launch_qkv_post(pbig, lay.qkv.splits, (size_t)M * Nqkv, ctrl, s, H, Hkv, hd, rope, qb, kown,
                                  vown, M, strm));
    if (drop & RKSC_DROP_Q_LO) HIP_TRY(rksc::launch_round_bf16(qb, (size_t)M * H * hd, strm));
    if (drop & RKSC_DROP_OWN_KV_LO) {
      HIP_TRY(rksc::launch_round_bf16(kown, (size_t)B * Hkv * s * hd, strm));
      HIP_TRY(rksc::launch_round_bf16(vown, (size_t)B * Hkv * s * hd, strm));
    }
    HIP_TRY(mark(l, 2));
    HIP_TRY(rksc::launch_attention(dt, lay.attn, qb, layer_view(chain, l, Hkv, hd, T), kown, vown, act, opart,
                                   mlpart, ctrl, s, H, Hkv, hd, B, strm, !(drop & RKSC_DROP_P_LO)));
    if (drop & RKSC_DROP_O_LO) HIP_TRY(drop_lo(act, (size_t)M * H * hd));
    HIP_TRY(mark(l, 3));
    HIP_TRY(mark(l, 4));
    HIP_TRY(rksc::launch_gemm(dt, lay.o, act, plane_lo(act, (size_t)M * H * hd), lw.w_o, pres, res_stride, ctrl, s,
                              M, d, H * hd, strm));
    HIP_TRY(mark(l, 5));
    HIP_TRY(rksc::launch_add_norm(dt, x_cur, pres, lay.o.splits, res_stride, false, ctrl, s, x_cur, act,
                                  lw.ffn_norm, d, c->rms_eps, M, strm));
    if (drop & RKSC_DROP_GATE_UP_LO) HIP_TRY(drop_lo(act, (size_t)M * d));
    HIP_TRY(mark(l, 6));
    if (event_at(l, 7) && !rksc::gate_up_fused(dt, lay.gu, 2 * F)) {
      // Profiled call: the class's closing event goes between the projection kernel and
      // its separate SwiGLU / split-K combine, so the pair brackets the projection alone.
      HIP_TRY(rksc::launch_gemm(dt, lay.gu, act, plane_lo(act, (size_t)M * d), lw.w_gate_up, pbig,
                                (size_t)M * 2 * F, ctrl, s, M, 2 * F, d, strm, lw.w_gate_up_tiled));
      HIP_TRY(mark(l, 7));
      HIP_TRY(rksc::launch_swiglu_post(dt, pbig, lay.gu.splits, (size_t)M * 2 * F, ctrl, s, F, ffn, M, strm));
    } else {
      HIP_TRY(rksc::launch_gate_up_swiglu(dt, lay.gu, act, plane_lo(act, (size_t)M * d), lw.w_gate_up, pbig,
                                          (size_t)M * 2 * F, ctrl, s, M, F, d, ffn, strm, lw.w_gate_up_tiled));
      HIP_TRY(mark(l, 7));
    }
    if (drop & RKSC_DROP_DOWN_LO) HIP_TRY(drop_lo(ffn, (size_t)M * F));
    HIP_TRY(mark(l, 8));
    HIP_TRY(rksc::launch_gemm(dt, lay.down, ffn, plane_lo(ffn, (size_t)M * F), lw.w_down, pres, res_stride, ctrl, s,
                              M, d, F, strm));
    HIP_TRY(mark(l, 9));
    if (l % win == win - 1 || l == L - 1) {   // window end: one lm_head stream for its layers
      HIP_TRY(rksc::launch_tap(dt, x_cur, pres, lay.down.splits, res_stride, ctrl, s, d, B, l, hidden_last,
                               w->final_norm, c->rms_eps, hn_a, hn_b, B, strm, l % win));
      const int kw = l % win + 1, first = l + 1 - kw;
      if (drop & RKSC_DROP_LM_HEAD_LO) HIP_TRY(hipMemsetAsync(hn_b, 0, (size_t)RKSC_MAX_BRANCHES * d * 2, strm));
      HIP_TRY(mark(l, 10));
      HIP_TRY(rksc::launch_entropy(dt, w->lm_head, hn_a, hn_b, ctrl, V, d, B, parts, strm, kw));
      HIP_TRY(mark(l, 11));
      HIP_TRY(rksc::launch_finalize_exit(parts, lay.nparts, ctrl, first + 1, kw, L, B, tau, patience, entropy,
                                         exit_layer, hidden_last, d, strm));
    }
  }
  return ok();
}

}  // namespace

RKSC_EXPORT rksc_status rksc_verify_forward(const rksc_weights* w, const rksc_prefix_kv* kv,
                                            const int32_t* branch_tokens, int32_t n_branches, int32_t branch_len,
                                            float tau, int32_t patience, float* entropy, int32_t* exit_layer,
                                            float* hidden_last, void* workspace, size_t workspace_bytes,
                                            void* stream) {
  return verify_impl(w, kv, branch_tokens, n_branches, branch_len, tau, patience, entropy, exit_layer,
                     hidden_last, workspace, workspace_bytes, stream, nullptr, kAutoWindow);
}

rksc_status rksc::verify_workspace(const rksc_model_config* cfg, int32_t n_branches, int32_t branch_len,
                                   int32_t n_prefix, size_t* bytes) {
  if (n_prefix < 0) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 0 (got %d)", n_prefix);
  Layout lay;
  const rksc_status st = make_layout(cfg, n_branches, branch_len, n_prefix, &lay);
  if (st != RKSC_OK) return st;
  *bytes = lay.total;
  return RKSC_OK;
}

rksc_status rksc::verify_call(const rksc_weights* w, const rksc_prefix_kv* kv, const int32_t* branch_tokens,
                              int32_t n_branches, int32_t branch_len, float tau, int32_t patience, float* entropy,
                              int32_t* exit_layer, float* hidden_last, void* workspace, size_t workspace_bytes,
                              void* stream) {
  return verify_impl(w, kv, branch_tokens, n_branches, branch_len, tau, patience, entropy, exit_layer,
                     hidden_last, workspace, workspace_bytes, stream, nullptr, kAutoWindow);
}

RKSC_EXPORT int32_t rksc_verify_window(const rksc_model_config* cfg, int32_t n_branches, int32_t branch_len,
                                       int32_t n_prefix) {
  if (check_config(cfg) != RKSC_OK) return 0;
  if (n_branches < 1 || n_branches > RKSC_MAX_BRANCHES || branch_len < 1 || n_prefix < 0) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "bad pass shape B = %d, s = %d, n = %d", n_branches, branch_len, n_prefix);
    return 0;
  }
  return exit_window(cfg, n_branches, branch_len, n_prefix);
}

RKSC_EXPORT rksc_status rksc_test_verify_precision(const rksc_weights* w, const rksc_prefix_kv* kv,
                                                   const int32_t* branch_tokens, int32_t n_branches,
                                                   int32_t branch_len, float tau, int32_t patience, float* entropy,
                                                   int32_t* exit_layer, float* hidden_last, void* workspace,
                                                   size_t workspace_bytes, void* stream, uint32_t drop_mask) {
  if (drop_mask & ~(uint32_t)RKSC_DROP_ALL) return fail(RKSC_ERR_INVALID_ARGUMENT, "unknown drop bits 0x%x", drop_mask);
  return verify_impl(w, kv, branch_tokens, n_branches, branch_len, tau, patience, entropy, exit_layer,
                     hidden_last, workspace, workspace_bytes, stream, nullptr, kAutoWindow, drop_mask);
}

RKSC_EXPORT rksc_status rksc_verify_forward_window(const rksc_weights* w, const rksc_prefix_kv* kv,
                                                   const int32_t* branch_tokens, int32_t n_branches,
                                                   int32_t branch_len, float tau, int32_t patience, float* entropy,
                                                   int32_t* exit_layer, float* hidden_last, void* workspace,
                                                   size_t workspace_bytes, void* stream, int32_t window) {
  if (window < 1)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "window must be in [1, %d] with window * n_branches <= 64 (got %d)",
                kMaxWindow, window);
  return verify_impl(w, kv, branch_tokens, n_branches, branch_len, tau, patience, entropy, exit_layer,
                     hidden_last, workspace, workspace_bytes, stream, nullptr, window);
}

RKSC_EXPORT rksc_status rksc_verify_forward_profiled(const rksc_weights* w, const rksc_prefix_kv* kv,
                                                     const int32_t* branch_tokens, int32_t n_branches,
                                                     int32_t branch_len, float tau, int32_t patience,
                                                     float* entropy, int32_t* exit_layer, float* hidden_last,
                                                     void* workspace, size_t workspace_bytes, void* stream,
                                                     void* const* events) {
  if (!events) return fail(RKSC_ERR_INVALID_ARGUMENT, "events is NULL");
  return verify_impl(w, kv, branch_tokens, n_branches, branch_len, tau, patience, entropy, exit_layer,
                     hidden_last, workspace, workspace_bytes, stream, events, kAutoWindow);
}

RKSC_EXPORT size_t rksc_prefill_workspace_size(const rksc_model_config* cfg, int32_t n_prefix) {
  if (n_prefix < 1) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 1 (got %d)", n_prefix);
    return 0;
  }
  Layout lay;
  if (make_layout(cfg, 1, n_prefix, 0, &lay) != RKSC_OK) return 0;
  return lay.total;
}

// Root forward (Eq. prefix_fwd): the verify pass's layer sequence for one
// "branch" of n tokens over an empty prefix, causal within itself, with the
// post-RoPE keys and the values of every layer stored as the prefix cache and
// the last token's layer outputs as the root hidden states. No entropy probe.
RKSC_EXPORT rksc_status rksc_prefill(const rksc_weights* w, const int32_t* tokens, int32_t n_prefix, void* k_out,
                                     void* v_out, float* h_root, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  if (!w) return fail(RKSC_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!tokens) return fail(RKSC_ERR_INVALID_ARGUMENT, "tokens is NULL");
  if (!k_out || !v_out) return fail(RKSC_ERR_INVALID_ARGUMENT, "k_out and v_out must not be NULL");
  if (!h_root) return fail(RKSC_ERR_INVALID_ARGUMENT, "h_root is NULL");
  if (!workspace) return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  if (n_prefix < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 1 (got %d)", n_prefix);
  const rksc_model_config* c = &w->cfg;
  Layout lay;
  rksc_status st = make_layout(c, 1, n_prefix, 0, &lay);
  if (st != RKSC_OK) return st;
  if (workspace_bytes < lay.total)
    return fail(RKSC_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, needs %zu", workspace_bytes, lay.total);
  if (!w->embed || !w->final_norm || !w->layers)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "embed, final_norm and layers must not be NULL");
  for (int l = 0; l < c->n_layers; ++l) {
    const rksc_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.w_qkv || !lw.w_o || !lw.ffn_norm || !lw.w_gate_up || !lw.w_down)
      return fail(RKSC_ERR_INVALID_ARGUMENT, "layer %d has a NULL weight pointer", l);
    if (const rksc_status e = check_tiled(c, lw, l); e != RKSC_OK) return e;
  }

  const DType dt = c->dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const size_t T = dt == DType::BF16 ? 2 : 4;
  const int L = c->n_layers, d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, hd = c->head_dim;
  const int F = c->d_ff, V = c->vocab, s = n_prefix;
  const int M = lay.max_rows;
  const int Nqkv = (H + 2 * Hkv) * hd;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  rksc::Ctrl* ctrl = reinterpret_cast<rksc::Ctrl*>(ws + lay.ctrl);
  float* x0 = reinterpret_cast<float*>(ws + lay.x0);
  float* x1 = reinterpret_cast<float*>(ws + lay.x1);
  float* act = reinterpret_cast<float*>(ws + lay.act);
  float* ffn = reinterpret_cast<float*>(ws + lay.ffn);
  float* qb = reinterpret_cast<float*>(ws + lay.q);
  float* kown = reinterpret_cast<float*>(ws + lay.kown);
  float* vown = reinterpret_cast<float*>(ws + lay.vown);
  float* pbig = reinterpret_cast<float*>(ws + lay.pbig);
  float* pres = reinterpret_cast<float*>(ws + lay.pres);
  float2* rope = reinterpret_cast<float2*>(ws + lay.rope);
  float* opart = reinterpret_cast<float*>(ws + lay.opart);
  float* mlpart = reinterpret_cast<float*>(ws + lay.mlpart);
  const size_t res_stride = (size_t)M * d;
  const size_t kv_layer = (size_t)Hkv * s * hd;
  auto plane_lo = [&](float* buf, size_t elems) -> const void* {
    return dt == DType::BF16 ? static_cast<const void*>(reinterpret_cast<const uint16_t*>(buf) + elems) : nullptr;
  };

  // One live "branch": h_root takes the tap's rows (hidden_last with B = 1).
  HIP_TRY(rksc::launch_init(ctrl, 1, L, nullptr, nullptr, h_root, (size_t)L * d, strm));
  HIP_TRY(rksc::launch_rope_table(rope, s, 0, hd, (double)c->rope_base, strm));
  HIP_TRY(rksc::launch_embed(dt, w->embed, tokens, V, x0, M, d, strm));
  for (int l = 0; l < L; ++l) {
    const rksc_layer_weights& lw = w->layers[l];
    float* x_prev = (l % 2 == 0) ? x0 : x1;
    float* x_cur = (l % 2 == 0) ? x1 : x0;
    // Also taps the previous layer's last row (the root hidden state of that layer).
    rksc::TapArgs tap;
    if (l > 0) {
      tap.gamma = w->final_norm;
      tap.hidden_last = h_root;
      tap.layer0 = l - 1;
      tap.B = 1;
      tap.hn_a = ws + lay.hn_a;
      tap.hn_b = ws + lay.hn_b;
    }
    HIP_TRY(rksc::launch_add_norm(dt, x_prev, pres, l == 0 ? 0 : lay.down.splits, res_stride, false, ctrl, s,
                                  x_cur, act, lw.attn_norm, d, c->rms_eps, M, strm, tap));
    HIP_TRY(rksc::launch_gemm(dt, lay.qkv, act, plane_lo(act, (size_t)M * d), lw.w_qkv, pbig, (size_t)M * Nqkv, ctrl,
                              s, M, Nqkv, d, strm));
    // The cache layer [Hkv, n, hd] is the branch-cache layout with one slot, cap = n.
    HIP_TRY(rksc::launch_qkv_post(pbig, lay.qkv.splits, (size_t)M * Nqkv, ctrl, s, H, Hkv, hd, rope, qb, kown,
                                  vown, M, strm, dt, static_cast<char*>(k_out) + l * kv_layer * T,
                                  static_cast<char*>(v_out) + l * kv_layer * T, s, 0));
    HIP_TRY(rksc::launch_attention(dt, lay.attn, qb, rksc::PrefixView{}, kown, vown, act, opart, mlpart, ctrl, s,
                                   H, Hkv, hd, 1, strm));
    HIP_TRY(rksc::launch_gemm(dt, lay.o, act, plane_lo(act, (size_t)M * H * hd), lw.w_o, pres, res_stride, ctrl, s,
                              M, d, H * hd, strm));
    HIP_TRY(rksc::launch_add_norm(dt, x_cur, pres, lay.o.splits, res_stride, false, ctrl, s, x_cur, act,
                                  lw.ffn_norm, d, c->rms_eps, M, strm));
    HIP_TRY(rksc::launch_gate_up_swiglu(dt, lay.gu, act, plane_lo(act, (size_t)M * d), lw.w_gate_up, pbig,
                                        (size_t)M * 2 * F, ctrl, s, M, F, d, ffn, strm, lw.w_gate_up_tiled));
    HIP_TRY(rksc::launch_gemm(dt, lay.down, ffn, plane_lo(ffn, (size_t)M * F), lw.w_down, pres, res_stride, ctrl, s,
                              M, d, F, strm));
    if (l == L - 1)
      HIP_TRY(rksc::launch_tap(dt, x_cur, pres, lay.down.splits, res_stride, ctrl, s, d, 1, l, h_root,
                               w->final_norm, c->rms_eps, ws + lay.hn_a, ws + lay.hn_b, 1, strm));
  }
  HIP_TRY(rksc::launch_unit_rows(h_root, L, d, strm));
  return ok();
}

RKSC_EXPORT size_t rksc_decode_workspace_size(const rksc_model_config* cfg, int32_t n_branches, int32_t suffix_len,
                                             int32_t n_prefix) {
  if (n_prefix < 0) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 0 (got %d)", n_prefix);
    return 0;
  }
  Layout a, b;
  if (make_layout(cfg, n_branches, suffix_len, n_prefix, &a) != RKSC_OK) return 0;
  if (make_layout(cfg, n_branches, 1, n_prefix, &b) != RKSC_OK) return 0;
  return a.total > b.total ? a.total : b.total;
}

namespace {

// Outputs of a branch pass; NULL members are not produced.
struct PassOut {
  int32_t* next_token;   // with p_top and conf: the last token's argmax and top-1 probability
  float* p_top;
  float* conf;
  float* h_out;          // [L, B, d]: every layer's output row of each branch's last token
};

// One pass of B branches of s tokens through all L layers (Sec. 2.2, "KV
// broadcast and batched decode"): the tokens sit at positions
// n + pos .. n + pos + s - 1, attend to the prefix cache `kv` and causally to
// each other, and their keys and values are written as entries off..off+s-1 of
// the per-branch cache layers ck/cv [L][B, Hkv, cap, hd]. `step` (s = 1, a
// decode step, pos = off) also attends to the cached entries 0..off-1;
// otherwise those entries are not read (a tree node's cache holds its parent's
// n entries first: off = n, pos = 0). With out.next_token, the last token's logits give the
// next token and its top-1 probability, summed into conf for Eq. gen_conf
// (set when off == 0 and not a step, else accumulated).
rksc_status branch_pass(const rksc_weights* w, const rksc_prefix_kv* kv, void* ck, void* cv, int cap, int off,
                        int pos, const int32_t* tokens, int32_t n_branches, int32_t s, bool step, const PassOut& out,
                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!w) return fail(RKSC_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!kv) return fail(RKSC_ERR_INVALID_ARGUMENT, "prefix_kv is NULL");
  if (!tokens) return fail(RKSC_ERR_INVALID_ARGUMENT, "tokens is NULL");
  if (!workspace) return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  Chain chain;
  rksc_status st = collect_chain(kv, &chain);
  if (st != RKSC_OK) return st;
  if (s < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "suffix_len must be >= 1 (got %d)", s);
  if (chain.n + pos + s > (1LL << 30)) return fail(RKSC_ERR_UNSUPPORTED, "positions above 2^30");
  const rksc_model_config* c = &w->cfg;
  Layout lay;
  st = make_layout(c, n_branches, s, (int)chain.n, &lay);
  if (st != RKSC_OK) return st;
  if (workspace_bytes < lay.total)
    return fail(RKSC_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, needs %zu", workspace_bytes, lay.total);
  if (!w->embed || !w->final_norm || !w->layers || (out.next_token && !w->lm_head))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "embed, final_norm, lm_head and layers must not be NULL");
  for (int l = 0; l < c->n_layers; ++l) {
    const rksc_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.w_qkv || !lw.w_o || !lw.ffn_norm || !lw.w_gate_up || !lw.w_down)
      return fail(RKSC_ERR_INVALID_ARGUMENT, "layer %d has a NULL weight pointer", l);
    if (const rksc_status e = check_tiled(c, lw, l); e != RKSC_OK) return e;
  }

  const DType dt = c->dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const size_t T = dt == DType::BF16 ? 2 : 4;
  const int L = c->n_layers, d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, hd = c->head_dim;
  const int F = c->d_ff, V = c->vocab, B = n_branches, n = (int)chain.n, len = off;
  const int M = lay.max_rows;
  const int Nqkv = (H + 2 * Hkv) * hd;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  rksc::Ctrl* ctrl = reinterpret_cast<rksc::Ctrl*>(ws + lay.ctrl);
  float* x0 = reinterpret_cast<float*>(ws + lay.x0);
  float* x1 = reinterpret_cast<float*>(ws + lay.x1);
  float* act = reinterpret_cast<float*>(ws + lay.act);
  float* ffn = reinterpret_cast<float*>(ws + lay.ffn);
  float* qb = reinterpret_cast<float*>(ws + lay.q);
  float* kown = reinterpret_cast<float*>(ws + lay.kown);
  float* vown = reinterpret_cast<float*>(ws + lay.vown);
  float* pbig = reinterpret_cast<float*>(ws + lay.pbig);
  float* pres = reinterpret_cast<float*>(ws + lay.pres);
  float* parts = reinterpret_cast<float*>(ws + lay.parts);
  float2* rope = reinterpret_cast<float2*>(ws + lay.rope);
  float* opart = reinterpret_cast<float*>(ws + lay.opart);
  float* mlpart = reinterpret_cast<float*>(ws + lay.mlpart);
  const size_t res_stride = (size_t)M * d;
  const size_t bkv_layer = (size_t)B * Hkv * cap * hd * T;
  auto plane_lo = [&](float* buf, size_t elems) -> const void* {
    return dt == DType::BF16 ? static_cast<const void*>(reinterpret_cast<const uint16_t*>(buf) + elems) : nullptr;
  };

  HIP_TRY(rksc::launch_init(ctrl, B, L, nullptr, nullptr, out.h_out, (size_t)L * B * d, strm));
  HIP_TRY(rksc::launch_rope_table(rope, s, n + pos, hd, (double)c->rope_base, strm));
  HIP_TRY(rksc::launch_embed(dt, w->embed, tokens, V, x0, M, d, strm));
  for (int l = 0; l < L; ++l) {
    const rksc_layer_weights& lw = w->layers[l];
    float* x_prev = (l % 2 == 0) ? x0 : x1;
    float* x_cur = (l % 2 == 0) ? x1 : x0;
    // With h_out, also taps the previous layer's last rows.
    rksc::TapArgs tap;
    if (l > 0 && out.h_out) {
      tap.gamma = w->final_norm;
      tap.hidden_last = out.h_out;
      tap.layer0 = l - 1;
      tap.B = B;
      tap.hn_a = ws + lay.hn_a;
      tap.hn_b = ws + lay.hn_b;
    }
    HIP_TRY(rksc::launch_add_norm(dt, x_prev, pres, l == 0 ? 0 : lay.down.splits, res_stride, false, ctrl, s,
                                  x_cur, act, lw.attn_norm, d, c->rms_eps, M, strm, tap));
    HIP_TRY(rksc::launch_gemm(dt, lay.qkv, act, plane_lo(act, (size_t)M * d), lw.w_qkv, pbig, (size_t)M * Nqkv, ctrl,
                              s, M, Nqkv, d, strm));
    char* bk = static_cast<char*>(ck) + l * bkv_layer;
    char* bv = static_cast<char*>(cv) + l * bkv_layer;
    HIP_TRY(rksc::launch_qkv_post(pbig, lay.qkv.splits, (size_t)M * Nqkv, ctrl, s, H, Hkv, hd, rope, qb, kown,
                                  vown, M, strm, dt, bk, bv, cap, len));
    const rksc::PrefixView pre = layer_view(chain, l, Hkv, hd, T);
    if (step)
      HIP_TRY(rksc::launch_attention_decode(dt, lay.attn, qb, pre, bk, bv, len, cap, kown, vown, act, opart,
                                            mlpart, ctrl, H, Hkv, hd, B, strm));
    else
      HIP_TRY(rksc::launch_attention(dt, lay.attn, qb, pre, kown, vown, act, opart, mlpart, ctrl, s, H, Hkv, hd, B,
                                     strm));
    HIP_TRY(rksc::launch_gemm(dt, lay.o, act, plane_lo(act, (size_t)M * H * hd), lw.w_o, pres, res_stride, ctrl, s,
                              M, d, H * hd, strm));
    HIP_TRY(rksc::launch_add_norm(dt, x_cur, pres, lay.o.splits, res_stride, false, ctrl, s, x_cur, act,
                                  lw.ffn_norm, d, c->rms_eps, M, strm));
    HIP_TRY(rksc::launch_gate_up_swiglu(dt, lay.gu, act, plane_lo(act, (size_t)M * d), lw.w_gate_up, pbig,
                                        (size_t)M * 2 * F, ctrl, s, M, F, d, ffn, strm, lw.w_gate_up_tiled));
    HIP_TRY(rksc::launch_gemm(dt, lay.down, ffn, plane_lo(ffn, (size_t)M * F), lw.w_down, pres, res_stride, ctrl, s,
                              M, d, F, strm));
    if (l == L - 1 && (out.h_out || out.next_token))
      HIP_TRY(rksc::launch_tap(dt, x_cur, pres, lay.down.splits, res_stride, ctrl, s, d, B, l, out.h_out,
                               w->final_norm, c->rms_eps, ws + lay.hn_a, ws + lay.hn_b, B, strm));
  }
  if (out.next_token) {
    HIP_TRY(rksc::launch_entropy_argmax(dt, w->lm_head, ws + lay.hn_a, ws + lay.hn_b, ctrl, V, d, B, parts, strm));
    HIP_TRY(rksc::launch_finalize_decode(parts, lay.nparts, B, out.next_token, out.p_top, out.conf,
                                         step || off > 0 ? 1 : 0, strm));
  }
  return ok();
}

rksc_status decode_impl(const rksc_weights* w, const rksc_prefix_kv* kv, rksc_branch_kv* bkv, const int32_t* tokens,
                        int32_t n_branches, int32_t s, bool step, int32_t* next_token, float* p_top, float* conf,
                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!bkv) return fail(RKSC_ERR_INVALID_ARGUMENT, "branch_kv is NULL");
  if (!bkv->k || !bkv->v) return fail(RKSC_ERR_INVALID_ARGUMENT, "branch_kv k/v are NULL");
  if (!next_token || !p_top || !conf)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "next_token, p_top and conf must not be NULL");
  if (bkv->length < 0) return fail(RKSC_ERR_INVALID_ARGUMENT, "branch_kv length must be >= 0 (got %d)", bkv->length);
  if (!step && bkv->length != 0)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "the suffix needs an empty branch cache (length %d)", bkv->length);
  if (s >= 1 && (long long)bkv->length + s > bkv->capacity)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "branch cache full: length %d + %d > capacity %d", bkv->length, s,
                bkv->capacity);
  const rksc_status st = branch_pass(w, kv, bkv->k, bkv->v, bkv->capacity, bkv->length, bkv->length, tokens,
                                     n_branches, s, step,
                                     PassOut{next_token, p_top, conf, nullptr}, workspace, workspace_bytes, stream);
  if (st == RKSC_OK) bkv->length += s;
  return st;
}

}  // namespace

RKSC_EXPORT rksc_status rksc_decode_suffix(const rksc_weights* w, const rksc_prefix_kv* kv, rksc_branch_kv* branch_kv,
                                           const int32_t* suffix_tokens, int32_t n_branches, int32_t suffix_len,
                                           int32_t* next_token, float* p_top, float* conf, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  return decode_impl(w, kv, branch_kv, suffix_tokens, n_branches, suffix_len, false, next_token, p_top, conf,
                     workspace, workspace_bytes, stream);
}

RKSC_EXPORT rksc_status rksc_decode_step(const rksc_weights* w, const rksc_prefix_kv* kv, rksc_branch_kv* branch_kv,
                                         const int32_t* tokens, int32_t n_branches, int32_t* next_token, float* p_top,
                                         float* conf, void* workspace, size_t workspace_bytes, void* stream) {
  return decode_impl(w, kv, branch_kv, tokens, n_branches, 1, true, next_token, p_top, conf, workspace,
                     workspace_bytes, stream);
}

RKSC_EXPORT size_t rksc_prefix_extend_workspace_size(const rksc_model_config* cfg, int32_t n_parent,
                                                    int32_t n_new) {
  if (n_parent < 0) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "n_parent must be >= 0 (got %d)", n_parent);
    return 0;
  }
  Layout lay;
  if (make_layout(cfg, 1, n_new, n_parent, &lay) != RKSC_OK) return 0;
  return lay.total;
}

// Tree sharing (Sec. 2.2; the paper shares a search-tree node's step among its
// children): the node's m tokens are run once over its ancestors' caches (the
// parent chain, read in place) and the node's own cache [L, Hkv, m, hd] receives
// their keys and values. Children read the chain root .. parent, node as their
// prefix (rksc_prefix_kv.parent); nothing of the parent is copied.
RKSC_EXPORT rksc_status rksc_prefix_extend(const rksc_weights* w, const rksc_prefix_kv* parent, const int32_t* tokens,
                                           int32_t n_new, void* k_out, void* v_out, float* h_node, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  if (!w) return fail(RKSC_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!parent) return fail(RKSC_ERR_INVALID_ARGUMENT, "parent is NULL");
  if (!k_out || !v_out) return fail(RKSC_ERR_INVALID_ARGUMENT, "k_out and v_out must not be NULL");
  if (n_new < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_new must be >= 1 (got %d)", n_new);
  const rksc_model_config* c = &w->cfg;
  rksc_status st = check_config(c);
  if (st != RKSC_OK) return st;
  Chain chain;
  st = collect_chain(parent, &chain);
  if (st != RKSC_OK) return st;
  if (chain.nseg == rksc::kMaxPrefixSegs)
    return fail(RKSC_ERR_UNSUPPORTED, "the node's children would read more than %d caches", rksc::kMaxPrefixSegs);
  if (chain.n + n_new > (1LL << 30)) return fail(RKSC_ERR_UNSUPPORTED, "positions above 2^30");
  const size_t T = c->dtype == RKSC_BF16 ? 2 : 4;
  const size_t per_entry = (size_t)c->n_layers * c->n_kv_heads * c->head_dim * T;
  const size_t child = per_entry * n_new;
  // The new entries are written while every cache of the chain is read: no overlap.
  auto overlap = [](const void* a, size_t na, const void* b, size_t nb) {
    const char *pa = static_cast<const char*>(a), *pb = static_cast<const char*>(b);
    return pa < pb + nb && pb < pa + na;
  };
  if (overlap(k_out, child, v_out, child)) return fail(RKSC_ERR_INVALID_ARGUMENT, "k_out overlaps v_out");
  for (int i = 0; i < chain.nseg; ++i) {
    const size_t par = per_entry * chain.seg[i]->n_prefix;
    const void* pk = chain.seg[i]->k;
    const void* pv = chain.seg[i]->v;
    if (overlap(pk, par, k_out, child) || overlap(pv, par, v_out, child) || overlap(pk, par, v_out, child) ||
        overlap(pv, par, k_out, child))
      return fail(RKSC_ERR_INVALID_ARGUMENT, "a parent cache overlaps the node's cache");
  }
  Layout lay;
  st = make_layout(c, 1, n_new, (int)chain.n, &lay);
  if (st != RKSC_OK) return st;
  if (workspace && workspace_bytes < lay.total)
    return fail(RKSC_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, needs %zu", workspace_bytes, lay.total);
  if (!tokens) return fail(RKSC_ERR_INVALID_ARGUMENT, "tokens is NULL");
  if (!workspace) return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!w->embed || !w->final_norm || !w->layers)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "embed, final_norm and layers must not be NULL");
  st = branch_pass(w, parent, k_out, v_out, n_new, 0, 0, tokens, 1, n_new, false,
                   PassOut{nullptr, nullptr, nullptr, h_node}, workspace, workspace_bytes, stream);
  if (st != RKSC_OK) return st;
  if (h_node) HIP_TRY(rksc::launch_unit_rows(h_node, c->n_layers, c->d_model, static_cast<hipStream_t>(stream)));
  return ok();
}

RKSC_EXPORT rksc_status rksc_asks_gate(const float* hidden, const float* h_root, int32_t n_layers, int32_t n_branches,
                                       int32_t d_model, float alpha, float tau, float* sigma, int32_t* shared,
                                       void* stream) {
  if (!hidden || !h_root || !sigma || !shared)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "hidden, h_root, sigma and shared must not be NULL");
  if (n_layers < 1 || n_branches < 1 || d_model < 1)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "L, B and d must be >= 1 (got %d, %d, %d)", n_layers, n_branches,
                d_model);
  if (n_branches > 65535) return fail(RKSC_ERR_UNSUPPORTED, "n_branches above 65535 (got %d)", n_branches);
  if (n_layers > 256 || d_model % 4)
    return fail(RKSC_ERR_UNSUPPORTED, "the gate needs L <= 256 and d %% 4 == 0 (got %d, %d)", n_layers, d_model);
  if (!std::isfinite(alpha)) return fail(RKSC_ERR_INVALID_ARGUMENT, "alpha must be finite");
  if (std::isnan(tau)) return fail(RKSC_ERR_INVALID_ARGUMENT, "tau must not be NaN");
  HIP_TRY(rksc::launch_asks_gate(hidden, h_root, n_layers, n_branches, d_model, alpha, tau, sigma, shared,
                                 static_cast<hipStream_t>(stream)));
  return ok();
}

RKSC_EXPORT rksc_status rksc_cgee_gate(const float* conf, int32_t n_branches, int32_t n_steps, float tau_conf,
                                       float r_gap, float* p_mean, int32_t* fired, int32_t* winner, float* stats,
                                       void* stream) {
  if (!conf) return fail(RKSC_ERR_INVALID_ARGUMENT, "conf is NULL");
  if (!fired || !winner) return fail(RKSC_ERR_INVALID_ARGUMENT, "fired and winner must not be NULL");
  if (n_branches < 1 || n_branches > RKSC_MAX_BRANCHES)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "n_branches must be in [1, %d] (got %d)", RKSC_MAX_BRANCHES, n_branches);
  if (n_steps < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_steps must be >= 1 (got %d)", n_steps);
  if (std::isnan(tau_conf) || std::isnan(r_gap))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "tau_conf and r_gap must not be NaN");
  HIP_TRY(rksc::launch_cgee_gate(conf, n_branches, n_steps, tau_conf, r_gap, p_mean, fired, winner, stats,
                                 static_cast<hipStream_t>(stream)));
  return ok();
}

RKSC_EXPORT rksc_status rksc_asks_similarity(const float* hidden, int32_t n_layers, int32_t n_branches,
                                             int32_t d_model, float alpha, float* S, void* stream) {
  if (!hidden || !S) return fail(RKSC_ERR_INVALID_ARGUMENT, "hidden and S must not be NULL");
  if (n_layers < 1 || n_branches < 1 || d_model < 1)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "L, B and d must be >= 1 (got %d, %d, %d)", n_layers, n_branches,
                d_model);
  if (n_branches > 65535) return fail(RKSC_ERR_UNSUPPORTED, "n_branches above 65535 (got %d)", n_branches);
  if (n_layers > 256) return fail(RKSC_ERR_UNSUPPORTED, "n_layers above 256 (got %d)", n_layers);
  if (!std::isfinite(alpha)) return fail(RKSC_ERR_INVALID_ARGUMENT, "alpha must be finite");
  HIP_TRY(rksc::launch_asks(hidden, n_layers, n_branches, d_model, alpha, S, static_cast<hipStream_t>(stream)));
  return ok();
}

// ------------------------------------------------------------------ kernel-level test entry points

RKSC_EXPORT rksc_status rksc_test_gemm_kind(int32_t dtype, const void* A, const void* A_lo, const void* W, float* P,
                                            int32_t M, int32_t N, int32_t K, int32_t splits, int32_t kind,
                                            int32_t* splits_used, void* stream) {
  if (!A || !W || !P) return fail(RKSC_ERR_INVALID_ARGUMENT, "A, W and P must not be NULL");
  if (dtype == RKSC_BF16 && !A_lo) return fail(RKSC_ERR_INVALID_ARGUMENT, "A_lo must not be NULL for bf16");
  if (dtype != RKSC_F32 && dtype != RKSC_BF16) return fail(RKSC_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (M < 1 || N < 1 || K < 8 || K % 8) return fail(RKSC_ERR_INVALID_ARGUMENT, "bad shape %d x %d x %d", M, N, K);
  if (splits < 0 || splits > 8) return fail(RKSC_ERR_INVALID_ARGUMENT, "splits must be in [0, 8]");
  if (kind < -1 || kind > 2) return fail(RKSC_ERR_INVALID_ARGUMENT, "kind must be -1, 0, 1 or 2 (got %d)", kind);
  if (kind >= 1 && dtype != RKSC_BF16) return fail(RKSC_ERR_UNSUPPORTED, "kind %d needs bf16 weights", kind);
  if (kind == 2 && (M > 32 || N % 4 || K > 32768 || (M > 16 && K > 16384)))
    return fail(RKSC_ERR_UNSUPPORTED, "kind 2 needs M <= 32, N %% 4 == 0 and K <= 32768 (K <= 16384 above 16 rows)");
  const DType dt = dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const GemmPlan p = rksc::plan_gemm_kind(dt, M, N, K, kind, splits);
  if (splits_used) *splits_used = p.splits;
  HIP_TRY(rksc::launch_gemm(dt, p, A, A_lo, W, P, (size_t)M * N, nullptr, 1, M, N, K,
                            static_cast<hipStream_t>(stream)));
  return ok();
}

RKSC_EXPORT rksc_status rksc_test_gemm_live(int32_t dtype, const void* A, const void* A_lo, const void* W, float* P,
                                            int32_t M, int32_t N, int32_t K, int32_t splits, int32_t kind,
                                            int32_t live_count, int32_t branch_len, void* ctrl_scratch,
                                            int32_t* splits_used, void* stream) {
  if (!A || !W || !P || !ctrl_scratch) return fail(RKSC_ERR_INVALID_ARGUMENT, "A, W, P and ctrl_scratch must not be NULL");
  if (dtype == RKSC_BF16 && !A_lo) return fail(RKSC_ERR_INVALID_ARGUMENT, "A_lo must not be NULL for bf16");
  if (dtype != RKSC_F32 && dtype != RKSC_BF16) return fail(RKSC_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (M < 1 || N < 1 || K < 8 || K % 8) return fail(RKSC_ERR_INVALID_ARGUMENT, "bad shape %d x %d x %d", M, N, K);
  if (splits < 0 || splits > 8) return fail(RKSC_ERR_INVALID_ARGUMENT, "splits must be in [0, 8]");
  if (kind < -1 || kind > 2) return fail(RKSC_ERR_INVALID_ARGUMENT, "kind must be -1, 0, 1 or 2 (got %d)", kind);
  if (kind >= 1 && dtype != RKSC_BF16) return fail(RKSC_ERR_UNSUPPORTED, "kind %d needs bf16 weights", kind);
  if (kind == 2 && (M > 32 || N % 4 || K > 32768 || (M > 16 && K > 16384)))
    return fail(RKSC_ERR_UNSUPPORTED, "kind 2 needs M <= 32, N %% 4 == 0 and K <= 32768 (K <= 16384 above 16 rows)");
  if (live_count < 1 || live_count > RKSC_MAX_BRANCHES || branch_len < 1 || (long long)live_count * branch_len > M)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "need 1 <= live_count <= %d, branch_len >= 1, live rows <= M",
                RKSC_MAX_BRANCHES);
  if (reinterpret_cast<uintptr_t>(ctrl_scratch) % 256)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "ctrl_scratch must be 256-byte aligned");
  static_assert(sizeof(rksc::Ctrl) <= 4096, "the control block fits the documented scratch size");
  const DType dt = dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const GemmPlan p = rksc::plan_gemm_kind(dt, M, N, K, kind, splits);
  if (splits_used) *splits_used = p.splits;
  hipStream_t st = static_cast<hipStream_t>(stream);
  rksc::Ctrl* ctrl = static_cast<rksc::Ctrl*>(ctrl_scratch);
  HIP_TRY(rksc::launch_init(ctrl, live_count, 1, nullptr, nullptr, nullptr, 0, st));
  HIP_TRY(rksc::launch_gemm(dt, p, A, A_lo, W, P, (size_t)M * N, ctrl, branch_len, M, N, K, st));
  return ok();
}

RKSC_EXPORT rksc_status rksc_test_gate_up_swiglu(const void* A, const void* A_lo, const void* W, void* a_out,
                                                 float* P, int32_t M, int32_t F, int32_t K, int32_t fused,
                                                 void* stream) {
  if (!A || !A_lo || !W || !a_out || !P) return fail(RKSC_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (M < 1 || F < 8 || F % 8 || K < 8 || K % 8)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "bad shape %d x %d x %d", M, F, K);
  if (fused != 0 && fused != 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "fused must be 0 or 1");
  GemmPlan p = rksc::plan_gemm_kind(DType::BF16, M, 2 * F, K, fused ? 1 : -1, fused ? 1 : 0);
  if (fused && !rksc::gate_up_fused(DType::BF16, p, 2 * F))
    return fail(RKSC_ERR_UNSUPPORTED, "no fused plan for this shape");
  if (!fused && rksc::gate_up_fused(DType::BF16, p, 2 * F)) {   // the unfused path: partials + SwiGLU kernel
    p.kind = 0;
    p.bm = 128;
    p.k_per_split = (K + 63) / 64 * 64;
  }
  HIP_TRY(rksc::launch_gate_up_swiglu(DType::BF16, p, A, A_lo, W, P, (size_t)M * 2 * F, nullptr, 1, M, F, K, a_out,
                                      static_cast<hipStream_t>(stream)));
  return ok();
}

RKSC_EXPORT rksc_status rksc_test_gemm_plan(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t splits,
                                            int32_t kind, int32_t* plan) {
  if (!plan) return fail(RKSC_ERR_INVALID_ARGUMENT, "plan must not be NULL");
  if (dtype != RKSC_F32 && dtype != RKSC_BF16) return fail(RKSC_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (M < 1 || N < 1 || K < 8 || K % 8) return fail(RKSC_ERR_INVALID_ARGUMENT, "bad shape %d x %d x %d", M, N, K);
  if (splits < 0 || splits > 8) return fail(RKSC_ERR_INVALID_ARGUMENT, "splits must be in [0, 8]");
  if (kind < -1 || kind > 2) return fail(RKSC_ERR_INVALID_ARGUMENT, "kind must be -1, 0, 1 or 2 (got %d)", kind);
  const GemmPlan p = rksc::plan_gemm_kind(dtype == RKSC_BF16 ? DType::BF16 : DType::F32, M, N, K, kind, splits);
  plan[0] = p.kind;
  plan[1] = p.bm;
  plan[2] = p.bn;
  plan[3] = p.splits;
  plan[4] = p.k_per_split;
  return ok();
}

RKSC_EXPORT rksc_status rksc_test_gemm(int32_t dtype, const void* A, const void* A_lo, const void* W, float* P,
                                       int32_t M, int32_t N, int32_t K, int32_t splits, int32_t* splits_used,
                                       void* stream) {
  return rksc_test_gemm_kind(dtype, A, A_lo, W, P, M, N, K, splits, -1, splits_used, stream);
}

RKSC_EXPORT size_t rksc_test_attention_scratch_size(int32_t dtype, int32_t B, int32_t n, int32_t s, int32_t H,
                                                   int32_t Hkv, int32_t hd) {
  if (B < 1 || s < 1 || n < 0 || H < 1 || Hkv < 1 || H % Hkv || hd < 1) return 0;
  const rksc::AttnPlan p = rksc::plan_attention(dtype == RKSC_BF16 ? DType::BF16 : DType::F32, B, n, s, H, Hkv);
  return 4096 + (size_t)p.partials * B * s * H * (hd + 2) * 4;
}

RKSC_EXPORT rksc_status rksc_test_attention(int32_t dtype, const void* q, const void* prefix_k, const void* prefix_v,
                                            const void* k_own, const void* v_own, void* o, int32_t B, int32_t n,
                                            int32_t s, int32_t H, int32_t Hkv, int32_t hd, void* scratch,
                                            size_t scratch_bytes, void* stream) {
  if (!q || !k_own || !v_own || !o || !scratch) return fail(RKSC_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (n > 0 && (!prefix_k || !prefix_v)) return fail(RKSC_ERR_INVALID_ARGUMENT, "NULL prefix with n > 0");
  if (dtype != RKSC_F32 && dtype != RKSC_BF16) return fail(RKSC_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (B < 1 || B > RKSC_MAX_BRANCHES || s < 1 || n < 0 || H < 1 || Hkv < 1 || H % Hkv)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "bad attention shape");
  if (hd != 64 && hd != 128) return fail(RKSC_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  hipStream_t st = static_cast<hipStream_t>(stream);
  rksc::Ctrl* ctrl = static_cast<rksc::Ctrl*>(scratch);
  const DType dt = dtype == RKSC_BF16 ? DType::BF16 : DType::F32;
  const rksc::AttnPlan plan = rksc::plan_attention(dt, B, n, s, H, Hkv);
  const size_t need = 4096 + (size_t)plan.partials * B * s * H * (hd + 2) * 4;
  if (scratch_bytes < need)
    return fail(RKSC_ERR_WORKSPACE_TOO_SMALL, "scratch has %zu bytes, needs %zu", scratch_bytes, need);
  char* sc = static_cast<char*>(scratch);
  float* opart = reinterpret_cast<float*>(sc + 4096);
  float* mlpart = opart + (size_t)plan.partials * B * s * H * hd;
  HIP_TRY(rksc::launch_init(ctrl, B, 1, nullptr, nullptr, nullptr, 0, st));
  rksc::PrefixView pre;
  if (n > 0) {
    pre.n = n;
    pre.nseg = 1;
    pre.len[0] = n;
    pre.k[0] = prefix_k;
    pre.v[0] = prefix_v;
  }
  HIP_TRY(rksc::launch_attention(dt, plan, q, pre, k_own, v_own, o, opart, mlpart, ctrl, s, H, Hkv, hd, B, st));
  return ok();
}
