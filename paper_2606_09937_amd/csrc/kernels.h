// Internal launch interface between the C-ABI layer (rksc_api.cpp) and the
// gfx950 kernels. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rksc {

// Per-call control block in the workspace. Slots are the compacted positions of
// the branches still being computed; `live_idx[slot]` is the caller's branch
// index, `gather_src[new_slot]` the previous layer's slot of a survivor.
struct Ctrl {
  int live_count;
  int pad0[63];
  int live_idx[64];
  int gather_src[64];
  int streak[64];     // indexed by branch
  float h_prev[64];   // indexed by branch
  float h_cur[64];    // indexed by slot
};

enum class DType { F32 = 0, BF16 = 1 };

// ---- setup
hipError_t launch_init(Ctrl* c, int B, int L, float* entropy, int* exit_layer, float* hidden_last,
                       size_t hidden_elems, hipStream_t st);
hipError_t launch_rope_table(float2* tab, int s, int n, int hd, double base, hipStream_t st);
hipError_t launch_embed(DType dt, const void* E, const int* tok, int V, float* x, int rows, int d,
                        hipStream_t st);

// ---- per-layer row kernels
// Projection inputs (xn, attention output o, SwiGLU output a) are written as bf16
// hi/lo planes for BF16 models (plane lo follows plane hi: max_rows rows each)
// and as fp32 for F32 models; q, k_own, v_own and the residual stream are fp32.
// The last-token tap of launch_tap, fused into launch_add_norm: layer layer0's
// output rows go to hidden_last and their RMSNorm(final_norm = gamma) to row
// jrow * live_count + slot of hn_a/hn_b. gamma NULL: no tap.
struct TapArgs {
  const float* gamma = nullptr;
  float* hidden_last = nullptr;
  int layer0 = 0, B = 0, jrow = 0;
  void* hn_a = nullptr;
  void* hn_b = nullptr;
};
// x_out[r] = x_in[src(r)] + sum_sp P[sp][src(r)] ; xn[r] = RMSNorm(x_out[r]; gamma).
// gather: src(r) = gather_src[r / s] * s + r % s, else src(r) = r (x_in may equal x_out).
// With tap.gamma set (no gather), each branch's last row x_out[slot * s + s - 1]
// is also tapped as described for TapArgs.
hipError_t launch_add_norm(DType dt, const float* x_in, const float* P, int nsplit, size_t split_stride,
                           bool gather, const Ctrl* c, int s, float* x_out, void* xn, const float* gamma, int d,
                           float eps, int max_rows, hipStream_t st, const TapArgs& tap = TapArgs{});
// q [rows, H, hd], k_own/v_own [B, Hkv, s, hd] from the summed QKV partials, RoPE on q and k.
// With k_cache/v_cache, the keys and values are also stored (type cache_dt) as
// entries off..off+s-1 of a cache layer [B, Hkv, cap, hd].
hipError_t launch_qkv_post(const float* P, int nsplit, size_t split_stride, const Ctrl* c, int s, int H,
                           int Hkv, int hd, const float2* rope, float* q, float* k_own, float* v_own,
                           int max_rows, hipStream_t st, DType cache_dt = DType::F32, void* k_cache = nullptr,
                           void* v_cache = nullptr, int cap = 0, int off = 0);
// a = silu(gate) * up from the summed gate|up partials.
hipError_t launch_swiglu_post(DType dt, const float* P, int nsplit, size_t split_stride, const Ctrl* c, int s,
                              int F, void* a, int max_rows, hipStream_t st);
// Last token of each live branch: h = x + sum_sp P; hidden_last[l][branch] = h;
// hn = RMSNorm(h; final_norm) as fp32 (F32) or as a bf16 hi+lo pair (BF16), at
// row jrow * live_count + slot (jrow: the layer's place in an exit window).
hipError_t launch_tap(DType dt, const float* x, const float* P, int nsplit, size_t split_stride,
                      const Ctrl* c, int s, int d, int B, int layer0, float* hidden_last,
                      const float* gamma, float eps, void* hn_a, void* hn_b, int max_branches,
                      hipStream_t st, int jrow = 0);

// ---- GEMM: P[split][m][n] = sum_{k in split} A[m][k] * W[n][k], rows m < live*s.
// BF16 models: A0/A1 are the bf16 hi/lo planes of the activation, W bf16.
// F32 models: A0 is the fp32 activation (A1 unused), W fp32.
constexpr int kMaxSplitsGemm = 8;   // the consumers of split partials sum at most this many
// kind: 0 = 128-row tiles (bn columns; HBM-bound skinny projections and mid
// sizes), 1 = 256 x 256 tiles (MFMA-bound projections with many rows).
struct GemmPlan {
  int kind, bm, bn, splits, k_per_split;
};
GemmPlan plan_gemm(DType dt, int max_rows, int N, int K);
// Test hook: kind -1 = the planner's choice, 0/1 = that kernel; splits > 0 forces the split count.
GemmPlan plan_gemm_kind(DType dt, int max_rows, int N, int K, int kind, int splits);
// W_tiled (may be null): the same weight pre-tiled by launch_tile_rows, read
// instead of W by the 128-row kernel's 256-column tiles (gemm_tiled says when).
hipError_t launch_gemm(DType dt, const GemmPlan& p, const void* A0, const void* A1, const void* W, float* P,
                       size_t split_stride, const Ctrl* c, int s, int max_rows, int N, int K, hipStream_t st,
                       const void* W_tiled = nullptr);
// Rows per column tile of the pre-tiled weight layout [N/kTileRows][K/64][kTileRows][64].
constexpr int kTileRows = 256;
// Whether launch_gemm reads W_tiled for this plan and shape.
bool gemm_tiled(DType dt, const GemmPlan& p, const void* W_tiled, int N, int K);
// out = W [N, K] (bf16) re-laid as [N/kTileRows][K/64][kTileRows][64]; N % kTileRows == 0, K % 64 == 0.
hipError_t launch_tile_rows(const void* W, void* out, int N, int K, hipStream_t st);
// The gate|up projection (W [2F, K]) and its SwiGLU: a = silu(gate) * up, written to `a`
// as the down projection's input (bf16 hi/lo planes [max_rows, F] for BF16 models). With
// the 256 x 256 kernel over one K split it is fused into the projection's epilogue (the
// fp32 gate|up product never reaches memory); otherwise the split partials go to P and
// launch_swiglu_post combines them.
bool gate_up_fused(DType dt, const GemmPlan& p, int N);
hipError_t launch_gate_up_swiglu(DType dt, const GemmPlan& p, const void* A0, const void* A1, const void* W,
                                 float* P, size_t split_stride, const Ctrl* c, int s, int max_rows, int F, int K,
                                 void* a, hipStream_t st, const void* W_tiled = nullptr);

// ---- the shared prefix of one layer
// Up to kMaxPrefixSegs caches in position order (a tree node's own entries after
// its ancestors'): segment i holds positions start[i] .. start[i] + len[i] - 1 as
// [Hkv, len[i], hd] in the model's storage type at k[i] / v[i]; n is the total.
constexpr int kMaxPrefixSegs = 8;
struct PrefixView {
  int n = 0, nseg = 0;
  int start[kMaxPrefixSegs] = {};
  int len[kMaxPrefixSegs] = {};
  const void* k[kMaxPrefixSegs] = {};
  const void* v[kMaxPrefixSegs] = {};
};

// ---- attention over [shared prefix ; own causal span]: q, k_own, v_own fp32; prefix of the
// model dtype; o is the projection input (bf16 hi/lo planes for BF16 models, fp32 otherwise).
// Split-KV plan: `chunks` workgroups share the keys of a query tile and write
// partials opart [partials, B*s, H, hd] and mlpart [partials, B*s, H, 2] that a
// combine kernel merges. `cross`: branches with G*s < 64 query rows per KV head
// are packed together into prefix-only tiles and their own spans are merged in
// the combine.
struct AttnPlan {
  int chunks, partials;
  bool cross;
};
AttnPlan plan_attention(DType dt, int B, int n, int s, int H, int Hkv);
// p_split = false: the probabilities enter P.V as bf16 alone instead of a hi/lo pair.
hipError_t launch_attention(DType dt, const AttnPlan& p, const void* q, const PrefixView& pre,
                            const void* k_own, const void* v_own, void* o, float* opart, float* mlpart,
                            const Ctrl* c, int s, int H, int Hkv, int hd, int max_branches, hipStream_t st,
                            bool p_split = true);
// x[i] = fp32(bf16(x[i])) for i < n: the value rounded to bf16 precision, kept in fp32.
hipError_t launch_round_bf16(float* x, size_t n, hipStream_t st);

// ---- entropy of the live branches' last-token logits
int entropy_parts(DType dt, int V, int max_branches);
// kmul: layers per exit window; the columns are kmul * live_count rows of hn.
hipError_t launch_entropy(DType dt, const void* W, const void* hn_a, const void* hn_b, const Ctrl* c,
                          int V, int d, int max_branches, float* parts, hipStream_t st, int kmul = 1);
// As launch_entropy, plus the vocabulary index of each column's maximum logit:
// parts become [grid, 64, 4] = (m, s, t, argmax as int bits).
hipError_t launch_entropy_argmax(DType dt, const void* W, const void* hn_a, const void* hn_b, const Ctrl* c, int V,
                                 int d, int max_branches, float* parts, hipStream_t st);
// Merges [nparts, 64, 4] statistics of B columns: next_token = argmax (smallest
// index among equal maxima; -1 if no finite logit), p_top = 1 / sum e^(z - max)
// (the top-1 softmax probability); conf = p_top (accumulate = 0) or conf + p_top.
hipError_t launch_finalize_decode(const float* parts, int nparts, int B, int* next_token, float* p_top, float* conf,
                                  int accumulate, hipStream_t st);
// Merges the partial statistics of an exit window of kw layers from layer1
// (1-based), writes entropy[l-1][branch], applies the exit rule layer by layer
// (NaN for the window's layers after an exit, in entropy and hidden_last) and
// compacts the live list.
hipError_t launch_finalize_exit(const float* parts, int nparts, Ctrl* c, int layer1, int kw, int L, int B,
                                float tau, int patience, float* entropy, int* exit_layer, float* hidden_last, int d,
                                hipStream_t st);

// ---- batched decode
// Attention of one new token per branch (s = 1) over the shared prefix (split-KV
// plan p, cross mode), the branch's cached entries 0..len-1 (model dtype, layer
// base [B, Hkv, cap, hd]) and its own key/value (fp32 k_own/v_own [B, Hkv, 1, hd]).
hipError_t launch_attention_decode(DType dt, const AttnPlan& p, const void* q, const PrefixView& pre,
                                   const void* ck, const void* cv, int len, int cap, const void* k_own,
                                   const void* v_own, void* o, float* opart, float* mlpart, const Ctrl* c,
                                   int H, int Hkv, int hd, int B, hipStream_t st);

// Level-1 / decode-level gate of Eq. cgee_gate over p = conf / n_steps of B <= 64
// branches; stats = (max, 2nd max, gap ratio) when not NULL.
hipError_t launch_cgee_gate(const float* conf, int B, int n_steps, float tau_conf, float r_gap, float* p_mean,
                            int* fired, int* winner, float* stats, hipStream_t st);

// ---- root forward (prefill)
// x[r] /= |x[r]| for rows r < rows of d floats (zero rows stay zero).
hipError_t launch_unit_rows(float* x, int rows, int d, hipStream_t st);

// ---- ASKS similarity
hipError_t launch_asks(const float* hidden, int L, int B, int d, float alpha, float* S, hipStream_t st);
// Alg. AsksGate against unit root rows: sigma [B], shared [B] = sigma >= tau.
hipError_t launch_asks_gate(const float* hidden, const float* root, int L, int B, int d, float alpha, float tau,
                            float* sigma, int* shared, hipStream_t st);

}  // namespace rksc
