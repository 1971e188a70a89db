// Row-wise kernels of the verify pass: setup, embedding, RMSNorm with the
// deferred residual adds and the live-branch gather, the QKV/RoPE and SwiGLU
// epilogues, the last-token tap, and the entropy merge + exit rule.
#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(bf16* p, float a, float b, float c, float d) {
  uint2 u;
  u.x = static_cast<uint32_t>(f32_to_bf16_bits(a)) | (static_cast<uint32_t>(f32_to_bf16_bits(b)) << 16);
  u.y = static_cast<uint32_t>(f32_to_bf16_bits(c)) | (static_cast<uint32_t>(f32_to_bf16_bits(d)) << 16);
  *reinterpret_cast<uint2*>(p) = u;
}

// ------------------------------------------------------------------ setup

__global__ void k_init(Ctrl* c, int B, int L, float* entropy, int* exit_layer, float* hidden_last,
                       size_t hidden_elems) {
  const size_t tid = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  if (tid == 0) c->live_count = B;
  if (tid < 64) {
    c->live_idx[tid] = (int)tid;
    c->gather_src[tid] = (int)tid;
    c->streak[tid] = 0;
    c->h_prev[tid] = INFINITY;
    c->h_cur[tid] = 0.f;
  }
  if (exit_layer && tid < (size_t)B) exit_layer[tid] = L;
  const float nan = __builtin_nanf("");
  if (entropy)
    for (size_t i = tid; i < (size_t)L * B; i += stride) entropy[i] = nan;
  if (hidden_last)
    for (size_t i = tid; i < hidden_elems; i += stride) hidden_last[i] = nan;
}

// cos/sin of (n + i) * base^(-2j/hd), evaluated in double precision.
__global__ void k_rope_table(float2* tab, int s, int n, int hd, double base) {
  const int half = hd / 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= s * half) return;
  const int i = idx / half, j = idx % half;
  const double theta = pow(base, -2.0 * (double)j / (double)hd);
  const double ang = (double)(n + i) * theta;
  tab[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

template <typename T>
__global__ void k_embed(const T* E, const int* tok, int V, float* x, int d) {
  const int r = blockIdx.x;
  const int t = tok[r];
  float* xr = x + (size_t)r * d;
  if (t < 0 || t >= V) {   // an id outside the vocabulary yields a NaN row, never a stray read
    for (int c = threadIdx.x; c < d; c += blockDim.x) xr[c] = __builtin_nanf("");
    return;
  }
  const T* e = E + (size_t)t * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) xr[c] = to_f32(e[c]);
}

// ------------------------------------------------------------------ last-token tap

// The tap of one residual row v (held as MAXC float4 chunks per thread of a
// 1024-thread block) with rinv = 1 / RMS(v): the row itself to hl_row (when not
// NULL) and RMSNorm(v; gamma) to row hrow of the normalised rows, as fp32
// (hn_a) or as a bf16 hi + lo pair (hn_a, hn_b): hi = bf16(hn), lo =
// bf16(hn - hi), so the lm_head product runs on bf16 MFMA with ~2^-16 relative
// error on the activation.
template <bool kSplitBf16, int MAXC>
__device__ __forceinline__ void tap_store(const float4 (&v)[MAXC], float rinv, const float* __restrict__ gamma,
                                          float* hl_row, void* hn_a, void* hn_b, size_t hrow, int d) {
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int col = (threadIdx.x + j * 1024) * 4;
    if (col >= d) continue;
    if (hl_row) *reinterpret_cast<float4*>(hl_row + col) = v[j];
    const float4 g = *reinterpret_cast<const float4*>(gamma + col);
    const float h0 = g.x * v[j].x * rinv, h1 = g.y * v[j].y * rinv, h2 = g.z * v[j].z * rinv, h3 = g.w * v[j].w * rinv;
    if (kSplitBf16) {
      uint16_t b0, b1, b2, b3, l0, l1, l2, l3;
      split2(h0, b0, l0);
      split2(h1, b1, l1);
      split2(h2, b2, l2);
      split2(h3, b3, l3);
      *reinterpret_cast<uint2*>(static_cast<bf16*>(hn_a) + hrow * d + col) = make_uint2(pack2(b0, b1), pack2(b2, b3));
      *reinterpret_cast<uint2*>(static_cast<bf16*>(hn_b) + hrow * d + col) = make_uint2(pack2(l0, l1), pack2(l2, l3));
    } else {
      *reinterpret_cast<float4*>(static_cast<float*>(hn_a) + hrow * d + col) = make_float4(h0, h1, h2, h3);
    }
  }
}

// ------------------------------------------------------------------ add + RMSNorm

// One 1024-thread block per row; each thread keeps up to MAXC float4 chunks of
// the row in registers, so every load of the row is issued before the first
// wait and the row is read exactly once.
constexpr int kMaxSplits = kMaxSplitsGemm;

// Writes 4 consecutive projection-input values: fp32, or (kSplit) as the bf16
// hi/lo planes, the lo plane starting plane_stride elements after the hi plane.
template <bool kSplit>
__device__ __forceinline__ void store_act4(void* base, size_t idx, size_t plane_stride, float a, float b, float c,
                                           float d) {
  if (kSplit) {
    uint16_t h0, l0, h1, l1, h2, l2, h3, l3;
    split2(a, h0, l0);
    split2(b, h1, l1);
    split2(c, h2, l2);
    split2(d, h3, l3);
    bf16* p = static_cast<bf16*>(base);
    *reinterpret_cast<uint2*>(p + idx) = make_uint2(pack2(h0, h1), pack2(h2, h3));
    *reinterpret_cast<uint2*>(p + plane_stride + idx) = make_uint2(pack2(l0, l1), pack2(l2, l3));
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(base) + idx) = make_float4(a, b, c, d);
  }
}

// With tap.gamma set, the last row of each branch (r % s == s - 1) is also
// tapped for the previous layer: x_out's row is that layer's output.
template <int MAXC, bool kSplit>
__global__ __launch_bounds__(1024) void k_add_norm(const float* __restrict__ x_in, const float* __restrict__ P,
                                                   int nsplit, size_t split_stride, int gather, const Ctrl* c,
                                                   int s, float* __restrict__ x_out, void* __restrict__ xn,
                                                   const float* __restrict__ gamma, int d, float eps, TapArgs tap) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  if (r >= c->live_count * s) return;
  const int src = gather ? c->gather_src[r / s] * s + (r % s) : r;
  const float* xi = x_in + (size_t)src * d;
  float4 v[MAXC];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int col = (threadIdx.x + j * 1024) * 4;
    v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (col < d) {
      v[j] = *reinterpret_cast<const float4*>(xi + col);
#pragma unroll
      for (int sp = 0; sp < kMaxSplits; ++sp) {
        if (sp < nsplit) {
          const float4 p = *reinterpret_cast<const float4*>(P + sp * split_stride + (size_t)src * d + col);
          v[j].x += p.x; v[j].y += p.y; v[j].z += p.z; v[j].w += p.w;
        }
      }
      ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
    }
  }
  const float tot = block_sum(ss, red);
  const float rinv = rsqrtf(tot / (float)d + eps);
  float* xo = x_out + (size_t)r * d;
  const size_t plane = (size_t)gridDim.x * d;
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int col = (threadIdx.x + j * 1024) * 4;
    if (col < d) {
      *reinterpret_cast<float4*>(xo + col) = v[j];
      const float4 g = *reinterpret_cast<const float4*>(gamma + col);
      store_act4<kSplit>(xn, (size_t)r * d + col, plane, g.x * v[j].x * rinv, g.y * v[j].y * rinv,
                         g.z * v[j].z * rinv, g.w * v[j].w * rinv);
    }
  }
  if (tap.gamma && r % s == s - 1) {
    const int slot = r / s, branch = c->live_idx[slot];
    tap_store<kSplit, MAXC>(v, rinv, tap.gamma,
                            tap.hidden_last ? tap.hidden_last + ((size_t)tap.layer0 * tap.B + branch) * d : nullptr,
                            tap.hn_a, tap.hn_b, (size_t)tap.jrow * c->live_count + slot, d);
  }
}

// ------------------------------------------------------------------ QKV epilogue

// Thread (unit u, row r): unit u covers columns (hh*hd + j, hh*hd + j + hd/2)
// of head hh of the [q | k | v] output; q and k pairs are rotated by RoPE.
// When kc is not NULL, the rotated keys and the values are also stored, in the
// cache type CT, as entries off..off+s-1 of the cache layer kc/vc
// [slots, Hkv, cap, hd] (the prefix cache of the root forward, or a branch
// cache of the decode).
template <typename T, typename CT>
__global__ __launch_bounds__(256) void k_qkv_post(const float* __restrict__ P, int nsplit, size_t split_stride,
                                                  const Ctrl* c, int s, int H, int Hkv, int hd,
                                                  const float2* __restrict__ rope, T* __restrict__ q,
                                                  T* __restrict__ k_own, T* __restrict__ v_own,
                                                  CT* __restrict__ kc, CT* __restrict__ vc, int cap, int off) {
  const int r = blockIdx.y;
  if (r >= c->live_count * s) return;
  const int half = hd / 2;
  const int units = (H + 2 * Hkv) * half;
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= units) return;
  const int slot = r / s, i = r % s;
  const int N = (H + 2 * Hkv) * hd;
  const float* pr = P + (size_t)r * N;
  const int hh = u / half, j = u % half;
  const int c1 = hh * hd + j, c2 = c1 + half;
  float x1 = 0.f, x2 = 0.f;
#pragma unroll
  for (int sp = 0; sp < kMaxSplits; ++sp) {
    if (sp < nsplit) {
      x1 += pr[sp * split_stride + c1];
      x2 += pr[sp * split_stride + c2];
    }
  }
  if (hh < H + Hkv) {
    const float2 cs = rope[i * half + j];
    const float y1 = x1 * cs.x - x2 * cs.y;
    const float y2 = x2 * cs.x + x1 * cs.y;
    x1 = y1;
    x2 = y2;
  }
  T* dst;
  CT* cdst = nullptr;
  if (hh < H) {
    dst = q + ((size_t)r * H + hh) * hd;
  } else if (hh < H + Hkv) {
    dst = k_own + (((size_t)slot * Hkv + (hh - H)) * s + i) * hd;
    if (kc) cdst = kc + (((size_t)slot * Hkv + (hh - H)) * cap + off + i) * hd;
  } else {
    dst = v_own + (((size_t)slot * Hkv + (hh - H - Hkv)) * s + i) * hd;
    if (vc) cdst = vc + (((size_t)slot * Hkv + (hh - H - Hkv)) * cap + off + i) * hd;
  }
  dst[j] = from_f32<T>(x1);
  dst[j + half] = from_f32<T>(x2);
  if (cdst) {
    cdst[j] = from_f32<CT>(x1);
    cdst[j + half] = from_f32<CT>(x2);
  }
}

// ------------------------------------------------------------------ SwiGLU epilogue

// Thread (4 columns, row r); F is a multiple of 8, so float4 groups never straddle.
template <bool kSplit>
__global__ __launch_bounds__(256) void k_swiglu_post(const float* __restrict__ P, int nsplit, size_t split_stride,
                                                     const Ctrl* c, int s, int F, void* __restrict__ a) {
  const int r = blockIdx.y;
  if (c && r >= c->live_count * s) return;   // no control block: every row is live, as in the GEMMs
  const int f = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (f >= F) return;
  const float* pr = P + (size_t)r * 2 * F;
  float4 g = make_float4(0.f, 0.f, 0.f, 0.f), u = g;
#pragma unroll
  for (int sp = 0; sp < kMaxSplits; ++sp) {
    if (sp < nsplit) {
      const float4 pg = *reinterpret_cast<const float4*>(pr + sp * split_stride + f);
      const float4 pu = *reinterpret_cast<const float4*>(pr + sp * split_stride + F + f);
      g.x += pg.x; g.y += pg.y; g.z += pg.z; g.w += pg.w;
      u.x += pu.x; u.y += pu.y; u.z += pu.z; u.w += pu.w;
    }
  }
  store_act4<kSplit>(a, (size_t)r * F + f, (size_t)gridDim.y * F, g.x / (1.f + expf(-g.x)) * u.x,
                     g.y / (1.f + expf(-g.y)) * u.y, g.z / (1.f + expf(-g.z)) * u.z, g.w / (1.f + expf(-g.w)) * u.w);
}

// ------------------------------------------------------------------ last-token tap kernel

template <bool kSplitBf16, int MAXC>
__global__ __launch_bounds__(1024) void k_tap(const float* __restrict__ x, const float* __restrict__ P, int nsplit,
                                              size_t split_stride, const Ctrl* c, int s, int d, int B, int layer0,
                                              float* __restrict__ hidden_last, const float* __restrict__ gamma,
                                              float eps, void* hn_a, void* hn_b, int jrow) {
  __shared__ float red[16];
  const int slot = blockIdx.x;
  if (slot >= c->live_count) return;
  const size_t hrow = (size_t)jrow * c->live_count + slot;   // row of the normalised rows (layer jrow of a window)
  const int branch = c->live_idx[slot];
  const size_t row = (size_t)slot * s + (s - 1);
  float4 v[MAXC];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int col = (threadIdx.x + j * 1024) * 4;
    v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (col < d) {
      v[j] = *reinterpret_cast<const float4*>(x + row * d + col);
#pragma unroll
      for (int sp = 0; sp < kMaxSplits; ++sp) {
        if (sp < nsplit) {
          const float4 p = *reinterpret_cast<const float4*>(P + sp * split_stride + row * d + col);
          v[j].x += p.x; v[j].y += p.y; v[j].z += p.z; v[j].w += p.w;
        }
      }
      ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
    }
  }
  const float tot = block_sum(ss, red);
  const float rinv = rsqrtf(tot / (float)d + eps);
  tap_store<kSplitBf16, MAXC>(v, rinv, gamma, hidden_last ? hidden_last + ((size_t)layer0 * B + branch) * d : nullptr,
                              hn_a, hn_b, hrow, d);
}

// ------------------------------------------------------------------ entropy merge + exit rule

// The exit rule over a window of kw layers layer1 .. layer1 + kw - 1 (1-based),
// whose entropies were streamed together: column j * Bl + slot holds layer
// layer1 + j of live slot `slot`. Each branch walks its layers in order; at an
// exit the later layers of the window (computed on the same live set) are
// discarded: their entropies stay NaN and their hidden rows are set back to
// NaN, so the outputs are those of a layer-by-layer schedule. Then the live
// list is compacted.
__global__ __launch_bounds__(256) void k_finalize_exit(const float* parts, int nparts, Ctrl* c, int layer1, int kw,
                                                       int L, int B, float tau, int patience, float* entropy,
                                                       int* exit_layer, float* hidden_last, int d) {
  __shared__ int exit_j[64], branch_of[64];
  const int Bl = c->live_count;
  if (Bl == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // One wave per column: lane p merges parts p, p + 64, ... in order, then a
  // fixed shuffle tree merges the lanes. The loads of kBatch parts are issued
  // together (one memory latency per batch, not per part).
  constexpr int kBatch = 8;
  for (int col = wid; col < Bl * kw; col += blockDim.x >> 6) {
    EntStats st = ent_empty();
    for (int p0 = lane; p0 < nparts; p0 += 64 * kBatch) {
      EntStats q[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int p = p0 + 64 * i;
        if (p < nparts) {
          const float* e = parts + ((size_t)p * 64 + col) * 3;
          q[i] = EntStats{e[0], e[1], e[2]};
        }
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i)
        if (p0 + 64 * i < nparts) st = ent_merge(st, q[i]);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const EntStats o{__shfl_xor(st.m, off, 64), __shfl_xor(st.s, off, 64), __shfl_xor(st.t, off, 64)};
      st = ent_merge(st, o);
    }
    if (lane == 0) c->h_cur[col] = logf(st.s) - st.t / st.s;
  }
  __syncthreads();
  if (tid < 64) {
    const int slot = tid;
    const bool live = slot < Bl;
    int branch = -1, ej = kw;
    bool keep = false;
    if (live) {
      branch = c->live_idx[slot];
      int streak = c->streak[branch];
      float prev = c->h_prev[branch];   // H_0 = +inf
      for (int j = 0; j < kw; ++j) {
        const float H = c->h_cur[j * Bl + slot];
        streak = fabsf(H - prev) < tau ? streak + 1 : 0;
        prev = H;
        entropy[(size_t)(layer1 - 1 + j) * B + branch] = H;
        if (streak >= patience) {
          exit_layer[branch] = layer1 + j;
          ej = j;
          break;
        }
      }
      c->streak[branch] = streak;
      c->h_prev[branch] = prev;
      keep = ej == kw && layer1 + kw - 1 < L;
    }
    exit_j[slot] = ej;
    branch_of[slot] = branch;
    const unsigned long long mask = __ballot(keep);
    if (keep) {
      const int ns = __popcll(mask & ((1ull << slot) - 1ull));
      c->gather_src[ns] = slot;
      c->live_idx[ns] = branch;
    }
    if (slot == 0) c->live_count = __popcll(mask);
  }
  __syncthreads();
  if (hidden_last) {
    const float nan = __builtin_nanf("");
    for (int slot = 0; slot < Bl; ++slot)
      for (int j = exit_j[slot] + 1; j < kw; ++j) {
        float* row = hidden_last + ((size_t)(layer1 - 1 + j) * B + branch_of[slot]) * d;
        for (int e = tid; e < d; e += blockDim.x) row[e] = nan;
      }
  }
}

// ------------------------------------------------------------------ batched decode

// Index of the larger maximum of two (statistics, index) pairs; the smaller
// index on equal maxima.
__device__ __forceinline__ int merge_argmax(const EntStats& a, int ia, const EntStats& b, int ib) {
  if (b.m > a.m) return ib;
  if (b.m < a.m) return ia;
  return min(ia, ib);
}

// Greedy token and top-1 probability of each branch's logits from the
// per-workgroup (m, s, t, argmax) of the lm_head stream (Eq. gen_conf's
// max_v Pr[y = v] = e^(z_max - LSE) = 1 / s). Fixed reduction order.
__global__ __launch_bounds__(256) void k_finalize_decode(const float* parts, int nparts, int B, int* next_token,
                                                         float* p_top, float* conf, int accumulate) {
  __shared__ EntStats red[256];
  __shared__ int red_am[256];
  const int tid = threadIdx.x;
  const int col = blockIdx.x;   // one workgroup per branch column
  EntStats st = ent_empty();
  int am = 0x7fffffff;
  for (int p = tid; p < nparts; p += blockDim.x) {
    const float* q = parts + ((size_t)p * 64 + col) * 4;
    const EntStats o{q[0], q[1], q[2]};
    am = merge_argmax(st, am, o, __float_as_int(q[3]));
    st = ent_merge(st, o);
  }
  red[tid] = st;
  red_am[tid] = am;
  __syncthreads();
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if (tid < off) {
      red_am[tid] = merge_argmax(red[tid], red_am[tid], red[tid + off], red_am[tid + off]);
      red[tid] = ent_merge(red[tid], red[tid + off]);
    }
    __syncthreads();
  }
  if (tid == 0) {
    const bool ok = red[0].m != -INFINITY && red_am[0] != 0x7fffffff;
    const float p = ok ? 1.f / red[0].s : __builtin_nanf("");
    next_token[col] = ok ? red_am[0] : -1;
    p_top[col] = p;
    if (conf) conf[col] = accumulate ? conf[col] + p : p;
  }
}

// ------------------------------------------------------------------ root forward

// Unit-normalises each row (the root hidden states are stored normalised).
__global__ __launch_bounds__(256) void k_unit_rows(float* __restrict__ x, int d) {
  __shared__ float red[16];
  float* row = x + (size_t)blockIdx.x * d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += blockDim.x) ss += row[c] * row[c];
  const float tot = block_sum(ss, red);
  const float inv = tot > 0.f ? rsqrtf(tot) : 0.f;
  for (int c = threadIdx.x; c < d; c += blockDim.x) row[c] *= inv;
}

// Eq. cgee_gate over the generation confidences p_b = conf_b / n_steps
// (Eq. gen_conf), one lane per branch: fires when max_b p >= tau_conf and
// (max - 2nd max) / max >= r_gap. The winner is the smallest index holding the
// maximum; the 2nd max is the largest p among the other branches (0 when there
// is none, so one branch is gated by tau_conf alone). NaN entries are ignored;
// with no valid entry the gate does not fire and winner = -1.
__global__ __launch_bounds__(64) void k_cgee_gate(const float* conf, int B, int n_steps, float tau_conf, float r_gap,
                                                  float* p_mean, int* fired, int* winner, float* stats) {
  const int lane = threadIdx.x;
  const float p = lane < B ? conf[lane] / (float)n_steps : __builtin_nanf("");
  if (p_mean && lane < B) p_mean[lane] = p;
  const bool valid = p == p;
  float m = valid ? p : -INFINITY;
  int idx = valid ? lane : 0x7fffffff;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float om = __shfl_xor(m, off, 64);
    const int oi = __shfl_xor(idx, off, 64);
    if (om > m || (om == m && oi < idx)) {
      m = om;
      idx = oi;
    }
  }
  float q = valid && lane != idx ? p : -INFINITY;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) q = fmaxf(q, __shfl_xor(q, off, 64));
  if (lane == 0) {
    const bool any = idx != 0x7fffffff;
    const float second = q == -INFINITY ? 0.f : q;
    const float gap = any && m > 0.f ? (m - second) / m : 0.f;
    fired[0] = any && m >= tau_conf && gap >= r_gap ? 1 : 0;
    winner[0] = any ? idx : -1;
    if (stats) {
      stats[0] = any ? m : __builtin_nanf("");
      stats[1] = second;
      stats[2] = gap;
    }
  }
}

}  // namespace

hipError_t launch_finalize_decode(const float* parts, int nparts, int B, int* next_token, float* p_top, float* conf,
                                  int accumulate, hipStream_t st) {
  hipLaunchKernelGGL(k_finalize_decode, dim3(B), dim3(256), 0, st, parts, nparts, B, next_token, p_top, conf,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_cgee_gate(const float* conf, int B, int n_steps, float tau_conf, float r_gap, float* p_mean,
                            int* fired, int* winner, float* stats, hipStream_t st) {
  hipLaunchKernelGGL(k_cgee_gate, dim3(1), dim3(64), 0, st, conf, B, n_steps, tau_conf, r_gap, p_mean, fired, winner,
                     stats);
  return hipGetLastError();
}

namespace {
__global__ void k_round_bf16(float* x, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    x[i] = bf16_to_f32(f32_to_bf16_bits(x[i]));
}
}  // namespace

hipError_t launch_round_bf16(float* x, size_t n, hipStream_t st) {
  const size_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(k_round_bf16, dim3(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096), dim3(256), 0, st, x, n);
  return hipGetLastError();
}

hipError_t launch_unit_rows(float* x, int rows, int d, hipStream_t st) {
  hipLaunchKernelGGL(k_unit_rows, dim3(rows), dim3(256), 0, st, x, d);
  return hipGetLastError();
}

hipError_t launch_init(Ctrl* c, int B, int L, float* entropy, int* exit_layer, float* hidden_last,
                       size_t hidden_elems, hipStream_t st) {
  size_t work = hidden_last ? hidden_elems : (size_t)L * B;
  int blocks = (int)((work + 255) / 256);
  blocks = blocks < 1 ? 1 : (blocks > 2048 ? 2048 : blocks);
  hipLaunchKernelGGL(k_init, dim3(blocks), dim3(256), 0, st, c, B, L, entropy, exit_layer, hidden_last,
                     hidden_elems);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* tab, int s, int n, int hd, double base, hipStream_t st) {
  const int total = s * hd / 2;
  hipLaunchKernelGGL(k_rope_table, dim3((total + 255) / 256), dim3(256), 0, st, tab, s, n, hd, base);
  return hipGetLastError();
}

hipError_t launch_embed(DType dt, const void* E, const int* tok, int V, float* x, int rows, int d,
                        hipStream_t st) {
  if (dt == DType::BF16)
    hipLaunchKernelGGL(k_embed<bf16>, dim3(rows), dim3(256), 0, st, static_cast<const bf16*>(E), tok, V, x, d);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3(rows), dim3(256), 0, st, static_cast<const float*>(E), tok, V, x, d);
  return hipGetLastError();
}

hipError_t launch_add_norm(DType dt, const float* x_in, const float* P, int nsplit, size_t split_stride,
                           bool gather, const Ctrl* c, int s, float* x_out, void* xn, const float* gamma, int d,
                           float eps, int max_rows, hipStream_t st, const TapArgs& tap) {
  if (gather && tap.gamma) return hipErrorInvalidValue;   // the tap reads rows in place
  const int chunks = (d / 4 + 1023) / 1024;
#define RKSC_NORM(MAXC, SPLIT)                                                                                   \
  hipLaunchKernelGGL((k_add_norm<MAXC, SPLIT>), dim3(max_rows), dim3(1024), 0, st, x_in, P, nsplit, split_stride, \
                     (int)gather, c, s, x_out, xn, gamma, d, eps, tap)
  const bool sp = dt == DType::BF16;
  if (chunks <= 1) { if (sp) RKSC_NORM(1, true); else RKSC_NORM(1, false); }
  else if (chunks <= 2) { if (sp) RKSC_NORM(2, true); else RKSC_NORM(2, false); }
  else { if (sp) RKSC_NORM(4, true); else RKSC_NORM(4, false); }
#undef RKSC_NORM
  return hipGetLastError();
}

hipError_t launch_qkv_post(const float* P, int nsplit, size_t split_stride, const Ctrl* c, int s, int H,
                           int Hkv, int hd, const float2* rope, float* q, float* k_own, float* v_own,
                           int max_rows, hipStream_t st, DType cache_dt, void* k_cache, void* v_cache, int cap,
                           int off) {
  const int units = (H + 2 * Hkv) * hd / 2;
  const dim3 grid((units + 255) / 256, max_rows);
  if (k_cache && cache_dt == DType::BF16)
    hipLaunchKernelGGL((k_qkv_post<float, bf16>), grid, dim3(256), 0, st, P, nsplit, split_stride, c, s, H, Hkv, hd,
                       rope, q, k_own, v_own, static_cast<bf16*>(k_cache), static_cast<bf16*>(v_cache), cap, off);
  else
    hipLaunchKernelGGL((k_qkv_post<float, float>), grid, dim3(256), 0, st, P, nsplit, split_stride, c, s, H, Hkv,
                       hd, rope, q, k_own, v_own, static_cast<float*>(k_cache), static_cast<float*>(v_cache), cap,
                       off);
  return hipGetLastError();
}

hipError_t launch_swiglu_post(DType dt, const float* P, int nsplit, size_t split_stride, const Ctrl* c, int s,
                              int F, void* a, int max_rows, hipStream_t st) {
  const dim3 grid((F / 4 + 255) / 256, max_rows);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(k_swiglu_post<true>, grid, dim3(256), 0, st, P, nsplit, split_stride, c, s, F, a);
  else
    hipLaunchKernelGGL(k_swiglu_post<false>, grid, dim3(256), 0, st, P, nsplit, split_stride, c, s, F, a);
  return hipGetLastError();
}

hipError_t launch_tap(DType dt, const float* x, const float* P, int nsplit, size_t split_stride, const Ctrl* c,
                      int s, int d, int B, int layer0, float* hidden_last, const float* gamma, float eps,
                      void* hn_a, void* hn_b, int max_branches, hipStream_t st, int jrow) {
  const int chunks = (d / 4 + 1023) / 1024;
#define RKSC_TAP(SPLIT, MAXC)                                                                                   \
  hipLaunchKernelGGL((k_tap<SPLIT, MAXC>), dim3(max_branches), dim3(1024), 0, st, x, P, nsplit, split_stride, c, \
                     s, d, B, layer0, hidden_last, gamma, eps, hn_a, hn_b, jrow)
  if (dt == DType::BF16) {
    if (chunks <= 1) RKSC_TAP(true, 1); else if (chunks <= 2) RKSC_TAP(true, 2); else RKSC_TAP(true, 4);
  } else {
    if (chunks <= 1) RKSC_TAP(false, 1); else if (chunks <= 2) RKSC_TAP(false, 2); else RKSC_TAP(false, 4);
  }
#undef RKSC_TAP
  return hipGetLastError();
}

hipError_t launch_finalize_exit(const float* parts, int nparts, Ctrl* c, int layer1, int kw, int L, int B, float tau,
                                int patience, float* entropy, int* exit_layer, float* hidden_last, int d,
                                hipStream_t st) {
  hipLaunchKernelGGL(k_finalize_exit, dim3(1), dim3(256), 0, st, parts, nparts, c, layer1, kw, L, B, tau, patience,
                     entropy, exit_layer, hidden_last, d);
  return hipGetLastError();
}

}  // namespace rksc
