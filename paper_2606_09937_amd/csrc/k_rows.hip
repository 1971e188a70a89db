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

// ------------------------------------------------------------------ add + RMSNorm

template <typename T>
__global__ __launch_bounds__(256) void k_add_norm(const float* x_in, const float* P, int nsplit,
                                                  size_t split_stride, int gather, const Ctrl* c, int s,
                                                  float* x_out, T* xn, const float* gamma, int d, float eps) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  if (r >= c->live_count * s) return;
  const int src = gather ? c->gather_src[r / s] * s + (r % s) : r;
  const float* xi = x_in + (size_t)src * d;
  float* xo = x_out + (size_t)r * d;
  float ss = 0.f;
  for (int col = threadIdx.x * 4; col < d; col += blockDim.x * 4) {
    float4 v = *reinterpret_cast<const float4*>(xi + col);
    for (int sp = 0; sp < nsplit; ++sp) {
      const float4 p = *reinterpret_cast<const float4*>(P + sp * split_stride + (size_t)src * d + col);
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    *reinterpret_cast<float4*>(xo + col) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float tot = block_sum(ss, red);
  const float rinv = rsqrtf(tot / (float)d + eps);
  T* xr = xn + (size_t)r * d;
  for (int col = threadIdx.x * 4; col < d; col += blockDim.x * 4) {
    const float4 v = *reinterpret_cast<const float4*>(xo + col);
    const float4 g = *reinterpret_cast<const float4*>(gamma + col);
    store4(xr + col, g.x * v.x * rinv, g.y * v.y * rinv, g.z * v.z * rinv, g.w * v.w * rinv);
  }
}

// ------------------------------------------------------------------ QKV epilogue

// One block per row. Pair unit u covers columns (hh*hd + j, hh*hd + j + hd/2) of
// head hh of the [q | k | v] output; q and k pairs are rotated by RoPE.
template <typename T>
__global__ __launch_bounds__(256) void k_qkv_post(const float* P, int nsplit, size_t split_stride,
                                                  const Ctrl* c, int s, int H, int Hkv, int hd,
                                                  const float2* rope, T* q, T* k_own, T* v_own) {
  const int r = blockIdx.x;
  if (r >= c->live_count * s) return;
  const int slot = r / s, i = r % s;
  const int half = hd / 2;
  const int N = (H + 2 * Hkv) * hd;
  const int units = (H + 2 * Hkv) * half;
  const float* pr = P + (size_t)r * N;
  for (int u = threadIdx.x; u < units; u += blockDim.x) {
    const int hh = u / half, j = u % half;
    const int c1 = hh * hd + j, c2 = c1 + half;
    float x1 = 0.f, x2 = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) {
      x1 += pr[sp * split_stride + c1];
      x2 += pr[sp * split_stride + c2];
    }
    if (hh < H + Hkv) {
      const float2 cs = rope[i * half + j];
      const float y1 = x1 * cs.x - x2 * cs.y;
      const float y2 = x2 * cs.x + x1 * cs.y;
      x1 = y1;
      x2 = y2;
    }
    T* dst;
    if (hh < H) {
      dst = q + ((size_t)r * H + hh) * hd;
    } else if (hh < H + Hkv) {
      dst = k_own + (((size_t)slot * Hkv + (hh - H)) * s + i) * hd;
    } else {
      dst = v_own + (((size_t)slot * Hkv + (hh - H - Hkv)) * s + i) * hd;
    }
    dst[j] = from_f32<T>(x1);
    dst[j + half] = from_f32<T>(x2);
  }
}

// ------------------------------------------------------------------ SwiGLU epilogue

template <typename T>
__global__ __launch_bounds__(256) void k_swiglu_post(const float* P, int nsplit, size_t split_stride,
                                                     const Ctrl* c, int s, int F, T* a) {
  const int r = blockIdx.x;
  if (r >= c->live_count * s) return;
  const float* pr = P + (size_t)r * 2 * F;
  T* ar = a + (size_t)r * F;
  for (int f = threadIdx.x; f < F; f += blockDim.x) {
    float g = 0.f, u = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) {
      g += pr[sp * split_stride + f];
      u += pr[sp * split_stride + F + f];
    }
    const float silu = g / (1.f + expf(-g));
    ar[f] = from_f32<T>(silu * u);
  }
}

// ------------------------------------------------------------------ last-token tap

template <bool kSplitBf16>
__global__ __launch_bounds__(256) void k_tap(const float* x, const float* P, int nsplit, size_t split_stride,
                                             const Ctrl* c, int s, int d, int B, int layer0,
                                             float* hidden_last, const float* gamma, float eps, void* hn_a,
                                             void* hn_b) {
  __shared__ float red[16];
  const int slot = blockIdx.x;
  if (slot >= c->live_count) return;
  const int branch = c->live_idx[slot];
  const size_t row = (size_t)slot * s + (s - 1);
  float ss = 0.f;
  for (int col = threadIdx.x * 4; col < d; col += blockDim.x * 4) {
    float4 v = *reinterpret_cast<const float4*>(x + row * d + col);
    for (int sp = 0; sp < nsplit; ++sp) {
      const float4 p = *reinterpret_cast<const float4*>(P + sp * split_stride + row * d + col);
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    if (hidden_last)
      *reinterpret_cast<float4*>(hidden_last + ((size_t)layer0 * B + branch) * d + col) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float tot = block_sum(ss, red);
  const float rinv = rsqrtf(tot / (float)d + eps);
  for (int col = threadIdx.x * 4; col < d; col += blockDim.x * 4) {
    // Second pass recomputes h (same additions in the same order, so the same value).
    float4 v = *reinterpret_cast<const float4*>(x + row * d + col);
    for (int sp = 0; sp < nsplit; ++sp) {
      const float4 p = *reinterpret_cast<const float4*>(P + sp * split_stride + row * d + col);
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    const float4 g = *reinterpret_cast<const float4*>(gamma + col);
    const float h0 = g.x * v.x * rinv, h1 = g.y * v.y * rinv, h2 = g.z * v.z * rinv, h3 = g.w * v.w * rinv;
    if (kSplitBf16) {
      // hn = hi + lo with hi = bf16(hn) and lo = bf16(hn - hi): the lm_head product
      // then runs on bf16 MFMA with ~2^-16 relative error on the activation.
      bf16* hi = static_cast<bf16*>(hn_a) + (size_t)slot * d + col;
      bf16* lo = static_cast<bf16*>(hn_b) + (size_t)slot * d + col;
      const uint16_t b0 = f32_to_bf16_bits(h0), b1 = f32_to_bf16_bits(h1);
      const uint16_t b2 = f32_to_bf16_bits(h2), b3 = f32_to_bf16_bits(h3);
      store4(hi, bf16_to_f32(b0), bf16_to_f32(b1), bf16_to_f32(b2), bf16_to_f32(b3));
      store4(lo, h0 - bf16_to_f32(b0), h1 - bf16_to_f32(b1), h2 - bf16_to_f32(b2), h3 - bf16_to_f32(b3));
    } else {
      store4(static_cast<float*>(hn_a) + (size_t)slot * d + col, h0, h1, h2, h3);
    }
  }
}

// ------------------------------------------------------------------ entropy merge + exit rule

__global__ __launch_bounds__(256) void k_finalize_exit(const float* parts, int nparts, Ctrl* c, int layer1,
                                                       int L, int B, float tau, int patience, float* entropy,
                                                       int* exit_layer) {
  __shared__ EntStats red[256];
  const int Bl = c->live_count;
  if (Bl == 0) return;
  const int tid = threadIdx.x;
  for (int col = 0; col < Bl; ++col) {
    EntStats st = ent_empty();
    for (int p = tid; p < nparts; p += blockDim.x) {
      const float* q = parts + ((size_t)p * 64 + col) * 3;
      st = ent_merge(st, EntStats{q[0], q[1], q[2]});
    }
    red[tid] = st;
    __syncthreads();
    for (int off = blockDim.x / 2; off > 0; off >>= 1) {
      if (tid < off) red[tid] = ent_merge(red[tid], red[tid + off]);
      __syncthreads();
    }
    if (tid == 0) c->h_cur[col] = logf(red[0].s) - red[0].t / red[0].s;
    __syncthreads();
  }
  if (tid < 64) {
    const int slot = tid;
    const bool live = slot < Bl;
    int branch = -1;
    bool keep = false;
    if (live) {
      branch = c->live_idx[slot];
      const float H = c->h_cur[slot];
      const float delta = fabsf(H - c->h_prev[branch]);      // H_0 = +inf
      const int streak = (delta < tau) ? c->streak[branch] + 1 : 0;
      c->streak[branch] = streak;
      c->h_prev[branch] = H;
      entropy[(size_t)(layer1 - 1) * B + branch] = H;
      const bool exits = streak >= patience;
      if (exits) exit_layer[branch] = layer1;
      keep = !exits && layer1 < L;
    }
    const unsigned long long mask = __ballot(keep);
    if (keep) {
      const int ns = __popcll(mask & ((1ull << slot) - 1ull));
      c->gather_src[ns] = slot;
      c->live_idx[ns] = branch;
    }
    if (slot == 0) c->live_count = __popcll(mask);
  }
}

}  // namespace

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

hipError_t launch_add_norm(const float* x_in, const float* P, int nsplit, size_t split_stride, bool gather,
                           const Ctrl* c, int s, float* x_out, float* xn, const float* gamma, int d, float eps,
                           int max_rows, hipStream_t st) {
  hipLaunchKernelGGL(k_add_norm<float>, dim3(max_rows), dim3(256), 0, st, x_in, P, nsplit, split_stride,
                     (int)gather, c, s, x_out, xn, gamma, d, eps);
  return hipGetLastError();
}

hipError_t launch_qkv_post(const float* P, int nsplit, size_t split_stride, const Ctrl* c, int s, int H,
                           int Hkv, int hd, const float2* rope, float* q, float* k_own, float* v_own,
                           int max_rows, hipStream_t st) {
  hipLaunchKernelGGL(k_qkv_post<float>, dim3(max_rows), dim3(256), 0, st, P, nsplit, split_stride, c, s, H, Hkv,
                     hd, rope, q, k_own, v_own);
  return hipGetLastError();
}

hipError_t launch_swiglu_post(const float* P, int nsplit, size_t split_stride, const Ctrl* c, int s, int F,
                              float* a, int max_rows, hipStream_t st) {
  hipLaunchKernelGGL(k_swiglu_post<float>, dim3(max_rows), dim3(256), 0, st, P, nsplit, split_stride, c, s, F, a);
  return hipGetLastError();
}

hipError_t launch_tap(DType dt, const float* x, const float* P, int nsplit, size_t split_stride, const Ctrl* c,
                      int s, int d, int B, int layer0, float* hidden_last, const float* gamma, float eps,
                      void* hn_a, void* hn_b, int max_branches, hipStream_t st) {
  if (dt == DType::BF16)
    hipLaunchKernelGGL(k_tap<true>, dim3(max_branches), dim3(256), 0, st, x, P, nsplit, split_stride, c, s, d, B,
                       layer0, hidden_last, gamma, eps, hn_a, hn_b);
  else
    hipLaunchKernelGGL(k_tap<false>, dim3(max_branches), dim3(256), 0, st, x, P, nsplit, split_stride, c, s, d,
                       B, layer0, hidden_last, gamma, eps, hn_a, hn_b);
  return hipGetLastError();
}

hipError_t launch_finalize_exit(const float* parts, int nparts, Ctrl* c, int layer1, int L, int B, float tau,
                                int patience, float* entropy, int* exit_layer, hipStream_t st) {
  hipLaunchKernelGGL(k_finalize_exit, dim3(1), dim3(256), 0, st, parts, nparts, c, layer1, L, B, tau, patience,
                     entropy, exit_layer);
  return hipGetLastError();
}

}  // namespace rksc
