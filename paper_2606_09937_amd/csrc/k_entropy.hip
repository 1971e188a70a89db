// Fused lm_head -> softmax-entropy statistics (Eq. entropy) for the live
// branches' last-token rows. The logits z = W_lm hn are consumed in registers
// as they are produced: each lane folds its logits into an online triple
// (m = max z, s = sum e^(z-m), t = sum e^(z-m)(z-m)), triples are merged across
// lanes with wavefront shuffles and across waves through LDS, and one triple
// per workgroup and branch is written. Logits never reach HBM. A separate
// single-workgroup kernel merges the per-workgroup triples: H = log s - t/s.
//
// bf16: the kernel streams W_lm [V, d] from HBM exactly once per layer. Each
// wave owns 16*NT vocabulary rows and contracts them against the normalised
// hidden rows with v_mfma_f32_16x16x32_bf16: W rows are the A operand, the
// branches the B columns (NCB blocks of 16). The hidden row is supplied as a
// bf16 hi + lo pair (two MFMAs into one fp32 accumulator), so the product keeps
// ~2^-16 relative accuracy while W_lm stays in its bf16 storage format.
// fp32: a plain wave-per-row dot-product kernel (fp32 models).
#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

constexpr int kEntWaves = 4;

__device__ __forceinline__ void stats_fold(EntStats& st, float mx, const float* z, int cnt) {
  // Fold `cnt` logits (all finite, max mx) into the running triple.
  const float mn = fmaxf(st.m, mx);
  float s_new, t_new;
  if (st.m == -INFINITY) {
    s_new = 0.f;
    t_new = 0.f;
  } else {
    const float dm = st.m - mn;
    const float sc = __expf(dm);
    s_new = st.s * sc;
    t_new = (st.t + st.s * dm) * sc;
  }
  for (int i = 0; i < cnt; ++i) {
    const float dz = z[i] - mn;
    const float e = __expf(dz);
    s_new += e;
    t_new = fmaf(e, dz, t_new);
  }
  st.m = mn;
  st.s = s_new;
  st.t = t_new;
}

// Wave triples -> block triple per column -> parts[block][col].
template <int NCB>
__device__ __forceinline__ void write_block_stats(EntStats (&st)[NCB], int Bl, float* parts) {
  __shared__ EntStats red[kEntWaves][16 * NCB];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    EntStats v = st[cb];
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
      EntStats o{__shfl_xor(v.m, off, 64), __shfl_xor(v.s, off, 64), __shfl_xor(v.t, off, 64)};
      v = ent_merge(v, o);
    }
    if (lane < 16) red[wid][16 * cb + lane] = v;
  }
  __syncthreads();
  const int col = threadIdx.x;
  if (col < 16 * NCB && col < Bl) {
    EntStats v = red[0][col];
    for (int w = 1; w < kEntWaves; ++w) v = ent_merge(v, red[w][col]);
    float* p = parts + ((size_t)blockIdx.x * 64 + col) * 3;
    p[0] = v.m;
    p[1] = v.s;
    p[2] = v.t;
  }
}

// W fragments of one 64-wide K step: NT row tiles, two 16-byte halves each.
template <int NT>
struct WStep {
  uint4 w[NT][2];
};

template <int NCB, int NT>
__global__ __launch_bounds__(256) void k_entropy_bf16(const bf16* __restrict__ W, const bf16* __restrict__ hi,
                                                      const bf16* __restrict__ lo, const Ctrl* c, int V, int d,
                                                      float* __restrict__ parts) {
  const int Bl = c->live_count;
  if (Bl == 0) return;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  constexpr int ROWS = 16 * NT;
  EntStats st[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) st[cb] = ent_empty();
  const uint4 zero = make_uint4(0, 0, 0, 0);
  bool cv[NCB];
  size_t hoff[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int col = 16 * cb + r16;
    cv[cb] = col < Bl;
    hoff[cb] = (size_t)(cv[cb] ? col : 0) * d + 16 * g;
  }

  for (int pass = blockIdx.x * kEntWaves + wid; pass * ROWS < V; pass += gridDim.x * kEntWaves) {
    const int v0 = pass * ROWS;
    const bf16* wrow[NT];
    bool rv[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int row = v0 + 16 * t + r16;
      rv[t] = row < V;
      wrow[t] = W + (size_t)(rv[t] ? row : 0) * d + 16 * g;
    }
    // Lane group g supplies k = k0 + 16g + 8ks + e in substep ks: each row's four
    // lane groups read 128 contiguous bytes per step.
    // Loads always hit valid memory (row clamped to 0, k clamped to the row start)
    // and are never masked, so no predicate forces an early wait on them:
    // weights past d meet zero hidden values, rows past V are left out of the
    // statistics.
    auto load = [&](WStep<NT>& f, int k0) {
      const int ka = k0 + 16 * g < d ? k0 : -16 * g, kb = k0 + 16 * g + 8 < d ? k0 + 8 : -16 * g;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f.w[t][0] = ldg16(wrow[t] + ka);
        f.w[t][1] = ldg16(wrow[t] + kb);
      }
    };
    floatx4 acc[NT][NCB];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[t][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto mma = [&](const WStep<NT>& f, int k0) {
      const bool in0 = k0 + 16 * g < d, in1 = k0 + 16 * g + 8 < d;
      const int ka = in0 ? k0 : -16 * g, kb = in1 ? k0 + 8 : -16 * g;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        // Hidden fragments (hi/lo): a few KB shared by every wave, served by the caches.
        const bool ok0 = cv[cb] && in0, ok1 = cv[cb] && in1;
        const uint4 xh0 = ldg16(hi + hoff[cb] + ka);
        const uint4 xh1 = ldg16(hi + hoff[cb] + kb);
        const uint4 xl0 = ldg16(lo + hoff[cb] + ka);
        const uint4 xl1 = ldg16(lo + hoff[cb] + kb);
        const bf16x8 h0 = __builtin_bit_cast(bf16x8, ok0 ? xh0 : zero);
        const bf16x8 h1 = __builtin_bit_cast(bf16x8, ok1 ? xh1 : zero);
        const bf16x8 l0 = __builtin_bit_cast(bf16x8, ok0 ? xl0 : zero);
        const bf16x8 l1 = __builtin_bit_cast(bf16x8, ok1 ? xl1 : zero);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const bf16x8 a0 = __builtin_bit_cast(bf16x8, f.w[t][0]), a1 = __builtin_bit_cast(bf16x8, f.w[t][1]);
          acc[t][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, h0, acc[t][cb], 0, 0, 0);
          acc[t][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, l0, acc[t][cb], 0, 0, 0);
          acc[t][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, h1, acc[t][cb], 0, 0, 0);
          acc[t][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, l1, acc[t][cb], 0, 0, 0);
        }
      }
    };
    // Two K steps of W in flight: while one step feeds the MFMAs, the next
    // step's loads are outstanding.
    WStep<NT> fa, fb;
    load(fa, 0);
    for (int k0 = 0; k0 < d; k0 += 128) {
      const bool has_b = k0 + 64 < d;
      if (has_b) load(fb, k0 + 64);
      mma(fa, k0);
      if (k0 + 128 < d) load(fa, k0 + 128);
      if (has_b) mma(fb, k0 + 64);
    }
    // Lane (r16, g) holds z[v0 + 16t + 4g + i] for branch column 16cb + r16.
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (v0 + 16 * t + 4 * g + i < V) mx = fmaxf(mx, acc[t][cb][i]);
      if (mx == -INFINITY) continue;
      const float mn = fmaxf(st[cb].m, mx);
      float s_new = 0.f, t_new = 0.f;
      if (st[cb].m != -INFINITY) {
        const float dm = st[cb].m - mn, sc = __expf(dm);
        s_new = st[cb].s * sc;
        t_new = (st[cb].t + st[cb].s * dm) * sc;
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (v0 + 16 * t + 4 * g + i < V) {
            const float dz = acc[t][cb][i] - mn, e = __expf(dz);
            s_new += e;
            t_new = fmaf(e, dz, t_new);
          }
      st[cb] = EntStats{mn, s_new, t_new};
    }
  }
  write_block_stats<NCB>(st, Bl, parts);
}

// fp32 models: each wave takes whole vocabulary rows, lanes stride over d.
__global__ __launch_bounds__(256) void k_entropy_f32(const float* __restrict__ W, const float* __restrict__ hn,
                                                     const Ctrl* c, int V, int d, float* __restrict__ parts) {
  const int Bl = c->live_count;
  if (Bl == 0) return;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  // Branch column `col` is owned by lane `col` (at most 64 branches).
  EntStats own = ent_empty();
  for (int row = blockIdx.x * kEntWaves + wid; row < V; row += gridDim.x * kEntWaves) {
    const float* wr = W + (size_t)row * d;
    for (int col = 0; col < Bl; ++col) {
      const float* hr = hn + (size_t)col * d;
      float acc = 0.f;
      for (int k = lane; k < d; k += 64) acc = fmaf(wr[k], hr[k], acc);
      acc = wave_sum(acc);
      if (lane == col) {
        float z = acc;
        stats_fold(own, z, &z, 1);
      }
    }
  }
  __shared__ EntStats red[kEntWaves][64];
  red[wid][lane] = own;
  __syncthreads();
  const int col = threadIdx.x;
  if (col < Bl) {
    EntStats v = red[0][col];
    for (int w = 1; w < kEntWaves; ++w) v = ent_merge(v, red[w][col]);
    float* p = parts + ((size_t)blockIdx.x * 64 + col) * 3;
    p[0] = v.m;
    p[1] = v.s;
    p[2] = v.t;
  }
}

// Vocabulary rows per wave pass: 64 for up to 16 branches, 32 beyond (register budget).
constexpr int kNT = 4;
constexpr int kNTWide = 2;

}  // namespace

int entropy_parts(DType dt, int V, int max_branches) {
  if (dt == DType::F32) {
    const int b = (V + kEntWaves - 1) / kEntWaves;
    return b < 256 ? b : 256;
  }
  const int rows_per_block = 16 * (max_branches <= 16 ? kNT : kNTWide) * kEntWaves;
  return (V + rows_per_block - 1) / rows_per_block;
}

hipError_t launch_entropy(DType dt, const void* W, const void* hn_a, const void* hn_b, const Ctrl* c, int V, int d,
                          int max_branches, float* parts, hipStream_t st) {
  const int blocks = entropy_parts(dt, V, max_branches);
  if (dt == DType::F32) {
    hipLaunchKernelGGL(k_entropy_f32, dim3(blocks), dim3(256), 0, st, static_cast<const float*>(W),
                       static_cast<const float*>(hn_a), c, V, d, parts);
    return hipGetLastError();
  }
  const bf16* w = static_cast<const bf16*>(W);
  const bf16* a = static_cast<const bf16*>(hn_a);
  const bf16* b = static_cast<const bf16*>(hn_b);
  if (max_branches <= 16)
    hipLaunchKernelGGL((k_entropy_bf16<1, kNT>), dim3(blocks), dim3(256), 0, st, w, a, b, c, V, d, parts);
  else if (max_branches <= 32)
    hipLaunchKernelGGL((k_entropy_bf16<2, kNTWide>), dim3(blocks), dim3(256), 0, st, w, a, b, c, V, d, parts);
  else
    hipLaunchKernelGGL((k_entropy_bf16<4, kNTWide>), dim3(blocks), dim3(256), 0, st, w, a, b, c, V, d, parts);
  return hipGetLastError();
}

}  // namespace rksc
