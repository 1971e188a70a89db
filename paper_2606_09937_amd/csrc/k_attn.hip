// Shared-prefix grouped-query attention of the verify pass.
//
// Query row (branch b, token i, head h) reads every key of the ONE shared prefix
// cache of KV head floor(h/G) (positions 0..n-1) and, causally, its own branch's
// keys 0..i (Sec. 3.2 "KV broadcast and batched decode": the cache is read by
// all branches, never copied per branch). Softmax uses the scale 1/sqrt(hd).
//
// bf16 kernel: one workgroup per (live slot, KV head, 64 query rows); the rows
// are token-major over the G query heads of the group, so every K/V tile staged
// in LDS serves all G heads. Scores are formed transposed, S^T = K Q^T, so that
// each lane owns one query column: the online-softmax statistics stay in the
// lane, and the probabilities are already in the operand layout of
// O^T = V^T P^T (V is staged transposed in LDS). All MFMAs are
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation; softmax runs in fp32.
// Queries, the branch's own keys/values and the probabilities are fp32 values
// carried as bf16 hi + lo pairs: a product with an exact bf16 prefix key/value
// takes two MFMAs (hi, lo), a product of two split values three (hi*hi, hi*lo,
// lo*hi), which keeps every score and output at fp32-level accuracy.
#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

template <int HD>
__global__ __launch_bounds__(256) void k_attn_bf16(const float* __restrict__ q, const bf16* __restrict__ pk,
                                                   const bf16* __restrict__ pv, const float* __restrict__ ko,
                                                   const float* __restrict__ vo, float* __restrict__ o,
                                                   const Ctrl* c, int n, int s, int H, int Hkv, float sl2) {
  constexpr int KT = 64;          // keys per tile
  constexpr int LDK = HD + 8;     // K tile row stride (elements)
  constexpr int LDV = KT + 8;     // V^T row stride (elements)
  constexpr int NC = HD / 32;     // 32-dim chunks of the QK^T contraction
  constexpr int ND = HD / 16;     // 16-dim tiles of the output
  // [0]: the prefix tile (exact bf16) or the hi part of an own-span tile; [1]: its lo part.
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KT * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][HD * LDV];

  const int slot = blockIdx.z;
  if (slot >= c->live_count) return;
  const int kvh = blockIdx.y;
  const int G = H / Hkv;
  const int rows = G * s;
  const int row0 = blockIdx.x * 64;
  if (row0 >= rows) return;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;

  // The query this lane owns as an MFMA column. Rows past the end compute a
  // duplicate of the last row and are not stored.
  const int rho_raw = row0 + 16 * wid + r16;
  const bool qvalid = rho_raw < rows;
  const int rho = qvalid ? rho_raw : rows - 1;
  const int qi = rho / G, h = kvh * G + rho % G;
  const size_t qrow = (size_t)slot * s + qi;
  bf16x8 qh[NC], ql[NC];
#pragma unroll
  for (int cc = 0; cc < NC; ++cc) {
    const float* qp = q + (qrow * H + h) * HD + 32 * cc + 8 * g;
    const float4 a = *reinterpret_cast<const float4*>(qp), b = *reinterpret_cast<const float4*>(qp + 4);
    uint16_t hh[8], ll[8];
    split2(a.x, hh[0], ll[0]); split2(a.y, hh[1], ll[1]); split2(a.z, hh[2], ll[2]); split2(a.w, hh[3], ll[3]);
    split2(b.x, hh[4], ll[4]); split2(b.y, hh[5], ll[5]); split2(b.z, hh[6], ll[6]); split2(b.w, hh[7], ll[7]);
    qh[cc] = __builtin_bit_cast(bf16x8, make_uint4(pack2(hh[0], hh[1]), pack2(hh[2], hh[3]), pack2(hh[4], hh[5]),
                                                   pack2(hh[6], hh[7])));
    ql[cc] = __builtin_bit_cast(bf16x8, make_uint4(pack2(ll[0], ll[1]), pack2(ll[2], ll[3]), pack2(ll[4], ll[5]),
                                                   pack2(ll[6], ll[7])));
  }

  floatx4 oacc[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) oacc[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;

  const bf16* Kp = pk + (size_t)kvh * n * HD;
  const bf16* Vp = pv + (size_t)kvh * n * HD;
  const float* Ko = ko + ((size_t)slot * Hkv + kvh) * s * HD;
  const float* Vo = vo + ((size_t)slot * Hkv + kvh) * s * HD;
  const int i_max = min(s - 1, (min(row0 + 63, rows - 1)) / G);
  const int n_ptiles = (n + KT - 1) / KT;
  const int n_tiles = n_ptiles + i_max / KT + 1;

  for (int t = 0; t < n_tiles; ++t) {
    const bool own = t >= n_ptiles;
    const int kbase = own ? (t - n_ptiles) * KT : t * KT;
    if (!own) {
      // Prefix tile: K rows as stored, V transposed (exact bf16, no split needed).
#pragma unroll
      for (int j = 0; j < KT * HD / 8 / 256; ++j) {
        const int idx = tid + 256 * j, key = idx / (HD / 8), dc = idx % (HD / 8);
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (kbase + key < n) {
          kv = *reinterpret_cast<const uint4*>(Kp + (size_t)(kbase + key) * HD + dc * 8);
          vv = *reinterpret_cast<const uint4*>(Vp + (size_t)(kbase + key) * HD + dc * 8);
        }
        *reinterpret_cast<uint4*>(&Ks[0][key * LDK + dc * 8]) = kv;
        const uint16_t* ve = reinterpret_cast<const uint16_t*>(&vv);
#pragma unroll
        for (int e = 0; e < 8; ++e) Vt[0][(dc * 8 + e) * LDV + key] = ve[e];
      }
    } else {
      // Own-span tile: fp32 keys/values of the branch, split into hi/lo.
#pragma unroll
      for (int j = 0; j < KT * HD / 4 / 256; ++j) {
        const int idx = tid + 256 * j, key = idx / (HD / 4), dq = idx % (HD / 4);
        float4 kf = make_float4(0.f, 0.f, 0.f, 0.f), vf = kf;
        if (kbase + key < s) {
          kf = *reinterpret_cast<const float4*>(Ko + (size_t)(kbase + key) * HD + dq * 4);
          vf = *reinterpret_cast<const float4*>(Vo + (size_t)(kbase + key) * HD + dq * 4);
        }
        uint16_t kh[4], kl[4], vh[4], vl[4];
        split2(kf.x, kh[0], kl[0]); split2(kf.y, kh[1], kl[1]); split2(kf.z, kh[2], kl[2]); split2(kf.w, kh[3], kl[3]);
        split2(vf.x, vh[0], vl[0]); split2(vf.y, vh[1], vl[1]); split2(vf.z, vh[2], vl[2]); split2(vf.w, vh[3], vl[3]);
        *reinterpret_cast<uint2*>(&Ks[0][key * LDK + dq * 4]) = make_uint2(pack2(kh[0], kh[1]), pack2(kh[2], kh[3]));
        *reinterpret_cast<uint2*>(&Ks[1][key * LDK + dq * 4]) = make_uint2(pack2(kl[0], kl[1]), pack2(kl[2], kl[3]));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          Vt[0][(dq * 4 + e) * LDV + key] = vh[e];
          Vt[1][(dq * 4 + e) * LDV + key] = vl[e];
        }
      }
    }
    __syncthreads();

    // S^T: lane holds scores of keys 16*kt + 4g + i for its query.
    floatx4 sc[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      sc[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) {
        const int off = (16 * kt + r16) * LDK + 32 * cc + 8 * g;
        const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(&Ks[0][off]);
        sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qh[cc], sc[kt], 0, 0, 0);
        sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, ql[cc], sc[kt], 0, 0, 0);
        if (own) {
          const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(&Ks[1][off]);
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qh[cc], sc[kt], 0, 0, 0);
        }
      }
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kbase + 16 * kt + 4 * g + i;
        const bool ok = own ? (key <= qi) : (key < n);
        if (!ok) sc[kt][i] = -INFINITY;
        mt = fmaxf(mt, sc[kt][i]);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    // Every query sees key 0 of its first tile, so mn is finite from the first tile on.
    const float mn = fmaxf(m, mt);
    const float alpha = exp2f((m - mn) * sl2);
    m = mn;
    l *= alpha;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) oacc[dt] *= alpha;
    float p[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[kt][i] = exp2f((sc[kt][i] - mn) * sl2);
        l += p[kt][i];
      }
    // O^T += V^T P^T over two 32-key blocks; lane group g supplies keys
    // {32kb + 4g + e, 32kb + 16 + 4g + e}, e = 0..3, in both operands.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      uint16_t ph[8], pl[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        split2(p[2 * kb][e], ph[e], pl[e]);
        split2(p[2 * kb + 1][e], ph[4 + e], pl[4 + e]);
      }
      const bf16x8 pbh = __builtin_bit_cast(bf16x8, make_uint4(pack2(ph[0], ph[1]), pack2(ph[2], ph[3]),
                                                               pack2(ph[4], ph[5]), pack2(ph[6], ph[7])));
      const bf16x8 pbl = __builtin_bit_cast(bf16x8, make_uint4(pack2(pl[0], pl[1]), pack2(pl[2], pl[3]),
                                                               pack2(pl[4], pl[5]), pack2(pl[6], pl[7])));
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const int off = (16 * dt + r16) * LDV + 32 * kb + 4 * g;
        const uint2 a0 = *reinterpret_cast<const uint2*>(&Vt[0][off]);
        const uint2 a1 = *reinterpret_cast<const uint2*>(&Vt[0][off + 16]);
        const bf16x8 v0 = __builtin_bit_cast(bf16x8, make_uint4(a0.x, a0.y, a1.x, a1.y));
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, pbh, oacc[dt], 0, 0, 0);
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, pbl, oacc[dt], 0, 0, 0);
        if (own) {
          const uint2 b0 = *reinterpret_cast<const uint2*>(&Vt[1][off]);
          const uint2 b1 = *reinterpret_cast<const uint2*>(&Vt[1][off + 16]);
          const bf16x8 v1 = __builtin_bit_cast(bf16x8, make_uint4(b0.x, b0.y, b1.x, b1.y));
          oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v1, pbh, oacc[dt], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (qvalid) {
    const float inv = 1.f / l;
    float* orow = o + (qrow * H + h) * HD;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
      *reinterpret_cast<float4*>(orow + 16 * dt + 4 * g) =
          make_float4(oacc[dt][0] * inv, oacc[dt][1] * inv, oacc[dt][2] * inv, oacc[dt][3] * inv);
  }
}

// fp32 models: one thread per (query row, head), plain online softmax.
template <int HD>
__global__ __launch_bounds__(128) void k_attn_f32(const float* __restrict__ q, const float* __restrict__ pk,
                                                  const float* __restrict__ pv, const float* __restrict__ ko,
                                                  const float* __restrict__ vo, float* __restrict__ o,
                                                  const Ctrl* c, int n, int s, int H, int Hkv, float scale) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= c->live_count * s * H) return;
  const int r = idx / H, h = idx % H;
  const int slot = r / s, i = r % s;
  const int kvh = h / (H / Hkv);
  const float* qr = q + ((size_t)r * H + h) * HD;
  float acc[HD];
  for (int d = 0; d < HD; ++d) acc[d] = 0.f;
  float m = -INFINITY, l = 0.f;
  auto visit = [&](const float* kr, const float* vr) {
    float sc = 0.f;
    for (int d = 0; d < HD; ++d) sc = fmaf(qr[d], kr[d], sc);
    sc *= scale;
    const float mn = fmaxf(m, sc);
    const float a = expf(m - mn), p = expf(sc - mn);
    l = l * a + p;
    for (int d = 0; d < HD; ++d) acc[d] = acc[d] * a + p * vr[d];
    m = mn;
  };
  const float* Kp = pk + (size_t)kvh * n * HD;
  const float* Vp = pv + (size_t)kvh * n * HD;
  for (int j = 0; j < n; ++j) visit(Kp + (size_t)j * HD, Vp + (size_t)j * HD);
  const float* Ko = ko + ((size_t)slot * Hkv + kvh) * s * HD;
  const float* Vo = vo + ((size_t)slot * Hkv + kvh) * s * HD;
  for (int j = 0; j <= i; ++j) visit(Ko + (size_t)j * HD, Vo + (size_t)j * HD);
  float* orow = o + ((size_t)r * H + h) * HD;
  for (int d = 0; d < HD; ++d) orow[d] = acc[d] / l;
}

}  // namespace

hipError_t launch_attention(DType dt, const void* q, const void* pk, const void* pv, const void* k_own,
                            const void* v_own, void* o, const Ctrl* c, int n, int s, int H, int Hkv, int hd,
                            int max_branches, hipStream_t st) {
  if (dt == DType::BF16) {
    const float sl2 = 1.4426950408889634f / sqrtf((float)hd);
    const dim3 grid(((H / Hkv) * s + 63) / 64, Hkv, max_branches);
    const float* qq = static_cast<const float*>(q);
    const bf16 *kk = static_cast<const bf16*>(pk), *vv = static_cast<const bf16*>(pv);
    const float *ko = static_cast<const float*>(k_own), *vo = static_cast<const float*>(v_own);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_bf16<128>, grid, dim3(256), 0, st, qq, kk, vv, ko, vo, static_cast<float*>(o), c,
                         n, s, H, Hkv, sl2);
    else
      hipLaunchKernelGGL(k_attn_bf16<64>, grid, dim3(256), 0, st, qq, kk, vv, ko, vo, static_cast<float*>(o), c, n,
                         s, H, Hkv, sl2);
  } else {
    const float scale = 1.f / sqrtf((float)hd);
    const int total = max_branches * s * H;
    const dim3 grid((total + 127) / 128);
    const float *qq = static_cast<const float*>(q), *kk = static_cast<const float*>(pk),
                *vv = static_cast<const float*>(pv), *ko = static_cast<const float*>(k_own),
                *vo = static_cast<const float*>(v_own);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_f32<128>, grid, dim3(128), 0, st, qq, kk, vv, ko, vo, static_cast<float*>(o), c,
                         n, s, H, Hkv, scale);
    else
      hipLaunchKernelGGL(k_attn_f32<64>, grid, dim3(128), 0, st, qq, kk, vv, ko, vo, static_cast<float*>(o), c, n,
                         s, H, Hkv, scale);
  }
  return hipGetLastError();
}

}  // namespace rksc
