// Shared-prefix grouped-query attention of the verify pass.
//
// Query row (branch b, token i, head h) reads every key of the ONE shared prefix
// cache of KV head floor(h/G) (positions 0..n-1) and, causally, its own branch's
// keys 0..i (Sec. 2.2 "KV broadcast and batched decode": the cache is read by
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

// a if c, else zero; component-wise so that no address is selected (a select
// of struct lvalues keeps register arrays in scratch memory).
__device__ __forceinline__ uint4 keep_if(bool c, const uint4& a) {
  return make_uint4(c ? a.x : 0u, c ? a.y : 0u, c ? a.z : 0u, c ? a.w : 0u);
}

// V^T tile layout: row = head dimension, column = key. The 4-key group of a
// row is XOR-swizzled by the row's 8-dimension block so that the packed stores
// (4 keys of one dimension) and the fragment reads are bank-conflict free.
__device__ __forceinline__ int vt_col(int dim, int key) { return key ^ (((dim >> 3) & 15) << 2); }

// Split-KV: the key tiles of a query tile -- the prefix tiles, then the own-span
// tiles up to its last query -- are divided evenly over `nchunks` workgroups,
// each writing an unnormalised partial output with its (max, sum) for
// k_attn_combine. (A merge by the last chunk to finish, found with an atomic
// ticket, needs device-scope release fences; on MI355X those write back the
// whole L2 and cost far more than the separate combine launch.)
// Tile loads are software-pipelined: the next tile's K/V (own-span tiles: K)
// are fetched into registers while the current tile is contracted; the masking
// and the hi/lo split happen when they are stored to LDS.
template <int HD>
__global__ __launch_bounds__(256, 2) void k_attn_bf16(const float* __restrict__ q, const bf16* __restrict__ pk,
                                                   const bf16* __restrict__ pv, const float* __restrict__ ko,
                                                   const float* __restrict__ vo, void* __restrict__ o,
                                                   float* __restrict__ opart, float* __restrict__ mlpart,
                                                   const Ctrl* c, int n, int s, int H, int Hkv, float sl2,
                                                   int nchunks, int max_rows) {
  constexpr int KT = 64;          // keys per tile
  constexpr int LDK = HD + 8;     // K tile row stride (elements)
  constexpr int LDV = KT + 8;     // V^T row stride (elements)
  constexpr int NC = HD / 32;     // 32-dim chunks of the QK^T contraction
  constexpr int ND = HD / 16;     // 16-dim tiles of the output
  // Register staging per thread: prefix tile (bf16) K in 16-byte row chunks and
  // V in units of 4 keys x 8 dimensions; own-span tile (fp32) K in 16-byte
  // chunks (4 dimensions); own-span V goes in units of 4 keys x 4 dimensions.
  constexpr int PK = KT * HD / 8 / 256;                  // K chunks per thread, prefix
  constexpr int PVU = (KT * HD / 32 + 255) / 256;        // V units per thread, prefix
  constexpr int OK = KT * HD / 4 / 256;                  // K chunks per thread, own span
  constexpr int OVU = (KT * HD / 16 + 255) / 256;        // V units per thread, own span
  // Own-span V is loaded when the tile is stored (2 of the ~n/64 + 2 tiles), which
  // keeps the staging at 8 registers x 16 B.
  constexpr int NSTAGE = (PK + 4 * PVU) > OK ? (PK + 4 * PVU) : OK;
  static_assert(KT * HD / 8 % 256 == 0 && KT * HD / 4 % 256 == 0, "tile staging assumes 256 threads");
  // [0]: the prefix tile (exact bf16) or the hi part of an own-span tile; [1]: its lo part.
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KT * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][HD * LDV];

  const int B_slots = gridDim.z / nchunks;
  const int slot = blockIdx.z % B_slots;
  const int chunk = blockIdx.z / B_slots;
  if (slot >= c->live_count) return;
  const int kvh = blockIdx.y;
  const int G = H / Hkv;
  const int rows = G * s;
  const int row0 = blockIdx.x * 64;
  if (row0 >= rows) return;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;

  const int i_max = min(s - 1, (min(row0 + 63, rows - 1)) / G);
  const int n_ptiles = (n + KT - 1) / KT;
  const int n_tiles = n_ptiles + i_max / KT + 1;
  const int t_begin = chunk * n_tiles / nchunks, t_end = (chunk + 1) * n_tiles / nchunks;

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

  // Fetch of tile t into registers (addresses clamped in bounds; out-of-range
  // keys are zeroed when stored).
  uint4 stg[NSTAGE];
  auto fetch = [&](int t) {
    if (t < n_ptiles) {
      const int kbase = t * KT;
#pragma unroll
      for (int j = 0; j < PK; ++j) {
        const int idx = tid + 256 * j, key = kbase + idx / (HD / 8), dc = idx % (HD / 8);
        stg[j] = ldg16(Kp + (size_t)(key < n ? key : 0) * HD + dc * 8);
      }
#pragma unroll
      for (int u = 0; u < PVU; ++u) {
        const int idx = tid + 256 * u;
        const int dc = idx % (HD / 8), kg = (idx < KT * HD / 32 ? idx : 0) / (HD / 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = kbase + 4 * kg + e;
          stg[PK + 4 * u + e] = ldg16(Vp + (size_t)(key < n ? key : 0) * HD + dc * 8);
        }
      }
    } else {
      const int kbase = (t - n_ptiles) * KT;
#pragma unroll
      for (int j = 0; j < OK; ++j) {
        const int idx = tid + 256 * j, key = kbase + idx / (HD / 4), dq = idx % (HD / 4);
        stg[j] = ldg16(Ko + (size_t)(key < s ? key : 0) * HD + dq * 4);
      }
    }
  };
  // Store of the fetched tile t to LDS: K rows and V^T, own-span tiles split into hi/lo.
  auto store = [&](int t) {
    if (t < n_ptiles) {
      const int kbase = t * KT;
#pragma unroll
      for (int j = 0; j < PK; ++j) {
        const int idx = tid + 256 * j, key = idx / (HD / 8), dc = idx % (HD / 8);
        *reinterpret_cast<uint4*>(&Ks[0][key * LDK + dc * 8]) = keep_if(kbase + key < n, stg[j]);
      }
#pragma unroll
      for (int u = 0; u < PVU; ++u) {
        const int idx = tid + 256 * u;
        if (idx < KT * HD / 32) {
          const int dc = idx % (HD / 8), kg = idx / (HD / 8);
          uint32_t w[4][4];   // w[e][j]: word j (elements 2j, 2j+1) of key 4kg + e
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint4 v = keep_if(kbase + 4 * kg + e < n, stg[PK + 4 * u + e]);
            w[e][0] = v.x; w[e][1] = v.y; w[e][2] = v.z; w[e][3] = v.w;
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // elements 2j (low halves) and 2j+1 (high halves) of the four keys
            const uint32_t lo01 = (w[0][j] & 0xffffu) | (w[1][j] << 16);
            const uint32_t lo23 = (w[2][j] & 0xffffu) | (w[3][j] << 16);
            const uint32_t hi01 = (w[0][j] >> 16) | (w[1][j] & 0xffff0000u);
            const uint32_t hi23 = (w[2][j] >> 16) | (w[3][j] & 0xffff0000u);
            const int d0 = dc * 8 + 2 * j, d1 = d0 + 1;
            *reinterpret_cast<uint2*>(&Vt[0][d0 * LDV + vt_col(d0, 4 * kg)]) = make_uint2(lo01, lo23);
            *reinterpret_cast<uint2*>(&Vt[0][d1 * LDV + vt_col(d1, 4 * kg)]) = make_uint2(hi01, hi23);
          }
        }
      }
    } else {
      const int kbase = (t - n_ptiles) * KT;
#pragma unroll
      for (int j = 0; j < OK; ++j) {
        const int idx = tid + 256 * j, key = idx / (HD / 4), dq = idx % (HD / 4);
        const float4 kf = __builtin_bit_cast(float4, keep_if(kbase + key < s, stg[j]));
        uint16_t kh[4], kl[4];
        split2(kf.x, kh[0], kl[0]); split2(kf.y, kh[1], kl[1]); split2(kf.z, kh[2], kl[2]); split2(kf.w, kh[3], kl[3]);
        *reinterpret_cast<uint2*>(&Ks[0][key * LDK + dq * 4]) = make_uint2(pack2(kh[0], kh[1]), pack2(kh[2], kh[3]));
        *reinterpret_cast<uint2*>(&Ks[1][key * LDK + dq * 4]) = make_uint2(pack2(kl[0], kl[1]), pack2(kl[2], kl[3]));
      }
#pragma unroll
      for (int u = 0; u < OVU; ++u) {
        const int idx = tid + 256 * u;
        if (idx < KT * HD / 16) {
          const int dq = idx % (HD / 4), kg = idx / (HD / 4);
          float x[4][4];   // x[e][k]: dimension 4dq + k of key 4kg + e
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = kbase + 4 * kg + e;
            const bool ok = key < s;
            const uint4 v = ldg16(Vo + (size_t)(ok ? key : 0) * HD + dq * 4);
            x[e][0] = ok ? __uint_as_float(v.x) : 0.f;
            x[e][1] = ok ? __uint_as_float(v.y) : 0.f;
            x[e][2] = ok ? __uint_as_float(v.z) : 0.f;
            x[e][3] = ok ? __uint_as_float(v.w) : 0.f;
          }
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int dim = dq * 4 + k;
            uint16_t hh[4], lw[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) split2(x[e][k], hh[e], lw[e]);
            const int col = vt_col(dim, 4 * kg);
            *reinterpret_cast<uint2*>(&Vt[0][dim * LDV + col]) = make_uint2(pack2(hh[0], hh[1]), pack2(hh[2], hh[3]));
            *reinterpret_cast<uint2*>(&Vt[1][dim * LDV + col]) = make_uint2(pack2(lw[0], lw[1]), pack2(lw[2], lw[3]));
          }
        }
      }
    }
  };

  if (t_begin < t_end) fetch(t_begin);
  for (int t = t_begin; t < t_end; ++t) {
    const bool own = t >= n_ptiles;
    const int kbase = own ? (t - n_ptiles) * KT : t * KT;
    store(t);
    __syncthreads();
    if (t + 1 < t_end) fetch(t + 1);   // in flight while this tile is contracted

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
    // A query may see no key in this chunk so far (an own-span tile past it):
    // then mn = -inf and everything stays zero.
    const float mn = fmaxf(m, mt);
    const float alpha = m == -INFINITY ? 0.f : exp2f((m - mn) * sl2);
    m = mn;
    l *= alpha;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) oacc[dt] *= alpha;
    float p[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[kt][i] = mn == -INFINITY ? 0.f : exp2f((sc[kt][i] - mn) * sl2);
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
        const int dim = 16 * dt + r16;
        const int off0 = dim * LDV + vt_col(dim, 32 * kb + 4 * g);
        const int off1 = dim * LDV + vt_col(dim, 32 * kb + 16 + 4 * g);
        const uint2 a0 = *reinterpret_cast<const uint2*>(&Vt[0][off0]);
        const uint2 a1 = *reinterpret_cast<const uint2*>(&Vt[0][off1]);
        const bf16x8 v0 = __builtin_bit_cast(bf16x8, make_uint4(a0.x, a0.y, a1.x, a1.y));
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, pbh, oacc[dt], 0, 0, 0);
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, pbl, oacc[dt], 0, 0, 0);
        if (own) {
          const uint2 b0 = *reinterpret_cast<const uint2*>(&Vt[1][off0]);
          const uint2 b1 = *reinterpret_cast<const uint2*>(&Vt[1][off1]);
          const bf16x8 v1 = __builtin_bit_cast(bf16x8, make_uint4(b0.x, b0.y, b1.x, b1.y));
          oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v1, pbh, oacc[dt], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  const size_t plane = (size_t)max_rows * H * HD;
  if (nchunks == 1) {
    if (!qvalid) return;
    // The output feeds the O projection: bf16 hi/lo planes [max_rows, H*hd] each.
    const float inv = 1.f / l;
    bf16* ob = reinterpret_cast<bf16*>(o);
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) {
      uint16_t h4[4], l4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) split2(oacc[dt][i] * inv, h4[i], l4[i]);
      const size_t idx = (qrow * H + h) * HD + 16 * dt + 4 * g;
      *reinterpret_cast<uint2*>(ob + idx) = make_uint2(pack2(h4[0], h4[1]), pack2(h4[2], h4[3]));
      *reinterpret_cast<uint2*>(ob + plane + idx) = make_uint2(pack2(l4[0], l4[1]), pack2(l4[2], l4[3]));
    }
    return;
  }
  // Unnormalised partial output and its (max, sum) for the combine kernel.
  if (!qvalid) return;
  const size_t prow = ((size_t)chunk * max_rows + qrow) * H + h;
  float* orow = opart + prow * HD;
#pragma unroll
  for (int dt = 0; dt < ND; ++dt)
    *reinterpret_cast<float4*>(orow + 16 * dt + 4 * g) = make_float4(oacc[dt][0], oacc[dt][1], oacc[dt][2], oacc[dt][3]);
  if (g == 0) *reinterpret_cast<float2*>(mlpart + prow * 2) = make_float2(m, l);
}

// Merges the split-KV partials of each (row, head):
// o = sum_c e^{(m_c - M) sl} o_c / sum_c e^{(m_c - M) sl} l_c, M = max_c m_c.
// A chunk that saw no key for a query (m = -inf) contributes nothing.
template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine(const float* __restrict__ opart, const float* __restrict__ mlpart,
                                                      void* __restrict__ o, const Ctrl* c, int s, int H, float sl2,
                                                      int nchunks, int max_rows) {
  const int rows = c->live_count * s * H;
  const int wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  if (wid >= rows) return;    // one wave per (row, head)
  float M = -INFINITY;
  for (int ch = 0; ch < nchunks; ++ch) M = fmaxf(M, mlpart[((size_t)ch * max_rows * H + wid) * 2]);
  float den = 0.f;
  float acc[HD / 64];
#pragma unroll
  for (int j = 0; j < HD / 64; ++j) acc[j] = 0.f;
  for (int ch = 0; ch < nchunks; ++ch) {
    const float2 ml = *reinterpret_cast<const float2*>(mlpart + ((size_t)ch * max_rows * H + wid) * 2);
    if (ml.x == -INFINITY) continue;
    const float w = exp2f((ml.x - M) * sl2);
    den += w * ml.y;
    const float* op = opart + ((size_t)ch * max_rows * H + wid) * HD;
#pragma unroll
    for (int j = 0; j < HD / 64; ++j) acc[j] += w * op[lane + 64 * j];
  }
  // bf16 hi/lo planes of the output, as in the single-chunk path.
  const float inv = 1.f / den;
  const size_t plane = (size_t)max_rows * H * HD;
  uint16_t* ob = reinterpret_cast<uint16_t*>(o);
#pragma unroll
  for (int j = 0; j < HD / 64; ++j) {
    uint16_t hb, lb;
    split2(acc[j] * inv, hb, lb);
    ob[(size_t)wid * HD + lane + 64 * j] = hb;
    ob[plane + (size_t)wid * HD + lane + 64 * j] = lb;
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

int attention_chunks(DType dt, int B, int n, int s, int H, int Hkv) {
  if (dt != DType::BF16 || n == 0) return 1;
  const int base = ((H / Hkv) * s + 63) / 64 * Hkv * B;
  // Tiles of the smallest query tile: every chunk gets at least one.
  const int min_tiles = (n + 63) / 64 + 1;
  int chunks = 1;
  // Split the keys until the launch has about two workgroups per CU.
  while (base * chunks < 512 && chunks < min_tiles) ++chunks;
  return chunks;
}

hipError_t launch_attention(DType dt, const void* q, const void* pk, const void* pv, const void* k_own,
                            const void* v_own, void* o, float* opart, float* mlpart, int nchunks, const Ctrl* c,
                            int n, int s, int H, int Hkv, int hd, int max_branches, hipStream_t st) {
  if (dt == DType::BF16) {
    const float sl2 = 1.4426950408889634f / sqrtf((float)hd);
    const dim3 grid(((H / Hkv) * s + 63) / 64, Hkv, max_branches * nchunks);
    const int max_rows = max_branches * s;
    const float* qq = static_cast<const float*>(q);
    const bf16 *kk = static_cast<const bf16*>(pk), *vv = static_cast<const bf16*>(pv);
    const float *ko = static_cast<const float*>(k_own), *vo = static_cast<const float*>(v_own);
    void* oo = o;
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_bf16<128>, grid, dim3(256), 0, st, qq, kk, vv, ko, vo, oo, opart, mlpart, c, n, s, H,
                         Hkv, sl2, nchunks, max_rows);
    else
      hipLaunchKernelGGL(k_attn_bf16<64>, grid, dim3(256), 0, st, qq, kk, vv, ko, vo, oo, opart, mlpart, c, n, s, H,
                         Hkv, sl2, nchunks, max_rows);
    if (nchunks > 1) {
      const int waves = max_rows * H;
      const dim3 cgrid((waves * 64 + 255) / 256);
      if (hd == 128)
        hipLaunchKernelGGL(k_attn_combine<128>, cgrid, dim3(256), 0, st, opart, mlpart, oo, c, s, H, sl2, nchunks,
                           max_rows);
      else
        hipLaunchKernelGGL(k_attn_combine<64>, cgrid, dim3(256), 0, st, opart, mlpart, oo, c, s, H, sl2, nchunks,
                           max_rows);
    }
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
