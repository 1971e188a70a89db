// Dense projections of the decoder layer: P[split][m][n] = sum_k A[m][k] * W[n][k]
// over the split's K range. A is the fp32 [rows, K] activation, W a [N, K]
// weight (torch Linear layout) in the model's storage type, P fp32. Split
// partials are summed by the consumer.
//
// bf16 weights: CDNA4 MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulate), LDS
// double buffered; both operands are K-contiguous, so every lane reads its
// fragment as one 16-byte LDS load.
// fp32 weights: a plain LDS-tiled FMA kernel.
#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

// bf16 weights W [N, K] times fp32 activations A [rows, K]. A is split into
// bf16 hi/lo tiles when it is staged into LDS, and every W fragment meets both
// (two v_mfma_f32_16x16x32_bf16 into one fp32 accumulator), so the product
// keeps fp32-level accuracy at twice the bf16 MFMA work.
template <int BM, int BN>
__global__ __launch_bounds__(256) void k_gemm_bf16(const float* __restrict__ A, const bf16* __restrict__ W,
                                                   float* __restrict__ P, size_t split_stride, const Ctrl* c,
                                                   int s, int max_rows, int N, int K, int kps) {
  constexpr int BK = 32, LDK = BK + 8;   // 80-byte LDS rows: conflict-free 16-byte fragment reads
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
  constexpr int AC = BM * 8 / 256;   // float4 chunks of A per thread per stage
  constexpr int WC = BN * 4 / 256;   // 16-byte chunks of W per thread per stage
  static_assert(AC >= 1 && WC >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) uint16_t Ah[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Al[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[2][BN * LDK];

  const int Ml = c ? min(c->live_count * s, max_rows) : max_rows;
  const int m0 = blockIdx.y * BM;
  if (m0 >= Ml) return;
  const int n0 = blockIdx.x * BN;
  const int kb = blockIdx.z * kps;
  const int ke = min(K, kb + kps);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm0 = (wid >> 1) * WM, wn0 = (wid & 1) * WN;
  const int r16 = lane & 15, g = lane >> 4;

  float4 ra[AC];
  uint4 rw[WC];
  auto gload = [&](int k0) {
#pragma unroll
    for (int j = 0; j < AC; ++j) {
      const int idx = tid + 256 * j, row = idx >> 3, gk = k0 + (idx & 7) * 4, gr = m0 + row;
      ra[j] = (gr < Ml && gk < ke) ? *reinterpret_cast<const float4*>(A + (size_t)gr * K + gk)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < WC; ++j) {
      const int idx = tid + 256 * j, row = idx >> 2, gk = k0 + (idx & 3) * 8, gr = n0 + row;
      rw[j] = (gr < N && gk < ke) ? *reinterpret_cast<const uint4*>(W + (size_t)gr * K + gk)
                                  : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < AC; ++j) {
      const int idx = tid + 256 * j, off = (idx >> 3) * LDK + (idx & 7) * 4;
      uint16_t h0, l0, h1, l1, h2, l2, h3, l3;
      split2(ra[j].x, h0, l0);
      split2(ra[j].y, h1, l1);
      split2(ra[j].z, h2, l2);
      split2(ra[j].w, h3, l3);
      *reinterpret_cast<uint2*>(&Ah[buf][off]) =
          make_uint2((uint32_t)h0 | ((uint32_t)h1 << 16), (uint32_t)h2 | ((uint32_t)h3 << 16));
      *reinterpret_cast<uint2*>(&Al[buf][off]) =
          make_uint2((uint32_t)l0 | ((uint32_t)l1 << 16), (uint32_t)l2 | ((uint32_t)l3 << 16));
    }
#pragma unroll
    for (int j = 0; j < WC; ++j) {
      const int idx = tid + 256 * j;
      *reinterpret_cast<uint4*>(&Ws[buf][(idx >> 2) * LDK + (idx & 3) * 8]) = rw[j];
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  gload(kb);
  sstore(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = kb; k0 < ke; k0 += BK) {
    const bool more = k0 + BK < ke;
    if (more) gload(k0 + BK);
    bf16x8 ah[TM], al[TM], bw[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int off = (wm0 + 16 * tm + r16) * LDK + 8 * g;
      ah[tm] = *reinterpret_cast<const bf16x8*>(&Ah[buf][off]);
      al[tm] = *reinterpret_cast<const bf16x8*>(&Al[buf][off]);
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
      bw[tn] = *reinterpret_cast<const bf16x8*>(&Ws[buf][(wn0 + 16 * tn + r16) * LDK + 8 * g]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[tm], bw[tn], acc[tm][tn], 0, 0, 0);
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[tm], bw[tn], acc[tm][tn], 0, 0, 0);
      }
    if (more) sstore(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // Lane (r16, g) holds C[4g + i][r16] of each 16x16 tile.
  float* out = P + blockIdx.z * split_stride;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col = n0 + wn0 + 16 * tn + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + wm0 + 16 * tm + 4 * g + i;
        if (row < Ml && col < N) out[(size_t)row * N + col] = acc[tm][tn][i];
      }
    }
}

__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, const float* __restrict__ W,
                                                  float* __restrict__ P, size_t split_stride, const Ctrl* c,
                                                  int s, int max_rows, int N, int K, int kps) {
  constexpr int T = 64, BK = 16;
  __shared__ float As[BK][T + 4];
  __shared__ float Ws[BK][T + 4];
  const int Ml = c ? min(c->live_count * s, max_rows) : max_rows;
  const int m0 = blockIdx.y * T;
  if (m0 >= Ml) return;
  const int n0 = blockIdx.x * T;
  const int kb = blockIdx.z * kps;
  const int ke = min(K, kb + kps);
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  float acc[4][4] = {};
  for (int k0 = kb; k0 < ke; k0 += BK) {
    for (int j = 0; j < 4; ++j) {
      const int idx = tid + 256 * j, row = idx / BK, kk = idx % BK, gk = k0 + kk;
      As[kk][row] = (m0 + row < Ml && gk < ke) ? A[(size_t)(m0 + row) * K + gk] : 0.f;
      Ws[kk][row] = (n0 + row < N && gk < ke) ? W[(size_t)(n0 + row) * K + gk] : 0.f;
    }
    __syncthreads();
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
      for (int j = 0; j < 4; ++j) b[j] = Ws[kk][tx * 4 + j];
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* out = P + blockIdx.z * split_stride;
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= Ml) continue;
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col < N) out[(size_t)row * N + col] = acc[i][j];
    }
  }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

GemmPlan plan_gemm(DType dt, int max_rows, int N, int K) {
  GemmPlan p;
  if (dt == DType::F32) {
    p.bm = 64; p.bn = 64;
  } else if (max_rows > 64) {
    p.bm = 128; p.bn = 128;
  } else {
    p.bm = 64; p.bn = 128;
  }
  const int kstep = dt == DType::BF16 ? 32 : 16;
  const int tiles = cdiv(N, p.bn) * cdiv(max_rows, p.bm);
  int splits = 1;
  while (tiles * splits < 256 && K / (splits * 2) >= 8 * kstep && splits < 8) splits *= 2;
  const int ktiles = cdiv(K, kstep);
  p.k_per_split = cdiv(ktiles, splits) * kstep;
  p.splits = cdiv(K, p.k_per_split);
  return p;
}

hipError_t launch_gemm(DType dt, const GemmPlan& p, const void* A, const void* W, float* P, size_t split_stride,
                       const Ctrl* c, int s, int max_rows, int N, int K, hipStream_t st) {
  const dim3 grid(cdiv(N, p.bn), cdiv(max_rows, p.bm), p.splits);
  if (dt == DType::F32) {
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, static_cast<const float*>(A),
                       static_cast<const float*>(W), P, split_stride, c, s, max_rows, N, K, p.k_per_split);
  } else if (p.bm == 128) {
    hipLaunchKernelGGL((k_gemm_bf16<128, 128>), grid, dim3(256), 0, st, static_cast<const float*>(A),
                       static_cast<const bf16*>(W), P, split_stride, c, s, max_rows, N, K, p.k_per_split);
  } else {
    hipLaunchKernelGGL((k_gemm_bf16<64, 128>), grid, dim3(256), 0, st, static_cast<const float*>(A),
                       static_cast<const bf16*>(W), P, split_stride, c, s, max_rows, N, K, p.k_per_split);
  }
  return hipGetLastError();
}

}  // namespace rksc
