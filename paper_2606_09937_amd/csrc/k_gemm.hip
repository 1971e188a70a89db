// Dense projections of the decoder layer: P[split][m][n] = sum_k A[m][k] * W[n][k]
// over the split's K range. A is the fp32 [rows, K] activation, W a [N, K]
// weight (torch Linear layout) in the model's storage type, P fp32. Split
// partials are summed by the consumer.
//
// bf16 weights: the activation arrives as two bf16 planes (hi + lo of the fp32
// value), and both meet every weight fragment in v_mfma_f32_16x16x32_bf16 with
// fp32 accumulation, so the product keeps fp32-level accuracy at twice the
// bf16 MFMA work. Operands stream through an LDS ring by direct DMA.
// fp32 weights: a plain LDS-tiled FMA kernel on fp32 activations.
#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

// ---------------------------------------------------------------------------
// Multi-stage LDS pipeline fed by direct global->LDS DMA (global_load_lds_dwordx4).
//
// The activation arrives pre-split as two bf16 planes (A = Ahi + Alo, both
// [rows, K]), the weight as bf16 [N, K]. Each K step of 32 moves three
// sub-tiles (Ahi, Alo: BM x 64 B; W: BN x 64 B) straight from memory into one
// slot of an R-deep LDS ring without touching registers, so R-1 steps of loads
// are in flight while the MFMAs consume the current slot. Within a 64-byte row
// the four 16-byte chunks are stored at position chunk ^ ((row >> 2) & 3): the
// DMA writes stay contiguous per wave and the 16-row fragment reads are
// bank-conflict free. Every wave issues the same number of DMA instructions
// per step, so "slot ready" is an explicit vmcnt wait followed by a barrier.
// K needs only to be a multiple of 8: a chunk that would start at or past the
// end of the split reads the split's first chunk instead (valid memory), and
// activation chunks past the end are zeroed before the last step is consumed.

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 2) & 3); }

template <int BM, int BN, int R>
__global__ __launch_bounds__(256) void k_gemm_dma(const bf16* __restrict__ Ahi, const bf16* __restrict__ Alo,
                                                  const bf16* __restrict__ W, float* __restrict__ P,
                                                  size_t split_stride, const Ctrl* c, int s, int max_rows, int N,
                                                  int K, int kps) {
  constexpr int BK = 32;
  constexpr int AI = BM / 16, WI = BN / 16;           // wave DMA instructions per sub-tile
  constexpr int NDMA = (2 * AI + WI) / 4;             // per wave per step
  static_assert((2 * AI + WI) % 4 == 0, "DMA instructions must split evenly over 4 waves");
  constexpr int A_BYTES = BM * 64, W_BYTES = BN * 64;
  constexpr int SLOT = 2 * A_BYTES + W_BYTES;
  constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 16, TN = WN / 16;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * SLOT];

  const int Ml = c ? min(c->live_count * s, max_rows) : max_rows;
  const int m0 = blockIdx.y * BM;
  if (m0 >= Ml) return;
  const int n0 = blockIdx.x * BN;
  const int kb = blockIdx.z * kps;
  const int ke = min(K, kb + kps);
  const int nsteps = (ke - kb + BK - 1) / BK;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm0 = (wid >> 1) * WM, wn0 = (wid & 1) * WN;
  const int r16 = lane & 15, g = lane >> 4;

  // Per-wave DMA sources: instruction j (global index wid + 4j) covers 16 rows of
  // one sub-tile; lane L fills chunk position L % 4 of row 16*i + L / 4, i.e.
  // the 8-element chunk swz(row, L % 4) of that row.
  const bf16* src[NDMA];
  int dst[NDMA];
  const int chunk_off = 8 * swz(lane >> 2, lane & 3);   // 16-row groups keep (row >> 2) & 3
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int ins = wid + 4 * j;
    const int row_in = lane >> 2;
    if (ins < 2 * AI) {
      const int plane = ins / AI, i = ins % AI;
      const int gr = min(m0 + 16 * i + row_in, max_rows - 1);
      src[j] = (plane ? Alo : Ahi) + (size_t)gr * K;
      dst[j] = plane * A_BYTES + i * 1024;
    } else {
      const int i = ins - 2 * AI;
      const int gn = min(n0 + 16 * i + row_in, N - 1);
      src[j] = W + (size_t)gn * K;
      dst[j] = 2 * A_BYTES + i * 1024;
    }
  }
  auto issue = [&](int step) {
    // Steps past the end re-read the split's first step (valid memory, never used);
    // a chunk starting at or past ke reads the split's first chunk instead.
    const int k = (step < nsteps ? kb + step * BK : kb) + chunk_off;
    const int col = k < ke ? k : kb;
    uint8_t* slot = smem + (step % R) * SLOT;
#pragma unroll
    for (int j = 0; j < NDMA; ++j) dma16(src[j] + col, slot + dst[j]);
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int st = 0; st < R - 1; ++st) issue(st);

  for (int st = 0; st < nsteps; ++st) {
    wait_vmcnt<NDMA * (R - 2)>();   // this thread's DMAs for step st have landed
    uint8_t* slot = smem + (st % R) * SLOT;
    const int kst = kb + st * BK;
    if (kst + BK > ke) {
      // Partial last step: zero activation chunks at k >= ke (both planes).
      for (int ci = tid; ci < 2 * BM * 4; ci += 256) {
        const int plane = ci / (BM * 4), row = (ci / 4) % BM, pos = ci & 3;
        const int chunk = swz(row, pos);
        if (kst + 8 * chunk >= ke)
          *reinterpret_cast<uint4*>(slot + plane * A_BYTES + row * 64 + pos * 16) = make_uint4(0, 0, 0, 0);
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the zeros are in LDS before the barrier
    }
    __builtin_amdgcn_s_barrier();        // every wave's DMAs for st landed; step st-1 fully consumed
    issue(st + R - 1);                   // refills the slot step st-1 used
    const uint8_t* ah_t = slot;
    const uint8_t* al_t = slot + A_BYTES;
    const uint8_t* w_t = slot + 2 * A_BYTES;
    bf16x8 ah[TM], al[TM], bw[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int row = wm0 + 16 * tm + r16;
      const int off = row * 64 + swz(row, g) * 16;
      ah[tm] = *reinterpret_cast<const bf16x8*>(ah_t + off);
      al[tm] = *reinterpret_cast<const bf16x8*>(al_t + off);
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int row = wn0 + 16 * tn + r16;
      bw[tn] = *reinterpret_cast<const bf16x8*>(w_t + row * 64 + swz(row, g) * 16);
    }
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[tm], bw[tn], acc[tm][tn], 0, 0, 0);
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[tm], bw[tn], acc[tm][tn], 0, 0, 0);
      }
  }
  wait_vmcnt<0>();   // drain the look-ahead DMAs before the workgroup can exit

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
  p.bm = 64;
  p.bn = dt == DType::F32 ? 64 : 128;
  if (dt == DType::BF16 && max_rows > 64) p.bm = 128;
  const int kstep = dt == DType::BF16 ? 32 : 16;
  const int tiles = cdiv(N, p.bn) * cdiv(max_rows, p.bm);
  // Split K until the launch has ~1.5 workgroups per CU (split partials are
  // summed by the consumer kernel), keeping at least 256 K per split.
  int splits = 1;
  while (tiles * splits < 384 && K / (splits * 2) >= 256 && splits < kMaxSplitsGemm) splits *= 2;
  const int ktiles = cdiv(K, kstep);
  p.k_per_split = cdiv(ktiles, splits) * kstep;
  p.splits = cdiv(K, p.k_per_split);
  return p;
}

hipError_t launch_gemm(DType dt, const GemmPlan& p, const void* A0, const void* A1, const void* W, float* P,
                       size_t split_stride, const Ctrl* c, int s, int max_rows, int N, int K, hipStream_t st) {
  const dim3 grid(cdiv(N, p.bn), cdiv(max_rows, p.bm), p.splits);
  if (dt == DType::F32) {
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, static_cast<const float*>(A0),
                       static_cast<const float*>(W), P, split_stride, c, s, max_rows, N, K, p.k_per_split);
  } else if (p.bm == 128) {
    hipLaunchKernelGGL((k_gemm_dma<128, 128, 3>), grid, dim3(256), 0, st, static_cast<const bf16*>(A0),
                       static_cast<const bf16*>(A1), static_cast<const bf16*>(W), P, split_stride, c, s, max_rows,
                       N, K, p.k_per_split);
  } else {
    hipLaunchKernelGGL((k_gemm_dma<64, 128, 3>), grid, dim3(256), 0, st, static_cast<const bf16*>(A0),
                       static_cast<const bf16*>(A1), static_cast<const bf16*>(W), P, split_stride, c, s, max_rows,
                       N, K, p.k_per_split);
  }
  return hipGetLastError();
}

}  // namespace rksc
