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
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

// ---------------------------------------------------------------------------
// Multi-stage LDS pipeline fed by direct global->LDS DMA (global_load_lds_dwordx4).
//
// The activation arrives pre-split as two bf16 planes (A = Ahi + Alo, both
// [rows, K]), the weight as bf16 [N, K]. A workgroup of 8 waves owns a
// 128-row x BN-column output tile and a K range. Each stage moves a 64-wide K
// slice (128 bytes per row) of three sub-tiles (Ahi, Alo: 128 rows; W: BN rows)
// straight from memory into one slot of an R-deep LDS ring, without touching
// registers: every DMA instruction covers 8 rows x 128 B, eight lanes per
// 128-byte line. Within a row the 16-byte chunk c is stored at position
// c ^ ((row >> 1) & 7), so the 16-row fragment reads of the MFMA operands are
// spread over the banks (the lanes fetch permuted chunks of the same line).
// The waves form a 2 x 4 grid of 64 x BN/4 tiles of v_mfma_f32_16x16x32_bf16;
// each weight fragment meets the hi and the lo fragment.
// Every wave issues the same number of DMA instructions per stage, so "slot
// ready" is an explicit vmcnt wait followed by a barrier. The fragment reads
// are typed bf16x8 loads, which the compiler does not order behind the
// untyped DMA stores (it would otherwise wait for every outstanding DMA).
// K needs only to be a multiple of 8: a chunk at or past the end of the split
// reads the split's first chunk instead (valid memory), and the activation
// chunks past the end are zeroed in LDS once the last, partial stage has
// landed.
//
// TILED: the weight is read from its pre-tiled copy [N/BN][K/64][BN][64]
// (launch_tile_rows), in which a stage's BN x 64 weight block is one
// contiguous run of BN * 128 bytes instead of BN runs of 128 bytes at a K * 2
// byte stride; the tile and the LDS layout are the same. The launcher takes
// this form only when N % BN == 0 and the split's K range is whole stages.

__device__ __forceinline__ int gswz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Waits until at most n_after stages of this thread's DMA instructions (IPW
// each) are outstanding, i.e. every earlier stage has landed; with LDS also
// every LDS access of the wave. n_after (0..3) is uniform: the stages issued
// after the one waited for, fewer near the end of a split, where no stage past
// the end is fetched.
template <int IPW, bool LDS>
__device__ __forceinline__ void wait_dma_after(int n_after) {
  if (n_after >= 3) {
    if constexpr (LDS) wait_vmcnt_lds<3 * IPW>(); else wait_vmcnt<3 * IPW>();
  } else if (n_after == 2) {
    if constexpr (LDS) wait_vmcnt_lds<2 * IPW>(); else wait_vmcnt<2 * IPW>();
  } else if (n_after == 1) {
    if constexpr (LDS) wait_vmcnt_lds<IPW>(); else wait_vmcnt<IPW>();
  } else {
    if constexpr (LDS) wait_vmcnt_lds<0>(); else wait_vmcnt<0>();
  }
}

constexpr int kGemmWaves = 8;

// XCD-aware grouped raster for grids with several row tiles. Workgroups are
// dealt to the 8 XCDs round robin (id % 8), and each XCD has its own L2. Each
// XCD is given a contiguous range of "virtual" tile ids, and virtual ids walk
// GM row tiles x all column tiles per group, so the ~32 workgroups resident on
// one XCD cover a compact GM-row block of tiles and re-read their activation
// and weight tiles from that XCD's L2 instead of from HBM/MALL.
template <int GM>
__device__ __forceinline__ void xcd_raster(int& tx, int& ty, int& tz) {
  const int NX = gridDim.x, NY = gridDim.y, T = NX * NY * gridDim.z;
  const int id = blockIdx.x + NX * (blockIdx.y + NY * blockIdx.z);
  const int x = id % 8, q = id / 8;
  const int v = x * (T / 8) + min(x, T % 8) + q;   // XCD x holds ids x, x+8, ...: T/8 (+1 for x < T%8)
  const int per_split = NX * NY;
  tz = v / per_split;
  const int r = v - tz * per_split;
  const int grp = r / (GM * NX), first_m = grp * GM, gm = min(GM, NY - first_m);
  const int rr = r - grp * GM * NX;
  ty = first_m + rr % gm;
  tx = rr / gm;
}

template <int BN, int R, bool TILED = false>
__global__ __launch_bounds__(kGemmWaves * 64) void k_gemm_dma(const bf16* __restrict__ Ahi,
                                                              const bf16* __restrict__ Alo,
                                                              const bf16* __restrict__ W, float* __restrict__ P,
                                                              size_t split_stride, const Ctrl* c, int s,
                                                              int max_rows, int N, int K, int kps) {
  constexpr int BM = 128, CB = 128, KEL = CB / 2;   // K elements per stage
  constexpr int A_BYTES = BM * CB, W_BYTES = BN * CB, SLOT = 2 * A_BYTES + W_BYTES;
  constexpr int NINS = SLOT / 1024;
  static_assert(NINS % kGemmWaves == 0, "DMA instructions must split evenly over the waves");
  constexpr int IPW = NINS / kGemmWaves;
  constexpr int WM = BM / 2, WN = BN / 4, TM = WM / 16, TN = WN / 16;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * SLOT];

  const int Ml = c ? min(c->live_count * s, max_rows) : max_rows;
  int tx = blockIdx.x, ty = blockIdx.y, tz = blockIdx.z;
  if (gridDim.y > 1) xcd_raster<4>(tx, ty, tz);
  const int m0 = ty * BM;
  if (m0 >= Ml) return;
  const int n0 = tx * BN;
  const int kb = tz * kps;
  const int ke = min(K, kb + kps);
  const int nsteps = (ke - kb + KEL - 1) / KEL;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm0 = (wid & 1) * WM, wn0 = (wid >> 1) * WN;
  const int r16 = lane & 15, g = lane >> 4;
  const bool wave_live = m0 + wm0 < Ml;   // waves whose 64 rows are all past the live rows skip the MFMAs

  // DMA sources: instruction ins covers rows 8*ins'.. of its sub-tile; lane L fills
  // physical chunk L & 7 of row L >> 3, i.e. logical chunk gswz(row, L & 7). src[j]
  // points at the lane's chunk of its row (K offset 0); the LDS destinations are
  // scalar (the wave index made uniform).
  const int widu = __builtin_amdgcn_readfirstlane(wid);
  // kstr[j]: elements from one stage's source to the next one's per K element
  // (1 in the row-major operands, BN in the tiled weight).
  const bf16* src[IPW];
  int dst[IPW], coff[IPW], kstr[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int off = (wid * IPW + j) * 1024;
    int row;
    kstr[j] = 1;
    if (off < 2 * A_BYTES) {
      const int plane = off / A_BYTES;
      row = (off % A_BYTES) / CB + (lane >> 3);
      src[j] = (plane ? Alo : Ahi) + (size_t)min(m0 + row, max_rows - 1) * K;
    } else {
      row = (off - 2 * A_BYTES) / CB + (lane >> 3);
      if constexpr (TILED) {
        src[j] = W + (size_t)tx * K * BN + (size_t)row * KEL;   // block row `row` of column tile tx
        kstr[j] = BN;
      } else {
        src[j] = W + (size_t)min(n0 + row, N - 1) * K;
      }
    }
    coff[j] = 8 * gswz(row, lane & 7);
    src[j] += coff[j];
    dst[j] = (widu * IPW + j) * 1024;
  }
  auto issue = [&](int step) {
    if (step >= nsteps) return;   // nothing past the split's end is fetched
    const int k = kb + step * KEL;
    uint8_t* slot = smem + (step % R) * SLOT;
    if (TILED || k + KEL <= ke) {   // a whole stage (the common case; always, when tiled)
#pragma unroll
      for (int j = 0; j < IPW; ++j) dma16(src[j] + (size_t)k * kstr[j], slot + dst[j]);
    } else {   // chunks at or past the split's end read the split's first chunk
#pragma unroll
      for (int j = 0; j < IPW; ++j) dma16(k + coff[j] < ke ? src[j] + k : src[j] - coff[j] + kb, slot + dst[j]);
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // The fragments of one 32-wide k substep sb of a stage: the hi/lo activation
  // fragments of the wave's row blocks and the weight fragments of its columns.
  struct Frag {
    bf16x8 ah[TM], al[TM], bw[TN];
  };
  auto load = [&](const uint8_t* slot, int sb, Frag& f) {
    const int ch = 4 * sb + g;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int row = wm0 + 16 * tm + r16;
      const int off = row * CB + gswz(row, ch) * 16;
      f.ah[tm] = *reinterpret_cast<const bf16x8*>(slot + off);
      f.al[tm] = *reinterpret_cast<const bf16x8*>(slot + A_BYTES + off);
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int row = wn0 + 16 * tn + r16;
      f.bw[tn] = *reinterpret_cast<const bf16x8*>(slot + 2 * A_BYTES + row * CB + gswz(row, ch) * 16);
    }
  };
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.ah[tm], f.bw[tn], acc[tm][tn], 0, 0, 0);
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.al[tm], f.bw[tn], acc[tm][tn], 0, 0, 0);
      }
  };
  // The next substep's TM * 2 + TN reads spread over the first MFMAs of a substep.
  constexpr int NRD = TM * 2 + TN, NMF = TM * TN * 2;
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < NRD / 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // two LDS reads
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NMF - NRD / 2, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  // The split's last, partial stage: the activation chunks at or past its end
  // (8-element chunks lie wholly inside or outside, K % 8 == 0) hold the split's
  // first chunk and are zeroed in LDS once the stage has landed, so that every
  // stage is contracted without a mask. Called by every thread.
  auto zero_tail = [&](int step) {
    const int kst = kb + step * KEL;
    if (TILED || kst + KEL <= ke) return;
    uint8_t* const slot = smem + (step % R) * SLOT;
    for (int idx = threadIdx.x; idx < 2 * BM * 8; idx += kGemmWaves * 64) {
      const int c = idx & 7, row = (idx >> 3) % BM, pl = idx / (BM * 8);
      if (kst + 8 * c >= ke)
        *reinterpret_cast<uint4*>(slot + pl * A_BYTES + row * CB + gswz(row, c) * 16) = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
  };

  // Software pipeline over the R-slot ring (all R slots filled up front). A
  // stage is two k substeps: the wave contracts substep 0 while it reads
  // substep 1's fragments; then (one barrier: stage st+1 has landed for every
  // thread, and every wave's reads of slot st are complete) slot st is refilled
  // with stage st+R, and the wave reads stage st+1's substep 0 while it
  // contracts substep 1. The barrier sits outside the wave_live guards. The
  // last stage also reads the next slot's fragments (in the ring, never used).
#pragma unroll
  for (int st = 0; st < R; ++st) issue(st);
  wait_dma_after<IPW, false>(min(R - 1, nsteps - 1));
  __builtin_amdgcn_s_barrier();
  zero_tail(0);
  Frag f0, f1;
  if (wave_live) load(smem, 0, f0);
  for (int st = 0; st < nsteps; ++st) {
    const uint8_t* const slot = smem + (st % R) * SLOT;
    const uint8_t* const nslot = smem + ((st + 1) % R) * SLOT;
    if (wave_live) {
      load(slot, 1, f1);
      mma(f0);
      interleave();
    }
    // This thread's DMAs of stage st+1 have landed and its reads of slot st are
    // complete; after the barrier every thread's are.
    wait_dma_after<IPW, true>(max(0, min(R - 2, nsteps - st - 2)));
    __builtin_amdgcn_s_barrier();
    issue(st + R);   // refills slot st
    if (st + 1 < nsteps) zero_tail(st + 1);
    if (wave_live) {
      load(nslot, 0, f0);
      mma(f1);
      interleave();
    }
  }
  wait_vmcnt<0>();   // no DMA is left in flight (none past the split's end); kept as a guard

  float* out = P + tz * split_stride;
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

// ---------------------------------------------------------------------------
// K-32 stage kernel: BM x BN tiles (256 x 256 for large row counts, 128 x 512
// or 128 x 256 for 128-row calls), stages of a 32-wide K slice (64 bytes per
// row), so that more stages fit the LDS and more bytes are in flight per CU.
//
// 8 waves as a (BM / 64) x (8 / (BM / 64)) grid of 64 x WN wave tiles. At
// 256 x 256 each wave reads 64 x 32 activation and 128 x 32 weight elements
// from LDS per 32-wide K step for 64 MFMAs, a third fewer LDS bytes per MFMA
// than the 128-row kernel's 64 x 64 wave tiles. A stage holds three sub-tiles
// (A hi, A lo: BM rows; W: BN rows) of 64-byte rows; R stages fit the LDS,
// all R are filled up front and R - 1 are in flight while one is contracted.
// Each DMA instruction moves 16 rows x 64 bytes.
//
// LDS layout of a sub-tile: rows 2q and 2q + 1 form the 128-byte line q, row r
// holding 16-byte slots 4 (r & 1) .. 4 (r & 1) + 3 of its line before the
// swizzle, and slot t of line q sits at t ^ (q & 7). A fragment read has lane
// (r16, g) read chunk g of row r16 of a 16-row block; a 128-bit LDS read is
// served eight lanes at a time (the even, then the odd lanes of each 16), and
// the eight even rows 0, 2, .., 14 lie on lines q = 0..7, so their chunks fall
// on eight distinct slots, i.e. all 32 banks. (With each row on its own 64-byte
// line, the even rows met only four distinct slots: a two-way bank conflict on
// every read.)
__device__ __forceinline__ int wlds(int row, int chunk) {
  const int q = row >> 1;
  return q * 128 + (((row & 1) * 4 + chunk) ^ (q & 7)) * 16;
}

// SWIGLU: the gate|up projection with its SwiGLU epilogue (one K split). W is
// [2F, K] (gate rows, then up rows, N = 2F); a workgroup's BN weight rows are
// gate rows n0..n0+BN/2-1 and the matching up rows F+n0.., so the waves of
// the first half of the wave columns hold gate values and those of the second
// half the up values of the same (row, column) in the same lanes. The up waves
// pass their accumulators through LDS and the gate waves write
// a = silu(gate) * up as the bf16 hi/lo planes [max_rows, F] at P (hi) and
// P + max_rows * F (lo), the down projection's input.
template <int BM, int BN, int R, bool SWIGLU = false>
__global__ __launch_bounds__(kGemmWaves * 64) void k_gemm_wide(const bf16* __restrict__ Ahi,
                                                               const bf16* __restrict__ Alo,
                                                               const bf16* __restrict__ W, float* __restrict__ P,
                                                               size_t split_stride, const Ctrl* c, int s,
                                                               int max_rows, int N, int K, int kps) {
  constexpr int KEL = 32, RB = KEL * 2;
  constexpr int SUB_A = BM * RB, SLOT = 2 * SUB_A + BN * RB;
  constexpr int IPW = SLOT / 1024 / kGemmWaves;   // DMA instructions per wave per stage
  constexpr int A_INS = SUB_A / 1024;             // instructions per activation plane
  constexpr int WGM = BM / 64, WGN = kGemmWaves / WGM;   // wave grid
  constexpr int WN = BN / WGN, TM = 4, TN = WN / 16;     // 64 x WN wave tile
  static_assert(A_INS % kGemmWaves == 0 && (SLOT / 1024) % kGemmWaves == 0,
                "every instruction of a wave stays in one sub-tile");
  static_assert(WGM * WGN == kGemmWaves && TN >= 1 && (!SWIGLU || WGN % 2 == 0), "wave grid");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * SLOT];

  const int Ml = c ? min(c->live_count * s, max_rows) : max_rows;
  int tx, ty, tz;
  xcd_raster<4>(tx, ty, tz);
  const int m0 = ty * BM;
  if (m0 >= Ml) return;
  const int F = N / 2;
  const int n0 = tx * (SWIGLU ? BN / 2 : BN);
  const int kb = tz * kps, ke = min(K, kb + kps);
  const int nsteps = (ke - kb + KEL - 1) / KEL;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int wm = wid % WGM, wn = wid / WGM;
  const bool wave_live = m0 + 64 * wm < Ml;
  // Weight row of tile row `row` (0..255).
  auto wrow = [&](int row) {
    if (!SWIGLU) return min(n0 + row, N - 1);
    return row < BN / 2 ? min(n0 + row, F - 1) : F + min(n0 + row - BN / 2, F - 1);
  };

  // DMA instruction j of this wave (ins = 8j + wid) fills 16 rows (8 lines) of
  // sub-tile plane(j) (0 A hi, 1 A lo, 2 W; fixed by j as A_INS is a multiple of
  // 8); lane L fills slot L & 7 of line L >> 3, i.e. logical slot
  // t = (L & 7) ^ (L >> 3): chunk t & 3 of row 2 (L >> 3) + (t >> 2) of the
  // block, the same for every j.
  // Row offsets in elements as size_t: rows x K passes 2^31 at large row counts.
  auto plane = [](int j) { return j * kGemmWaves < A_INS ? 0 : (j * kGemmWaves < 2 * A_INS ? 1 : 2); };
  size_t rowoff[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int pl = plane(j);
    const int t = (lane & 7) ^ (lane >> 3);
    const int row = (j * kGemmWaves + wid - pl * A_INS) * 16 + 2 * (lane >> 3) + (t >> 2);
    rowoff[j] = (size_t)(pl < 2 ? min(m0 + row, max_rows - 1) : wrow(row)) * K;
  }
  const int ccol = 8 * (((lane & 7) ^ (lane >> 3)) & 3);
  // The wave index made uniform, so that the LDS destinations are scalar (M0) values.
  const int widu = __builtin_amdgcn_readfirstlane(wid);
  auto issue = [&](int step) {
    // Steps past the end re-read the split's first step (valid memory, never
    // used; fetching nothing there measured 1-2% slower for this kernel, which
    // runs several rounds of workgroups); chunks at or past the end of the last,
    // partial stage read the split's first chunk and are zeroed in LDS.
    const int k = kb + (step < nsteps ? step : 0) * KEL;
    uint8_t* slot = smem + (step % R) * SLOT;
    const int col = k + ccol < ke ? k + ccol : kb;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const bf16* base = plane(j) == 0 ? Ahi : (plane(j) == 1 ? Alo : W);
      dma16(base + rowoff[j] + col, slot + (j * kGemmWaves + widu) * 1024);
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // Fragment reads of one stage: the weight fragments of the wave's columns,
  // and the hi/lo activation fragments of row block tm.
  auto load_w = [&](const uint8_t* slot, bf16x8 (&bw)[TN]) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int row = wn * WN + 16 * tn + r16;
      bw[tn] = *reinterpret_cast<const bf16x8*>(slot + 2 * SUB_A + wlds(row, g));
    }
  };
  auto load_a = [&](const uint8_t* slot, int tm, bf16x8& ah, bf16x8& al) {
    const int row = wm * 64 + 16 * tm + r16;
    const int off = wlds(row, g);
    ah = *reinterpret_cast<const bf16x8*>(slot + off);
    al = *reinterpret_cast<const bf16x8*>(slot + SUB_A + off);
  };
  auto mma = [&](int tm, const bf16x8& ah, const bf16x8& al, const bf16x8 (&bw)[TN]) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
      acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bw[tn], acc[tm][tn], 0, 0, 0);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
      acc[tm][tn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bw[tn], acc[tm][tn], 0, 0, 0);
  };
  // The split's last, partial stage: the activation chunks at or past its end
  // (8-element chunks lie wholly inside or outside, K % 8 == 0) hold the split's
  // first chunk and are zeroed in LDS once the stage has landed, so that every
  // stage is contracted without a mask. Called by every thread.
  auto zero_tail = [&](int step) {
    const int kst = kb + step * KEL;
    if (kst + KEL <= ke) return;
    uint8_t* const slot = smem + (step % R) * SLOT;
    for (int idx = threadIdx.x; idx < 2 * BM * 4; idx += kGemmWaves * 64) {
      const int c = idx & 3, row = (idx >> 2) % BM, pl = idx / (BM * 4);
      if (kst + 8 * c >= ke)
        *reinterpret_cast<uint4*>(slot + pl * SUB_A + wlds(row, c)) = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
  };

  // Software pipeline over the R-slot ring (all R slots filled up front). In
  // stage st a wave contracts row blocks 0..2 while reading the next block's
  // fragments; then (barrier A: stage st+1 has landed for every thread) it
  // reads stage st+1's weight and first activation fragments while contracting
  // row block 3, so the LDS reads of one stage overlap the MFMAs of the last;
  // then (barrier B: every wave is done reading slot st) slot st is refilled
  // with stage st+R. Barriers sit outside the wave_live guards.
#pragma unroll
  for (int st = 0; st < R; ++st) issue(st);
  wait_vmcnt<IPW * (R - 1)>();
  __builtin_amdgcn_s_barrier();
  zero_tail(0);
  // Two register sets for the weight fragments, used alternately by even and
  // odd stages. The last stage also reads the next slot's fragments; those
  // reads land in the ring (in bounds) and are never used.
  bf16x8 bwa[TN], bwb[TN], h0, l0, h1, l1, h2, l2, h3, l3;
  if (wave_live) {
    load_w(smem, bwa);
    load_a(smem, 0, h0, l0);
  }
  auto stage = [&](int st, const bf16x8 (&bwc)[TN], bf16x8 (&bwn)[TN]) {
    const uint8_t* const slot = smem + (st % R) * SLOT;
    const uint8_t* const nslot = smem + ((st + 1) % R) * SLOT;
    // sched_barrier(0) keeps the compiler from hoisting a row block's MFMAs
    // above the previous block's, which would wait on reads just issued.
    if (wave_live) {
      load_a(slot, 1, h1, l1);
      mma(0, h0, l0, bwc);
      __builtin_amdgcn_sched_barrier(0);
      load_a(slot, 2, h2, l2);
      mma(1, h1, l1, bwc);
      __builtin_amdgcn_sched_barrier(0);
      load_a(slot, 3, h3, l3);
      mma(2, h2, l2, bwc);
      __builtin_amdgcn_sched_barrier(0);
    }
    // A: this thread's DMAs of stage st+1 have landed; after the barrier every thread's have.
    wait_vmcnt<IPW * (R - 2)>();
    __builtin_amdgcn_s_barrier();
    if (st + 1 < nsteps) zero_tail(st + 1);
    if (wave_live) {
      load_w(nslot, bwn);
      load_a(nslot, 0, h0, l0);
      mma(3, h3, l3, bwc);
      // The next stage's TN + 2 reads spread over the first MFMAs of this block.
#pragma unroll
      for (int i = 0; i < (TN + 2) / 2; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // two LDS reads
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * TN - (TN + 2) / 2, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // B: this wave's reads of slot st are complete; after the barrier every wave's are.
    wait_vmcnt_lds<63>();
    __builtin_amdgcn_s_barrier();
    issue(st + R);   // refills slot st
  };
  for (int st = 0; st < nsteps; st += 2) {
    stage(st, bwa, bwb);
    if (st + 1 < nsteps) stage(st + 1, bwb, bwa);
  }
  wait_vmcnt<0>();   // drain the look-ahead DMAs before the workgroup can exit
  if constexpr (SWIGLU) {
    // Up accumulators of wave (wm, wn) with wn >= WGN / 2 to LDS (the ring is
    // free once every wave is past its last stage), read back by wave
    // (wm, wn - WGN / 2) lane for lane.
    constexpr int HG = WGN / 2;
    __syncthreads();
    floatx4* xch = reinterpret_cast<floatx4*>(smem);   // [WGM][HG][TM][TN][64 lanes]
    static_assert(WGM * HG * TM * TN * 64 * 16 <= R * SLOT, "the exchange fits in the ring");
    const int pair = wm * HG + wn % HG;
    if (wn >= HG) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) xch[((pair * TM + tm) * TN + tn) * 64 + lane] = acc[tm][tn];
    }
    __syncthreads();
    if (wn >= HG || !wave_live) return;
    bf16* hi = reinterpret_cast<bf16*>(P);
    bf16* lo = hi + (size_t)max_rows * F;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const floatx4 u = xch[((pair * TM + tm) * TN + tn) * 64 + lane];
        const int col = n0 + wn * WN + 16 * tn + r16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + wm * 64 + 16 * tm + 4 * g + i;
          if (row < Ml && col < F) {
            const float gt = acc[tm][tn][i];
            const float a = gt / (1.f + expf(-gt)) * u[i];
            uint16_t h, l;
            split2(a, h, l);
            const size_t idx = (size_t)row * F + col;
            hi[idx] = __builtin_bit_cast(bf16, h);
            lo[idx] = __builtin_bit_cast(bf16, l);
          }
        }
      }
    return;
  }
  if (!wave_live) return;

  float* out = P + tz * split_stride;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col = n0 + wn * WN + 16 * tn + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + wm * 64 + 16 * tm + 4 * g + i;
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

// ---------------------------------------------------------------- skinny GEMM
//
// At most 32 activation rows (one decode token per branch): the product is a
// stream of the weight matrix, and the kernel is laid out like the lm_head
// stream. RB blocks of 16 activation rows (RB = 2 from 17 rows) meet every
// weight fragment read from LDS. The weights pass through an R-deep LDS ring of 16 KB units (16 rows x
// 512 K, one 1 KB row segment per DMA instruction, chunk c of row r at position
// c ^ r), while the activation stays in registers: a workgroup covers a K range
// of 2048 * KH (one split of the output) and wave w holds the hi and lo bf16
// fragments of the 16 rows over its KH half-slices of 256 K, loaded once. A unit
// (tile t, slice s) is contracted by the owners of the slice's two halves (8
// k-substeps x 2 MFMAs each); after every kSkGroup tiles the waves' partial
// tiles are summed through LDS and stored as fp32 partials P[split][row][n].
// Workgroup (split, j) takes a contiguous range of the 16-row weight tiles.
// Rows past N are clamped (fetched, never stored); activation rows past the
// live rows are zero; chunks past K read the row start and meet zero fragments.
// With two row blocks the ring has 6 units, so that the doubled reduction area
// still fits the 160 KB of LDS, and the K range of a split is 2048 (KH = 1).
constexpr int kSkUnit = 16 * 1024;
constexpr int kSkGroup = 4;
constexpr int kSkRedBytes = kGemmWaves * kSkGroup * 1024;   // per row block
constexpr int kSkMaxRows = 32;

template <int KH, int RB>
__global__ __launch_bounds__(kGemmWaves * 64) void k_gemm_skinny(const bf16* __restrict__ Ahi,
                                                                 const bf16* __restrict__ Alo,
                                                                 const bf16* __restrict__ W, float* __restrict__ P,
                                                                 size_t split_stride, const Ctrl* c, int s,
                                                                 int max_rows, int N, int K, int wgps) {
  constexpr int NW = kGemmWaves, R = RB == 1 ? 7 : 6, IPW = 16 / NW;
  constexpr int KSPLIT = 2048 * KH;
  static_assert(16 % NW == 0, "a unit's 16 rows split evenly over the waves");
  static_assert(RB == 1 || (RB == 2 && KH == 1), "two row blocks with one half-slice per wave");
  static_assert(NW * 64 == RB * kSkGroup * 64 || RB == 1, "one merging thread per (block, tile, lane)");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * kSkUnit + RB * kSkRedBytes];

  const int Ml = c ? min(c->live_count * s, max_rows) : max_rows;
  const int sp = blockIdx.x / wgps, jw = blockIdx.x - sp * wgps;
  const int k0 = sp * KSPLIT;
  const int ns = min(4 * KH, (K - k0 + 511) / 512);   // 512-wide slices of this split
  const int T = (N + 15) / 16;
  const int t0 = (int)((long long)jw * T / wgps), t1 = (int)((long long)(jw + 1) * T / wgps);
  const int ntile = t1 - t0, nunits = ntile * ns;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;

  // Issue cursor: unit iu = (tile t0 + it, slice isl); past the end unit 0 is
  // fetched again (never consumed). A unit inside the matrix is addressed as a
  // scalar base (its tile's first row, its slice) plus this lane's fixed offset
  // wlane[j] (row r of the tile, chunk lane ^ r); only a tile past row N - 1 or a
  // slice past K takes the clamped path.
  const int widu = __builtin_amdgcn_readfirstlane(wid);
  size_t wlane[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int r = IPW * wid + j;
    wlane[j] = (size_t)r * K + 8 * (lane ^ r);
  }
  int iu = 0, it = 0, isl = 0;
  auto issue = [&](int slot_idx) {
    uint8_t* slot = smem + slot_idx * kSkUnit;
    const bool past = iu >= nunits;
    const int t = t0 + (past ? 0 : it), sl = past ? 0 : isl;
    const int kbase = k0 + 512 * sl;
    if (16 * t + 15 < N && kbase + 512 <= K) {
      const bf16* base = W + (size_t)(16 * t) * K + kbase;
#pragma unroll
      for (int j = 0; j < IPW; ++j) dma16(base + wlane[j], slot + (IPW * widu + j) * 1024);
    } else {
#pragma unroll
      for (int j = 0; j < IPW; ++j) {
        const int r = IPW * wid + j;
        const int k = kbase + 8 * (lane ^ r);
        const int row = min(16 * t + r, N - 1);
        dma16(W + (size_t)row * K + (k < K ? k : 0), slot + (IPW * widu + j) * 1024);
      }
    }
    ++iu;
    if (++isl == ns) {
      isl = 0;
      ++it;
    }
  };
#pragma unroll
  for (int i = 0; i < R - 1; ++i) issue(i);

  // The activation fragments (after the ring's first units, so that both are in
  // flight together); the empty asm makes the compiler wait for them here, once.
  const bf16x8 zero = {};
  bf16x8 ah[RB][KH][8], al[RB][KH][8];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int ar = 16 * rb + r16;
    const int arow = min(ar, max_rows - 1);
#pragma unroll
    for (int q = 0; q < KH; ++q) {
      const int kb = k0 + 256 * (wid * KH + q);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = kb + 32 * j + 8 * g;
        const bool ok = k < K && ar < Ml;
        const size_t off = (size_t)arow * K + (ok ? k : 0);
        const bf16x8 h = *reinterpret_cast<const bf16x8*>(Ahi + off);
        const bf16x8 l = *reinterpret_cast<const bf16x8*>(Alo + off);
        ah[rb][q][j] = ok ? h : zero;
        al[rb][q][j] = ok ? l : zero;
      }
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int q = 0; q < KH; ++q)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const u32x4 hv = __builtin_bit_cast(u32x4, ah[rb][q][j]), lv = __builtin_bit_cast(u32x4, al[rb][q][j]);
        asm volatile("" ::"v"(hv), "v"(lv));
      }

  int qs = 0;   // ring slot of the next unit consumed (units consumed mod R)
  auto step = [&]() -> const uint8_t* {
    wait_vmcnt_lds<IPW * (R - 2)>();
    __builtin_amdgcn_s_barrier();
    issue(qs == 0 ? R - 1 : qs - 1);   // refills the slot the previous unit used
    const uint8_t* slot = smem + qs * kSkUnit;
    qs = qs == R - 1 ? 0 : qs + 1;
    return slot;
  };

  floatx4* red = reinterpret_cast<floatx4*>(smem + R * kSkUnit);
  for (int gi = 0; gi < ntile; gi += kSkGroup) {
    const int gt = min(kSkGroup, ntile - gi);
    floatx4 acc[RB][kSkGroup];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int m = 0; m < kSkGroup; ++m) acc[rb][m] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < kSkGroup; ++m) {
      if (m < gt) {
        for (int sl = 0; sl < ns; ++sl) {
          const uint8_t* slot = step();
#pragma unroll
          for (int q = 0; q < KH; ++q) {
            const int hs = wid * KH + q;   // half-slice: slice hs / 2, K half hs % 2
            if ((hs >> 1) == sl) {
              const int kh = hs & 1;
#pragma unroll
              for (int j = 0; j < 8; ++j) {
                const int lc = 4 * (8 * kh + j) + g;
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(slot + r16 * 1024 + (lc ^ r16) * 16);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                  acc[rb][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, ah[rb][q][j], acc[rb][m], 0, 0, 0);
                  acc[rb][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, al[rb][q][j], acc[rb][m], 0, 0, 0);
                }
              }
            }
          }
        }
      }
    }
    // Lane (r16, g) of every wave holds, for activation row 16 rb + r16, its K
    // part of weight rows 16 t + 4 g + i. The group's partial tiles meet in LDS;
    // the area is rewritten only after the next group's first ring barrier.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int m = 0; m < kSkGroup; ++m) red[((rb * NW + wid) * kSkGroup + m) * 64 + lane] = acc[rb][m];
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the partials are in LDS
    __builtin_amdgcn_s_barrier();
    {
      const int rb = tid / (kSkGroup * 64), m = (tid >> 6) % kSkGroup, l = tid & 63;
      if (rb < RB && m < gt) {
        floatx4 z = red[((rb * NW) * kSkGroup + m) * 64 + l];
#pragma unroll
        for (int w = 1; w < NW; ++w) z += red[((rb * NW + w) * kSkGroup + m) * 64 + l];
        const int row = 16 * rb + (l & 15), n = 16 * (t0 + gi + m) + 4 * (l >> 4);
        if (row < Ml && n < N)
          *reinterpret_cast<float4*>(P + sp * split_stride + (size_t)row * N + n) =
              make_float4(z[0], z[1], z[2], z[3]);
      }
    }
  }
  wait_vmcnt<0>();   // drain the look-ahead DMAs before the workgroup can exit
}

namespace {
// Half-slices per wave of the skinny kernel: the K range of a split is 2048 * KH
// and the consumers sum at most kMaxSplitsGemm splits.
int skinny_kh(int K) { return cdiv(K, 2048) <= kMaxSplitsGemm ? 1 : 2; }
// From 17 rows the two-block stream is taken only for wide projections: at 32
// rows it beat the 128-row tiles on the 28672-column gate|up (71 -> 53 us) and
// lost on the 4096- and 6144-column ones (15 -> 19 us for O), whose short
// stream per workgroup does not amortise the ring's fill and the reductions.
bool skinny_fits(DType dt, int max_rows, int N, int K) {
  const bool rows_ok = max_rows <= 16 || (max_rows <= kSkMaxRows && skinny_kh(K) == 1 && N >= 16384);
  return dt == DType::BF16 && rows_ok && N % 4 == 0 && K % 8 == 0 && cdiv(K, 2048 * skinny_kh(K)) <= kMaxSplitsGemm;
}
}  // namespace

// From 512 rows the projections are MFMA-bound (2 * 128 = 256 flops per weight
// byte with the hi/lo split), and what decides is how evenly the workgroups
// fill whole rounds of the 256 CUs. (Used from 512 to 1024 rows, where it was
// measured; with many rounds the 256 x 256 tiles' lead grows beyond the fixed
// rates below, and the whole-round rule after this function decides.) Modelled time of a plan: rounds of
// workgroups x one workgroup's MFMA work at the issue rate measured on MI355X
// (~45% of peak for the 128-row tiles, ~50% for 256 x 256), plus the split
// partials (written by the GEMM, about half of it hidden behind the MFMAs, and
// read back by the row kernel after it, at ~6 TB/s). The 128-row plan `p0`
// competes with 256 x 256 tiles over 1 to 8 K splits; the latter are taken
// only if the model puts them at least 5% ahead. Measured at 1024 rows: the
// 3584-wide QKV of the 28-layer shape went from 108 to 71 µs (3 splits), the
// 7B down projection from 202 to 197 µs; at 512 rows the 7B gate|up from 259
// to 224 µs.
static GemmPlan plan_mfma_bound(GemmPlan p0, int max_rows, int N, int K) {
  constexpr double kCuFlops = 2.5e15 / kComputeUnits;   // dense bf16 MFMA per CU
  auto rounds = [](long long wgs) { return (double)((wgs + kComputeUnits - 1) / kComputeUnits); };
  auto partials = [&](int sp) { return sp * (double)max_rows * N * 4.0 * 1.5 / 6e12; };
  const int mt0 = cdiv(max_rows, p0.bm);
  const double t0 = rounds((long long)cdiv(N, p0.bn) * mt0 * p0.splits) * 4.0 * p0.bm * p0.bn * p0.k_per_split /
                        (kCuFlops * 0.45) + partials(p0.splits);
  GemmPlan best = p0;
  double t_best = t0;
  for (int sp : {1, 2, 3, 4, 6, 8}) {
    const int kps = cdiv(cdiv(K, 32), sp) * 32;
    if (cdiv(K, kps) != sp || (sp > 1 && kps < 256)) continue;
    const double t = rounds((long long)cdiv(N, 256) * cdiv(max_rows, 256) * sp) * 4.0 * 256 * 256 * kps /
                         (kCuFlops * 0.50) + partials(sp);
    if (t < t_best && t < 0.95 * t0) {
      best = GemmPlan{1, 256, 256, sp, kps};
      t_best = t;
    }
  }
  return best;
}

GemmPlan plan_gemm(DType dt, int max_rows, int N, int K) {
  GemmPlan p;
  p.kind = 0;
  if (dt == DType::F32) {
    p.bm = 64;
    p.bn = 64;
    const int tiles = cdiv(N, p.bn) * cdiv(max_rows, p.bm);
    int splits = 1;
    while (tiles * splits < 384 && K / (splits * 2) >= 256 && splits < kMaxSplitsGemm) splits *= 2;
    p.k_per_split = cdiv(cdiv(K, 16), splits) * 16;
    p.splits = cdiv(K, p.k_per_split);
    return p;
  }
  // bf16 with at most 16 rows (a decode step): the weight stream.
  if (skinny_fits(dt, max_rows, N, K)) {
    p.kind = 2;
    p.bm = max_rows <= 16 ? 16 : 32;
    p.bn = 16;
    p.k_per_split = 2048 * skinny_kh(K);
    p.splits = cdiv(K, p.k_per_split);
    return p;
  }
  // bf16: one 8-wave workgroup per compute unit at a time. Take the widest weight
  // tile (256, 192 or 128 columns: wider tiles read fewer activation bytes from
  // LDS per MFMA) whose launch still reaches ~224 workgroups with at most 8
  // K splits; split K until it does, keeping at least 256 K per split.
  p.bm = 128;
  const int mt = cdiv(max_rows, p.bm);
  auto splits_for = [&](int bn) {
    int sp = 1;
    while (cdiv(N, bn) * mt * sp < 224 && K / (sp * 2) >= 256 && sp < kMaxSplitsGemm) sp *= 2;
    return sp;
  };
  p.bn = 128;
  for (int bn : {256, 192}) {
    if (cdiv(N, bn) * mt * splits_for(bn) >= 224) {
      p.bn = bn;
      break;
    }
  }
  const int splits = splits_for(p.bn);
  p.k_per_split = cdiv(cdiv(K, 64), splits) * 64;
  p.splits = cdiv(K, p.k_per_split);
  if (max_rows >= 512 && max_rows <= 1024) return plan_mfma_bound(p, max_rows, N, K);
  // 256 x 256 tiles when they fill at least one full round of workgroups without
  // splitting K and, counted in rounds of 256 workgroups, finish sooner: measured
  // on MI355X (split MFMA work, 4096 rows) the 256 x 256 kernel issues MFMAs at
  // ~50% of peak and the 128 x 256 kernel at ~45%.
  const int wide_wgs = cdiv(N, 256) * cdiv(max_rows, 256);
  if (p.splits == 1 && p.bn == 256 && wide_wgs >= kComputeUnits) {
    const double t_wide = cdiv(wide_wgs, kComputeUnits) * 2.0 / 0.50;
    const double t_dma = cdiv(cdiv(N, 256) * mt, kComputeUnits) * 1.0 / 0.45;
    if (t_wide < t_dma) {
      p.kind = 1;
      p.bm = 256;
      p.k_per_split = cdiv(K, 32) * 32;
    }
  }
  return p;
}

GemmPlan plan_gemm_kind(DType dt, int max_rows, int N, int K, int kind, int splits) {
  if (kind == 2) {   // the skinny kernel fixes its own splits (callers check skinny_fits)
    GemmPlan p{2, max_rows <= 16 ? 16 : 32, 16, 1, 2048 * skinny_kh(K)};
    p.splits = cdiv(K, p.k_per_split);
    return p;
  }
  GemmPlan p = plan_gemm(dt, max_rows, N, K);
  if (p.kind == 2 && kind < 0) return p;   // the planner's weight stream keeps its own splits
  if (p.kind == 2) {   // a forced dense kernel for a shape the planner streams
    p.kind = 0;
    p.bm = 128;
    p.bn = 128;
    int sp = 1;
    while (cdiv(N, 128) * sp < 224 && K / (sp * 2) >= 256 && sp < kMaxSplitsGemm) sp *= 2;
    p.k_per_split = cdiv(cdiv(K, 64), sp) * 64;
    p.splits = cdiv(K, p.k_per_split);
  }
  if (dt == DType::BF16 && kind == 1) {
    p.kind = 1;
    p.bm = 256;
    p.bn = 256;
  } else if (dt == DType::BF16 && kind == 0 && p.kind == 1) {
    p.kind = 0;
    p.bm = 128;
    p.k_per_split = cdiv(cdiv(K, 64), p.splits) * 64;
  }
  if (splits > 0 || p.kind == 1) {
    const int sp = splits > 0 ? splits : p.splits;
    const int kstep = dt == DType::F32 ? 16 : (p.kind == 1 ? 32 : 64);   // K elements per pipeline stage
    p.k_per_split = cdiv(cdiv(K, kstep), sp) * kstep;
    p.splits = cdiv(K, p.k_per_split);
  }
  return p;
}

namespace {
// The K-32 stage kernel for the plan's tile: 256 x 256, 128 x 512 or 128 x 256.
template <bool SWIGLU>
void launch_wide(const GemmPlan& p, dim3 grid, hipStream_t st, const void* A0, const void* A1, const void* W,
                 float* P, size_t split_stride, const Ctrl* c, int s, int max_rows, int N, int K) {
  const bf16 *a0 = static_cast<const bf16*>(A0), *a1 = static_cast<const bf16*>(A1), *w = static_cast<const bf16*>(W);
  const dim3 blk(kGemmWaves * 64);
  if (p.bm == 256)
    hipLaunchKernelGGL((k_gemm_wide<256, 256, 3, SWIGLU>), grid, blk, 0, st, a0, a1, w, P, split_stride, c, s,
                       max_rows, N, K, p.k_per_split);
  else if (p.bn == 512)
    hipLaunchKernelGGL((k_gemm_wide<128, 512, 3, SWIGLU>), grid, blk, 0, st, a0, a1, w, P, split_stride, c, s,
                       max_rows, N, K, p.k_per_split);
  else
    hipLaunchKernelGGL((k_gemm_wide<128, 256, 4, SWIGLU>), grid, blk, 0, st, a0, a1, w, P, split_stride, c, s,
                       max_rows, N, K, p.k_per_split);
}
}  // namespace

bool gate_up_fused(DType dt, const GemmPlan& p, int N) {
  return dt == DType::BF16 && p.kind == 1 && p.splits == 1 && N % 2 == 0;
}

hipError_t launch_gate_up_swiglu(DType dt, const GemmPlan& p, const void* A0, const void* A1, const void* W,
                                 float* P, size_t split_stride, const Ctrl* c, int s, int max_rows, int F, int K,
                                 void* a, hipStream_t st, const void* W_tiled) {
  if (!gate_up_fused(dt, p, 2 * F)) {
    hipError_t e = launch_gemm(dt, p, A0, A1, W, P, split_stride, c, s, max_rows, 2 * F, K, st, W_tiled);
    if (e != hipSuccess) return e;
    return launch_swiglu_post(dt, P, p.splits, split_stride, c, s, F, a, max_rows, st);
  }
  const dim3 grid(cdiv(F, p.bn / 2), cdiv(max_rows, p.bm), 1);
  launch_wide<true>(p, grid, st, A0, A1, W, static_cast<float*>(a), split_stride, c, s, max_rows, 2 * F, K);
  return hipGetLastError();
}

bool gemm_tiled(DType dt, const GemmPlan& p, const void* W_tiled, int N, int K) {
  return W_tiled && dt == DType::BF16 && p.kind == 0 && p.bn == kTileRows && N % kTileRows == 0 && K % 64 == 0 &&
         p.k_per_split % 64 == 0;
}

namespace {
// Column tile tx, K block kb (64 wide), row r, element e of the tiled copy sits
// at ((tx * (K / 64) + kb) * kTileRows + r) * 64 + e; one thread moves 16 bytes.
__global__ __launch_bounds__(256) void k_tile_rows(const bf16* __restrict__ W, bf16* __restrict__ out, int N, int K) {
  const size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x;   // 16-byte chunk of `out`
  if (idx >= (size_t)N * K / 8) return;
  const int e8 = (int)(idx % 8), r = (int)((idx / 8) % kTileRows);
  const size_t blk = idx / (8 * kTileRows);
  const int kb = (int)(blk % (size_t)(K / 64)), tx = (int)(blk / (size_t)(K / 64));
  *reinterpret_cast<uint4*>(out + idx * 8) =
      *reinterpret_cast<const uint4*>(W + ((size_t)tx * kTileRows + r) * K + (size_t)kb * 64 + e8 * 8);
}
}  // namespace

hipError_t launch_tile_rows(const void* W, void* out, int N, int K, hipStream_t st) {
  if (N % kTileRows || K % 64) return hipErrorInvalidValue;
  const size_t chunks = (size_t)N * K / 8;
  hipLaunchKernelGGL(k_tile_rows, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, st,
                     static_cast<const bf16*>(W), static_cast<bf16*>(out), N, K);
  return hipGetLastError();
}

hipError_t launch_gemm(DType dt, const GemmPlan& p, const void* A0, const void* A1, const void* W, float* P,
                       size_t split_stride, const Ctrl* c, int s, int max_rows, int N, int K, hipStream_t st,
                       const void* W_tiled) {
  if (dt == DType::BF16 && p.kind == 2) {
    const int wgps = std::max(1, std::min(cdiv(N, 16), kComputeUnits / p.splits));
    const dim3 sgrid(p.splits * wgps);
    const bf16 *a0 = static_cast<const bf16*>(A0), *a1 = static_cast<const bf16*>(A1);
    if (p.k_per_split != 2048 && p.k_per_split != 4096) return hipErrorInvalidValue;
    if (max_rows > kSkMaxRows || (max_rows > 16 && (p.bm != 32 || p.k_per_split != 2048)))
      return hipErrorInvalidValue;
    if (p.bm == 32)
      hipLaunchKernelGGL((k_gemm_skinny<1, 2>), sgrid, dim3(kGemmWaves * 64), 0, st, a0, a1,
                         static_cast<const bf16*>(W), P, split_stride, c, s, max_rows, N, K, wgps);
    else if (p.k_per_split == 2048)
      hipLaunchKernelGGL((k_gemm_skinny<1, 1>), sgrid, dim3(kGemmWaves * 64), 0, st, a0, a1,
                         static_cast<const bf16*>(W), P, split_stride, c, s, max_rows, N, K, wgps);
    else
      hipLaunchKernelGGL((k_gemm_skinny<2, 1>), sgrid, dim3(kGemmWaves * 64), 0, st, a0, a1,
                         static_cast<const bf16*>(W), P, split_stride, c, s, max_rows, N, K, wgps);
    return hipGetLastError();
  }
  const dim3 grid(cdiv(N, p.bn), cdiv(max_rows, p.bm), p.splits);
  if (dt == DType::BF16 && p.kind == 1) {
    launch_wide<false>(p, grid, st, A0, A1, W, P, split_stride, c, s, max_rows, N, K);
  } else if (dt == DType::F32) {
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, static_cast<const float*>(A0),
                       static_cast<const float*>(W), P, split_stride, c, s, max_rows, N, K, p.k_per_split);
  } else {
    const bf16 *a0 = static_cast<const bf16*>(A0), *a1 = static_cast<const bf16*>(A1);
    const bf16* w = static_cast<const bf16*>(W);
    // LDS: 144 KB (128 columns, 3 slots), 112 KB (192, 2), 128 KB (256, 2).
    if (gemm_tiled(dt, p, W_tiled, N, K))
      hipLaunchKernelGGL((k_gemm_dma<256, 2, true>), grid, dim3(kGemmWaves * 64), 0, st, a0, a1,
                         static_cast<const bf16*>(W_tiled), P, split_stride, c, s, max_rows, N, K, p.k_per_split);
    else if (p.bn == 256)
      hipLaunchKernelGGL((k_gemm_dma<256, 2>), grid, dim3(kGemmWaves * 64), 0, st, a0, a1, w, P, split_stride, c, s,
                         max_rows, N, K, p.k_per_split);
    else if (p.bn == 192)
      hipLaunchKernelGGL((k_gemm_dma<192, 2>), grid, dim3(kGemmWaves * 64), 0, st, a0, a1, w, P, split_stride, c, s,
                         max_rows, N, K, p.k_per_split);
    else
      hipLaunchKernelGGL((k_gemm_dma<128, 3>), grid, dim3(kGemmWaves * 64), 0, st, a0, a1, w, P, split_stride, c, s,
                         max_rows, N, K, p.k_per_split);
  }
  return hipGetLastError();
}

}  // namespace rksc
