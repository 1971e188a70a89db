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

// Wave triples -> block triple per column -> parts[block][col]. `red` is LDS
// scratch of kEntWaves * 16 * NCB triples that no DMA is still writing.
template <int NCB>
__device__ __forceinline__ void write_block_stats(EntStats (&st)[NCB], int Bl, float* parts, EntStats* red) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    EntStats v = st[cb];
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
      EntStats o{__shfl_xor(v.m, off, 64), __shfl_xor(v.s, off, 64), __shfl_xor(v.t, off, 64)};
      v = ent_merge(v, o);
    }
    if (lane < 16) red[wid * 16 * NCB + 16 * cb + lane] = v;
  }
  __syncthreads();
  const int col = threadIdx.x;
  if (col < 16 * NCB && col < Bl) {
    EntStats v = red[col];
    for (int w = 1; w < kEntWaves; ++w) v = ent_merge(v, red[w * 16 * NCB + col]);
    float* p = parts + ((size_t)blockIdx.x * 64 + col) * 3;
    p[0] = v.m;
    p[1] = v.s;
    p[2] = v.t;
  }
}

// lm_head stream through an R-deep LDS ring fed by direct DMA.
//
// A workgroup (4 waves) owns vocabulary tiles of 128 rows; the tiles of one
// workgroup are blockIdx.x, blockIdx.x + gridDim.x, ... and its K steps of 64
// run back to back across tiles, so the ring never drains between tiles. One
// ring slot holds the W tile's 64-wide K slice (128 rows x 128 B) and the same
// slice of the normalised hidden columns (NCB blocks of 16 columns, hi and lo
// planes, 128 B per column). Every DMA instruction moves 8 rows x 128 B, eight
// lanes per 128-byte line, so HBM reads are whole lines. Within a row the
// 16-byte chunk c is stored at position c ^ (row & 7); the swizzle is applied
// to the global address each lane fetches (the DMA writes lane L at 16 L), so
// the MFMA fragment reads of 16 consecutive rows spread over the banks.
// Wave w computes rows 32w .. 32w+31 of the tile (two 16-row MFMA tiles):
// per K step two k-substeps of 32, each tile times the hi and the lo plane.
// Chunks at or past d are fetched from the row start (valid memory) and the
// hidden fragment is zeroed on read; rows past V are clamped and left out of
// the statistics; hidden columns past the live count read column 0 and their
// statistics are never written.
// The explicit vmcnt wait + barrier is what orders the DMA writes before the
// fragment reads. The reads are typed bf16x8 loads: the compiler then treats
// them as not aliasing the untyped DMA stores and adds no wait of its own
// (with untyped reads it waits for every outstanding DMA, draining the ring).
constexpr int kEntRows = 128;

__device__ __forceinline__ int ent_swz(int row, int chunk) { return chunk ^ (row & 7); }

template <int NCB, int R>
__global__ __launch_bounds__(256) void k_entropy_bf16(const bf16* __restrict__ W, const bf16* __restrict__ hi,
                                                      const bf16* __restrict__ lo, const Ctrl* c, int V, int d,
                                                      float* __restrict__ parts) {
  constexpr int W_BYTES = kEntRows * 128;          // 16 KB
  constexpr int H_BYTES = NCB * 2 * 16 * 128;      // NCB x (hi, lo) x 16 columns x 128 B
  constexpr int SLOT = W_BYTES + H_BYTES;
  constexpr int W_INS = W_BYTES / 1024 / 4;        // DMA instructions per wave per step
  constexpr int H_INS = H_BYTES / 1024 / 4;
  constexpr int NDMA = W_INS + H_INS;
  static_assert(H_BYTES % 4096 == 0, "hidden slice must split evenly over 4 waves");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * SLOT];

  const int Bl = c->live_count;
  if (Bl == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ntiles = (V + kEntRows - 1) / kEntRows;
  const int nk = (d + 63) / 64;
  const int my_tiles = blockIdx.x < ntiles ? (ntiles - 1 - blockIdx.x) / gridDim.x + 1 : 0;
  const int total = my_tiles * nk;

  // DMA lane roles: lane L fills row/column (L >> 3) of its instruction's 8,
  // physical chunk L & 7, i.e. logical chunk (L & 7) ^ (L >> 3).
  const int sub = lane >> 3;
  const int lchunk = (lane & 7) ^ sub;
  const bf16* hsrc[H_INS];
  int hdst[H_INS];
#pragma unroll
  for (int j = 0; j < H_INS; ++j) {
    const int ins = wid * H_INS + j;           // 0 .. NCB*4-1: (cb, plane, 8-column group)
    const int cb = ins >> 2, plane = (ins >> 1) & 1, grp = ins & 1;
    const int col = 16 * cb + 8 * grp + sub;
    hsrc[j] = (plane ? lo : hi) + (size_t)(col < Bl ? col : 0) * d;
    hdst[j] = W_BYTES + ins * 1024;
  }
  auto issue = [&](int q) {
    uint8_t* slot = smem + (q % R) * SLOT;
    // Steps past the end re-read the block's first step (valid memory, never
    // used), which keeps every iteration's wait count the same.
    if (q >= total) q = 0;
    const int t = q / nk, ks = q - t * nk;
    const int v0 = (blockIdx.x + t * gridDim.x) * kEntRows;
    const int k = 64 * ks + 8 * lchunk;
    const int kk = k < d ? k : 0;
#pragma unroll
    for (int j = 0; j < W_INS; ++j) {
      const int ins = wid * W_INS + j;          // rows 8*ins .. 8*ins+7 of the tile
      const int row = min(v0 + 8 * ins + sub, V - 1);
      dma16(W + (size_t)row * d + kk, slot + ins * 1024);
    }
#pragma unroll
    for (int j = 0; j < H_INS; ++j) dma16(hsrc[j] + kk, slot + hdst[j]);
  };

  EntStats st[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) st[cb] = ent_empty();
  floatx4 acc[2][NCB];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[t][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
  const bf16x8 zero = {};

#pragma unroll
  for (int q = 0; q < R - 1; ++q) issue(q);

  for (int q = 0; q < total; ++q) {
    wait_vmcnt<NDMA * (R - 2)>();     // this thread's DMAs for step q have landed
    __builtin_amdgcn_s_barrier();     // every wave's DMAs for q landed; step q-1 fully consumed
    issue(q + R - 1);   // refills the slot step q-1 used
    const uint8_t* slot = smem + (q % R) * SLOT;
    const int t_loc = q / nk, ks = q - t_loc * nk;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
      const int chunk = 4 * kh + g;
      const bool kin = 64 * ks + 8 * chunk < d;
      bf16x8 a[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int row = 32 * wid + 16 * t + r16;
        a[t] = *reinterpret_cast<const bf16x8*>(slot + row * 128 + ent_swz(row, chunk) * 16);
      }
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        // Column r16 of block cb, plane p: instruction (cb, p, r16 >> 3), row r16 & 7.
        const int hoff = cb * 4096 + (r16 >> 3) * 1024 + (r16 & 7) * 128 + ent_swz(r16, chunk) * 16;
        const bf16x8 xh = *reinterpret_cast<const bf16x8*>(slot + W_BYTES + hoff);
        const bf16x8 xl = *reinterpret_cast<const bf16x8*>(slot + W_BYTES + hoff + 2048);
        const bf16x8 bh = kin ? xh : zero;
        const bf16x8 bl = kin ? xl : zero;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          acc[t][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], bh, acc[t][cb], 0, 0, 0);
          acc[t][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], bl, acc[t][cb], 0, 0, 0);
        }
      }
    }
    if (ks == nk - 1) {
      // Tile done: lane (r16, g) holds z[v0 + 32 wid + 16 t + 4 g + i] of column 16 cb + r16.
      const int vb = (blockIdx.x + t_loc * gridDim.x) * kEntRows + 32 * wid + 4 * g;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (vb + 16 * t + i < V) mx = fmaxf(mx, acc[t][cb][i]);
        if (mx != -INFINITY) {
          const float mn = fmaxf(st[cb].m, mx);
          float s_new = 0.f, t_new = 0.f;
          if (st[cb].m != -INFINITY) {
            const float dm = st[cb].m - mn, sc = __expf(dm);
            s_new = st[cb].s * sc;
            t_new = (st[cb].t + st[cb].s * dm) * sc;
          }
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (vb + 16 * t + i < V) {
                const float dz = acc[t][cb][i] - mn, e = __expf(dz);
                s_new += e;
                t_new = fmaf(e, dz, t_new);
              }
          st[cb] = EntStats{mn, s_new, t_new};
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[t][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  // Drain the look-ahead DMAs and let every wave finish its reads, then reuse
  // the ring for the cross-wave reduction.
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  write_block_stats<NCB>(st, Bl, parts, reinterpret_cast<EntStats*>(smem));
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

// Persistent grid: as many workgroups as are resident at once on MI355X's 256
// compute units (LDS per workgroup: 60 KB for <= 16 columns, 72 KB for <= 32,
// 96 KB for <= 64).
constexpr int kComputeUnits = 256;
constexpr int kEntRing = 3;

int ent_ncb(int max_branches) { return max_branches <= 16 ? 1 : max_branches <= 32 ? 2 : 4; }

}  // namespace

int entropy_parts(DType dt, int V, int max_branches) {
  if (dt == DType::F32) {
    const int b = (V + kEntWaves - 1) / kEntWaves;
    return b < 256 ? b : 256;
  }
  const int tiles = (V + kEntRows - 1) / kEntRows;
  const int grid = (ent_ncb(max_branches) <= 2 ? 2 : 1) * kComputeUnits;
  return tiles < grid ? tiles : grid;
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
  switch (ent_ncb(max_branches)) {
    case 1:
      hipLaunchKernelGGL((k_entropy_bf16<1, kEntRing>), dim3(blocks), dim3(256), 0, st, w, a, b, c, V, d, parts);
      break;
    case 2:
      hipLaunchKernelGGL((k_entropy_bf16<2, kEntRing>), dim3(blocks), dim3(256), 0, st, w, a, b, c, V, d, parts);
      break;
    default:
      hipLaunchKernelGGL((k_entropy_bf16<4, kEntRing>), dim3(blocks), dim3(256), 0, st, w, a, b, c, V, d, parts);
      break;
  }
  return hipGetLastError();
}

}  // namespace rksc
