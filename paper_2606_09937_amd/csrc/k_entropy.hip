// Fused lm_head -> softmax-entropy statistics (Eq. entropy) for the live
// branches' last-token rows. The logits z = W_lm hn are consumed in registers
// as they are produced: each lane folds its logits into an online triple
// (m = max z, s = sum e^(z-m), t = sum e^(z-m)(z-m)), triples are merged across
// lanes with wavefront shuffles and across waves through LDS, and one triple
// per workgroup and branch is written. Logits never reach HBM. A separate
// single-workgroup kernel merges the per-workgroup triples: H = log s - t/s.
//
// bf16: the kernel streams W_lm [V, d] from HBM exactly once per layer and
// contracts it against the normalised hidden rows with
// v_mfma_f32_16x16x32_bf16: W rows are the A operand, the branches the B
// columns (NCB blocks of 16). The hidden row is supplied as a bf16 hi + lo
// pair (two MFMAs into one fp32 accumulator), so the product keeps ~2^-16
// relative accuracy while W_lm stays in its bf16 storage format.
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

// Folds one MFMA output fragment into a lane's running triple: the lane holds
// z[row0 + i], i = 0..3, of its column; rows at or past V are left out.
__device__ __forceinline__ void fold4(EntStats& st, const floatx4& z, int row0, int V) {
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (row0 + i < V) mx = fmaxf(mx, z[i]);
  if (mx == -INFINITY) return;
  const float mn = fmaxf(st.m, mx);
  float s_new = 0.f, t_new = 0.f;
  if (st.m != -INFINITY) {
    const float dm = st.m - mn, sc = __expf(dm);
    s_new = st.s * sc;
    t_new = (st.t + st.s * dm) * sc;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (row0 + i < V) {
      const float dz = z[i] - mn, e = __expf(dz);
      s_new += e;
      t_new = fmaf(e, dz, t_new);
    }
  st = EntStats{mn, s_new, t_new};
}

// fold4 that also keeps the vocabulary index of the running maximum (the
// greedy token): the first row among equal maxima wins, as rows are visited in
// increasing order within a lane and merges keep the smaller index on ties.
__device__ __forceinline__ void fold4_am(EntStats& st, int& am, const floatx4& z, int row0, int V) {
  float mx = -INFINITY;
  int ix = 0x7fffffff;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (row0 + i < V && z[i] > mx) {
      mx = z[i];
      ix = row0 + i;
    }
  if (mx == -INFINITY) return;
  if (mx > st.m) am = ix;
  else if (mx == st.m) am = min(am, ix);
  fold4(st, z, row0, V);
}

// Index of the larger maximum of two (statistics, index) pairs; the smaller
// index on equal maxima; an empty side (m = -inf) has no index.
__device__ __forceinline__ int merge_am(const EntStats& a, int ia, const EntStats& b, int ib) {
  if (b.m > a.m) return ib;
  if (b.m < a.m) return ia;
  return min(ia, ib);
}

// lm_head stream through an R-deep LDS ring fed by direct DMA.
//
// The unit of the ring is 16 rows x 1 KB: a 512-wide K slice of 16 vocabulary
// rows of W, or of 16 hidden columns of one plane (hi or lo). Each DMA
// instruction moves one 1 KB row segment, so HBM sees 1 KB contiguous runs:
// runs of 128-512 B per row cost up to a fifth of the bandwidth on MI355X.
// Within a row the 16-byte chunk c sits at position c ^ (row & 15) (the lanes
// fetch permuted chunks of the same segment), so a 16-row fragment read hits
// 16 distinct bank groups.
//
// A workgroup (8 waves) owns a contiguous range of 16-row vocabulary tiles
// (the ranges of the grid differ by at most one tile) and walks it in groups
// of G tiles. Wave w serves column block w % NCB, K half (w / NCB) % 2 of the
// slice and owner group w / (2 NCB). For each 512-wide K slice of a group, the
// 2*NCB hidden units come first: every wave copies its column block's K half
// into registers (8 k-substeps x hi/lo). The group's G weight units follow;
// unit i is contracted by the 2*NCB waves of owner group i mod (4 / NCB), each
// over its K half (16 MFMAs), so a unit's work is spread over two SIMDs and
// the barrier of the next unit waits for at most that. After the group the two
// K halves of each tile are summed through LDS (one barrier per group) and
// the first-half wave folds the logits into its running statistics.
//
// Chunks at or past d are fetched from the row start (valid memory) and the
// hidden fragment is zeroed; rows past V are clamped and left out of the
// statistics; hidden columns past the live count read stale (allocated) rows
// and their statistics are never written.
// The explicit vmcnt wait + barrier is what orders the DMA writes before the
// fragment reads. The reads are typed bf16x8 loads: the compiler then treats
// them as not aliasing the untyped DMA stores and adds no wait of its own
// (with untyped reads it waits for every outstanding DMA, draining the ring).
constexpr int kUnitBytes = 16 * 1024;
constexpr int kEntRing = 7;
constexpr int kEntWaves8 = 8;                         // waves per workgroup
constexpr int kEntRedTiles = 4;                       // tiles per wave per reduction round
constexpr int kRedBytes = kEntWaves8 * kEntRedTiles * 1024;
constexpr int kFinBytes = kEntWaves8 * 16 * 16;       // one triple (+ argmax) per column per wave

// AM: also track the argmax (greedy token) and write (m, s, t, index) per
// column instead of the triple.
template <int NCB, int G, int R, bool AM>
__global__ __launch_bounds__(512) void k_entropy_bf16(const bf16* __restrict__ W, const bf16* __restrict__ hi,
                                                      const bf16* __restrict__ lo, const Ctrl* c, int V, int d,
                                                      int kmul, float* __restrict__ parts) {
  constexpr int NW = kEntWaves8;
  constexpr int IPW = 16 / NW;        // DMA instructions per wave per unit
  constexpr int TPW = NW / (2 * NCB); // owner groups; unit i goes to group i % TPW
  constexpr int LT = G / TPW;         // tiles per wave per group
  constexpr int HU = 2 * NCB;         // hidden units per slice
  static_assert(G % TPW == 0 && LT % kEntRedTiles == 0, "tile group must split over the waves and rounds");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * kUnitBytes + kRedBytes + kFinBytes];

  const int Bl = c->live_count * kmul;   // columns: kmul layers' rows of every live branch
  if (Bl == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int cbw = wid % NCB, kh = (wid / NCB) & 1, own = wid / (2 * NCB);
  const int T = (V + 15) / 16;
  const int t0 = (int)((long long)blockIdx.x * T / gridDim.x);
  const int t1 = (int)((long long)(blockIdx.x + 1) * T / gridDim.x);
  const int ntile = t1 - t0;
  const int ns = (d + 511) / 512;
  const int ng = (ntile + G - 1) / G;

  // Issue cursor (group, slice, unit) of the next ring unit; past the end the
  // first unit is fetched again (never consumed) so every step has the same
  // number of DMAs in flight.
  int cg = 0, cs = 0, cu = 0;
  auto issue = [&](int slot_idx) {
    uint8_t* slot = smem + slot_idx * kUnitBytes;
    const bool past = cg >= ng;
    const int g_ = past ? 0 : cg, s_ = past ? 0 : cs, u_ = past ? 0 : cu;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int r = IPW * wid + j;                // unit row filled by this instruction
      const int k = 512 * s_ + 8 * (lane ^ r);    // logical chunk lane ^ r of the segment
      const int kk = k < d ? k : 0;
      const bf16* src;
      if (u_ < HU) {
        const int col = 16 * (u_ >> 1) + r;
        src = ((u_ & 1) ? lo : hi) + (size_t)col * d + kk;   // rows past Bl: stale, never used
      } else {
        const int row = min(16 * (t0 + g_ * G + (u_ - HU)) + r, V - 1);
        src = W + (size_t)row * d + kk;
      }
      dma16(src, slot + r * 1024);
    }
    if (!past) {
      const int gt = min(G, ntile - cg * G);
      if (++cu == HU + gt) {
        cu = 0;
        if (++cs == ns) {
          cs = 0;
          ++cg;
        }
      }
    }
  };
  int qc = 0;   // ring units consumed
  auto step = [&]() -> const uint8_t* {
    // This thread's DMAs for unit qc have landed and its reads of unit qc-1
    // are complete; after the barrier every wave's are.
    wait_vmcnt_lds<IPW * (R - 2)>();
    __builtin_amdgcn_s_barrier();
    issue((qc + R - 1) % R);          // refills the slot unit qc-1 used
    const uint8_t* slot = smem + (qc % R) * kUnitBytes;
    ++qc;
    return slot;
  };
#pragma unroll
  for (int i = 0; i < R - 1; ++i) issue(i);

  const bf16x8 zero = {};
  EntStats st = ent_empty();
  int am = 0x7fffffff;
  bf16x8 hreg[2][8];
  floatx4 acc[LT];
  for (int gi = 0; gi < ng; ++gi) {
    const int gt = min(G, ntile - gi * G);
#pragma unroll
    for (int m = 0; m < LT; ++m) acc[m] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < ns; ++s) {
#pragma unroll
      for (int u = 0; u < HU; ++u) {
        const uint8_t* slot = step();
        if ((u >> 1) == cbw) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int lc = 4 * (8 * kh + j) + g;
            const bf16x8 v = *reinterpret_cast<const bf16x8*>(slot + r16 * 1024 + (lc ^ r16) * 16);
            hreg[u & 1][j] = 512 * s + 8 * lc < d ? v : zero;
          }
        }
      }
#pragma unroll
      for (int ii = 0; ii < G; ++ii) {
        if (ii < gt) {
          const uint8_t* slot = step();
          if (ii % TPW == own) {
            floatx4& ac = acc[ii / TPW];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const int lc = 4 * (8 * kh + j) + g;
              const bf16x8 a = *reinterpret_cast<const bf16x8*>(slot + r16 * 1024 + (lc ^ r16) * 16);
              ac = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hreg[0][j], ac, 0, 0, 0);
              ac = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hreg[1][j], ac, 0, 0, 0);
            }
          }
        }
      }
    }
    // Lane (r16, g) holds, over its K half, z[16 tile + 4 g + i] of column
    // 16 cbw + r16 for the wave's tiles ii = m * TPW + own. The second-half
    // wave hands its partials to its partner (wave - NCB) through LDS, four
    // tiles per round; after the last round the area is rewritten only at the
    // end of the next group, many barriers on.
    floatx4* red = reinterpret_cast<floatx4*>(smem + R * kUnitBytes);
#pragma unroll
    for (int rr = 0; rr < LT / kEntRedTiles; ++rr) {
      if (rr > 0) __builtin_amdgcn_s_barrier();   // the previous round is read
      if (kh == 1) {
#pragma unroll
        for (int m = 0; m < kEntRedTiles; ++m)
          red[((wid - NCB) * kEntRedTiles + m) * 64 + lane] = acc[rr * kEntRedTiles + m];
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the partials are in LDS
      __builtin_amdgcn_s_barrier();
      if (kh == 0) {
#pragma unroll
        for (int m = 0; m < kEntRedTiles; ++m) {
          const int ii = (rr * kEntRedTiles + m) * TPW + own;
          if (ii < gt) {
            const floatx4 z = acc[rr * kEntRedTiles + m] + red[(wid * kEntRedTiles + m) * 64 + lane];
            if constexpr (AM) fold4_am(st, am, z, 16 * (t0 + gi * G + ii) + 4 * g, V);
            else fold4(st, z, 16 * (t0 + gi * G + ii) + 4 * g, V);
          }
        }
      }
    }
  }
  wait_vmcnt<0>();   // drain the look-ahead DMAs before the workgroup can exit

  // Column triples: merge the four lane groups, then the waves of each column
  // block in a fixed order (second-half waves hold empty triples).
#pragma unroll
  for (int off = 16; off < 64; off <<= 1) {
    EntStats o{__shfl_xor(st.m, off, 64), __shfl_xor(st.s, off, 64), __shfl_xor(st.t, off, 64)};
    if constexpr (AM) am = merge_am(st, am, o, __shfl_xor(am, off, 64));
    st = ent_merge(st, o);
  }
  EntStats* fin = reinterpret_cast<EntStats*>(smem + R * kUnitBytes + kRedBytes);
  int* fin_am = reinterpret_cast<int*>(fin + NW * 16);
  if (lane < 16) {
    fin[wid * 16 + lane] = st;
    if constexpr (AM) fin_am[wid * 16 + lane] = am;
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the triples are in LDS
  __builtin_amdgcn_s_barrier();
  const int col = tid;
  if (col < 16 * NCB && col < Bl) {
    const int cb = col >> 4;
    EntStats v = fin[cb * 16 + (col & 15)];
    int va = AM ? fin_am[cb * 16 + (col & 15)] : 0;
#pragma unroll
    for (int p = 1; p < NW / NCB; ++p) {
      const EntStats o = fin[(p * NCB + cb) * 16 + (col & 15)];
      if constexpr (AM) va = merge_am(v, va, o, fin_am[(p * NCB + cb) * 16 + (col & 15)]);
      v = ent_merge(v, o);
    }
    if constexpr (AM) {
      float* pp = parts + ((size_t)blockIdx.x * 64 + col) * 4;
      pp[0] = v.m;
      pp[1] = v.s;
      pp[2] = v.t;
      pp[3] = __int_as_float(va);
    } else {
      float* pp = parts + ((size_t)blockIdx.x * 64 + col) * 3;
      pp[0] = v.m;
      pp[1] = v.s;
      pp[2] = v.t;
    }
  }
}

// fp32 models: each wave takes whole vocabulary rows, lanes stride over d.
template <bool AM>
__global__ __launch_bounds__(256) void k_entropy_f32(const float* __restrict__ W, const float* __restrict__ hn,
                                                     const Ctrl* c, int V, int d, int kmul,
                                                     float* __restrict__ parts) {
  const int Bl = c->live_count * kmul;
  if (Bl == 0) return;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  // Branch column `col` is owned by lane `col` (at most 64 branches).
  EntStats own = ent_empty();
  int own_am = 0x7fffffff;
  for (int row = blockIdx.x * kEntWaves + wid; row < V; row += gridDim.x * kEntWaves) {
    const float* wr = W + (size_t)row * d;
    for (int col = 0; col < Bl; ++col) {
      const float* hr = hn + (size_t)col * d;
      float acc = 0.f;
      for (int k = lane; k < d; k += 64) acc = fmaf(wr[k], hr[k], acc);
      acc = wave_sum(acc);
      if (lane == col) {
        float z = acc;
        if (AM && z > own.m) own_am = row;   // rows ascend within a wave: the first maximum is kept
        stats_fold(own, z, &z, 1);
      }
    }
  }
  __shared__ EntStats red[kEntWaves][64];
  __shared__ int red_am[kEntWaves][64];
  red[wid][lane] = own;
  red_am[wid][lane] = own_am;
  __syncthreads();
  const int col = threadIdx.x;
  if (col < Bl) {
    EntStats v = red[0][col];
    int va = red_am[0][col];
    for (int w = 1; w < kEntWaves; ++w) {
      if (AM) va = merge_am(v, va, red[w][col], red_am[w][col]);
      v = ent_merge(v, red[w][col]);
    }
    if (AM) {
      float* p = parts + ((size_t)blockIdx.x * 64 + col) * 4;
      p[0] = v.m;
      p[1] = v.s;
      p[2] = v.t;
      p[3] = __int_as_float(va);
    } else {
      float* p = parts + ((size_t)blockIdx.x * 64 + col) * 3;
      p[0] = v.m;
      p[1] = v.s;
      p[2] = v.t;
    }
  }
}

// Persistent grid: one 8-wave workgroup (146 KB of LDS: a 7-unit ring keeps
// 96 KB of the stream in flight) per compute unit (kComputeUnits).

int ent_ncb(int max_branches) { return max_branches <= 16 ? 1 : max_branches <= 32 ? 2 : 4; }

}  // namespace

int entropy_parts(DType dt, int V, int max_branches) {
  if (dt == DType::F32) {
    const int b = (V + kEntWaves - 1) / kEntWaves;
    return b < 256 ? b : 256;
  }
  const int tiles = (V + 15) / 16;
  const int grid = kComputeUnits;
  return tiles < grid ? tiles : grid;
}

namespace {
template <bool AM>
hipError_t launch_entropy_t(DType dt, const void* W, const void* hn_a, const void* hn_b, const Ctrl* c, int V,
                            int d, int max_branches, int kmul, float* parts, hipStream_t st) {
  const int blocks = entropy_parts(dt, V, max_branches);
  if (dt == DType::F32) {
    hipLaunchKernelGGL(k_entropy_f32<AM>, dim3(blocks), dim3(256), 0, st, static_cast<const float*>(W),
                       static_cast<const float*>(hn_a), c, V, d, kmul, parts);
    return hipGetLastError();
  }
  const bf16* w = static_cast<const bf16*>(W);
  const bf16* a = static_cast<const bf16*>(hn_a);
  const bf16* b = static_cast<const bf16*>(hn_b);
  switch (ent_ncb(max_branches)) {
    case 1:
      hipLaunchKernelGGL((k_entropy_bf16<1, 32, kEntRing, AM>), dim3(blocks), dim3(512), 0, st, w, a, b, c, V, d,
                         kmul, parts);
      break;
    case 2:
      hipLaunchKernelGGL((k_entropy_bf16<2, 64, kEntRing, AM>), dim3(blocks), dim3(512), 0, st, w, a, b, c, V, d,
                         kmul, parts);
      break;
    default:
      hipLaunchKernelGGL((k_entropy_bf16<4, 32, kEntRing, AM>), dim3(blocks), dim3(512), 0, st, w, a, b, c, V, d,
                         kmul, parts);
      break;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_entropy(DType dt, const void* W, const void* hn_a, const void* hn_b, const Ctrl* c, int V, int d,
                          int max_branches, float* parts, hipStream_t st, int kmul) {
  return launch_entropy_t<false>(dt, W, hn_a, hn_b, c, V, d, max_branches * kmul, kmul, parts, st);
}

hipError_t launch_entropy_argmax(DType dt, const void* W, const void* hn_a, const void* hn_b, const Ctrl* c, int V,
                                 int d, int max_branches, float* parts, hipStream_t st) {
  return launch_entropy_t<true>(dt, W, hn_a, hn_b, c, V, d, max_branches, 1, parts, st);
}

}  // namespace rksc
