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

#include <type_traits>

namespace rksc {

namespace {

constexpr int kAttnWaves = 8;    // waves per attention workgroup (16 query rows each)
constexpr int kAttnRing = 4;     // prefix K/V tiles in the LDS ring
constexpr float kLazyLog2 = 8.f; // slack of the softmax reference (log2 units): p <= 2^8
#ifndef RKSC_ATTN_XCD_ORDER
#define RKSC_ATTN_XCD_ORDER 1
#endif

// Maximum and sum over the four 16-lane rows of a wave (lanes l, l ^ 16, l ^ 32,
// l ^ 48), with the gfx950 row-swap moves instead of LDS permutes: with both
// operands x, v_permlane16_swap yields x's rows (0, 0, 2, 2) and (1, 1, 3, 3),
// and v_permlane32_swap its halves (lo, lo) and (hi, hi) (checked on the device).
__device__ __forceinline__ float rows_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// a if c, else zero; component-wise so that no address is selected (a select
// of struct lvalues keeps register arrays in scratch memory).
__device__ __forceinline__ uint4 keep_if(bool c, const uint4& a) {
  return make_uint4(c ? a.x : 0u, c ? a.y : 0u, c ? a.z : 0u, c ? a.w : 0u);
}

// Row `key` (a position in the shared prefix) of KV head kvh: the segment that
// holds the position (segments are in position order; the loop bound is uniform,
// so with one segment it is a single compare) and the row within it.
template <typename T, int HD>
__device__ __forceinline__ const T* prefix_row(const PrefixView& P, bool isv, int kvh, int key) {
  const void* base = isv ? P.v[0] : P.k[0];
  int off = key, ln = P.len[0];
  for (int j = 1; j < P.nseg; ++j) {
    if (key >= P.start[j]) {
      base = isv ? P.v[j] : P.k[j];
      off = key - P.start[j];
      ln = P.len[j];
    }
  }
  return static_cast<const T*>(base) + ((size_t)kvh * ln + off) * HD;
}

// V^T tile layout: row = head dimension, column = key position. Within each
// 32-key block the eight keys that one lane group feeds to a P.V MFMA
// ({4g..4g+3} and {16+4g..16+4g+3}, the keys whose probabilities the lane
// holds) are made adjacent, so a fragment is one 16-byte read; the 8-key groups
// are XOR-swizzled by the row's 8-dimension block so that the 4-key stores of
// neighbouring dimension blocks land in different banks.
__device__ __forceinline__ int vt_col(int dim, int key) {
  const int k = key & 31;
  const int pos = (key & 32) + ((k & 15) >> 2) * 8 + (k >> 4) * 4 + (k & 3);
  return pos ^ (((dim >> 3) & 7) << 3);
}

// Prefix K/V tiles are moved by DMA (global_load_lds) in their natural
// [key][dim] layout into R-slot LDS rings (one for K, one for V), several tiles ahead of the
// contraction. The 16-byte chunks of a key row are XOR-swizzled by the key:
// K by key & (CPR - 1), so that the 16 rows of a fragment read hit distinct
// banks; V by (key & (CPR/2 - 1)) << 1, which keeps chunk pairs together for
// the transposing reads. V^T fragments for O^T += V^T P^T come from
// ds_read_b64_tr_b16: within each 16-lane group, result lane i, element t is
// element (i mod 4) of source lane 4t + i/4, so a group whose lane j points at
// dims 4(j mod 4)..+3 of key k0 + j/4 receives dim i of keys k0..k0+3.
__device__ __forceinline__ int swz_k(int key, int cpr) { return key & (cpr - 1); }
__device__ __forceinline__ int swz_v(int key, int cpr) { return (key & (cpr / 2 - 1)) << 1; }

// The transposing reads are issued as inline assembly: the compiler cannot
// tell that the builtin's LDS read does not alias the ring's in-flight DMA
// writes and would drain the whole ring (vmcnt(0)) before every such read. The
// kernel's own wait + barrier already guarantee that the tile has landed; the
// results are made valid by an explicit lgkmcnt(0) that takes the fragments as
// operands, so no use of them can be scheduled before it.
typedef short shortx4 __attribute__((ext_vector_type(4)));
template <int OFF0, int OFF1>
__device__ __forceinline__ void lds_read_tr16_pair(uint32_t addr, shortx4& a, shortx4& b) {
  static_assert(OFF0 >= 0 && OFF1 < 65536, "ds offsets are 16-bit immediates");
  // Early-clobber outputs: the first read's destination must not share a
  // register with the address that the second read still uses.
  asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%3\n\tds_read_b64_tr_b16 %1, %2 offset:%4"
               : "=&v"(a), "=&v"(b)
               : "v"(addr), "i"(OFF0), "i"(OFF1));
}
template <int ND>
__device__ __forceinline__ void lds_wait_pairs(shortx4 (&a)[ND], shortx4 (&b)[ND]) {
  static_assert(ND == 4 || ND == 8, "head_dim 64 or 128");
  if constexpr (ND == 8)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(a[0]), "+v"(b[0]), "+v"(a[1]), "+v"(b[1]), "+v"(a[2]), "+v"(b[2]), "+v"(a[3]), "+v"(b[3]),
                   "+v"(a[4]), "+v"(b[4]), "+v"(a[5]), "+v"(b[5]), "+v"(a[6]), "+v"(b[6]), "+v"(a[7]), "+v"(b[7]));
  else
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(a[0]), "+v"(b[0]), "+v"(a[1]), "+v"(b[1]), "+v"(a[2]), "+v"(b[2]), "+v"(a[3]), "+v"(b[3]));
}

// Split-KV: the key tiles of a query tile -- the prefix tiles, then the own-span
// tiles up to its last query -- are divided evenly over `nchunks` workgroups,
// each writing an unnormalised partial output with its (max, sum) for the
// combine. (A merge by the last chunk to finish, found with an atomic ticket,
// needs device-scope release fences; on MI355X those write back the whole L2
// and cost far more than the separate combine launch.)
// Own-span tiles (fp32 keys/values of the branch itself) are staged through
// registers, split into bf16 hi/lo and stored to padded LDS tiles that reuse
// the ring's memory once the prefix tiles of the chunk are done; the next own
// tile is fetched while the current one is contracted.
// The contraction is instantiated per tile kind (full prefix tile, last
// partial prefix tile, own-span tile), so the MFMA sequences carry no branches
// and full prefix tiles no masking.
// Scores are formed in log2 units: the queries are pre-multiplied by
// log2(e)/sqrt(hd) before their hi/lo split, and the partial maxima in mlpart
// are in the same units.
// 8 waves x 16 query columns = 128 query rows per workgroup.
// PS: the probabilities meet V as a bf16 hi/lo pair (two MFMAs); without it, as
// bf16(p) alone (one MFMA, ~2^-9 relative rounding of each weight).
template <int HD, bool XB, bool PS = true, bool MS = false>
__global__ __launch_bounds__(512) void k_attn_bf16(const float* __restrict__ q, const PrefixView pre,
                                                   const float* __restrict__ ko,
                                                   const float* __restrict__ vo, void* __restrict__ o,
                                                   float* __restrict__ opart, float* __restrict__ mlpart,
                                                   const Ctrl* c, int s, int H, int Hkv, float sl2,
                                                   int nchunks, int max_rows) {
  const int n = pre.n;
  constexpr int NW = kAttnWaves, NT = NW * 64, QT = 16 * NW;
  constexpr int KT = 64;                   // keys per tile
  constexpr int CPR = HD / 8;              // 16-byte chunks per key row
  constexpr int ROW = HD * 2;              // bytes per key row
  constexpr int TB = KT * ROW;             // bytes of a K (or V) tile
  constexpr int SLOT = 2 * TB;             // one tile: K (in the K ring), V (in the V ring)
  constexpr int R = kAttnRing;
  constexpr int IPT = SLOT / 1024;         // 1 KB DMA instructions per tile
  static_assert(IPT % NW == 0, "every wave issues the same number of DMA instructions");
  constexpr int IPW = IPT / NW;
  constexpr int RPI = 1024 / ROW;          // key rows per DMA instruction
  constexpr int LDK = HD + 8;              // own-span K tile row stride (elements)
  constexpr int LDV = KT + 8;              // own-span V^T row stride (elements)
  constexpr int NC = HD / 32;              // 32-dim chunks of the QK^T contraction
  constexpr int ND = HD / 16;              // 16-dim tiles of the output
  constexpr int OK = KT * HD / 4 / NT;     // own-span K: 16-byte chunks (4 fp32) per thread
  constexpr int OVU = (KT * HD / 16 + NT - 1) / NT;   // own-span V: units of 4 keys x 4 dims
  static_assert(OK >= 1 && KT * HD / 4 % NT == 0, "own-span staging");
  static_assert((2 * KT * LDK + 2 * HD * LDV) * 2 <= R * SLOT, "own-span tiles fit in the ring");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[R * SLOT];
  uint16_t* const Ks0 = reinterpret_cast<uint16_t*>(smem);   // own span: K hi [KT][LDK]
  uint16_t* const Ks1 = Ks0 + KT * LDK;                        //            K lo
  uint16_t* const Vt0 = Ks1 + KT * LDK;                        //            V^T hi [HD][LDV]
  uint16_t* const Vt1 = Vt0 + HD * LDV;                        //            V^T lo

  // Work order. The hardware deals workgroups to the 8 XCDs round robin by
  // linear id, and each XCD has its own L2. In fused mode every branch's query
  // tiles of a KV head walk the same prefix tiles, so the linear ids are
  // re-dealt KV-head-major: XCD x takes a contiguous range of (head, branch,
  // query tile) work items, i.e. the workgroups of one head (Hkv = 8) or of a
  // part of one (fewer heads), and the head's prefix is fetched from HBM about
  // once per XCD instead of once per branch.
  int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
#if RKSC_ATTN_XCD_ORDER
  if constexpr (!XB) {
    const int NX = gridDim.x, NY = gridDim.y, NZ = gridDim.z, T = NX * NY * NZ;
    const int id = bx + NX * (by + NY * bz);
    const int x = id % 8, qq = id / 8;
    const int v = x * (T / 8) + min(x, T % 8) + qq;   // XCD x holds ids x, x+8, ...: T/8 (+1 for x < T%8)
    by = v / (NX * NZ);
    const int rr = v - by * NX * NZ;
    bx = rr % NX;
    bz = rr / NX;
  }
#endif
  // Fused mode: bz = chunk * slots + slot, rows of one branch.
  // XB mode: bz = chunk, rows of all live branches, prefix tiles only.
  const int B_slots = XB ? 1 : gridDim.z / nchunks;
  const int chunk = bz / B_slots;
  const int bslot = bz % B_slots;
  if (!XB && bslot >= c->live_count) return;
  const int kvh = by;
  const int G = H / Hkv;
  const int rows = XB ? c->live_count * s * G : G * s;
  const int row0 = bx * QT;
  if (row0 >= rows) return;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  // A wave whose 16 query rows all lie past the last row (a packed decode tile
  // of few branches) still issues its share of every tile's DMA and meets every
  // barrier, but forms no scores and contracts nothing.
  const bool wave_live = row0 + 16 * __builtin_amdgcn_readfirstlane(wid) < rows;

  const int i_max = min(s - 1, (min(row0 + QT - 1, rows - 1)) / G);
  const int n_ptiles = (n + KT - 1) / KT;
  const int n_full = n / KT;      // prefix tiles with no key past n - 1
  // Split-KV chunks by cost: an own-span tile (fp32 keys and values staged through
  // registers, three MFMAs per product) counts as two prefix tiles, so that the
  // chunk holding the own span is not the straggler. f(x) = tiles whose cost
  // interval starts below x (prefix tile i at i, own tile j at n_ptiles + 2j).
  const int n_own = XB ? 0 : i_max / KT + 1;
  const int cost = n_ptiles + 2 * n_own;
  auto tiles_below = [&](int x) { return min(n_ptiles, x) + min(n_own, max(0, (x - n_ptiles + 1) / 2)); };
  const int t_begin = tiles_below(chunk * cost / nchunks), t_end = tiles_below((chunk + 1) * cost / nchunks);

  // The query this lane owns as an MFMA column. Rows past the end compute a
  // duplicate of the last row and are not stored.
  const int rho_raw = row0 + 16 * wid + r16;
  const bool qvalid = rho_raw < rows;
  const int rho = qvalid ? rho_raw : rows - 1;
  const int slot = XB ? rho / (s * G) : bslot;
  const int rin = XB ? rho - slot * s * G : rho;
  const int qi = rin / G, h = kvh * G + rin % G;
  const size_t qrow = (size_t)slot * s + qi;
  // The lane's query, scaled to log2 units and split into hi/lo, is loaded
  // after the chunk's first tiles are requested, so that the two memory round
  // trips overlap.
  bf16x8 qh[NC], ql[NC];
  auto load_q = [&]() {
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const float* qp = q + (qrow * H + h) * HD + 32 * cc + 8 * g;
      const float4 a = *reinterpret_cast<const float4*>(qp), b = *reinterpret_cast<const float4*>(qp + 4);
      const float x[8] = {a.x * sl2, a.y * sl2, a.z * sl2, a.w * sl2, b.x * sl2, b.y * sl2, b.z * sl2, b.w * sl2};
      uint16_t hh[8], ll[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) split2(x[e], hh[e], ll[e]);
      qh[cc] = __builtin_bit_cast(bf16x8, make_uint4(pack2(hh[0], hh[1]), pack2(hh[2], hh[3]), pack2(hh[4], hh[5]),
                                                     pack2(hh[6], hh[7])));
      ql[cc] = __builtin_bit_cast(bf16x8, make_uint4(pack2(ll[0], ll[1]), pack2(ll[2], ll[3]), pack2(ll[4], ll[5]),
                                                     pack2(ll[6], ll[7])));
    }
  };

  floatx4 oacc[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) oacc[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;

  const float* Ko = ko + ((size_t)slot * Hkv + kvh) * s * HD;
  const float* Vo = vo + ((size_t)slot * Hkv + kvh) * s * HD;

  // ---- prefix DMA: instruction ins = j * NW + wid of a tile moves RPI key rows
  // of K (ins < IPT/2) or V; lane L fills physical chunk L % CPR of row L / CPR.
  // The first half of a wave's instructions move K, the rest V (IPT/2 is a
  // multiple of NW). The wave index is made uniform so that the LDS
  // destinations are scalar (M0) values; a full tile is addressed as a scalar
  // tile base plus this lane's fixed 32-bit byte offset dlane[j].
  static_assert((IPT / 2) % NW == 0, "K and V instructions of a wave are fixed by j");
  const int widu = __builtin_amdgcn_readfirstlane(wid);
  int dkey[IPW], dsrc[IPW], ddst[IPW];
  uint32_t dlane[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const bool isv = j * NW >= IPT / 2;
    const int i_in = j * NW + (isv ? widu - IPT / 2 : widu);
    const int key = (j * NW + wid - (isv ? IPT / 2 : 0)) * RPI + lane / CPR;
    const int ph = lane % CPR;
    const int lc = ph ^ (isv ? swz_v(key, CPR) : swz_k(key, CPR));
    dkey[j] = key;
    dsrc[j] = lc * 8;
    dlane[j] = (uint32_t)(key * ROW + lc * 16);
    ddst[j] = (isv ? R * TB : 0) + i_in * 1024;
  }
  // Transposing V reads: this lane points at key 4g + r16/4 of each 32-key
  // block (and 16 keys further, an immediate offset), dims 16dt + 4 (r16 % 4)
  // .. +3, i.e. logical 16-byte chunk 2dt + (r16 % 4)/2, half r16 % 2; with the
  // V swizzle 2m, m = key & (CPR/2 - 1) (the same for key + 16 and key + 32),
  // the physical chunk is 2 (dt ^ m) + (r16 % 4)/2.
  uint32_t voff[ND];
  {
    const int vk = 4 * g + (r16 >> 2);
    const int mv = swz_v(vk, CPR) >> 1;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
      voff[dt] = vk * ROW + 32 * (dt ^ mv) + 16 * ((r16 & 3) >> 1) + 8 * (r16 & 1);
  }
  // LDS byte address of the V ring, and of this lane's reads in a V tile at slot 0.
  const uint32_t vring = (uint32_t)reinterpret_cast<uintptr_t>(smem) + R * TB;
  uint32_t vaddr[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) vaddr[dt] = vring + voff[dt];

  // One segment (MS = false): every row from the one base, straight-line code.
  // Several (MS): a tile inside one segment addresses its rows from that
  // segment's base, found once per tile with scalar compares; only a tile that
  // straddles a segment boundary looks up each row. A per-row lookup in the
  // one-segment kernel cost it 13-18% (branches between the DMAs of a tile).
  const bf16* const Kp0 = static_cast<const bf16*>(pre.k[0]) + (size_t)kvh * pre.len[0] * HD;
  const bf16* const Vp0 = static_cast<const bf16*>(pre.v[0]) + (size_t)kvh * pre.len[0] * HD;
  auto issue = [&](int pt, int sl) {
    const int kbase = pt * KT;
    if constexpr (!MS) {
      if (kbase + KT <= n) {
        const char* const kt0 = reinterpret_cast<const char*>(Kp0 + (size_t)kbase * HD);
        const char* const vt0 = reinterpret_cast<const char*>(Vp0 + (size_t)kbase * HD);
#pragma unroll
        for (int j = 0; j < IPW; ++j) dma16((j * NW >= IPT / 2 ? vt0 : kt0) + dlane[j], smem + sl * TB + ddst[j]);
      } else {
#pragma unroll
        for (int j = 0; j < IPW; ++j) {
          const int key = min(kbase + dkey[j], n - 1);   // rows past n - 1 are masked in the contraction
          dma16((j * NW >= IPT / 2 ? Vp0 : Kp0) + (size_t)key * HD + dsrc[j], smem + sl * TB + ddst[j]);
        }
      }
    } else {
      int sg = 0;
      for (int j = 1; j < pre.nseg; ++j) sg = kbase >= pre.start[j] ? j : sg;
      const int klast = min(kbase + KT, n) - 1;
      if (sg + 1 == pre.nseg || klast < pre.start[sg + 1]) {
        const int kofs = kbase - pre.start[sg];   // row of the tile's first key within its segment
        const bf16* Kt = static_cast<const bf16*>(pre.k[sg]) + ((size_t)kvh * pre.len[sg] + kofs) * HD;
        const bf16* Vt = static_cast<const bf16*>(pre.v[sg]) + ((size_t)kvh * pre.len[sg] + kofs) * HD;
#pragma unroll
        for (int j = 0; j < IPW; ++j) {
          const int key = min(kbase + dkey[j], n - 1);
          dma16((j * NW >= IPT / 2 ? Vt : Kt) + (size_t)(key - kbase) * HD + dsrc[j], smem + sl * TB + ddst[j]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < IPW; ++j) {
          const int key = min(kbase + dkey[j], n - 1);
          dma16(prefix_row<bf16, HD>(pre, j * NW >= IPT / 2, kvh, key) + dsrc[j], smem + sl * TB + ddst[j]);
        }
      }
    }
  };

  // ---- own-span staging (fused mode): fetch_own loads a tile's fp32 keys and
  // values into registers (in flight while the previous tile is contracted),
  // store_own splits them into hi/lo and stores the padded LDS tiles.
  uint4 stg[OK];
  uint4 vstg[OVU][4];
  auto fetch_own = [&](int kbase) {
    const float* kt = Ko + (size_t)kbase * HD;
    const int kmax = s - 1 - kbase;
#pragma unroll
    for (int j = 0; j < OK; ++j) {
      const int idx = tid + NT * j, key = idx / (HD / 4), dq = idx % (HD / 4);
      stg[j] = ldg16(kt + (key <= kmax ? key : kmax) * HD + dq * 4);
    }
#pragma unroll
    for (int u = 0; u < OVU; ++u) {
      const int idx = min(tid + NT * u, KT * HD / 16 - 1);   // units past the tile repeat its last (unused)
      const int dq = idx % (HD / 4), kg = idx / (HD / 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kbase + 4 * kg + e;
        vstg[u][e] = ldg16(Vo + (size_t)(key < s ? key : 0) * HD + dq * 4);
      }
    }
  };
  auto store_own = [&](int kbase) {
#pragma unroll
    for (int j = 0; j < OK; ++j) {
      const int idx = tid + NT * j, key = idx / (HD / 4), dq = idx % (HD / 4);
      const float4 kf = __builtin_bit_cast(float4, keep_if(kbase + key < s, stg[j]));
      uint16_t kh[4], kl[4];
      split2(kf.x, kh[0], kl[0]); split2(kf.y, kh[1], kl[1]); split2(kf.z, kh[2], kl[2]); split2(kf.w, kh[3], kl[3]);
      *reinterpret_cast<uint2*>(&Ks0[key * LDK + dq * 4]) = make_uint2(pack2(kh[0], kh[1]), pack2(kh[2], kh[3]));
      *reinterpret_cast<uint2*>(&Ks1[key * LDK + dq * 4]) = make_uint2(pack2(kl[0], kl[1]), pack2(kl[2], kl[3]));
    }
#pragma unroll
    for (int u = 0; u < OVU; ++u) {
      const int idx = tid + NT * u;
      if (idx < KT * HD / 16) {
        const int dq = idx % (HD / 4), kg = idx / (HD / 4);
        float x[4][4];   // x[e][k]: dimension 4dq + k of key 4kg + e
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ok = kbase + 4 * kg + e < s;
          const uint4 v = keep_if(ok, vstg[u][e]);
          x[e][0] = __uint_as_float(v.x);
          x[e][1] = __uint_as_float(v.y);
          x[e][2] = __uint_as_float(v.z);
          x[e][3] = __uint_as_float(v.w);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int dim = dq * 4 + k;
          uint16_t hh[4], lw[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) split2(x[e][k], hh[e], lw[e]);
          const int col = vt_col(dim, 4 * kg);
          *reinterpret_cast<uint2*>(&Vt0[dim * LDV + col]) = make_uint2(pack2(hh[0], hh[1]), pack2(hh[2], hh[3]));
          *reinterpret_cast<uint2*>(&Vt1[dim * LDV + col]) = make_uint2(pack2(lw[0], lw[1]), pack2(lw[2], lw[3]));
        }
      }
    }
  };

  // Contraction of one tile with this lane's query, in three parts so that the
  // prefix loop can overlap them across tiles:
  // - scores: S^T = K Q^T relative to the lane's softmax reference (the MFMA
  //   accumulator starts at -m, or at 0 while no key has been seen), so the
  //   lane holds score - m of keys 16*kt + 4g + i of its query;
  // - stats: mask, tile maximum, reference update;
  // - pv: p = 2^(score - m), then O^T += V^T P^T.
  // OWN: a padded own-span tile whose keys and values are hi/lo pairs (three
  // MFMAs per product), causal mask; otherwise the prefix tile in ring slot
  // `sl`: an int, or a std::integral_constant so that every LDS offset of the
  // tile is an instruction immediate. MASKED: some keys of the tile are invalid
  // for some query.
  auto scores = [&](auto own_c, auto sl, floatx4 (&sc)[4]) {
    constexpr bool OWN = decltype(own_c)::value;
    const float bias = m == -INFINITY ? 0.f : -m;
    const uint8_t* Kt = smem + (int)sl * TB;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      sc[kt] = floatx4{bias, bias, bias, bias};
      const int key = 16 * kt + r16;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) {
        if constexpr (OWN) {
          const int off = key * LDK + 32 * cc + 8 * g;
          const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(&Ks0[off]);
          const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(&Ks1[off]);
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qh[cc], sc[kt], 0, 0, 0);
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, ql[cc], sc[kt], 0, 0, 0);
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qh[cc], sc[kt], 0, 0, 0);
        } else {
          const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(Kt + key * ROW + ((4 * cc + g) ^ swz_k(key, CPR)) * 16);
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qh[cc], sc[kt], 0, 0, 0);
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, ql[cc], sc[kt], 0, 0, 0);
        }
      }
    }
  };
  // Online softmax with a lazily moved reference: the probabilities are
  // p = 2^(score - m) for a per-query reference m that moves only when a tile's
  // maximum exceeds it by more than kLazyLog2 (then to that maximum, rescaling
  // l and the accumulator by 2^(m_old - m_new)). Otherwise p <= 2^kLazyLog2 and
  // the tile needs no rescale: the accumulators are exact sums relative to m
  // either way, and the final normalisation by l (or the combine's weights
  // 2^(m_c - M)) cancels the choice of m. The move is decided per lane (the four
  // lanes of a query see the same tile maximum), and the rescale runs behind a
  // wave-uniform branch that, past the first tiles, is rarely taken. The
  // scores arrive relative to the reference in force when they were formed,
  // which is the current one (no update comes between a tile's scores and its
  // stats); a move shifts them to the new reference.
  auto stats = [&](auto own_c, auto masked_c, int kbase, floatx4 (&sc)[4]) {
    constexpr bool OWN = decltype(own_c)::value;
    constexpr bool MASKED = decltype(masked_c)::value;
    if constexpr (MASKED) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kbase + 16 * kt + 4 * g + i;
          if (!(OWN ? key <= qi : key < n)) sc[kt][i] = -INFINITY;
        }
    }
    float mt = fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3]));
#pragma unroll
    for (int kt = 1; kt < 4; ++kt) mt = fmaxf(mt, fmaxf(fmaxf(sc[kt][0], sc[kt][1]), fmaxf(sc[kt][2], sc[kt][3])));
    mt = rows_max(mt);
    // mt is relative to the scores' reference: m, or 0 while m = -inf (then any
    // finite maximum moves it; a fully masked tile, mt = -inf, never does).
    const bool fresh = m == -INFINITY;
    const bool up = fresh ? mt > -INFINITY : mt > kLazyLog2;
    if (__builtin_amdgcn_ballot_w64(up) != 0) {
      const float shift = up ? mt : 0.f;                 // new reference - old, in score units
      const float alpha = up && !fresh ? __builtin_amdgcn_exp2f(-mt) : (fresh ? 0.f : 1.f);
      m = up ? (fresh ? mt : m + mt) : m;
      l *= alpha;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) oacc[dt] *= alpha;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) sc[kt] -= shift;
    }
  };
  auto pv = [&](auto own_c, auto sl, floatx4 (&sc)[4]) {
    constexpr bool OWN = decltype(own_c)::value;
    float p[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[kt][i] = __builtin_amdgcn_exp2f(sc[kt][i]);   // masked (and no key yet): exp2(-inf) = 0
        l += p[kt][i];
      }
    // O^T += V^T P^T over two 32-key blocks; lane group g supplies keys
    // {32kb + 4g + e, 32kb + 16 + 4g + e}, e = 0..3, in both operands.
    auto block = [&](auto kb_c) {
      constexpr int kb = decltype(kb_c)::value;
      // hi/lo split of the probabilities, two at a time: hi = bf16(p) packed
      // by one conversion, lo = bf16(p - hi) likewise.
      uint32_t ph[4], pl[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const float p0 = p[2 * kb + (e2 >> 1)][2 * (e2 & 1)], p1 = p[2 * kb + (e2 >> 1)][2 * (e2 & 1) + 1];
        if constexpr (PS) {
          split2x2(p0, p1, ph[e2], pl[e2]);
        } else {
          typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
          typedef float floatx2_t __attribute__((ext_vector_type(2)));
          ph[e2] = __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{p0, p1}, bf16x2_t));
        }
      }
      const bf16x8 pbh = __builtin_bit_cast(bf16x8, make_uint4(ph[0], ph[1], ph[2], ph[3]));
      const bf16x8 pbl = __builtin_bit_cast(bf16x8, make_uint4(pl[0], pl[1], pl[2], pl[3]));
      shortx4 vlo[ND], vhi[ND];
      if constexpr (!OWN) {
        if constexpr (std::is_integral_v<decltype(sl)>) {
          const uint32_t vb = vring + sl * TB + kb * 32 * ROW;
#pragma unroll
          for (int dt = 0; dt < ND; ++dt) lds_read_tr16_pair<0, 16 * ROW>(vb + voff[dt], vlo[dt], vhi[dt]);
        } else {
          constexpr int IMM = decltype(sl)::value * TB + kb * 32 * ROW;
#pragma unroll
          for (int dt = 0; dt < ND; ++dt) lds_read_tr16_pair<IMM, IMM + 16 * ROW>(vaddr[dt], vlo[dt], vhi[dt]);
        }
        lds_wait_pairs<ND>(vlo, vhi);
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        bf16x8 v0;
        if constexpr (OWN) {
          const int dim = 16 * dt + r16;
          v0 = *reinterpret_cast<const bf16x8*>(&Vt0[dim * LDV + vt_col(dim, 32 * kb + 4 * g)]);
        } else {
          v0 = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vlo[dt], vhi[dt], 0, 1, 2, 3, 4, 5, 6, 7));
        }
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, pbh, oacc[dt], 0, 0, 0);
        if constexpr (PS) oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v0, pbl, oacc[dt], 0, 0, 0);
        if constexpr (OWN) {
          const int dim = 16 * dt + r16;
          const bf16x8 v1 = *reinterpret_cast<const bf16x8*>(&Vt1[dim * LDV + vt_col(dim, 32 * kb + 4 * g)]);
          oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v1, pbh, oacc[dt], 0, 0, 0);
        }
      }
    };
    block(std::integral_constant<int, 0>{});
    block(std::integral_constant<int, 1>{});
  };
  auto contract = [&](auto own_c, auto masked_c, int sl, int kbase) {
    floatx4 sc[4];
    scores(own_c, sl, sc);
    stats(own_c, masked_c, kbase, sc);
    pv(own_c, sl, sc);
  };

  // ---- prefix tiles of this chunk through the ring, software-pipelined: the
  // scores of tile i+1 (MFMA) are formed in the same scheduling region as the
  // softmax of tile i (VALU), so the two overlap on the SIMD. Every step issues
  // one tile (past the end: a harmless re-fetch of the first); at step i the
  // DMA instructions behind tile i+1 are those of tiles i+2 .. i+R-2. The loop
  // is unrolled R times so that tile i's slot, i % R, is a compile-time
  // constant; the score arrays alternate between two register sets.
  const int p_end = min(t_end, n_ptiles);
  const int np = p_end - t_begin;
  if (np > 0) {
    static_assert(R >= 3 && R % 2 == 0, "the pipelined loop needs a slot for tile i+1 and one being refilled");
#pragma unroll
    for (int u = 0; u < R - 1; ++u) issue(t_begin + (u < np ? u : 0), u);
    if (wave_live) load_q();   // loads complete in order: the wait for the query covers these tiles too
    wait_vmcnt_lds<IPW * (R - 2)>();   // tile 0
    __builtin_amdgcn_s_barrier();
    floatx4 sca[4], scb[4];
    if (wave_live) scores(std::false_type{}, std::integral_constant<int, 0>{}, sca);
    // Tiles before the chunk's last are never partial (only the prefix's last
    // tile can be, and it is the last of its chunk).
    int i = 0;
    auto step = [&](auto sl_c) {
      constexpr int SL = decltype(sl_c)::value;
      wait_vmcnt_lds<IPW * (R - 3)>();   // tile i+1 has landed; every wave is done with slot (i-1) % R
      __builtin_amdgcn_s_barrier();
      const int nx = i + R - 1;
      issue(t_begin + (nx < np ? nx : 0), (SL + R - 1) % R);
      auto body = [&](floatx4 (&cur)[4], floatx4 (&nxt)[4]) {
        if (!wave_live) return;
        stats(std::false_type{}, std::false_type{}, (t_begin + i) * KT, cur);
        scores(std::false_type{}, std::integral_constant<int, (SL + 1) % R>{}, nxt);
        pv(std::false_type{}, sl_c, cur);
      };
      if constexpr (SL % 2 == 0) body(sca, scb);
      else body(scb, sca);
      ++i;
    };
    static_assert(R == 4, "the unrolled loop below has R steps");
    while (true) {
      if (i + 1 >= np) break;
      step(std::integral_constant<int, 0>{});
      if (i + 1 >= np) break;
      step(std::integral_constant<int, 1>{});
      if (i + 1 >= np) break;
      step(std::integral_constant<int, 2>{});
      if (i + 1 >= np) break;
      step(std::integral_constant<int, 3>{});
    }
    const int pl = t_begin + np - 1;
    auto finish = [&](floatx4 (&last)[4]) {
      if (!wave_live) return;
      if (pl < n_full) stats(std::false_type{}, std::false_type{}, pl * KT, last);
      else stats(std::false_type{}, std::true_type{}, pl * KT, last);
      pv(std::false_type{}, (np - 1) % R, last);
    };
    if ((np - 1) % 2 == 0) finish(sca);   // two copies: register arrays cannot be selected at run time
    else finish(scb);
    // The trailing re-fetches must land before the ring memory is reused or the
    // workgroup ends.
    wait_vmcnt<0>();
    __syncthreads();
  }

  // ---- own-span tiles of this chunk (fused mode)
  const int o_begin = max(t_begin, n_ptiles);
  if (!XB && o_begin < t_end) {
    fetch_own((o_begin - n_ptiles) * KT);
    if (np <= 0 && wave_live) load_q();   // a chunk of own-span tiles only
    for (int t = o_begin; t < t_end; ++t) {
      const int kbase = (t - n_ptiles) * KT;
      store_own(kbase);
      __syncthreads();
      if (t + 1 < t_end) fetch_own(kbase + KT);   // in flight while this tile is contracted
      if (wave_live) contract(std::true_type{}, std::true_type{}, 0, kbase);
      __syncthreads();
    }
  }

  l = rows_sum(l);
  const size_t plane = (size_t)max_rows * H * HD;
  if (!XB && nchunks == 1) {
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

// Merges the split-KV partials of each (row, head), with maxima in log2 units:
// o = sum_c 2^{m_c - M} o_c / sum_c 2^{m_c - M} l_c, M = max_c m_c.
// A chunk that saw no key for a query (m = -inf) contributes nothing. One wave
// per (row, head): lane c < nchunks reads chunk c's (m, l), the wave reduces
// the maximum, and each lane then sums its HD/64 dimensions over the chunks.
template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine(const float* __restrict__ opart, const float* __restrict__ mlpart,
                                                      void* __restrict__ o, const Ctrl* c, int s, int H,
                                                      int nchunks, int max_rows) {
  const int rows = c->live_count * s * H;
  const int wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  if (wid >= rows) return;    // one wave per (row, head)
  const size_t cstride = (size_t)max_rows * H;
  float acc[HD / 64];
#pragma unroll
  for (int j = 0; j < HD / 64; ++j) acc[j] = 0.f;
  float den = 0.f;
  float Mx = -INFINITY;
  if (nchunks <= 8) {
    // Up to 8 chunks: every load (the partials and each chunk's (m, l)) is issued
    // before the first wait, so the merge costs one memory round trip.
    float v[8][HD / 64];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int j = 0; j < HD / 64; ++j)
        v[u][j] = u < nchunks ? opart[((size_t)u * cstride + wid) * HD + lane + 64 * j] : 0.f;
    float2 ml = make_float2(-INFINITY, 0.f);
    if (lane < nchunks) ml = *reinterpret_cast<const float2*>(mlpart + (lane * cstride + wid) * 2);
    float M = ml.x;
#pragma unroll
    for (int off = 4; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
    const float w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - M);
    float wl = w * ml.y;
#pragma unroll
    for (int off = 4; off >= 1; off >>= 1) wl += __shfl_xor(wl, off, 64);
    den = __shfl(wl, 0, 64);   // lanes 0..7 hold the chunks' sum
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float wk = __shfl(w, u, 64);
#pragma unroll
      for (int j = 0; j < HD / 64; ++j) acc[j] += wk * v[u][j];
    }
    nchunks = 0;   // skips the general loops below
  }
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int ch = c0 + lane;
    const float mc = ch < nchunks ? mlpart[(ch * cstride + wid) * 2] : -INFINITY;
    float M = mc;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
    Mx = fmaxf(Mx, M);
  }
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int ch = c0 + lane;
    float w = 0.f, wl = 0.f;
    if (ch < nchunks) {
      const float2 ml = *reinterpret_cast<const float2*>(mlpart + (ch * cstride + wid) * 2);
      w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - Mx);
      wl = w * ml.y;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) wl += __shfl_xor(wl, off, 64);
    den += wl;
    // Every chunk wrote its partial (zeros where it saw no key), so the loads
    // are independent of the weights and can all be in flight.
    const int cn = min(64, nchunks - c0);
    int k = 0;
    for (; k + 8 <= cn; k += 8) {
      float v[8][HD / 64];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float* op = opart + ((size_t)(c0 + k + u) * cstride + wid) * HD;
#pragma unroll
        for (int j = 0; j < HD / 64; ++j) v[u][j] = op[lane + 64 * j];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float wk = __shfl(w, k + u, 64);
#pragma unroll
        for (int j = 0; j < HD / 64; ++j) acc[j] += wk * v[u][j];
      }
    }
    for (; k < cn; ++k) {
      const float wk = __shfl(w, k, 64);
      const float* op = opart + ((size_t)(c0 + k) * cstride + wid) * HD;
#pragma unroll
      for (int j = 0; j < HD / 64; ++j) acc[j] += wk * op[lane + 64 * j];
    }
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

// XB-mode merge: the prefix partials of each (row, head) plus the row's own
// causal span, whose few keys (G * s < 64, so s < 64) are scored here in fp32:
// o = (sum_c 2^{m_c - M} o_c + sum_{j <= i} 2^{t_j - M} v_j) / (sum_c 2^{m_c - M} l_c + sum_j 2^{t_j - M}),
// t_j = log2(e)/sqrt(hd) q.k_j, M the maximum of all m_c and t_j. One wave per (row, head).
template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine_own(const float* __restrict__ opart,
                                                          const float* __restrict__ mlpart,
                                                          const float* __restrict__ q, const float* __restrict__ ko,
                                                          const float* __restrict__ vo, void* __restrict__ o,
                                                          const Ctrl* c, int s, int H, int Hkv, float sl2,
                                                          int nchunks, int max_rows) {
  constexpr int E = HD / 64;   // dimensions per lane
  const int rows = c->live_count * s * H;
  const int wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  if (wid >= rows) return;
  const int qrow = wid / H, h = wid - qrow * H;
  const int slot = qrow / s, qi = qrow - slot * s, kvh = h / (H / Hkv);
  const size_t cstride = (size_t)max_rows * H;
  float Mx = -INFINITY;
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int ch = c0 + lane;
    float M = ch < nchunks ? mlpart[(ch * cstride + wid) * 2] : -INFINITY;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
    Mx = fmaxf(Mx, M);
  }
  float qv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) qv[e] = q[(size_t)wid * HD + lane + 64 * e] * sl2;
  const float* kb = ko + ((size_t)slot * Hkv + kvh) * s * HD;
  const float* vb = vo + ((size_t)slot * Hkv + kvh) * s * HD;
  float my_t = -INFINITY;   // lane j keeps the score of own key j
  for (int j = 0; j <= qi; ++j) {
    float part = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) part = fmaf(qv[e], kb[(size_t)j * HD + lane + 64 * e], part);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
    if (lane == j) my_t = part;
    Mx = fmaxf(Mx, part);
  }
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  float den = 0.f;
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int ch = c0 + lane;
    float w = 0.f, wl = 0.f;
    if (ch < nchunks) {
      const float2 ml = *reinterpret_cast<const float2*>(mlpart + (ch * cstride + wid) * 2);
      w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - Mx);
      wl = w * ml.y;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) wl += __shfl_xor(wl, off, 64);
    den += wl;
    // Every chunk wrote its partial (zeros where it saw no key), so the loads
    // do not depend on the weights and can all be in flight.
    const int cn = min(64, nchunks - c0);
    int k = 0;
    for (; k + 8 <= cn; k += 8) {
      float v[8][E];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float* op = opart + ((size_t)(c0 + k + u) * cstride + wid) * HD;
#pragma unroll
        for (int e = 0; e < E; ++e) v[u][e] = op[lane + 64 * e];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float wk = __shfl(w, k + u, 64);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] += wk * v[u][e];
      }
    }
    for (; k < cn; ++k) {
      const float wk = __shfl(w, k, 64);
      const float* op = opart + ((size_t)(c0 + k) * cstride + wid) * HD;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] += wk * op[lane + 64 * e];
    }
  }
  for (int j = 0; j <= qi; ++j) {
    const float p = __builtin_amdgcn_exp2f(__shfl(my_t, j, 64) - Mx);
    den += p;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += p * vb[(size_t)j * HD + lane + 64 * e];
  }
  const float inv = 1.f / den;
  const size_t plane = (size_t)max_rows * H * HD;
  uint16_t* ob = reinterpret_cast<uint16_t*>(o);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    uint16_t hb, lb;
    split2(acc[e] * inv, hb, lb);
    ob[(size_t)wid * HD + lane + 64 * e] = hb;
    ob[plane + (size_t)wid * HD + lane + 64 * e] = lb;
  }
}

// Decode merge: one new token per branch (s = 1). One wave per (branch, head)
// combines the prefix partials of the split-KV chunks with the branch's own
// keys -- its cached entries 0..len-1 (bf16) and the new token's own key
// (fp32, entry len) -- in log2 units:
// o = (sum_c 2^{m_c - M} o_c + sum_j 2^{t_j - M} v_j) / (sum_c 2^{m_c - M} l_c + sum_j 2^{t_j - M}),
// t_j = log2(e)/sqrt(hd) q.k_j. The cached keys are scored 64 at a time, one
// per lane (16-byte loads of the key row; the query address is wave-uniform),
// with an online maximum across the blocks of 64; the own key is scored by the
// whole wave. Value rows and chunk partials are loaded DEC_BATCH at a time so
// that their loads are in flight together.
constexpr int kDecBatch = 16;

template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine_dec(const float* __restrict__ opart,
                                                          const float* __restrict__ mlpart,
                                                          const float* __restrict__ q, const bf16* __restrict__ ck,
                                                          const bf16* __restrict__ cv, int len, int cap,
                                                          const float* __restrict__ ko, const float* __restrict__ vo,
                                                          void* __restrict__ o, const Ctrl* c, int H, int Hkv,
                                                          float sl2, int nchunks, int max_rows) {
  constexpr int E = HD / 64;   // dimensions per lane
  const int rows = c->live_count * H;
  const int wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  if (wid >= rows) return;
  const int b = wid / H, h = wid - b * H, kvh = h / (H / Hkv);
  const float* qr = q + (size_t)wid * HD;
  const uint16_t* kb = reinterpret_cast<const uint16_t*>(ck) + ((size_t)b * Hkv + kvh) * cap * HD;
  const uint16_t* vb = reinterpret_cast<const uint16_t*>(cv) + ((size_t)b * Hkv + kvh) * cap * HD;
  const float* kc = ko + ((size_t)b * Hkv + kvh) * HD;   // the new token's own key (s = 1)
  const float* vc = vo + ((size_t)b * Hkv + kvh) * HD;
  const size_t cstride = (size_t)max_rows * H;

  // Up to 8 prefix chunks: their (m, l) and partials do not depend on the rest,
  // so they are requested first and are in registers by the time they are merged.
  const bool few = nchunks <= 8;
  float2 ml8 = make_float2(-INFINITY, 0.f);
  float op8[8][E];
  if (few) {
    if (lane < nchunks) ml8 = *reinterpret_cast<const float2*>(mlpart + (lane * cstride + wid) * 2);
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int e = 0; e < E; ++e) op8[k][e] = k < nchunks ? opart[((size_t)k * cstride + wid) * HD + lane + 64 * e] : 0.f;
  }

  // The own key's score, reduced over the wave.
  float t_own = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) t_own = fmaf(qr[lane + 64 * e], kc[lane + 64 * e], t_own);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) t_own += __shfl_xor(t_own, off, 64);
  t_own *= sl2;

  float Mr = -INFINITY, den = 0.f, acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  const int nkeys = len + 1;
  for (int j0 = 0; j0 < nkeys; j0 += 64) {
    const int j = j0 + lane;
    float t = -INFINITY;
    if (j < len) {
      const uint4* kr = reinterpret_cast<const uint4*>(kb + (size_t)j * HD);
      uint4 w[HD / 8];
#pragma unroll
      for (int u = 0; u < HD / 8; ++u) w[u] = kr[u];
      float dot = 0.f;
#pragma unroll
      for (int u = 0; u < HD / 8; ++u) {
        const float4 qa = *reinterpret_cast<const float4*>(qr + 8 * u);
        const float4 qb = *reinterpret_cast<const float4*>(qr + 8 * u + 4);
        dot = fmaf(qa.x, __uint_as_float(w[u].x << 16), dot);
        dot = fmaf(qa.y, __uint_as_float(w[u].x & 0xffff0000u), dot);
        dot = fmaf(qa.z, __uint_as_float(w[u].y << 16), dot);
        dot = fmaf(qa.w, __uint_as_float(w[u].y & 0xffff0000u), dot);
        dot = fmaf(qb.x, __uint_as_float(w[u].z << 16), dot);
        dot = fmaf(qb.y, __uint_as_float(w[u].z & 0xffff0000u), dot);
        dot = fmaf(qb.z, __uint_as_float(w[u].w << 16), dot);
        dot = fmaf(qb.w, __uint_as_float(w[u].w & 0xffff0000u), dot);
      }
      t = dot * sl2;
    } else if (j == len) {
      t = t_own;
    }
    float bm = t;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) bm = fmaxf(bm, __shfl_xor(bm, off, 64));
    const float Mn = fmaxf(Mr, bm);   // finite: every block holds at least one key
    const float alpha = __builtin_amdgcn_exp2f(Mr - Mn);   // Mr = -inf gives 0
    const float p = j < nkeys ? __builtin_amdgcn_exp2f(t - Mn) : 0.f;
    float ps = p;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) ps += __shfl_xor(ps, off, 64);
    den = den * alpha + ps;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= alpha;
    // Cached values of the block: one load path (rows clamped to len - 1, weight 0
    // past the block), so a batch's loads are all in flight together.
    const int cnt = min(64, len - j0);
    for (int u0 = 0; u0 < cnt; u0 += kDecBatch) {
      float v[kDecBatch][E];
#pragma unroll
      for (int uu = 0; uu < kDecBatch; ++uu) {
        const size_t row = (size_t)min(j0 + u0 + uu, len - 1) * HD;
#pragma unroll
        for (int e = 0; e < E; ++e) v[uu][e] = __uint_as_float((uint32_t)vb[row + lane + 64 * e] << 16);
      }
#pragma unroll
      for (int uu = 0; uu < kDecBatch; ++uu) {
        const float pu = __shfl(p, (u0 + uu) & 63, 64);
        const float pv = u0 + uu < cnt ? pu : 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(pv, v[uu][e], acc[e]);
      }
    }
    if (len - j0 < 64) {   // the own key is in this block, at lane len - j0
      const float po = __shfl(p, len - j0, 64);
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(po, vc[lane + 64 * e], acc[e]);
    }
    Mr = Mn;
  }
  // The prefix chunks' partials (zeros where a chunk saw no key).
  float Mx = Mr;
  if (few) {
    float M = ml8.x;
#pragma unroll
    for (int off = 4; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
    Mx = fmaxf(Mx, __shfl(M, 0, 64));
    const float own_w = __builtin_amdgcn_exp2f(Mr - Mx);
    const float w = ml8.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml8.x - Mx);
    float wl = w * ml8.y;
#pragma unroll
    for (int off = 4; off >= 1; off >>= 1) wl += __shfl_xor(wl, off, 64);
    den = den * own_w + __shfl(wl, 0, 64);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= own_w;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float wk = __shfl(w, k, 64);
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(wk, op8[k][e], acc[e]);
    }
    nchunks = 0;   // skips the general merge below
  }
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int ch = c0 + lane;
    float M = ch < nchunks ? mlpart[(ch * cstride + wid) * 2] : -INFINITY;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
    Mx = fmaxf(Mx, M);
  }
  if (!few) {
    const float own_w = __builtin_amdgcn_exp2f(Mr - Mx);
    den *= own_w;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= own_w;
  }
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int ch = c0 + lane;
    float w = 0.f, wl = 0.f;
    if (ch < nchunks) {
      const float2 ml = *reinterpret_cast<const float2*>(mlpart + (ch * cstride + wid) * 2);
      w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - Mx);
      wl = w * ml.y;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) wl += __shfl_xor(wl, off, 64);
    den += wl;
    const int cn = min(64, nchunks - c0);
    for (int k0 = 0; k0 < cn; k0 += kDecBatch) {
      float v[kDecBatch][E];
#pragma unroll
      for (int kk = 0; kk < kDecBatch; ++kk) {
        const float* op = opart + ((size_t)(c0 + min(k0 + kk, cn - 1)) * cstride + wid) * HD;
#pragma unroll
        for (int e = 0; e < E; ++e) v[kk][e] = op[lane + 64 * e];
      }
#pragma unroll
      for (int kk = 0; kk < kDecBatch; ++kk) {
        const float wk = __shfl(w, (k0 + kk) & 63, 64);
        const float wv = k0 + kk < cn ? wk : 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(wv, v[kk][e], acc[e]);
      }
    }
  }
  const float inv = 1.f / den;
  const size_t plane = (size_t)max_rows * H * HD;
  uint16_t* ob = reinterpret_cast<uint16_t*>(o);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    uint16_t hb, lb;
    split2(acc[e] * inv, hb, lb);
    ob[(size_t)wid * HD + lane + 64 * e] = hb;
    ob[plane + (size_t)wid * HD + lane + 64 * e] = lb;
  }
}

// fp32 models, decode: one thread per (branch, head) over the prefix, the
// branch's cached entries 0..len-1 and its own new key.
template <int HD>
__global__ __launch_bounds__(128) void k_attn_f32_dec(const float* __restrict__ q, const PrefixView pre,
                                                      const float* __restrict__ ck,
                                                      const float* __restrict__ cv, int len, int cap,
                                                      const float* __restrict__ ko, const float* __restrict__ vo,
                                                      float* __restrict__ o, const Ctrl* c, int H, int Hkv,
                                                      float scale) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= c->live_count * H) return;
  const int b = idx / H, h = idx % H;
  const int kvh = h / (H / Hkv);
  const float* qr = q + (size_t)idx * HD;
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
  for (int sg = 0; sg < pre.nseg; ++sg) {
    const float* Kp = static_cast<const float*>(pre.k[sg]) + (size_t)kvh * pre.len[sg] * HD;
    const float* Vp = static_cast<const float*>(pre.v[sg]) + (size_t)kvh * pre.len[sg] * HD;
    for (int j = 0; j < pre.len[sg]; ++j) visit(Kp + (size_t)j * HD, Vp + (size_t)j * HD);
  }
  const float* Kc = ck + ((size_t)b * Hkv + kvh) * cap * HD;
  const float* Vc = cv + ((size_t)b * Hkv + kvh) * cap * HD;
  for (int j = 0; j < len; ++j) visit(Kc + (size_t)j * HD, Vc + (size_t)j * HD);
  visit(ko + ((size_t)b * Hkv + kvh) * HD, vo + ((size_t)b * Hkv + kvh) * HD);
  float* orow = o + (size_t)idx * HD;
  for (int d = 0; d < HD; ++d) orow[d] = acc[d] / l;
}

// fp32 models: one thread per (query row, head), plain online softmax.
template <int HD>
__global__ __launch_bounds__(128) void k_attn_f32(const float* __restrict__ q, const PrefixView pre,
                                                  const float* __restrict__ ko,
                                                  const float* __restrict__ vo, float* __restrict__ o,
                                                  const Ctrl* c, int s, int H, int Hkv, float scale) {
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
  for (int sg = 0; sg < pre.nseg; ++sg) {
    const float* Kp = static_cast<const float*>(pre.k[sg]) + (size_t)kvh * pre.len[sg] * HD;
    const float* Vp = static_cast<const float*>(pre.v[sg]) + (size_t)kvh * pre.len[sg] * HD;
    for (int j = 0; j < pre.len[sg]; ++j) visit(Kp + (size_t)j * HD, Vp + (size_t)j * HD);
  }
  const float* Ko = ko + ((size_t)slot * Hkv + kvh) * s * HD;
  const float* Vo = vo + ((size_t)slot * Hkv + kvh) * s * HD;
  for (int j = 0; j <= i; ++j) visit(Ko + (size_t)j * HD, Vo + (size_t)j * HD);
  float* orow = o + ((size_t)r * H + h) * HD;
  for (int d = 0; d < HD; ++d) orow[d] = acc[d] / l;
}

}  // namespace

AttnPlan plan_attention(DType dt, int B, int n, int s, int H, int Hkv) {
  AttnPlan p{1, 0, false};
  if (dt != DType::BF16) return p;
  const int G = H / Hkv;
  const int n_ptiles = (n + 63) / 64;
  // A branch with fewer than 64 query rows per KV head (G * s < 64, e.g. decode
  // or short verify spans) would leave most of a 64-row tile empty and make every
  // branch stream the prefix on its own: its rows are packed with other
  // branches' into shared tiles that see only the prefix, and the short own span
  // is merged in the combine.
  p.cross = G * s < 64;
  constexpr int QT = 16 * kAttnWaves;   // query rows per workgroup
  const int base = p.cross ? (B * s * G + QT - 1) / QT * Hkv : (G * s + QT - 1) / QT * Hkv * B;
  const int min_tiles = p.cross ? n_ptiles : n_ptiles + 1;   // key tiles of the smallest query tile
  if (p.cross && n == 0) {
    p.chunks = 0;
    return p;
  }
  // Split the keys while the launch still fits one round of workgroups (one
  // fits per CU), keeping at least 2 tiles per chunk: a split that spills into
  // a second round costs more than it shares out (224 query tiles of the
  // 28-layer shapes: one chunk, 30.4 ms per call, against 31.0 ms with two).
  while (base * (p.chunks + 1) <= kComputeUnits && (p.chunks + 1) * 2 <= min_tiles) ++p.chunks;
  p.partials = (p.cross || p.chunks > 1) ? p.chunks : 0;
  return p;
}

namespace {
// k_attn_bf16 with the probabilities split into hi/lo (p_split) or not, over a
// prefix of one segment or of several (multi_seg).
template <int HD, bool XB, typename... Args>
void launch_attn_tiles(bool p_split, bool multi_seg, dim3 grid, hipStream_t st, Args... args) {
  const dim3 blk(64 * kAttnWaves);
  if (p_split && !multi_seg) hipLaunchKernelGGL((k_attn_bf16<HD, XB, true, false>), grid, blk, 0, st, args...);
  else if (p_split) hipLaunchKernelGGL((k_attn_bf16<HD, XB, true, true>), grid, blk, 0, st, args...);
  else if (!multi_seg) hipLaunchKernelGGL((k_attn_bf16<HD, XB, false, false>), grid, blk, 0, st, args...);
  else hipLaunchKernelGGL((k_attn_bf16<HD, XB, false, true>), grid, blk, 0, st, args...);
}
}  // namespace

hipError_t launch_attention_decode(DType dt, const AttnPlan& p, const void* q, const PrefixView& pre,
                                   const void* ck, const void* cv, int len, int cap, const void* k_own,
                                   const void* v_own, void* o, float* opart, float* mlpart, const Ctrl* c,
                                   int H, int Hkv, int hd, int B, hipStream_t st) {
  const float* qq = static_cast<const float*>(q);
  const float *ko = static_cast<const float*>(k_own), *vo = static_cast<const float*>(v_own);
  if (dt == DType::BF16) {
    const float sl2 = 1.4426950408889634f / sqrtf((float)hd);
    const int G = H / Hkv;
    const int max_rows = B;   // one token per branch
    const bf16 *cka = static_cast<const bf16*>(ck), *cva = static_cast<const bf16*>(cv);
    if (p.chunks > 0) {
      const dim3 grid((max_rows * G + 16 * kAttnWaves - 1) / (16 * kAttnWaves), Hkv, p.chunks);
      if (hd == 128)
        launch_attn_tiles<128, true>(true, pre.nseg > 1, grid, st, qq, pre, ko, vo, o, opart, mlpart, c, 1, H, Hkv,
                                     sl2, p.chunks, max_rows);
      else
        launch_attn_tiles<64, true>(true, pre.nseg > 1, grid, st, qq, pre, ko, vo, o, opart, mlpart, c, 1, H, Hkv,
                                    sl2, p.chunks, max_rows);
    }
    const dim3 cgrid((B * H * 64 + 255) / 256);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_combine_dec<128>, cgrid, dim3(256), 0, st, opart, mlpart, qq, cka, cva, len,
                         cap, ko, vo, o, c, H, Hkv, sl2, p.chunks, max_rows);
    else
      hipLaunchKernelGGL(k_attn_combine_dec<64>, cgrid, dim3(256), 0, st, opart, mlpart, qq, cka, cva, len,
                         cap, ko, vo, o, c, H, Hkv, sl2, p.chunks, max_rows);
  } else {
    const float scale = 1.f / sqrtf((float)hd);
    const dim3 grid((B * H + 127) / 128);
    const float *cka = static_cast<const float*>(ck), *cva = static_cast<const float*>(cv);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_f32_dec<128>, grid, dim3(128), 0, st, qq, pre, cka, cva, len, cap, ko, vo,
                         static_cast<float*>(o), c, H, Hkv, scale);
    else
      hipLaunchKernelGGL(k_attn_f32_dec<64>, grid, dim3(128), 0, st, qq, pre, cka, cva, len, cap, ko, vo,
                         static_cast<float*>(o), c, H, Hkv, scale);
  }
  return hipGetLastError();
}

hipError_t launch_attention(DType dt, const AttnPlan& p, const void* q, const PrefixView& pre,
                            const void* k_own, const void* v_own, void* o, float* opart, float* mlpart,
                            const Ctrl* c, int s, int H, int Hkv, int hd, int max_branches, hipStream_t st,
                            bool p_split) {
  if (dt == DType::BF16) {
    const float sl2 = 1.4426950408889634f / sqrtf((float)hd);
    const int G = H / Hkv;
    const int max_rows = max_branches * s;
    const float* qq = static_cast<const float*>(q);
    const float *ko = static_cast<const float*>(k_own), *vo = static_cast<const float*>(v_own);
    void* oo = o;
    const int waves = max_rows * H;
    const dim3 cgrid((waves * 64 + 255) / 256);
    const bool ms = pre.nseg > 1;
    if (p.cross) {
      const dim3 grid((max_rows * G + 16 * kAttnWaves - 1) / (16 * kAttnWaves), Hkv, p.chunks);
      if (p.chunks > 0) {
        if (hd == 128)
          launch_attn_tiles<128, true>(p_split, ms, grid, st, qq, pre, ko, vo, oo, opart, mlpart, c, s, H, Hkv, sl2,
                                       p.chunks, max_rows);
        else
          launch_attn_tiles<64, true>(p_split, ms, grid, st, qq, pre, ko, vo, oo, opart, mlpart, c, s, H, Hkv, sl2,
                                      p.chunks, max_rows);
      }
      if (hd == 128)
        hipLaunchKernelGGL(k_attn_combine_own<128>, cgrid, dim3(256), 0, st, opart, mlpart, qq, ko, vo, oo, c, s, H,
                           Hkv, sl2, p.chunks, max_rows);
      else
        hipLaunchKernelGGL(k_attn_combine_own<64>, cgrid, dim3(256), 0, st, opart, mlpart, qq, ko, vo, oo, c, s, H,
                           Hkv, sl2, p.chunks, max_rows);
      return hipGetLastError();
    }
    const dim3 grid((G * s + 16 * kAttnWaves - 1) / (16 * kAttnWaves), Hkv, max_branches * p.chunks);
    if (hd == 128)
      launch_attn_tiles<128, false>(p_split, ms, grid, st, qq, pre, ko, vo, oo, opart, mlpart, c, s, H, Hkv, sl2,
                                    p.chunks, max_rows);
    else
      launch_attn_tiles<64, false>(p_split, ms, grid, st, qq, pre, ko, vo, oo, opart, mlpart, c, s, H, Hkv, sl2,
                                   p.chunks, max_rows);
    if (p.chunks > 1) {
      if (hd == 128)
        hipLaunchKernelGGL(k_attn_combine<128>, cgrid, dim3(256), 0, st, opart, mlpart, oo, c, s, H, p.chunks,
                           max_rows);
      else
        hipLaunchKernelGGL(k_attn_combine<64>, cgrid, dim3(256), 0, st, opart, mlpart, oo, c, s, H, p.chunks,
                           max_rows);
    }
  } else {
    const float scale = 1.f / sqrtf((float)hd);
    const int total = max_branches * s * H;
    const dim3 grid((total + 127) / 128);
    const float *qq = static_cast<const float*>(q), *ko = static_cast<const float*>(k_own),
                *vo = static_cast<const float*>(v_own);
    if (hd == 128)
      hipLaunchKernelGGL(k_attn_f32<128>, grid, dim3(128), 0, st, qq, pre, ko, vo, static_cast<float*>(o), c, s, H,
                         Hkv, scale);
    else
      hipLaunchKernelGGL(k_attn_f32<64>, grid, dim3(128), 0, st, qq, pre, ko, vo, static_cast<float*>(o), c, s, H,
                         Hkv, scale);
  }
  return hipGetLastError();
}

}  // namespace rksc
