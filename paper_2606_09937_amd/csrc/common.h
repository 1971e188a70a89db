// Device-side helpers shared by the gfx950 kernels: bf16 conversion, vector
// types, wavefront reductions and the MFMA operand types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rksc {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

// 16-byte load through a global-address-space pointer (keeps the compiler from
// falling back to flat loads when it cannot infer the address space).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16(const void* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  const u32x4 v = *(const __attribute__((address_space(1))) u32x4*)p;
#else
  const u32x4 v = *static_cast<const u32x4*>(p);
#endif
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Direct global->LDS DMA of 16 bytes per lane (global_load_lds_dwordx4): lane L's
// bytes land at lds_base + 16 * L. lds_base must be uniform across the wave.
// The transfer counts on the vector-memory counter like an ordinary load.
__device__ __forceinline__ void dma16(const void* gsrc, void* lds_base) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)gsrc,
                                   (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Vector-memory counter <= N and every LDS access of this wave complete.
template <int N>
__device__ __forceinline__ void wait_vmcnt_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

// Round-to-nearest-even fp32 -> bf16 bits (NaN stays NaN): gfx950's
// v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// Split of an fp32 value into bf16 hi + lo (hi = RNE(x), lo = RNE(x - hi); x - hi
// is exact in fp32). hi + lo carries x to ~2^-17 relative, and a bf16 value
// times each part is exact in the MFMA's fp32 products, so two bf16 MFMAs give
// an fp32-accurate product with a bf16 operand.
__device__ __forceinline__ void split2(float x, uint16_t& hi, uint16_t& lo) {
  const __bf16 h = static_cast<__bf16>(x);
  hi = __builtin_bit_cast(uint16_t, h);
  lo = __builtin_bit_cast(uint16_t, static_cast<__bf16>(x - static_cast<float>(h)));
}

// split2 of two values at once, packed: hi2 = (bf16(x1) << 16) | bf16(x0), lo2
// likewise for the residuals (one v_cvt_pk_bf16_f32 each).
__device__ __forceinline__ void split2x2(float x0, float x1, uint32_t& hi2, uint32_t& lo2) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float floatx2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t h = __builtin_convertvector(floatx2_t{x0, x1}, bf16x2_t);
  hi2 = __builtin_bit_cast(uint32_t, h);
  const float h0 = __uint_as_float(hi2 << 16), h1 = __uint_as_float(hi2 & 0xffff0000u);
  lo2 = __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{x0 - h0, x1 - h1}, bf16x2_t));
}

__device__ __forceinline__ uint32_t pack2(uint16_t a, uint16_t b) {
  return static_cast<uint32_t>(a) | (static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return static_cast<float>(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) {
  uint16_t b = f32_to_bf16_bits(v);
  return __builtin_bit_cast(bf16, b);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); every thread gets the result.
// Fixed reduction order, so the result is deterministic.
__device__ __forceinline__ float block_sum(float v, float* smem /* >= 16 floats */) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) smem[wid] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += smem[i];
  return t;
}

// Online softmax statistics of a set of logits z: m = max z,
// s = sum exp(z - m), t = sum exp(z - m) * (z - m). Entropy = log(s) - t/s.
struct EntStats {
  float m, s, t;
};

__device__ __forceinline__ EntStats ent_empty() { return {-INFINITY, 0.f, 0.f}; }

// Compute units of an MI355X (8 XCDs x 32): the size of a one-wave-of-workgroups grid.
constexpr int kComputeUnits = 256;

// Merge of two statistic triples (associative up to rounding).
__device__ __forceinline__ EntStats ent_merge(EntStats a, EntStats b) {
  if (b.m == -INFINITY) return a;
  if (a.m == -INFINITY) return b;
  const float m = fmaxf(a.m, b.m);
  const float da = a.m - m, db = b.m - m;
  const float ea = __expf(da), eb = __expf(db);
  EntStats r;
  r.m = m;
  r.s = a.s * ea + b.s * eb;
  r.t = (a.t + a.s * da) * ea + (b.t + b.s * db) * eb;
  return r;
}

}  // namespace rksc
