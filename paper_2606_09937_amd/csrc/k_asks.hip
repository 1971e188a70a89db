// ASKS similarity (Eq. asks_sim with the exponential layer weights of
// Alg. AsksGate), for every pair of branches:
//   S[i][j] = sum_l w_l <h_i^l, h_j^l> / (|h_i^l| |h_j^l|),
//   w_l = exp(alpha l / L) / sum_l' exp(alpha l' / L), l = 1..L.
// One workgroup per pair (i, j). Each layer's dot product and both squared
// norms are reduced in one pass over d by one wave, in a fixed order, so
// S[i][j] and S[j][i] are computed identically (S is exactly symmetric).
#include "common.h"
#include "kernels.h"

namespace rksc {

namespace {

constexpr int kAsksWaves = 8;
constexpr int kAsksMaxLayers = 256;

__global__ __launch_bounds__(kAsksWaves * 64) void k_asks(const float* __restrict__ hidden, int L, int B, int d,
                                                          float alpha, float* __restrict__ S) {
  __shared__ float cosl[kAsksMaxLayers];
  const int i = blockIdx.x, j = blockIdx.y;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  // Wave w takes the layers w, w + 8, ...; the weighted sum then runs over the
  // layers in order, so S[i][j] and S[j][i] see the same operations.
  for (int l = wid; l < L; l += kAsksWaves) {
    const float* hi = hidden + ((size_t)l * B + i) * d;
    const float* hj = hidden + ((size_t)l * B + j) * d;
    float dot = 0.f, ni = 0.f, nj = 0.f;
    for (int k = lane; k < d; k += 64) {
      const float x = hi[k], y = hj[k];
      dot = fmaf(x, y, dot);
      ni = fmaf(x, x, ni);
      nj = fmaf(y, y, nj);
    }
    dot = wave_sum(dot);
    ni = wave_sum(ni);
    nj = wave_sum(nj);
    // The two norms enter symmetrically (ni*nj), so S[i][j] == S[j][i] bit for bit.
    if (lane == 0) cosl[l] = (ni > 0.f && nj > 0.f) ? dot / sqrtf(ni * nj) : 0.f;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // Weights in double with the largest exponent subtracted (no overflow for large |alpha|).
    const double a = (double)alpha;
    const double top = a >= 0.0 ? a : a / (double)L;
    double wsum = 0.0;
    for (int l = 1; l <= L; ++l) wsum += exp(a * (double)l / (double)L - top);
    float acc = 0.f;
    for (int l = 0; l < L; ++l) acc = fmaf((float)(exp(a * (double)(l + 1) / (double)L - top) / wsum), cosl[l], acc);
    S[(size_t)i * B + j] = acc;
  }
}

// Alg. AsksGate against the root: sigma_b = sum_l w_l <h_b^l / |h_b^l|, r^l>
// with the root rows r^l stored unit-normalised (Eq. prefix_fwd; they are not
// normalised again), shared[b] = sigma_b >= tau. One workgroup per branch; wave
// w reduces the layers l = w, w + 8, ... (float4 loads, d % 4 == 0) and the
// weighted sum runs over the layers in order, so the result does not depend on
// the wave schedule. A zero branch row contributes 0.
constexpr int kGateWaves = 8;
constexpr int kGateMaxLayers = 256;

__global__ __launch_bounds__(kGateWaves * 64) void k_asks_gate(const float* __restrict__ hidden,
                                                               const float* __restrict__ root, int L, int B, int d,
                                                               float alpha, float tau, float* __restrict__ sigma,
                                                               int* __restrict__ shared) {
  __shared__ float cosl[kGateMaxLayers];
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  for (int l = wid; l < L; l += kGateWaves) {
    const float4* hb = reinterpret_cast<const float4*>(hidden + ((size_t)l * B + b) * d);
    const float4* r = reinterpret_cast<const float4*>(root + (size_t)l * d);
    float dot = 0.f, nb = 0.f;
    for (int k = lane; k < d / 4; k += 64) {
      const float4 x = hb[k], y = r[k];
      dot = fmaf(x.x, y.x, fmaf(x.y, y.y, fmaf(x.z, y.z, fmaf(x.w, y.w, dot))));
      nb = fmaf(x.x, x.x, fmaf(x.y, x.y, fmaf(x.z, x.z, fmaf(x.w, x.w, nb))));
    }
    dot = wave_sum(dot);
    nb = wave_sum(nb);
    if (lane == 0) cosl[l] = nb > 0.f ? dot / sqrtf(nb) : 0.f;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double a = (double)alpha;
    const double top = a >= 0.0 ? a : a / (double)L;
    double wsum = 0.0;
    for (int l = 1; l <= L; ++l) wsum += exp(a * (double)l / (double)L - top);
    float acc = 0.f;
    for (int l = 0; l < L; ++l) acc = fmaf((float)(exp(a * (double)(l + 1) / (double)L - top) / wsum), cosl[l], acc);
    sigma[b] = acc;
    shared[b] = acc >= tau ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_asks(const float* hidden, int L, int B, int d, float alpha, float* S, hipStream_t st) {
  hipLaunchKernelGGL(k_asks, dim3(B, B), dim3(kAsksWaves * 64), 0, st, hidden, L, B, d, alpha, S);
  return hipGetLastError();
}

hipError_t launch_asks_gate(const float* hidden, const float* root, int L, int B, int d, float alpha, float tau,
                            float* sigma, int* shared, hipStream_t st) {
  hipLaunchKernelGGL(k_asks_gate, dim3(B), dim3(kGateWaves * 64), 0, st, hidden, root, L, B, d, alpha, tau, sigma, shared);
  return hipGetLastError();
}

}  // namespace rksc
