// 16 x 16 x 4 MFMA tiles in fp32 and fp64 for the SIMT-shaped kernels (the
// general chunked path, third order).  Included by their .hip files only.
//
// v_mfma_f32_16x16x4_f32: lane l = 16 g + n supplies A[n][k_g] and B[k_g][n]
// (k_g: the g-th of the four contraction indices of the step) and holds
// D[4 g + i][n] in element i.  v_mfma_f64_16x16x4_f64 takes its operands the
// same way but holds D[4 i + g][n] in element i; a product whose A rows are
// supplied in the order pr(n) = 4 (n % 4) + n / 4 (lane n gives row pr(n))
// therefore returns D[4 g + i][n] in element i, the fp32 layout.
#pragma once
#include <hip/hip_runtime.h>

namespace hla {

typedef float f32x4c __attribute__((ext_vector_type(4)));
typedef double f64x4c __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int mfma_pr(int n) { return 4 * (n & 3) + (n >> 2); }

__device__ __forceinline__ f32x4c mfma4(float a, float b, const f32x4c& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f64x4c mfma4(double a, double b, const f64x4c& c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// acc += sum_{k < K} A(k) B(k) for this lane's operands, K a multiple of 16,
// af(k) = A[row][k], bf(k) = B[k][n0 + n]; both from LDS, four k steps'
// loads issued ahead of their products.
template <typename E, typename V, typename AF, typename BF>
__device__ __forceinline__ void mma_lds(V& acc, int K, int g, AF af, BF bf) {
  for (int k0 = 0; k0 < K; k0 += 16) {
    E x[4], y[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      x[u] = af(k0 + 4 * u + g);
      y[u] = bf(k0 + 4 * u + g);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) acc = mfma4(x[u], y[u], acc);
  }
}

// The same with B from global memory (K <= 128): all of the lane's B loads
// are issued before the first product.
template <typename E, typename V, typename AF, typename BF>
__device__ __forceinline__ void mma_glb(V& acc, int K, int g, AF af, BF bf) {
  float y[32];
#pragma unroll
  for (int s = 0; s < 32; ++s)
    if (4 * s < K) y[s] = bf(4 * s + g);
#pragma unroll
  for (int s = 0; s < 32; ++s)
    if (4 * s < K) acc = mfma4(af(4 * s + g), (E)y[s], acc);
}

}  // namespace hla
