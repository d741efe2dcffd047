// Exclusive scan of second-order segment states under the masked semidirect
// product, Eq. (semidirect):
//   (S_A+S_B, C_A+C_B, m_A+m_B, G_A+G_B+S_B C_A, h_A+h_B+S_B m_A).
// For each head the input is a sequence of M segment states (chunk or segment
// summaries, record layout S|C|m|G|h); the output holds, for every segment,
// E (+) init (+) x_0 (+) ... (+) x_{c-1} (Rem. scan-modes), and optionally the
// inclusive total.
//
// The only cross-segment product is S_c C_acc, where C_acc is an additive
// prefix, so the work splits over column blocks of C and G.  One workgroup
// owns (head, column block) and streams the head's segments in order; block
// 0 also carries S, m and h.  The column blocks of one head are placed on the
// same XCD so the segment's S tile, read by each of them, is served from
// that XCD's L2.
#include "common.h"

namespace hla {

constexpr int kScanCols = 16;   // value columns of C and G per workgroup

// One workgroup per (head, 16 columns of C/G); block 0 also carries S, m, h.
// The next segment's loads are issued before the current segment's
// cross-term product, so memory latency overlaps the arithmetic.
template <int d>
__global__ __launch_bounds__(256) void k_scan(const float* __restrict__ states, const float* __restrict__ init,
                                              float* __restrict__ prefix, float* __restrict__ total,
                                              int BH, int M, int dv, int nblk, size_t in_stride,
                                              size_t pre_stride, size_t tot_stride) {
  constexpr int CB = kScanCols;
  constexpr int ldS = d + 4;
  constexpr int nSS = (d * d + 255) / 256;      // S elements per thread
  constexpr int nCC = (d * CB + 255) / 256;     // C-block elements per thread
  extern __shared__ float smem[];
  float* ScT = smem;                       // [d][d+4]: ScT[a'][a] = S_c[a][a']
  float* Cacc = ScT + d * ldS;             // [d][CB]
  float* Cnew = Cacc + d * CB;             // [d][CB]
  float* macc = Cnew + d * CB;             // [d]
  const int tid = threadIdx.x;
  const int L = blockIdx.x;
  const int group = L / (8 * nblk), within = L % (8 * nblk);
  const int bh = group * 8 + within % 8;
  const int blk = within / 8;
  if (bh >= BH) return;
  const int c0 = blk * CB;
  const size_t F = state_floats(d, dv);
  const size_t oC = off_C(d, dv), om = off_m(d, dv), oG = off_G(d, dv), oh = off_h(d, dv);
  const float* in = states + (size_t)bh * in_stride;
  float* pre = prefix + (size_t)bh * pre_stride;
  const float* ini = init ? init + (size_t)bh * F : nullptr;
  // cross-term tile: thread -> rows 4*aq .. 4*aq+3, columns 4*jq .. 4*jq+3 of the block
  const int jq = tid % (CB / 4), aq = tid / (CB / 4);
  const bool active = aq * 4 < d;
  const int gr = active ? aq * 4 : 0;

  float sacc[nSS], gacc[4][4], hacc = 0.f;
#pragma unroll
  for (int r = 0; r < nSS; ++r) {
    const int idx = tid + 256 * r;
    sacc[r] = (ini && blk == 0 && idx < d * d) ? ini[idx] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      gacc[i][j] = (ini && active) ? ini[oG + (size_t)(gr + i) * dv + c0 + jq * 4 + j] : 0.f;
#pragma unroll
  for (int r = 0; r < nCC; ++r) {
    const int idx = tid + 256 * r;
    if (idx < d * CB) Cacc[idx] = ini ? ini[oC + (size_t)(idx / CB) * dv + c0 + idx % CB] : 0.f;
  }
  if (tid < d) {
    macc[tid] = ini ? ini[om + tid] : 0.f;
    hacc = (ini && blk == 0) ? ini[oh + tid] : 0.f;
  }

  // registers holding segment c (loaded one step ahead)
  float sv[nSS], cv[nCC], gv[4][4], mv = 0.f, hv = 0.f;
  auto load = [&](int c) {
    const float* x = in + (size_t)c * F;
#pragma unroll
    for (int r = 0; r < nSS; ++r) {
      const int idx = tid + 256 * r;
      sv[r] = idx < d * d ? x[idx] : 0.f;
    }
#pragma unroll
    for (int r = 0; r < nCC; ++r) {
      const int idx = tid + 256 * r;
      cv[r] = idx < d * CB ? x[oC + (size_t)(idx / CB) * dv + c0 + idx % CB] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) gv[i][j] = active ? x[oG + (size_t)(gr + i) * dv + c0 + jq * 4 + j] : 0.f;
    if (tid < d) {
      mv = x[om + tid];
      hv = x[oh + tid];
    }
  };
  if (M > 0) load(0);
  __syncthreads();

  for (int c = 0; c <= M; ++c) {
    float* dst = (c < M) ? pre + (size_t)c * F : (total ? total + (size_t)bh * tot_stride : nullptr);
    // the exclusive prefix of segment c (or the total after the last)
    if (dst) {
      if (blk == 0) {
#pragma unroll
        for (int r = 0; r < nSS; ++r) {
          const int idx = tid + 256 * r;
          if (idx < d * d) dst[idx] = sacc[r];
        }
        if (tid < d) {
          dst[om + tid] = macc[tid];
          dst[oh + tid] = hacc;
        }
      }
#pragma unroll
      for (int r = 0; r < nCC; ++r) {
        const int idx = tid + 256 * r;
        if (idx < d * CB) dst[oC + (size_t)(idx / CB) * dv + c0 + idx % CB] = Cacc[idx];
      }
      if (active)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) dst[oG + (size_t)(gr + i) * dv + c0 + jq * 4 + j] = gacc[i][j];
    }
    if (c == M) break;
    // consume segment c's registers: stage S_c, C_new = C_acc + C_c, add G_c, h_c, S_c
#pragma unroll
    for (int r = 0; r < nSS; ++r) {
      const int idx = tid + 256 * r;
      if (idx < d * d) ScT[(idx % d) * ldS + idx / d] = sv[r];
      if (blk == 0) sacc[r] += sv[r];
    }
#pragma unroll
    for (int r = 0; r < nCC; ++r) {
      const int idx = tid + 256 * r;
      if (idx < d * CB) Cnew[idx] = Cacc[idx] + cv[r];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) gacc[i][j] += gv[i][j];
    const float m_c = mv;
    hacc += hv;
    __syncthreads();
    if (c + 1 < M) load(c + 1);
    // G_acc += S_c C_acc   (segment A = accumulated prefix, B = segment c)
    if (active) {
      float acc[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
#pragma unroll 8
      for (int ap = 0; ap < d; ++ap) {
        const float4 s4 = *reinterpret_cast<const float4*>(&ScT[ap * ldS + gr]);
        const float4 c4 = *reinterpret_cast<const float4*>(&Cacc[ap * CB + jq * 4]);
        const float svv[4] = {s4.x, s4.y, s4.z, s4.w};
        const float cvv[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] += svv[i] * cvv[j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) gacc[i][j] += acc[i][j];
    }
    // h_acc += S_c m_acc
    if (blk == 0 && tid < d) {
      float e = 0.f;
#pragma unroll 8
      for (int ap = 0; ap < d; ++ap) e += ScT[ap * ldS + tid] * macc[ap];
      hacc += e;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < nCC; ++r) {
      const int idx = tid + 256 * r;
      if (idx < d * CB) Cacc[idx] = Cnew[idx];
    }
    if (tid < d) macc[tid] += m_c;
    __syncthreads();
  }
}

hipError_t launch_scan(const float* states, const float* init, float* prefix, float* total,
                       int BH, int M, int d, int dv, hipStream_t s) {
  const size_t F = state_floats(d, dv);
  return launch_scan_strided(states, init, prefix, total, BH, M, d, dv, (size_t)M * F, (size_t)M * F, F, s);
}

hipError_t launch_scan_strided(const float* states, const float* init, float* prefix, float* total, int BH, int M,
                               int d, int dv, size_t in_stride, size_t pre_stride, size_t tot_stride,
                               hipStream_t s) {
  const int nblk = (dv + kScanCols - 1) / kScanCols;
  const int groups = (BH + 7) / 8;
  const size_t lds = sizeof(float) * ((size_t)d * (d + 4) + 2 * (size_t)d * kScanCols + d);
  const void* kern = nullptr;
  switch (d) {
    case 16: kern = (const void*)k_scan<16>; break;
    case 32: kern = (const void*)k_scan<32>; break;
    case 64: kern = (const void*)k_scan<64>; break;
    case 128: kern = (const void*)k_scan<128>; break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(groups * 8 * nblk), block(256);
  switch (d) {
    case 16: hipLaunchKernelGGL(k_scan<16>, grid, block, lds, s, states, init, prefix, total, BH, M, dv, nblk, in_stride, pre_stride, tot_stride); break;
    case 32: hipLaunchKernelGGL(k_scan<32>, grid, block, lds, s, states, init, prefix, total, BH, M, dv, nblk, in_stride, pre_stride, tot_stride); break;
    case 64: hipLaunchKernelGGL(k_scan<64>, grid, block, lds, s, states, init, prefix, total, BH, M, dv, nblk, in_stride, pre_stride, tot_stride); break;
    default: hipLaunchKernelGGL(k_scan<128>, grid, block, lds, s, states, init, prefix, total, BH, M, dv, nblk, in_stride, pre_stride, tot_stride); break;
  }
  return hipGetLastError();
}

}  // namespace hla
