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

static inline int scan_cols(int d, int dv) {
  int cb = 4096 / d;            // d*cb/16 threads, at most 256
  if (cb > dv) cb = dv;
  return cb;
}

__global__ __launch_bounds__(256) void k_scan(const float* __restrict__ states, const float* __restrict__ init,
                                              float* __restrict__ prefix, float* __restrict__ total,
                                              int BH, int M, int d, int dv, int CB, int nblk, size_t in_stride,
                                              size_t pre_stride, size_t tot_stride) {
  extern __shared__ float smem[];
  const int ldS = d + 4;
  float* ScT = smem;                       // [d][d+4]: ScT[a'][a] = S_c[a][a']
  float* Cacc = smem + d * ldS;            // [d][CB]
  float* macc = Cacc + d * CB;             // [d]
  const int tid = threadIdx.x;
  const int L = blockIdx.x;
  const int group = L / (8 * nblk), within = L % (8 * nblk);
  const int bh = group * 8 + within % 8;
  const int blk = within / 8;
  if (bh >= BH) return;
  const int c0 = blk * CB;
  const int ncol = min(CB, dv - c0);
  const size_t F = state_floats(d, dv);
  const size_t oC = off_C(d, dv), om = off_m(d, dv), oG = off_G(d, dv), oh = off_h(d, dv);
  const float* in = states + (size_t)bh * in_stride;
  float* pre = prefix + (size_t)bh * pre_stride;
  const float* ini = init ? init + (size_t)bh * F : nullptr;

  // cross-term tile: thread -> (a-quad, j-quad)
  const int nj4 = CB / 4;
  const int jq = tid % nj4, aq = tid / nj4;
  const bool active = (aq * 4 < d) && (jq * 4 < ncol);
  float gacc[4][4];
  // S accumulator of block 0: element idx = tid + 256 r
  const int nS = (d * d + 255) / 256;
  float sacc[64];
  float hacc = 0.f;

  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) gacc[i][j] = 0.f;
  if (ini) {
    if (active)
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) gacc[i][j] = ini[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j];
  }
  for (int idx = tid; idx < d * CB; idx += blockDim.x) {
    const int a = idx / CB, j = idx % CB;
    Cacc[idx] = (ini && j < ncol) ? ini[oC + (size_t)a * dv + c0 + j] : 0.f;
  }
  for (int a = tid; a < d; a += blockDim.x) macc[a] = ini ? ini[om + a] : 0.f;
  if (blk == 0) {
    for (int r = 0; r < nS; ++r) {
      const int idx = tid + 256 * r;
      sacc[r] = (ini && idx < d * d) ? ini[idx] : 0.f;
    }
    if (tid < d) hacc = ini ? ini[oh + tid] : 0.f;
  }
  __syncthreads();

  for (int c = 0; c <= M; ++c) {
    float* dst = (c < M) ? pre + (size_t)c * F : (total ? total + (size_t)bh * tot_stride : nullptr);
    // write the exclusive prefix of segment c (or the total after the last)
    if (dst) {
      if (blk == 0) {
        for (int r = 0; r < nS; ++r) {
          const int idx = tid + 256 * r;
          if (idx < d * d) dst[idx] = sacc[r];
        }
        if (tid < d) {
          dst[om + tid] = macc[tid];
          dst[oh + tid] = hacc;
        }
      }
      for (int idx = tid; idx < d * CB; idx += blockDim.x) {
        const int a = idx / CB, j = idx % CB;
        if (j < ncol) dst[oC + (size_t)a * dv + c0 + j] = Cacc[idx];
      }
      if (active)
        for (int i = 0; i < 4; ++i)
          for (int j = 0; j < 4; ++j) dst[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j] = gacc[i][j];
    }
    if (c == M) break;
    const float* x = in + (size_t)c * F;
    // stage S_c transposed
    for (int idx = tid; idx < d * d; idx += blockDim.x) {
      const int a = idx / d, ap = idx % d;
      ScT[ap * ldS + a] = x[idx];
    }
    __syncthreads();
    // G_acc += G_c + S_c C_acc   (segment A = accumulated prefix, B = segment c)
    if (active) {
      float acc[4][4];
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) acc[i][j] = x[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j];
      for (int ap = 0; ap < d; ++ap) {
        const float4 s4 = *reinterpret_cast<const float4*>(&ScT[ap * ldS + aq * 4]);
        const float4 c4 = *reinterpret_cast<const float4*>(&Cacc[ap * CB + jq * 4]);
        const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
        const float cv[4] = {c4.x, c4.y, c4.z, c4.w};
        for (int i = 0; i < 4; ++i)
          for (int j = 0; j < 4; ++j) acc[i][j] += sv[i] * cv[j];
      }
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) gacc[i][j] += acc[i][j];
    }
    if (blk == 0) {
      if (tid < d) {
        float s = x[oh + tid];
        for (int ap = 0; ap < d; ++ap) s += ScT[ap * ldS + tid] * macc[ap];
        hacc += s;
      }
      for (int r = 0; r < nS; ++r) {
        const int idx = tid + 256 * r;
        if (idx < d * d) sacc[r] += x[idx];
      }
    }
    __syncthreads();
    for (int idx = tid; idx < d * CB; idx += blockDim.x) {
      const int a = idx / CB, j = idx % CB;
      if (j < ncol) Cacc[idx] += x[oC + (size_t)a * dv + c0 + j];
    }
    for (int a = tid; a < d; a += blockDim.x) macc[a] += x[om + a];
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
  const int CB = scan_cols(d, dv);
  const int nblk = (dv + CB - 1) / CB;
  const int groups = (BH + 7) / 8;
  const size_t lds = sizeof(float) * ((size_t)d * (d + 4) + (size_t)d * CB + d);
  hipError_t e = hipFuncSetAttribute((const void*)k_scan, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_scan, dim3(groups * 8 * nblk), dim3(256), lds, s, states, init, prefix, total, BH, M, d,
                     dv, CB, nblk, in_stride, pre_stride, tot_stride);
  return hipGetLastError();
}

}  // namespace hla
