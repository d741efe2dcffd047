// Chunk-parallel second-order HLA, general path (fp32 SIMT arithmetic).
//
// Two kernels, one workgroup per (head, chunk):
//   k_chunk_summary  the chunk's masked summary (S, C, m, G, h) with zero
//                    carry-in, built from dense intra-chunk products
//                    (prefix summaries of Sec. 3 and the masking summaries G, h
//                    of Sec. 3.1, restricted to the chunk).
//   k_readout        per-token outputs of a chunk from its exclusive carry-in
//                    state (Thm. 1 applied to carry (+) local prefix, Eq.
//                    (semidirect); Rem. scan-modes, inter-chunk parallelism).
// Any d, dv <= 128 and chunk <= 128 are accepted; fp32 or bf16 inputs.
#include "common.h"

namespace hla {

// ----------------------------------------------------------------------------
// Chunk summary.  With A_s[i][j] = [j < i] k_i . q_j (strictly lower):
//   S = K^T K,  C = Q^T V,  m = Q^T 1,  G = K^T (A_s V),  h = K^T (A_s 1).
// G is sum_i k_i k_i^T C_{i-1} with C local to the chunk (Sec. 3.1).
// LDS: A_s [chunk][chunk] and Y = [A_s V | A_s 1]  [chunk][dv+1].
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_chunk_summary(const T* __restrict__ q, const T* __restrict__ k,
                                                       const T* __restrict__ v, float* __restrict__ states,
                                                       int n, int d, int dv, int chunk, int M) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0);
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  float* As = smem;                       // [L][L]
  float* Y = smem + chunk * chunk;        // [L][dv+1]
  const int ldY = dv + 1;
  float* st = states + ((size_t)bh * M + c) * state_floats(d, dv);
  float* S = st;
  float* Cc = st + off_C(d, dv);
  float* m = st + off_m(d, dv);
  float* G = st + off_G(d, dv);
  float* h = st + off_h(d, dv);

  for (int idx = tid; idx < L * L; idx += blockDim.x) {
    const int i = idx / L, j = idx % L;
    float s = 0.f;
    if (j < i)
      for (int a = 0; a < d; ++a) s += ldf(k, qk_base + (size_t)i * d + a) * ldf(q, qk_base + (size_t)j * d + a);
    As[i * L + j] = s;
  }
  __syncthreads();
  for (int idx = tid; idx < L * ldY; idx += blockDim.x) {
    const int i = idx / ldY, b = idx % ldY;
    float s = 0.f;
    for (int j = 0; j < i; ++j) s += As[i * L + j] * (b < dv ? ldf(v, v_base + (size_t)j * dv + b) : 1.f);
    Y[i * ldY + b] = s;
  }
  __syncthreads();
  for (int idx = tid; idx < d * d; idx += blockDim.x) {
    const int a = idx / d, b = idx % d;
    float s = 0.f;
    for (int t = 0; t < L; ++t) s += ldf(k, qk_base + (size_t)t * d + a) * ldf(k, qk_base + (size_t)t * d + b);
    S[idx] = s;
  }
  for (int idx = tid; idx < d * dv; idx += blockDim.x) {
    const int a = idx / dv, b = idx % dv;
    float sc = 0.f, sg = 0.f;
    for (int t = 0; t < L; ++t) {
      sc += ldf(q, qk_base + (size_t)t * d + a) * ldf(v, v_base + (size_t)t * dv + b);
      sg += ldf(k, qk_base + (size_t)t * d + a) * Y[t * ldY + b];
    }
    Cc[idx] = sc;
    G[idx] = sg;
  }
  for (int a = tid; a < d; a += blockDim.x) {
    float sm = 0.f, sh = 0.f;
    for (int t = 0; t < L; ++t) {
      sm += ldf(q, qk_base + (size_t)t * d + a);
      sh += ldf(k, qk_base + (size_t)t * d + a) * Y[t * ldY + dv];
    }
    m[a] = sm;
    h[a] = sh;
  }
}

// ----------------------------------------------------------------------------
// Readout of one chunk from its carry-in (S0, C0, m0, G0, h0).
// With p_t = S0 q_t and r_j = S_j q_j = p_j + sum_{i<=j, i in chunk} (k_i.q_j) k_i:
//   masked:   o_t = q_t^T (S0 C0 - G0) + sum_{j<=t} (q_t . r_j) v_j
//             den_t = q_t^T (S0 m0 - h0) + sum_{j<=t} (q_t . r_j)
//   unmasked: o_t = r_t^T C0 + sum_{j<=t} (r_t . q_j) v_j,   den_t = r_t . m0 + sum_{j<=t} r_t . q_j
// (q_t^T S_t = r_t^T since S is symmetric.)  These are Thm. 1 evaluated on
// the inclusive state carry (+) local prefix, grouped so that no d x dv
// product of states is formed.
// LDS: R [chunk][d], W/T [chunk][chunk], den [chunk].
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_readout(const T* __restrict__ q, const T* __restrict__ k,
                                                 const T* __restrict__ v, const float* __restrict__ prefix,
                                                 float* __restrict__ out, int n, int d, int dv, int chunk,
                                                 int M, int masked, int normalized, float eps) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0);
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  float* R = smem;                       // [L][d]
  float* W = smem + chunk * d;           // [L][L]
  float* dn = W + chunk * chunk;         // [L]
  const float* st = prefix + ((size_t)bh * M + c) * state_floats(d, dv);
  const float* S0 = st;
  const float* C0 = st + off_C(d, dv);
  const float* m0 = st + off_m(d, dv);
  const float* G0 = st + off_G(d, dv);
  const float* h0 = st + off_h(d, dv);
  float* o = out + v_base;

  // P = Q S0 into R;  W[t][i] = [i <= t] q_t . k_i
  for (int idx = tid; idx < L * d; idx += blockDim.x) {
    const int t = idx / d, a = idx % d;
    float s = 0.f;
    for (int b = 0; b < d; ++b) s += ldf(q, qk_base + (size_t)t * d + b) * S0[(size_t)b * d + a];
    R[idx] = s;
  }
  for (int idx = tid; idx < L * L; idx += blockDim.x) {
    const int t = idx / L, i = idx % L;
    float s = 0.f;
    if (i <= t)
      for (int a = 0; a < d; ++a) s += ldf(q, qk_base + (size_t)t * d + a) * ldf(k, qk_base + (size_t)i * d + a);
    W[idx] = s;
  }
  __syncthreads();
  if (masked) {
    // carry term q_t^T S0 C0 - q_t^T G0 (and its denominator)
    for (int idx = tid; idx < L * dv; idx += blockDim.x) {
      const int t = idx / dv, b = idx % dv;
      float s = 0.f;
      for (int a = 0; a < d; ++a)
        s += R[t * d + a] * C0[(size_t)a * dv + b] - ldf(q, qk_base + (size_t)t * d + a) * G0[(size_t)a * dv + b];
      o[(size_t)t * dv + b] = s;
    }
    for (int t = tid; t < L; t += blockDim.x) {
      float s = 0.f;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * m0[a] - ldf(q, qk_base + (size_t)t * d + a) * h0[a];
      dn[t] = s;
    }
  }
  __syncthreads();
  // R += W K  (r_j = S_j q_j)
  for (int idx = tid; idx < L * d; idx += blockDim.x) {
    const int j = idx / d, a = idx % d;
    float s = R[idx];
    for (int i = 0; i <= j; ++i) s += W[j * L + i] * ldf(k, qk_base + (size_t)i * d + a);
    R[idx] = s;
  }
  __syncthreads();
  // T[t][j] = [j <= t] (q_t . r_j)  (masked)  or  (r_t . q_j)  (unmasked)
  for (int idx = tid; idx < L * L; idx += blockDim.x) {
    const int t = idx / L, j = idx % L;
    float s = 0.f;
    if (j <= t) {
      if (masked)
        for (int a = 0; a < d; ++a) s += ldf(q, qk_base + (size_t)t * d + a) * R[j * d + a];
      else
        for (int a = 0; a < d; ++a) s += R[t * d + a] * ldf(q, qk_base + (size_t)j * d + a);
    }
    W[idx] = s;
  }
  if (!masked) {
    for (int idx = tid; idx < L * dv; idx += blockDim.x) {
      const int t = idx / dv, b = idx % dv;
      float s = 0.f;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * C0[(size_t)a * dv + b];
      o[(size_t)t * dv + b] = s;
    }
    for (int t = tid; t < L; t += blockDim.x) {
      float s = 0.f;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * m0[a];
      dn[t] = s;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < L * dv; idx += blockDim.x) {
    const int t = idx / dv, b = idx % dv;
    float s = o[(size_t)t * dv + b];
    for (int j = 0; j <= t; ++j) s += W[t * L + j] * ldf(v, v_base + (size_t)j * dv + b);
    o[(size_t)t * dv + b] = s;
  }
  if (normalized) {
    for (int t = tid; t < L; t += blockDim.x) {
      float s = dn[t];
      for (int j = 0; j <= t; ++j) s += W[t * L + j];
      dn[t] = s;
    }
    __syncthreads();
    for (int idx = tid; idx < L * dv; idx += blockDim.x) {
      const int t = idx / dv, b = idx % dv;
      o[(size_t)t * dv + b] = o[(size_t)t * dv + b] / (dn[t] + eps);
    }
  }
}

// ----------------------------------------------------------------------------
static size_t summary_lds(int chunk, int dv) { return sizeof(float) * ((size_t)chunk * chunk + (size_t)chunk * (dv + 1)); }
static size_t readout_lds(int chunk, int d) { return sizeof(float) * ((size_t)chunk * d + (size_t)chunk * chunk + chunk); }

hipError_t launch_chunk_summaries(const void* q, const void* k, const void* v, float* states,
                                  int BH, int n, int d, int dv, int chunk, int dtype, hipStream_t s) {
  const int M = (n + chunk - 1) / chunk;
  const size_t lds = summary_lds(chunk, dv);
  dim3 grid(M, BH), block(256);
  if (dtype == 1) {
    auto kern = k_chunk_summary<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, block, lds, s, (const uint16_t*)q, (const uint16_t*)k,
                       (const uint16_t*)v, states, n, d, dv, chunk, M);
  } else {
    auto kern = k_chunk_summary<float>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, block, lds, s, (const float*)q, (const float*)k, (const float*)v,
                       states, n, d, dv, chunk, M);
  }
  return hipGetLastError();
}

hipError_t launch_readout(const Fwd& f, const float* prefix, hipStream_t s) {
  const int M = (f.n + f.chunk - 1) / f.chunk;
  const size_t lds = readout_lds(f.chunk, f.d);
  dim3 grid(M, f.BH), block(256);
  if (f.dtype == 1) {
    auto kern = k_readout<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, block, lds, s, (const uint16_t*)f.q, (const uint16_t*)f.k,
                       (const uint16_t*)f.v, prefix, f.out, f.n, f.d, f.dv, f.chunk, M, f.masked,
                       f.normalized, f.eps);
  } else {
    auto kern = k_readout<float>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, block, lds, s, (const float*)f.q, (const float*)f.k, (const float*)f.v,
                       prefix, f.out, f.n, f.d, f.dv, f.chunk, M, f.masked, f.normalized, f.eps);
  }
  return hipGetLastError();
}

}  // namespace hla
