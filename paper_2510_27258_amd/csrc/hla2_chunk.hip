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
//
// Decay gamma in (0, 1] (decay section; decay-aware monoid): the pair (i, j)
// enters row t with weight gamma^{(t-i)+(t-j)}, the masked operator keeping
// i <= j.  A chunk's summary is then taken relative to its last token, and
// the scan composes chunks with attenuation rho = gamma^length (G and h by
// rho^2, the cross term by rho).  gamma = 1 is the undecayed operator: every
// power below is exp2(0) = 1 exactly.
#include "common.h"
#include "profile.h"

namespace hla {

// ----------------------------------------------------------------------------
// Chunk summary.  With A_s[i][j] = [j < i] k_i . q_j (strictly lower):
//   S = K^T K,  C = Q^T V,  m = Q^T 1,  G = K^T (A_s V),  h = K^T (A_s 1).
// G is sum_i k_i k_i^T C_{i-1} with C local to the chunk (Sec. 3.1).
// With decay every token t of a chunk of L tokens carries w_t = gamma^(L-1-t)
// in S, C, m and the pair (i, j) carries w_i w_j in G, h.
// LDS: A_s [chunk][chunk] and Y = [A_s V | A_s 1]  [chunk][dv+1].
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_chunk_summary(const T* __restrict__ q, const T* __restrict__ k,
                                                       const T* __restrict__ v, float* __restrict__ states,
                                                       int n, int d, int dv, int chunk, int M, float lg2g) {
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

  auto w = [&](int t) { return exp2f(lg2g * (float)(L - 1 - t)); };   // gamma^(L-1-t)
  for (int idx = tid; idx < L * L; idx += blockDim.x) {
    const int i = idx / L, j = idx % L;
    float s = 0.f;
    if (j < i) {
      for (int a = 0; a < d; ++a) s += ldf(k, qk_base + (size_t)i * d + a) * ldf(q, qk_base + (size_t)j * d + a);
      s *= exp2f(lg2g * (float)(2 * L - 2 - i - j));
    }
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
    for (int t = 0; t < L; ++t) s += w(t) * ldf(k, qk_base + (size_t)t * d + a) * ldf(k, qk_base + (size_t)t * d + b);
    S[idx] = s;
  }
  for (int idx = tid; idx < d * dv; idx += blockDim.x) {
    const int a = idx / dv, b = idx % dv;
    float sc = 0.f, sg = 0.f;
    for (int t = 0; t < L; ++t) {
      sc += w(t) * ldf(q, qk_base + (size_t)t * d + a) * ldf(v, v_base + (size_t)t * dv + b);
      sg += ldf(k, qk_base + (size_t)t * d + a) * Y[t * ldY + b];
    }
    Cc[idx] = sc;
    G[idx] = sg;
  }
  for (int a = tid; a < d; a += blockDim.x) {
    float sm = 0.f, sh = 0.f;
    for (int t = 0; t < L; ++t) {
      sm += w(t) * ldf(q, qk_base + (size_t)t * d + a);
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
// product of states is formed.  With decay (local index a of token t, carry
// taken at the token before the chunk):
//   r_j = g^(a_j+1) S0 q_j + sum_{i<=j} g^(a_j-a_i) (k_i.q_j) k_i,
//   masked:   o_t = g^(2(a+1)) q_t^T (S0 C0 - G0) + sum_{j<=t} g^(2(a-a_j)) (q_t . r_j) v_j
//   unmasked: o_t = g^(a+1) r_t^T C0 + sum_{j<=t} g^(a-a_j) (r_t . q_j) v_j
// (the decayed inclusive state is g^(a+1) S0 + S_loc etc., and the S_loc C0
// terms of S C - G still cancel).
// LDS: R [chunk][d], W/T [chunk][chunk], den [chunk].
// ----------------------------------------------------------------------------
// The dot products over d accumulate in fp64 and R is held in fp64: a row
// whose value is far below the size of its terms (row 0 is (q_0.k_0)^2 v_0,
// with q_0.k_0 a cancelling dot product) keeps the fp32-input bar only when
// r_j and q_t . r_j are not rounded to fp32 on the way.  Chunks of up to 64
// tokens (the forward paths cut larger chunks, exact by Thm. 2).
// LDS: R [chunk][d] fp64, W/T [chunk][chunk] fp32, den [chunk] fp32.
template <typename T>
__global__ __launch_bounds__(256) void k_readout(const T* __restrict__ q, const T* __restrict__ k,
                                                 const T* __restrict__ v, const float* __restrict__ prefix,
                                                 float* __restrict__ out, float* __restrict__ den_out, int n,
                                                 int d, int dv, int chunk, int M, int masked, int normalized,
                                                 float eps, float lg2g) {
  extern __shared__ double smemd[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0);
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  double* R = smemd;                                        // [L][d]
  float* W = reinterpret_cast<float*>(smemd + chunk * d);   // [L][L]
  float* dn = W + chunk * chunk;                            // [L]
  const float* st = prefix + ((size_t)bh * M + c) * state_floats(d, dv);
  const float* S0 = st;
  const float* C0 = st + off_C(d, dv);
  const float* m0 = st + off_m(d, dv);
  const float* G0 = st + off_G(d, dv);
  const float* h0 = st + off_h(d, dv);
  float* o = out + v_base;
  auto qf = [&](int t, int a) { return (double)ldf(q, qk_base + (size_t)t * d + a); };
  auto kf = [&](int t, int a) { return (double)ldf(k, qk_base + (size_t)t * d + a); };

  // P = Q S0 into R;  W[t][i] = [i <= t] g^(t-i) q_t . k_i
  for (int idx = tid; idx < L * d; idx += blockDim.x) {
    const int t = idx / d, a = idx % d;
    double s = 0.0;
    for (int b = 0; b < d; ++b) s += qf(t, b) * (double)S0[(size_t)b * d + a];
    R[idx] = s;
  }
  for (int idx = tid; idx < L * L; idx += blockDim.x) {
    const int t = idx / L, i = idx % L;
    double s = 0.0;
    if (i <= t) {
      for (int a = 0; a < d; ++a) s += qf(t, a) * kf(i, a);
      s *= (double)exp2f(lg2g * (float)(t - i));
    }
    W[idx] = (float)s;
  }
  __syncthreads();
  if (masked) {
    // carry term g^(2(a+1)) (q_t^T S0 C0 - q_t^T G0) (and its denominator)
    for (int idx = tid; idx < L * dv; idx += blockDim.x) {
      const int t = idx / dv, b = idx % dv;
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * (double)C0[(size_t)a * dv + b] - qf(t, a) * (double)G0[(size_t)a * dv + b];
      o[(size_t)t * dv + b] = (float)s * exp2f(lg2g * (float)(2 * t + 2));
    }
    for (int t = tid; t < L; t += blockDim.x) {
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * (double)m0[a] - qf(t, a) * (double)h0[a];
      dn[t] = (float)s * exp2f(lg2g * (float)(2 * t + 2));
    }
  }
  __syncthreads();
  // the carry part of r_t decays by g^(a+1); then R += W K  (r_j = S_j q_j)
  for (int idx = tid; idx < L * d; idx += blockDim.x) {
    const int j = idx / d, a = idx % d;
    double s = R[idx] * (double)exp2f(lg2g * (float)(j + 1));
    for (int i = 0; i <= j; ++i) s += (double)W[j * L + i] * kf(i, a);
    R[idx] = s;
  }
  __syncthreads();
  // T[t][j] = [j <= t] g^(2(t-j)) (q_t . r_j)  (masked)  or  g^(t-j) (r_t . q_j)  (unmasked)
  for (int idx = tid; idx < L * L; idx += blockDim.x) {
    const int t = idx / L, j = idx % L;
    double s = 0.0;
    if (j <= t) {
      if (masked)
        for (int a = 0; a < d; ++a) s += qf(t, a) * R[j * d + a];
      else
        for (int a = 0; a < d; ++a) s += R[t * d + a] * qf(j, a);
      s *= (double)exp2f(lg2g * (float)((masked ? 2 : 1) * (t - j)));
    }
    W[idx] = (float)s;
  }
  if (!masked) {
    for (int idx = tid; idx < L * dv; idx += blockDim.x) {
      const int t = idx / dv, b = idx % dv;
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * (double)C0[(size_t)a * dv + b];
      o[(size_t)t * dv + b] = (float)s * exp2f(lg2g * (float)(t + 1));
    }
    for (int t = tid; t < L; t += blockDim.x) {
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += R[t * d + a] * (double)m0[a];
      dn[t] = (float)s * exp2f(lg2g * (float)(t + 1));
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
      if (den_out) den_out[(size_t)bh * n + t0 + t] = s;
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
static size_t readout_lds(int chunk, int d) {
  return sizeof(double) * (size_t)chunk * d + sizeof(float) * ((size_t)chunk * chunk + chunk);
}

hipError_t launch_chunk_summaries(const void* q, const void* k, const void* v, float* states,
                                  int BH, int n, int d, int dv, int chunk, int dtype, hipStream_t s, float gamma) {
  const float lg2g = log2f(gamma);
  const int M = (n + chunk - 1) / chunk;
  const size_t lds = summary_lds(chunk, dv);
  dim3 grid(M, BH), block(256);
  if (dtype == 1) {
    auto kern = k_chunk_summary<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const uint16_t*)q, (const uint16_t*)k,
                       (const uint16_t*)v, states, n, d, dv, chunk, M, lg2g);
  } else {
    auto kern = k_chunk_summary<float>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const float*)q, (const float*)k, (const float*)v,
                       states, n, d, dv, chunk, M, lg2g);
  }
  return hipGetLastError();
}

hipError_t launch_readout(const Fwd& f, const float* prefix, hipStream_t s) {
  if (f.chunk > kReadoutMaxChunk) return hipErrorInvalidValue;
  const float lg2g = log2f(f.gamma);
  const int M = (f.n + f.chunk - 1) / f.chunk;
  const size_t lds = readout_lds(f.chunk, f.d);
  dim3 grid(M, f.BH), block(256);
  if (f.dtype == 1) {
    auto kern = k_readout<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const uint16_t*)f.q, (const uint16_t*)f.k,
                       (const uint16_t*)f.v, prefix, f.out, f.den_out, f.n, f.d, f.dv, f.chunk, M, f.masked,
                       f.normalized, f.eps, lg2g);
  } else {
    auto kern = k_readout<float>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const float*)f.q, (const float*)f.k, (const float*)f.v,
                       prefix, f.out, f.den_out, f.n, f.d, f.dv, f.chunk, M, f.masked, f.normalized, f.eps, lg2g);
  }
  return hipGetLastError();
}

}  // namespace hla
