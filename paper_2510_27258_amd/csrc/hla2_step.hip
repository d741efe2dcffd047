// Decode step of second-order HLA: one token per head, state updated in place.
//
// The online updates of Sec. 3.1 and the readout of Thm. 1 in the order of
// Sec. 5 (u = q^T S_t, num = u C_t - q^T G_t, den = u m_t - q^T h_t):
//   w = k^T C_{t-1},  s = k^T m_{t-1}
//   G += k w^T,  h += s k,  S += k k^T,  C += q v^T,  m += q
// One workgroup per head.  Every state element is read once and written
// once: all of S, C and G are loaded up front (16-byte vector loads, up to
// 48 per thread), then three dependent reductions over rows run through LDS.
// The state (all heads together larger than the last-level cache) is
// streamed once per step, so its loads and stores are non-temporal.
#include "common.h"
#include "profile.h"

namespace hla {

constexpr int kStepThreads = 256;
typedef float nf4 __attribute__((ext_vector_type(4)));
// 16-byte non-temporal load and store
__device__ __forceinline__ float4 ntld(const float4* p) {
  const nf4 x = __builtin_nontemporal_load(reinterpret_cast<const nf4*>(p));
  return make_float4(x[0], x[1], x[2], x[3]);
}
__device__ __forceinline__ void ntst(const float4& v, float4* p) {
  __builtin_nontemporal_store(nf4{v.x, v.y, v.z, v.w}, reinterpret_cast<nf4*>(p));
}
constexpr int kStepMaxVec = 16;   // d*d/4/256 and d*dv/4/256 at d = dv = 128

template <typename T>
__global__ __launch_bounds__(kStepThreads) void k_step(float* __restrict__ state, const T* __restrict__ q,
                                                       const T* __restrict__ k, const T* __restrict__ v,
                                                       float* __restrict__ out, int d, int dv, int masked,
                                                       int normalized, float eps) {
  __shared__ float qs[128], ks[128], vs[128], us[128], ws[128], mk[128], dterm[128];
  __shared__ float red1[1024], red2[1024];
  const int bh = blockIdx.x, tid = threadIdx.x;
  const size_t F = state_floats(d, dv);
  float* st = state + (size_t)bh * F;
  float* S = st;
  float* C = st + off_C(d, dv);
  float* m = st + off_m(d, dv);
  float* G = st + off_G(d, dv);
  float* h = st + off_h(d, dv);
  const int nS4 = d * d / 4, nC4 = d * dv / 4;

  float4 Sv[kStepMaxVec], Cv[kStepMaxVec], Gv[kStepMaxVec];
#pragma unroll
  for (int r = 0; r < kStepMaxVec; ++r) {
    const int f = tid + kStepThreads * r;
    if (f < nS4) Sv[r] = ntld(reinterpret_cast<const float4*>(S) + f);
    if (f < nC4) {
      Cv[r] = ntld(reinterpret_cast<const float4*>(C) + f);
      Gv[r] = ntld(reinterpret_cast<const float4*>(G) + f);
    }
  }
  float m_old = 0.f, h_old = 0.f;
  if (tid < d) {
    qs[tid] = ldf(q, (size_t)bh * d + tid);
    ks[tid] = ldf(k, (size_t)bh * d + tid);
    m_old = m[tid];
    h_old = h[tid];
    mk[tid] = ks[tid] * m_old;
  }
  if (tid < dv) vs[tid] = ldf(v, (size_t)bh * dv + tid);
  __syncthreads();

  // S pass: S_t = S_{t-1} + k k^T, partial u = q^T S_t over this thread's rows
  {
    const int col = (tid * 4) % d, rg = (tid * 4) / d;
    float up[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < kStepMaxVec; ++r) {
      const int f = tid + kStepThreads * r;
      if (f < nS4) {
        const int a = (f * 4) / d;
        const float ka = ks[a], qa = qs[a];
        float4 s = Sv[r];
        s.x += ka * ks[col + 0];
        s.y += ka * ks[col + 1];
        s.z += ka * ks[col + 2];
        s.w += ka * ks[col + 3];
        ntst(s, reinterpret_cast<float4*>(S) + f);
        up[0] += qa * s.x; up[1] += qa * s.y; up[2] += qa * s.z; up[3] += qa * s.w;
      }
    }
    if (tid < nS4 && tid * 4 < 1024)
      for (int i = 0; i < 4; ++i) red1[rg * d + col + i] = up[i];
  }
  // C pass: w = k^T C_{t-1} (old values), then C_t = C_{t-1} + q v^T (kept in registers)
  {
    const int col = (tid * 4) % dv, rg = (tid * 4) / dv;
    float wp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < kStepMaxVec; ++r) {
      const int f = tid + kStepThreads * r;
      if (f < nC4) {
        const int a = (f * 4) / dv;
        const float ka = ks[a], qa = qs[a];
        float4 c = Cv[r];
        wp[0] += ka * c.x; wp[1] += ka * c.y; wp[2] += ka * c.z; wp[3] += ka * c.w;
        c.x += qa * vs[col + 0];
        c.y += qa * vs[col + 1];
        c.z += qa * vs[col + 2];
        c.w += qa * vs[col + 3];
        Cv[r] = c;
        ntst(c, reinterpret_cast<float4*>(C) + f);
      }
    }
    if (tid < nC4 && tid * 4 < 1024)
      for (int i = 0; i < 4; ++i) red2[rg * dv + col + i] = wp[i];
  }
  __syncthreads();

  // finish u, w; update m, h; denominator terms
  if (tid < d) {
    float u = 0.f;
    const int ngS = min(1024, nS4 * 4) / d;
    for (int g = 0; g < ngS; ++g) u += red1[g * d + tid];
    us[tid] = u;
    float s = 0.f;
    for (int a = 0; a < d; ++a) s += mk[a];
    const float m_new = m_old + qs[tid];
    const float h_new = h_old + s * ks[tid];
    m[tid] = m_new;
    h[tid] = h_new;
    dterm[tid] = u * m_new - (masked ? qs[tid] * h_new : 0.f);
  }
  if (tid < dv) {
    float w = 0.f;
    const int ngC = min(1024, nC4 * 4) / dv;
    for (int g = 0; g < ngC; ++g) w += red2[g * dv + tid];
    ws[tid] = w;
  }
  __syncthreads();

  // num = u C_t - q^T G_t, with G_t = G_{t-1} + k w^T
  {
    const int col = (tid * 4) % dv, rg = (tid * 4) / dv;
    float np[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < kStepMaxVec; ++r) {
      const int f = tid + kStepThreads * r;
      if (f < nC4) {
        const int a = (f * 4) / dv;
        const float ka = ks[a], qa = qs[a], ua = us[a];
        const float4 c = Cv[r];
        float4 g = Gv[r];
        g.x += ka * ws[col + 0];
        g.y += ka * ws[col + 1];
        g.z += ka * ws[col + 2];
        g.w += ka * ws[col + 3];
        ntst(g, reinterpret_cast<float4*>(G) + f);
        np[0] += ua * c.x; np[1] += ua * c.y; np[2] += ua * c.z; np[3] += ua * c.w;
        if (masked) {
          np[0] -= qa * g.x; np[1] -= qa * g.y; np[2] -= qa * g.z; np[3] -= qa * g.w;
        }
      }
    }
    __syncthreads();   // red1 was read above; reuse it
    if (tid < nC4 && tid * 4 < 1024)
      for (int i = 0; i < 4; ++i) red1[rg * dv + col + i] = np[i];
  }
  __syncthreads();
  if (tid < dv) {
    float num = 0.f;
    const int ngC = min(1024, nC4 * 4) / dv;
    for (int g = 0; g < ngC; ++g) num += red1[g * dv + tid];
    if (normalized) {
      float den = 0.f;
      for (int a = 0; a < d; ++a) den += dterm[a];
      num = num / (den + eps);
    }
    out[(size_t)bh * dv + tid] = num;
  }
}

__global__ __launch_bounds__(256) void k_zero(float4* __restrict__ p, size_t n4) {
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) p[i] = z;
}

hipError_t launch_zero(float* p, size_t n4, hipStream_t s) {
  if (n4 == 0) return hipSuccess;
  const size_t blocks = (n4 + 255) / 256;
  HLA_LAUNCH(k_zero, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, s, reinterpret_cast<float4*>(p), n4);
  return hipGetLastError();
}

hipError_t launch_step(float* state, const void* q, const void* k, const void* v, float* out, int BH, int d,
                       int dv, int masked, int normalized, float eps, int dtype, hipStream_t s) {
  if (dtype == 1)
    HLA_LAUNCH(k_step<uint16_t>, dim3(BH), dim3(kStepThreads), 0, s, state, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, out, d, dv, masked, normalized, eps);
  else
    HLA_LAUNCH(k_step<float>, dim3(BH), dim3(kStepThreads), 0, s, state, (const float*)q,
                       (const float*)k, (const float*)v, out, d, dv, masked, normalized, eps);
  return hipGetLastError();
}

}  // namespace hla
