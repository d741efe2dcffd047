// Decode step of second-order HLA: one token per head, state updated in place.
//
// The online updates of Sec. 3.1 and the readout of Thm. 1 in the order of
// Sec. 5 (u = q^T S_t, num = u C_t - q^T G_t, den = u m_t - q^T h_t):
//   w = k^T C_{t-1},  s = k^T m_{t-1}
//   G += k w^T,  h += s k,  S += k k^T,  C += q v^T,  m += q
// Every state element is read once and written once per step.  The state is
// the paper's 5-tuple with S packed symmetric (Sec. 5: its upper triangle,
// d(d+1)/2 floats in folded row pairs; layout in common.h), which cuts a
// head's bytes from 2 (d^2 + 2 d dv + 2d) 4 to 2 (d(d+1)/2 + 2 d dv + 2d) 4.
//
// One workgroup per CU walks heads blockIdx.x, blockIdx.x + gridDim.x, ...
// A head is three streaming passes over its state (S, then C, then G), each
// held in registers (16-byte pieces, 1024/d rows apart per thread for C and
// G); while one pass is computed, the next pass's matrix is already loading
// into the other register buffer (C during the S pass, G during the C pass,
// the next head's S during the G pass), so every workgroup keeps one to two
// matrices of loads in flight.  The reductions between passes go through
// LDS behind barriers that do not drain global memory.
//   S pass: S_t = S_{t-1} + k k^T on the triangle, mirrored into LDS in
//           full; u = q^T S_t from the LDS copy (a fixed summation order)
//   C pass: w = k^T C_{t-1},  C_t = C_{t-1} + q v^T,  num = u C_t
//   G pass: G_t = G_{t-1} + k w^T,  num -= q^T G_t (masked)
// Launch shape and cache policy were measured on 2048 heads at d = dv = 128
// with the full S (812 MB per step): one workgroup per CU streamed at 0.85 of
// HBM peak, two at 0.77, four at 0.80; non-temporal loads dropped two per CU
// to 0.67.  The
// stores are non-temporal (the state, larger than the last-level cache, is
// not read again within the step).
#include "common.h"
#include "profile.h"

namespace hla {

constexpr int kStepThreads = 256;
constexpr int kStepMaxVec = 16;   // d*d/4/256 and d*dv/4/256 at d = dv = 128
constexpr int kStepWGsPerCU = 1;
constexpr int kCUs = 256;   // MI355X

typedef __amdgpu_buffer_rsrc_t step_rsrc;
constexpr int kStoreNT = 2;   // buffer cache policy bit: non-temporal

struct StepSmall {
  float q, k, v, m, h;
};

// One head's state as a buffer resource (offsets in bytes from the head's S).
__device__ __forceinline__ step_rsrc step_res(float* st, size_t F) {
  return __builtin_amdgcn_make_buffer_rsrc(st, (short)0, (int)(F * 4), 0x00020000);
}

// Offsets (floats) of the packed decode record's fields.
template <int D, int DV>
struct StepRec {
  static constexpr size_t nS = (size_t)D * (D + 1) / 2;
  static constexpr size_t oC = nS, om = nS + (size_t)D * DV, oG = om + D, oh = oG + (size_t)D * DV;
  static constexpr size_t F = oh + D;
  static_assert(nS % 4 == 0, "C, m, G, h stay 16-byte aligned");
};

template <typename T, int D, int DV>
__device__ __forceinline__ void step_small(StepSmall& x, const T* q, const T* k, const T* v, const float* st,
                                           int bh, int tid) {
  if (tid < D) {
    x.q = ldf(q, (size_t)bh * D + tid);
    x.k = ldf(k, (size_t)bh * D + tid);
    x.m = st[StepRec<D, DV>::om + tid];
    x.h = st[StepRec<D, DV>::oh + tid];
  }
  if (tid < DV) x.v = ldf(v, (size_t)bh * DV + tid);
}

// Matrix of N4 float4 at byte offset base of the head: element tid + 256 r
// of thread tid in slot r.
template <int N4>
struct StepMat {
  static constexpr int R = N4 >= kStepThreads ? N4 / kStepThreads : 1;
  static __device__ __forceinline__ bool lane_ok(int tid) { return N4 >= kStepThreads || tid < N4; }
};

template <int N4>
__device__ __forceinline__ void step_load(float4 (&X)[kStepMaxVec], step_rsrc res, uint32_t base, int tid) {
  if (!StepMat<N4>::lane_ok(tid)) return;
#pragma unroll
  for (int r = 0; r < StepMat<N4>::R; ++r) {
    const auto x = __builtin_amdgcn_raw_buffer_load_b128(res, (int)(base + tid * 16), r * kStepThreads * 16, 0);
    X[r] = make_float4(__uint_as_float(x[0]), __uint_as_float(x[1]), __uint_as_float(x[2]), __uint_as_float(x[3]));
  }
}

// Whole offset in the lane offset and a zero soffset: with an SGPR soffset
// the compiler may place a VALU write of a 16-byte store's data registers
// right after the store, and on gfx950 such a write was seen to reach memory
// in place of the data.
// The packed S of a head: element tid + 256 r in slot r, the last slot partial.
template <int N4>
__device__ __forceinline__ void step_load_s(float4 (&X)[kStepMaxVec], step_rsrc res, int tid) {
  static_assert((N4 + kStepThreads - 1) / kStepThreads <= kStepMaxVec, "packed S fits the slots");
#pragma unroll
  for (int r = 0; r < (N4 + kStepThreads - 1) / kStepThreads; ++r)
    if (tid + kStepThreads * r < N4) {
      const auto x = __builtin_amdgcn_raw_buffer_load_b128(res, (int)((tid + kStepThreads * r) * 16), 0, 0);
      X[r] = make_float4(__uint_as_float(x[0]), __uint_as_float(x[1]), __uint_as_float(x[2]), __uint_as_float(x[3]));
    }
}

__device__ __forceinline__ void step_store(const float4& v, step_rsrc res, uint32_t base, int tid, int r) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(
      u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)}, res,
      (int)(base + tid * 16 + r * kStepThreads * 16), 0, kStoreNT);
}

struct StepLds {
  float vec[2][4][128];     // per head slot: q, k, v, k_a m_a
  float us[128], ws[128], dterm[128];
  float redA[1024], redB[1024];
  float Sm[128 * 129];      // S_t in full (row stride d + 1), mirrored from the packed triangle
};

// One head.  On entry X holds (or is loading) the head's packed S and x its
// small vectors; on exit Y holds (or is loading) the next head's S and x its
// small vectors.  The head's C goes to Y, then its G to X once the S pass has
// read X, and the next head's S to Y once the C pass has read Y.
template <typename T, int D, int DV>
__device__ __forceinline__ void step_head(float4 (&X)[kStepMaxVec], float4 (&Y)[kStepMaxVec], StepSmall& x,
                                          StepLds& L, int slot, float* __restrict__ state, const T* q,
                                          const T* k, const T* v, float* __restrict__ out, int bh, int nb,
                                          int masked, int normalized, float eps) {
  using Rec = StepRec<D, DV>;
  constexpr int nSp4 = (int)(Rec::nS / 4), nC4 = D * DV / 4;
  constexpr size_t F = Rec::F;
  constexpr uint32_t oC = 4 * Rec::oC, oG = 4 * Rec::oG;
  const int tid = threadIdx.x;
  float* st = state + (size_t)bh * F;
  const step_rsrc res = step_res(st, F);
  // C loads go out first: the small vectors below were loaded after this
  // head's S, so waiting for them waits for S as well
  step_load<nC4>(Y, res, oC, tid);
  float* qs = L.vec[slot][0];
  float* ks = L.vec[slot][1];
  float* vs = L.vec[slot][2];
  float* mk = L.vec[slot][3];
  const float m_old = x.m, h_old = x.h;
  if (tid < D) {
    qs[tid] = x.q;
    ks[tid] = x.k;
    mk[tid] = x.k * x.m;
  }
  if (tid < DV) vs[tid] = x.v;
  lds_barrier();

  // S pass: S_t = S_{t-1} + k k^T on the stored triangle, each updated value
  // mirrored into the full matrix in LDS; then u = q^T S_t by columns
  {
    constexpr int RS = (nSp4 + kStepThreads - 1) / kStepThreads;
#pragma unroll
    for (int r = 0; r < RS; ++r) {
      const int f = tid + kStepThreads * r;
      if (f < nSp4) {
        float x4[4] = {X[r].x, X[r].y, X[r].z, X[r].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int a, j;
          packed_s_index(4 * f + i, D, a, j);
          x4[i] += ks[a] * ks[j];
          L.Sm[a * (D + 1) + j] = x4[i];
          L.Sm[j * (D + 1) + a] = x4[i];
        }
        step_store(make_float4(x4[0], x4[1], x4[2], x4[3]), res, 0, tid, r);
      }
    }
  }
  step_load<nC4>(X, res, oG, tid);   // X is free: this head's G
  lds_barrier();
  {
    constexpr int NG = kStepThreads / D, RPG = D / NG;   // row groups, rows per group
    const int j = tid % D, g = tid / D;
    float up = 0.f;
#pragma unroll 8
    for (int a = g * RPG; a < (g + 1) * RPG; ++a) up += qs[a] * L.Sm[a * (D + 1) + j];
    L.redA[g * D + j] = up;
  }
  lds_barrier();
  if (tid < D) {
    float u = 0.f;
    for (int g = 0; g < kStepThreads / D; ++g) u += L.redA[g * D + tid];
    L.us[tid] = u;
    float s = 0.f;
    for (int a = 0; a < D; ++a) s += mk[a];
    const float m_new = m_old + qs[tid];
    const float h_new = h_old + s * ks[tid];
    st[Rec::om + tid] = m_new;
    st[Rec::oh + tid] = h_new;
    L.dterm[tid] = u * m_new - (masked ? qs[tid] * h_new : 0.f);
  }
  lds_barrier();

  constexpr int rstepC = kStepThreads * 4 / DV;
  constexpr int ngC = (kStepThreads * 4 < D * DV ? kStepThreads * 4 : D * DV) / DV;
  const int colC = (tid * 4) % DV, rgC = (tid * 4) / DV;
  // C pass
  if (StepMat<nC4>::lane_ok(tid)) {
    float wp[4] = {0.f, 0.f, 0.f, 0.f}, np[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < StepMat<nC4>::R; ++r) {
      const int a = rgC + r * rstepC;
      const float ka = ks[a], qa = qs[a], ua = L.us[a];
      float4 c = Y[r];
      wp[0] += ka * c.x; wp[1] += ka * c.y; wp[2] += ka * c.z; wp[3] += ka * c.w;
      c.x += qa * vs[colC + 0];
      c.y += qa * vs[colC + 1];
      c.z += qa * vs[colC + 2];
      c.w += qa * vs[colC + 3];
      step_store(c, res, oC, tid, r);
      np[0] += ua * c.x; np[1] += ua * c.y; np[2] += ua * c.z; np[3] += ua * c.w;
    }
    for (int i = 0; i < 4; ++i) {
      L.redA[rgC * DV + colC + i] = wp[i];
      L.redB[rgC * DV + colC + i] = np[i];
    }
  }
  if (nb >= 0) {                 // Y is free: the next head's S and small vectors
    float* nst = state + (size_t)nb * F;
    step_load_s<nSp4>(Y, step_res(nst, F), tid);
    step_small<T, D, DV>(x, q, k, v, nst, nb, tid);
  }
  lds_barrier();
  float num = 0.f;
  if (tid < DV) {
    float w = 0.f;
    for (int g = 0; g < ngC; ++g) {
      w += L.redA[g * DV + tid];
      num += L.redB[g * DV + tid];
    }
    L.ws[tid] = w;
  }
  lds_barrier();

  // G pass
  if (StepMat<nC4>::lane_ok(tid)) {
    float gp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < StepMat<nC4>::R; ++r) {
      const int a = rgC + r * rstepC;
      const float ka = ks[a], qa = qs[a];
      float4 g = X[r];
      g.x += ka * L.ws[colC + 0];
      g.y += ka * L.ws[colC + 1];
      g.z += ka * L.ws[colC + 2];
      g.w += ka * L.ws[colC + 3];
      step_store(g, res, oG, tid, r);
      gp[0] += qa * g.x; gp[1] += qa * g.y; gp[2] += qa * g.z; gp[3] += qa * g.w;
    }
    if (masked)
      for (int i = 0; i < 4; ++i) L.redA[rgC * DV + colC + i] = gp[i];
  }
  lds_barrier();
  if (tid < DV) {
    if (masked)
      for (int g = 0; g < ngC; ++g) num -= L.redA[g * DV + tid];
    if (normalized) {
      float den = 0.f;
      for (int a = 0; a < D; ++a) den += L.dterm[a];
      num = num / (den + eps);
    }
    out[(size_t)bh * DV + tid] = num;
  }
}

template <typename T, int D, int DV>
__global__ __launch_bounds__(kStepThreads) void k_step_pipe(float* __restrict__ state, const T* __restrict__ q,
                                                            const T* __restrict__ k, const T* __restrict__ v,
                                                            float* __restrict__ out, int BH, int masked,
                                                            int normalized, float eps) {
  __shared__ StepLds L;
  constexpr size_t F = StepRec<D, DV>::F;
  float4 A[kStepMaxVec], B[kStepMaxVec];
  StepSmall x{0.f, 0.f, 0.f, 0.f, 0.f};
  const int tid = threadIdx.x, G = gridDim.x;
  int bh = blockIdx.x;
  step_load_s<(int)(StepRec<D, DV>::nS / 4)>(A, step_res(state + (size_t)bh * F, F), tid);
  step_small<T, D, DV>(x, q, k, v, state + (size_t)bh * F, bh, tid);
  for (int slot = 0;; slot ^= 1) {
    int nb = bh + G < BH ? bh + G : -1;
    step_head<T, D, DV>(A, B, x, L, slot, state, q, k, v, out, bh, nb, masked, normalized, eps);
    if (nb < 0) break;
    bh = nb;
    slot ^= 1;
    nb = bh + G < BH ? bh + G : -1;
    step_head<T, D, DV>(B, A, x, L, slot, state, q, k, v, out, bh, nb, masked, normalized, eps);
    if (nb < 0) break;
    bh = nb;
  }
}

template <typename T, int D, int DV>
hipError_t launch_step_pipe(float* state, const void* q, const void* k, const void* v, float* out, int BH,
                            int masked, int normalized, float eps, int grid, hipStream_t s) {
  HLA_LAUNCH((k_step_pipe<T, D, DV>), dim3(grid), dim3(kStepThreads), 0, s, state, (const T*)q, (const T*)k,
             (const T*)v, out, BH, masked, normalized, eps);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t step_dv(int dv, float* state, const void* q, const void* k, const void* v, float* out, int BH,
                   int masked, int normalized, float eps, int grid, hipStream_t s) {
  switch (dv) {
    case 16: return launch_step_pipe<T, D, 16>(state, q, k, v, out, BH, masked, normalized, eps, grid, s);
    case 32: return launch_step_pipe<T, D, 32>(state, q, k, v, out, BH, masked, normalized, eps, grid, s);
    case 64: return launch_step_pipe<T, D, 64>(state, q, k, v, out, BH, masked, normalized, eps, grid, s);
    case 128: return launch_step_pipe<T, D, 128>(state, q, k, v, out, BH, masked, normalized, eps, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t step_d(int d, int dv, float* state, const void* q, const void* k, const void* v, float* out, int BH,
                  int masked, int normalized, float eps, int grid, hipStream_t s) {
  switch (d) {
    case 16: return step_dv<T, 16>(dv, state, q, k, v, out, BH, masked, normalized, eps, grid, s);
    case 32: return step_dv<T, 32>(dv, state, q, k, v, out, BH, masked, normalized, eps, grid, s);
    case 64: return step_dv<T, 64>(dv, state, q, k, v, out, BH, masked, normalized, eps, grid, s);
    case 128: return step_dv<T, 128>(dv, state, q, k, v, out, BH, masked, normalized, eps, grid, s);
  }
  return hipErrorInvalidValue;
}

// Full decode records [BH][state_floats] <-> packed [BH][dstate_floats]
// (S's upper triangle in folded row pairs, then C | m | G | h).  grid
// (blocks, BH); S is symmetric, so packing takes the upper triangle and
// unpacking writes both (a, j) and (j, a).
template <bool PACK>
__global__ __launch_bounds__(256) void k_state_pack(const float* __restrict__ src, float* __restrict__ dst, int d,
                                                    int dv) {
  const int bh = blockIdx.y;
  const size_t F = state_floats(d, dv), FP = dstate_floats(d, dv), nS = packed_s_floats(d);
  const float* in = src + (size_t)bh * (PACK ? F : FP);
  float* out = dst + (size_t)bh * (PACK ? FP : F);
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < FP; e += (size_t)gridDim.x * 256) {
    if (e < nS) {
      int a, j;
      packed_s_index((int)e, d, a, j);
      if (PACK) {
        out[e] = in[(size_t)a * d + j];
      } else {
        const float x = in[e];
        out[(size_t)a * d + j] = x;
        out[(size_t)j * d + a] = x;
      }
    } else {
      const size_t r = e - nS, dd = (size_t)d * d;
      if (PACK) out[e] = in[dd + r];
      else out[dd + r] = in[e];
    }
  }
}

hipError_t launch_state_pack(const float* full, float* packed, int BH, int d, int dv, hipStream_t s) {
  const size_t blocks = (dstate_floats(d, dv) + 255) / 256;
  HLA_LAUNCH(k_state_pack<true>, dim3((unsigned)(blocks < 64 ? blocks : 64), BH), dim3(256), 0, s, full, packed, d, dv);
  return hipGetLastError();
}

hipError_t launch_state_unpack(const float* packed, float* full, int BH, int d, int dv, hipStream_t s) {
  const size_t blocks = (dstate_floats(d, dv) + 255) / 256;
  HLA_LAUNCH(k_state_pack<false>, dim3((unsigned)(blocks < 64 ? blocks : 64), BH), dim3(256), 0, s, packed, full, d, dv);
  return hipGetLastError();
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
  const int grid = BH < kStepWGsPerCU * kCUs ? BH : kStepWGsPerCU * kCUs;
  if (dtype == 1) return step_d<uint16_t>(d, dv, state, q, k, v, out, BH, masked, normalized, eps, grid, s);
  return step_d<float>(d, dv, state, q, k, v, out, BH, masked, normalized, eps, grid, s);
}

}  // namespace hla
