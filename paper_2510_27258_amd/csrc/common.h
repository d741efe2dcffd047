// Shared device/host definitions for the HLA HIP library (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace hla {

// Record layout of one second-order state (one head or one chunk), fp32:
//   S [d][d] | C [d][dv] | m [d] | G [d][dv] | h [d]
__host__ __device__ inline size_t state_floats(int d, int dv) {
  return (size_t)d * d + 2 * (size_t)d * dv + 2 * (size_t)d;
}
__host__ __device__ inline size_t off_C(int d, int dv) { return (size_t)d * d; }
__host__ __device__ inline size_t off_m(int d, int dv) { return (size_t)d * d + (size_t)d * dv; }
__host__ __device__ inline size_t off_G(int d, int dv) { return (size_t)d * d + (size_t)d * dv + d; }
__host__ __device__ inline size_t off_h(int d, int dv) { return (size_t)d * d + 2 * (size_t)d * dv + d; }

// Record of one head of a decode state (hla2_state): the same fields with S
// packed symmetric (Sec. 5: only the upper triangle is stored), d(d+1)/2
// floats in d/2 folded row pairs: pair p holds row p of S from column p
// (d - p values), then row d-1-p from column d-1-p (p + 1 values); then
// C | m | G | h as above.  Element (a, j), a <= j, sits at p (d+1) + c with
// p = a, c = j - a when a < d/2, else p = d-1-a, c = j + 1.
__host__ __device__ inline size_t packed_s_floats(int d) { return (size_t)d * (d + 1) / 2; }
__host__ __device__ inline size_t dstate_floats(int d, int dv) {
  return packed_s_floats(d) + 2 * (size_t)d * dv + 2 * (size_t)d;
}
// (a, j), a <= j, of packed S element e
__host__ __device__ inline void packed_s_index(int e, int d, int& a, int& j) {
  const int p = e / (d + 1), c = e - p * (d + 1);
  const bool first = c < d - p;
  a = first ? p : d - 1 - p;
  j = first ? p + c : c - 1;
}

// Element loads converting the storage type to fp32.  bf16 is held as its
// 16-bit pattern; widening is exact.
__device__ __forceinline__ float ldf(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float ldf(const uint16_t* p, size_t i) {
  return __uint_as_float(((uint32_t)p[i]) << 16);
}

// Workgroup barrier that orders LDS only: it waits for this wave's LDS
// operations but not for its outstanding global loads and stores, so
// prefetches and output stores stay in flight across it (__syncthreads()
// also drains global memory).  Use it only where no wave reads global memory
// that another wave of the workgroup wrote before the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace hla

// Launchers implemented in the .hip files (host code, called by the C ABI).
namespace hla {
struct Fwd {
  const void* q; const void* k; const void* v; float* out;
  int BH, n, d, dv, chunk, masked, normalized, dtype;
  float eps;
  float gamma = 1.f;   // decay; 1 = none
  float* den_out = nullptr;   // [BH, n]: den_t without eps (normalized only), or null
};
// gamma: decay in (0, 1]; the summaries are taken relative to each chunk's last token.
hipError_t launch_chunk_summaries(const void* q, const void* k, const void* v, float* states,
                                  int BH, int n, int d, int dv, int chunk, int dtype,
                                  hipStream_t s, float gamma = 1.f);
// rho, rho_last: attenuation gamma^length of every segment but the last, and of
// the last (the decayed concatenation; 1 = none).
hipError_t launch_scan(const float* states, const float* init, float* prefix, float* total,
                       int BH, int M, int d, int dv, hipStream_t s, float rho = 1.f, float rho_last = 1.f);
// Strided form: head h's segment c is states[h*in_stride + c*F]; its prefix
// goes to prefix[h*pre_stride + c*F] and its total to total[h*tot_stride].
hipError_t launch_scan_strided(const float* states, const float* init, float* prefix, float* total, int BH, int M,
                               int d, int dv, size_t in_stride, size_t pre_stride, size_t tot_stride,
                               hipStream_t s, float rho = 1.f, float rho_last = 1.f);
// Chunks of at most kReadoutMaxChunk tokens (the forward paths cut larger ones).
constexpr int kReadoutMaxChunk = 64;
hipError_t launch_readout(const Fwd& f, const float* prefix, hipStream_t s);
hipError_t launch_step(float* state, const void* q, const void* k, const void* v, float* out,
                       int BH, int d, int dv, int masked, int normalized, float eps, int dtype,
                       hipStream_t s);
// p[0 .. n4) = 0 as float4 stores (a fill kernel, so it may be captured in a graph).
hipError_t launch_zero(float* p, size_t n4, hipStream_t s);
// Decode states: full records [BH][state_floats] <-> packed [BH][dstate_floats].
hipError_t launch_state_pack(const float* full, float* packed, int BH, int d, int dv, hipStream_t s);
hipError_t launch_state_unpack(const float* packed, float* full, int BH, int d, int dv, hipStream_t s);
}  // namespace hla
