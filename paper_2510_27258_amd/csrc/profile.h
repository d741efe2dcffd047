// Kernel-level timing used by the C ABI when profiling is enabled.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

namespace hla {
void prof_start(const char* name, hipStream_t s);
void prof_stop(hipStream_t s);
// The open bracket's two events for the first kernel launched inside it (the
// dispatch records its own start and end time into them); false when no
// bracket is open or a kernel already took them.
bool prof_take(hipEvent_t* start, hipEvent_t* stop);
// hipLaunchKernel, through prof_take.
hipError_t prof_launch(const void* fn, dim3 grid, dim3 block, void** args, size_t lds, hipStream_t s);
// Brackets one launcher call: PROF("name", stream, expr)
#define HLA_PROF(name, s, expr) \
  (hla::prof_start(name, s), [&]() { auto _r = (expr); hla::prof_stop(s); return _r; }())
// hipLaunchKernelGGL, through prof_take.
#define HLA_LAUNCH(kernel, grid, block, lds, stream, ...)                                        \
  do {                                                                                             \
    hipEvent_t hla_e0_, hla_e1_;                                                                   \
    if (hla::prof_take(&hla_e0_, &hla_e1_))                                                        \
      hipExtLaunchKernelGGL(kernel, grid, block, lds, stream, hla_e0_, hla_e1_, 0, __VA_ARGS__);   \
    else                                                                                           \
      hipLaunchKernelGGL(kernel, grid, block, lds, stream, __VA_ARGS__);                           \
  } while (0)
}  // namespace hla
