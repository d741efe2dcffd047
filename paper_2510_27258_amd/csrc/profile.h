// Kernel-level event bracketing used by the C ABI when profiling is enabled.
#pragma once
#include <hip/hip_runtime.h>

namespace hla {
void prof_start(const char* name, hipStream_t s);
void prof_stop(hipStream_t s);
// Brackets one launcher call: PROF("name", stream, expr)
#define HLA_PROF(name, s, expr) \
  (hla::prof_start(name, s), [&]() { auto _r = (expr); hla::prof_stop(s); return _r; }())
}  // namespace hla
