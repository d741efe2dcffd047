// Gradients of the masked second-order HLA for bf16 inputs (MFMA).  See hla2_backward.hip.
#pragma once
#include "common.h"

namespace hla {
struct Bwd {
  const void* q; const void* k; const void* v;   // bf16 [BH][n][d]
  const float* g;                                 // upstream gradient, fp32 [BH][n][dv]
  float* dq; float* dk; float* dv;                // fp32 [BH][n][d] (dv: [BH][n][dv])
  int BH, n, d, dvd, dtype;                      // dvd: value width
};
bool backward_supported(int n, int d, int dv, int dtype);
size_t backward_workspace_bytes(int BH, int n, int d);
hipError_t launch_backward(const Bwd& b, void* workspace, hipStream_t s);
}  // namespace hla
