// Fused segment-walk forward for bf16 inputs (MFMA).  See fused.hip.
#pragma once
#include "common.h"

namespace hla {
bool fused_supported(int n, int d, int dv, int chunk, int dtype, int masked);
// the decayed operator (Fwd::gamma != 1) on the fused path: row-split shapes only
bool fused_decay_supported(int n, int d, int dv, int chunk, int dtype, int masked);
size_t fused_workspace_bytes(int BH, int n, int d, int dv, int chunk);
// segments per head and token tile of the plan for these arguments (false if no shape covers them)
bool fused_plan_query(int BH, int n, int d, int dv, int chunk, int* P, int* tile, int* first, int* per);
// init/final: optional [BH][F] states (carry-in of token 0 / state after the last token).
hipError_t launch_fused(const Fwd& f, const float* init, float* final_state, void* workspace, hipStream_t s);
}  // namespace hla
