// Masked third-order HLA forward (fp32 arithmetic).  See hla3.hip.
#pragma once
#include "common.h"

namespace hla {
bool hla3_supported(int d, int dv, int chunk, int masked);
size_t hla3_workspace(int BH, int n, int d, int dv, int chunk);
hipError_t launch_hla3(const Fwd& f, void* workspace, hipStream_t s);
}  // namespace hla
