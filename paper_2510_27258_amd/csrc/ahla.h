// AHLA (Sec. 6) forward for bf16 inputs (MFMA).  See ahla.hip.
#pragma once
#include "common.h"

namespace hla {
bool ahla_supported(int n, int d, int dv, int chunk, int dtype);
size_t ahla_workspace_bytes(int BH, int n, int d);
hipError_t launch_ahla(const Fwd& f, void* workspace, hipStream_t s);
}  // namespace hla
