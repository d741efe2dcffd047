// hla2_forward_noalloc: hla2_forward for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc).  Its workspace is a fixed array in the library's own
// device memory, `scratch`, one copy per GPU (each GPU the library runs on
// holds it until the process ends).  Kernels and validation are those of
// hla2_forward_ex; only the workspace pointer differs.
//
// The array's name is a host-side stand-in in host code, not a device
// address: host code uses only the pointer hipGetSymbolAddress returns for
// the current device, taken once per device on the entry point's first call
// there.
#include <mutex>

#include "../../include/hla.h"
#include "common.h"

namespace hla {
int api_fail(int code, const char* msg);
}

namespace {

constexpr size_t kScratchBytes = HLA_NOALLOC_SCRATCH_BYTES;   // per GPU
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (null on failure, with the reason in
// *err).  Looked up once per device, with that device current.
void* scratch_ptr(hipError_t* err) {
  int dev = -1;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) return nullptr;
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" {

int hla2_forward_noalloc(const void* q, const void* k, const void* v, float* out, int B, int H, int n, int d, int dv,
                         int chunk, int masked, int normalized, float eps, int dtype, void* stream) {
  // the workspace of the algorithm HLA_ALGO_AUTO takes for these arguments
  // (the fused path when it covers them, with the call's masked flag)
  const int algo = hla2_algo_supported(HLA_ALGO_FUSED, n, d, dv, chunk, dtype, masked) ? HLA_ALGO_FUSED
                                                                                        : HLA_ALGO_CHUNKED;
  size_t need = 0;
  const int rc = hla2_workspace_query(B, H, n, d, dv, chunk, dtype, algo, &need);
  if (rc != HLA_OK) return rc;
  if (need > kScratchBytes) {
    char msg[256];
    snprintf(msg, sizeof(msg),
             "hla2_forward_noalloc: these sizes need %zu bytes of workspace, above the library's fixed %zu-byte "
             "scratch; call hla2_forward with a caller-owned workspace instead",
             need, kScratchBytes);
    return hla::api_fail(HLA_ERR_WORKSPACE, msg);
  }
  hipError_t e;
  void* ws = scratch_ptr(&e);
  if (!ws) return hla::api_fail(HLA_ERR_HIP, hipGetErrorString(e));
  return hla2_forward_ex(q, k, v, out, nullptr, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws,
                         kScratchBytes, algo, stream);
}

}  // extern "C"
