// C ABI of the HLA library: argument validation, workspace carving and kernel
// dispatch.  No call allocates, synchronises or throws across the boundary.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/hla.h"
#include "ahla.h"
#include "backward.h"
#include "common.h"
#include "fused.h"
#include "hla3.h"
#include "profile.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return HLA_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(HLA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool pow2_in(int x, int lo, int hi) { return x >= lo && x <= hi && (x & (x - 1)) == 0; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int check_dims(int B, int H, int n, int d, int dv, int chunk, int dtype, bool need_n) {
  if (B < 1 || H < 1) return fail(HLA_ERR_INVALID, "B and H must be >= 1 (got B=%d H=%d)", B, H);
  if ((long long)B * H > 65535) return fail(HLA_ERR_UNSUPPORTED, "B*H=%lld exceeds 65535", (long long)B * H);
  if (need_n && n < 1) return fail(HLA_ERR_INVALID, "n must be >= 1 (got %d)", n);
  if (!pow2_in(d, 16, 128) || !pow2_in(dv, 16, 128))
    return fail(HLA_ERR_UNSUPPORTED, "d and dv must be one of 16, 32, 64, 128 (got d=%d dv=%d)", d, dv);
  // kernels address one head's rows with 32-bit byte offsets
  if (need_n && (long long)n * (d > dv ? d : dv) * 4 >= (1LL << 31))
    return fail(HLA_ERR_UNSUPPORTED, "n=%d is too long: n*max(d,dv)*4 must stay below 2^31 bytes", n);
  if (chunk != 0 && !pow2_in(chunk, 16, 128))
    return fail(HLA_ERR_UNSUPPORTED, "chunk must be one of 16, 32, 64, 128 (got %d)", chunk);
  if (dtype != HLA_FP32 && dtype != HLA_BF16) return fail(HLA_ERR_INVALID, "dtype must be HLA_FP32 or HLA_BF16");
  return HLA_OK;
}

int check_flags(int masked, int normalized, float eps) {
  if ((masked != 0 && masked != 1) || (normalized != 0 && normalized != 1))
    return fail(HLA_ERR_INVALID, "masked and normalized must be 0 or 1");
  if (!std::isfinite(eps) || eps < 0.f) return fail(HLA_ERR_INVALID, "eps must be finite and >= 0");
  return HLA_OK;
}

int check_ptr(const void* p, const char* name) {
  if (!p) return fail(HLA_ERR_INVALID, "%s is NULL", name);
  if (!aligned16(p)) return fail(HLA_ERR_INVALID, "%s is not 16-byte aligned", name);
  return HLA_OK;
}

// Chunk of the chunked path's summaries and readout: the caller's chunk, cut
// to the readout's maximum (exact for any chunking, Thm. 2).
int path_chunk(int chunk) { return chunk < hla::kReadoutMaxChunk ? chunk : hla::kReadoutMaxChunk; }

size_t chunked_ws(int BH, int n, int d, int dv, int chunk) {
  const size_t M = (size_t)(n + path_chunk(chunk) - 1) / path_chunk(chunk);
  return 2 * align256(sizeof(float) * (size_t)BH * M * hla::state_floats(d, dv));
}

int select_algo(int algo, int n, int d, int dv, int chunk, int dtype, int masked) {
  if (algo == HLA_ALGO_AUTO) return hla::fused_supported(n, d, dv, chunk, dtype, masked) ? HLA_ALGO_FUSED : HLA_ALGO_CHUNKED;
  return algo;
}

}  // namespace

namespace hla {
// Sets the thread's last error from another source file of the library.
int api_fail(int code, const char* msg) { return fail(code, "%s", msg); }
}  // namespace hla

extern "C" {

const char* hla_last_error(void) { return g_err; }

size_t hla2_state_floats(int d, int dv) { return hla::state_floats(d, dv); }

int hla2_algo_supported(int algo, int n, int d, int dv, int chunk, int dtype, int masked) {
  if (check_dims(1, 1, n, d, dv, chunk, dtype, true) != HLA_OK || chunk == 0) return 0;
  if (algo == HLA_ALGO_AUTO || algo == HLA_ALGO_CHUNKED) return 1;
  if (algo == HLA_ALGO_FUSED) return hla::fused_supported(n, d, dv, chunk, dtype, masked) ? 1 : 0;
  return 0;
}

size_t hla2_workspace_bytes_ex(int B, int H, int n, int d, int dv, int chunk, int dtype, int algo) {
  if (check_dims(B, H, n, d, dv, chunk, dtype, true) != HLA_OK) return 0;
  if (chunk == 0) { fail(HLA_ERR_INVALID, "chunk must be set"); return 0; }
  if (algo < HLA_ALGO_AUTO || algo > HLA_ALGO_FUSED) { fail(HLA_ERR_INVALID, "unknown algo %d", algo); return 0; }
  if (algo == HLA_ALGO_FUSED && !hla::fused_supported(n, d, dv, chunk, dtype, 1)) {
    fail(HLA_ERR_UNSUPPORTED, "the fused path does not cover d=%d dv=%d chunk=%d dtype=%d", d, dv, chunk, dtype);
    return 0;
  }
  const int a = select_algo(algo, n, d, dv, chunk, dtype, 1);
  if (a == HLA_ALGO_FUSED) return hla::fused_workspace_bytes(B * H, n, d, dv, chunk);
  return chunked_ws(B * H, n, d, dv, chunk);
}

size_t hla2_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype) {
  // large enough for whichever algorithm AUTO selects for either flag value
  size_t a = hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype, HLA_ALGO_AUTO);
  size_t b = hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype, HLA_ALGO_CHUNKED);
  return a > b ? a : b;
}

int hla2_forward_ex(const void* q, const void* k, const void* v, float* out, float* den, int B, int H, int n, int d,
                    int dv, int chunk, int masked, int normalized, float eps, int dtype, void* workspace,
                    size_t workspace_bytes, int algo, void* stream) {
  int rc;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if ((rc = check_flags(masked, normalized, eps)) != HLA_OK) return rc;
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v")) ||
      (rc = check_ptr(out, "out")))
    return rc;
  if (den && !normalized) return fail(HLA_ERR_INVALID, "den is written only with normalized = 1");
  if (den && !aligned16(den)) return fail(HLA_ERR_INVALID, "den is not 16-byte aligned");
  if (algo < HLA_ALGO_AUTO || algo > HLA_ALGO_FUSED) return fail(HLA_ERR_INVALID, "unknown algo %d", algo);
  const int a = select_algo(algo, n, d, dv, chunk, dtype, masked);
  const int BH = B * H;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hla::Fwd f{q, k, v, out, BH, n, d, dv, chunk, masked, normalized, dtype, eps};
  f.den_out = den;
  if (a == HLA_ALGO_FUSED) {
    if (!hla::fused_supported(n, d, dv, chunk, dtype, masked))
      return fail(HLA_ERR_UNSUPPORTED, "fused path needs bf16 inputs, masked=1 and (d, dv, chunk) in its "
                                       "instantiated set (got d=%d dv=%d chunk=%d dtype=%d)", d, dv, chunk, dtype);
    const size_t need = hla::fused_workspace_bytes(BH, n, d, dv, chunk);
    if (!workspace || workspace_bytes < need)
      return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
    hipError_t e = hla::launch_fused(f, nullptr, nullptr, workspace, s);
    if (e != hipSuccess) return hip_fail(e, "fused forward");
    return ok();
  }
  const size_t need = chunked_ws(BH, n, d, dv, chunk);
  if (!workspace || workspace_bytes < need)
    return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  f.chunk = path_chunk(chunk);
  const int M = (n + f.chunk - 1) / f.chunk;
  float* states = static_cast<float*>(workspace);
  float* prefix = reinterpret_cast<float*>(static_cast<char*>(workspace) + need / 2);
  hipError_t e = HLA_PROF("chunk_summary", s,
                          hla::launch_chunk_summaries(q, k, v, states, BH, n, d, dv, f.chunk, dtype, s));
  if (e != hipSuccess) return hip_fail(e, "chunk summaries");
  e = HLA_PROF("scan", s, hla::launch_scan(states, nullptr, prefix, nullptr, BH, M, d, dv, s));
  if (e != hipSuccess) return hip_fail(e, "scan");
  e = HLA_PROF("readout", s, hla::launch_readout(f, prefix, s));
  if (e != hipSuccess) return hip_fail(e, "readout");
  return ok();
}

int hla2_forward(const void* q, const void* k, const void* v, float* out, int B, int H, int n, int d, int dv,
                 int chunk, int masked, int normalized, float eps, int dtype, void* workspace,
                 size_t workspace_bytes, void* stream) {
  return hla2_forward_ex(q, k, v, out, nullptr, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, workspace,
                         workspace_bytes, HLA_ALGO_AUTO, stream);
}

int hla2_workspace_query(int B, int H, int n, int d, int dv, int chunk, int dtype, int algo, size_t* bytes) {
  if (!bytes) return fail(HLA_ERR_INVALID, "bytes is NULL");
  *bytes = 0;
  int rc;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if (algo < HLA_ALGO_AUTO || algo > HLA_ALGO_FUSED) return fail(HLA_ERR_INVALID, "unknown algo %d", algo);
  if (algo == HLA_ALGO_FUSED && !hla::fused_supported(n, d, dv, chunk, dtype, 1))
    return fail(HLA_ERR_UNSUPPORTED, "the fused path does not cover d=%d dv=%d chunk=%d dtype=%d", d, dv, chunk,
                dtype);
  *bytes = hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype, algo);
  return ok();
}

int hla2_fused_plan(int B, int H, int n, int d, int dv, int chunk, int* segments, int* tile, int* first_tiles,
                    int* tiles_per_segment) {
  int rc;
  if (!segments || !tile) return fail(HLA_ERR_INVALID, "segments and tile must not be NULL");
  if ((rc = check_dims(B, H, n, d, dv, chunk, HLA_BF16, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if (!hla::fused_supported(n, d, dv, chunk, HLA_BF16, 1) || !hla::fused_plan_query(B * H, n, d, dv, chunk, segments, tile, first_tiles, tiles_per_segment))
    return fail(HLA_ERR_UNSUPPORTED, "the fused path does not cover d=%d dv=%d chunk=%d", d, dv, chunk);
  return ok();
}

size_t hla2_forward_decay_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype) {
  if (check_dims(B, H, n, d, dv, chunk, dtype, true) != HLA_OK) return 0;
  if (chunk == 0) { fail(HLA_ERR_INVALID, "chunk must be set"); return 0; }
  // the larger of the two paths: the masked flag is not an argument here
  const size_t fused = hla::fused_decay_supported(n, d, dv, chunk, dtype, 1)
                           ? hla::fused_workspace_bytes(B * H, n, d, dv, chunk) : 0;
  const size_t chunked = chunked_ws(B * H, n, d, dv, chunk);
  return fused > chunked ? fused : chunked;
}

int hla2_forward_decay(const void* q, const void* k, const void* v, float* out, int B, int H, int n, int d, int dv,
                       int chunk, int masked, int normalized, float eps, float gamma, int dtype, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int rc;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if ((rc = check_flags(masked, normalized, eps)) != HLA_OK) return rc;
  if (!std::isfinite(gamma) || gamma <= 0.f || gamma > 1.f)
    return fail(HLA_ERR_INVALID, "gamma must be finite with 0 < gamma <= 1 (got %g)", (double)gamma);
  // both paths walk tiles of min(chunk, 64) tokens and scale by gamma^(2 (a + 1)), a < tile: keep that a
  // normal number
  const int tile = chunk < 64 ? chunk : 64;
  if (2.0 * tile * std::log2((double)gamma) < -125.0)
    return fail(HLA_ERR_UNSUPPORTED, "gamma^(2*%d) underflows fp32 (gamma=%g chunk=%d)", tile, (double)gamma, chunk);
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v")) ||
      (rc = check_ptr(out, "out")))
    return rc;
  const int BH = B * H;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (hla::fused_decay_supported(n, d, dv, chunk, dtype, masked)) {
    // bf16, masked, d = dv in {64, 128}: the fused segment walk with decay
    const size_t need = hla::fused_workspace_bytes(BH, n, d, dv, chunk);
    if (!workspace || workspace_bytes < need)
      return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
    hla::Fwd f{q, k, v, out, BH, n, d, dv, chunk, masked, normalized, dtype, eps, gamma};
    const hipError_t e = hla::launch_fused(f, nullptr, nullptr, workspace, s);
    if (e != hipSuccess) return hip_fail(e, "decayed fused forward");
    return ok();
  }
  const size_t need = chunked_ws(BH, n, d, dv, chunk);
  if (!workspace || workspace_bytes < need)
    return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  const int cc = path_chunk(chunk);
  hla::Fwd f{q, k, v, out, BH, n, d, dv, cc, masked, normalized, dtype, eps, gamma};
  const int M = (n + cc - 1) / cc;
  const int last = n - (M - 1) * cc;
  const float rho = (float)std::pow((double)gamma, (double)cc), rho_last = (float)std::pow((double)gamma, (double)last);
  float* states = static_cast<float*>(workspace);
  float* prefix = reinterpret_cast<float*>(static_cast<char*>(workspace) + need / 2);
  hipError_t e = HLA_PROF("chunk_summary", s,
                          hla::launch_chunk_summaries(q, k, v, states, BH, n, d, dv, cc, dtype, s, gamma));
  if (e != hipSuccess) return hip_fail(e, "chunk summaries");
  e = HLA_PROF("scan", s, hla::launch_scan(states, nullptr, prefix, nullptr, BH, M, d, dv, s, rho, rho_last));
  if (e != hipSuccess) return hip_fail(e, "scan");
  e = HLA_PROF("readout", s, hla::launch_readout(f, prefix, s));
  if (e != hipSuccess) return hip_fail(e, "readout");
  return ok();
}

size_t hla2_backward_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype) {
  if (check_dims(B, H, n, d, dv, chunk, dtype, true) != HLA_OK) return 0;
  if (!hla::backward_supported(n, d, dv, dtype)) {
    fail(HLA_ERR_UNSUPPORTED, "the backward covers bf16 q/k/v with d = dv in {64, 128} (got d=%d dv=%d dtype=%d)", d,
         dv, dtype);
    return 0;
  }
  return hla::backward_workspace_bytes(B * H, n, d);
}

int hla2_backward(const void* q, const void* k, const void* v, const float* g, float* dq, float* dk, float* dv,
                  int B, int H, int n, int d, int dv_dim, int chunk, int dtype, void* workspace,
                  size_t workspace_bytes, void* stream) {
  int rc;
  if ((rc = check_dims(B, H, n, d, dv_dim, chunk, dtype, true)) != HLA_OK) return rc;
  if (!hla::backward_supported(n, d, dv_dim, dtype))
    return fail(HLA_ERR_UNSUPPORTED, "the backward covers bf16 q/k/v with d = dv in {64, 128} (got d=%d dv=%d dtype=%d)",
                d, dv_dim, dtype);
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v")) || (rc = check_ptr(g, "g")) ||
      (rc = check_ptr(dq, "dq")) || (rc = check_ptr(dk, "dk")) || (rc = check_ptr(dv, "dv")))
    return rc;
  const int BH = B * H;
  const size_t need = hla::backward_workspace_bytes(BH, n, d);
  if (!workspace || workspace_bytes < need)
    return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  hla::Bwd b{q, k, v, g, dq, dk, dv, BH, n, d, dv_dim, dtype};
  const hipError_t e = hla::launch_backward(b, workspace, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "backward");
  return ok();
}

size_t ahla_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype) {
  if (check_dims(B, H, n, d, dv, chunk, dtype, true) != HLA_OK) return 0;
  if (chunk == 0 || !hla::ahla_supported(n, d, dv, chunk, dtype)) {
    fail(HLA_ERR_UNSUPPORTED, "AHLA covers bf16, d = dv in {64, 128}, chunk in {64, 128} (got d=%d dv=%d chunk=%d "
         "dtype=%d)", d, dv, chunk, dtype);
    return 0;
  }
  return hla::ahla_workspace_bytes(B * H, n, d);
}

int ahla_forward(const void* q, const void* k, const void* v, float* out, int B, int H, int n, int d, int dv,
                 int chunk, int normalized, float eps, int dtype, void* workspace, size_t workspace_bytes,
                 void* stream) {
  int rc;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if ((rc = check_flags(1, normalized, eps)) != HLA_OK) return rc;
  if (!hla::ahla_supported(n, d, dv, chunk, dtype))
    return fail(HLA_ERR_UNSUPPORTED, "AHLA covers bf16, d = dv in {64, 128}, chunk in {64, 128} "
                "(got d=%d dv=%d chunk=%d dtype=%d)", d, dv, chunk, dtype);
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v")) ||
      (rc = check_ptr(out, "out")))
    return rc;
  const int BH = B * H;
  const size_t need = hla::ahla_workspace_bytes(BH, n, d);
  if (!workspace || workspace_bytes < need)
    return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  hla::Fwd f{q, k, v, out, BH, n, d, dv, chunk, 1, normalized, dtype, eps};
  const hipError_t e = hla::launch_ahla(f, workspace, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "ahla forward");
  return ok();
}

int hla2_chunk_summaries(const void* q, const void* k, const void* v, float* states, int B, int H, int n, int d,
                         int dv, int chunk, int dtype, void* stream) {
  int rc;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v")) ||
      (rc = check_ptr(states, "states")))
    return rc;
  hipError_t e = hla::launch_chunk_summaries(q, k, v, states, B * H, n, d, dv, chunk, dtype,
                                             reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "chunk summaries");
  return ok();
}

int hla2_scan(const float* states, const float* init, float* prefix, float* total, int B, int H, int M, int d,
              int dv, void* stream) {
  int rc;
  if ((rc = check_dims(B, H, 1, d, dv, 0, HLA_FP32, false)) != HLA_OK) return rc;
  if (M < 1) return fail(HLA_ERR_INVALID, "M must be >= 1 (got %d)", M);
  if ((rc = check_ptr(states, "states")) || (rc = check_ptr(prefix, "prefix"))) return rc;
  if (init && !aligned16(init)) return fail(HLA_ERR_INVALID, "init is not 16-byte aligned");
  if (total && !aligned16(total)) return fail(HLA_ERR_INVALID, "total is not 16-byte aligned");
  hipError_t e = hla::launch_scan(states, init, prefix, total, B * H, M, d, dv, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "scan");
  return ok();
}

// ---------------------------------------------------------------------------
// Decode state descriptor.  The check word hashes every other field, so a
// descriptor edited after hla2_state_init (a flag flipped between a prefill
// and a step, say) is rejected.
static unsigned long long state_check(const hla2_state* st) {
  unsigned long long h = 1469598103934665603ull;
  auto mix = [&](unsigned long long x) {
    for (int b = 0; b < 8; ++b) {
      h ^= (x >> (8 * b)) & 0xffu;
      h *= 1099511628211ull;
    }
  };
  uint32_t eb;
  std::memcpy(&eb, &st->eps, 4);
  mix((unsigned long long)st->B); mix((unsigned long long)st->H); mix((unsigned long long)st->d);
  mix((unsigned long long)st->dv); mix((unsigned long long)st->masked); mix((unsigned long long)st->normalized);
  mix((unsigned long long)st->dtype); mix(eb); mix((unsigned long long)(uintptr_t)st->data);
  mix((unsigned long long)st->head_floats);
  const float* f[5] = {st->S, st->C, st->m, st->G, st->h};
  for (const float* p : f) mix((unsigned long long)(uintptr_t)p);
  return h ^ 0x484c4132u;     // "HLA2"
}

static int check_state(const hla2_state* st) {
  if (!st) return fail(HLA_ERR_INVALID, "state descriptor is NULL");
  if (st->check != state_check(st))
    return fail(HLA_ERR_INVALID, "state descriptor was not set by hla2_state_init or has changed since");
  return HLA_OK;
}

size_t hla2_state_bytes(int B, int H, int d, int dv) {
  if (check_dims(B, H, 1, d, dv, 0, HLA_FP32, false) != HLA_OK) return 0;
  return sizeof(float) * (size_t)B * H * hla::dstate_floats(d, dv);
}

int hla2_state_init(hla2_state* st, void* buf, size_t buf_bytes, int B, int H, int d, int dv, int masked,
                    int normalized, float eps, int dtype, void* stream) {
  int rc;
  if (!st) return fail(HLA_ERR_INVALID, "state descriptor is NULL");
  if ((rc = check_dims(B, H, 1, d, dv, 0, dtype, false)) != HLA_OK) return rc;
  if ((rc = check_flags(masked, normalized, eps)) != HLA_OK) return rc;
  if ((rc = check_ptr(buf, "buf")) != HLA_OK) return rc;
  const size_t need = hla2_state_bytes(B, H, d, dv);
  if (buf_bytes < need) return fail(HLA_ERR_INVALID, "state buffer of %zu bytes needed, %zu given", need, buf_bytes);
  hla2_state s{};
  s.B = B; s.H = H; s.d = d; s.dv = dv;
  s.masked = masked; s.normalized = normalized; s.dtype = dtype; s.eps = eps;
  s.data = static_cast<float*>(buf);
  s.head_floats = hla::dstate_floats(d, dv);
  s.S = s.data;
  s.C = s.S + hla::packed_s_floats(d);
  s.m = s.C + (size_t)d * dv;
  s.G = s.m + d;
  s.h = s.G + (size_t)d * dv;
  s.check = state_check(&s);
  const hipError_t e = hla::launch_zero(s.data, need / 16, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "state zeroing");
  *st = s;
  return ok();
}

static size_t prefill_ws(int BH, int n, int d, int dv, int chunk) {
  const size_t a = chunked_ws(BH, n, d, dv, chunk);
  const size_t b = align256(hla::fused_workspace_bytes(BH, n, d, dv, chunk));
  return (a > b ? a : b) + 2 * align256(sizeof(float) * (size_t)BH * hla::state_floats(d, dv));
}

size_t hla2_prefill_workspace_bytes(const hla2_state* st, int n, int chunk) {
  if (check_state(st) != HLA_OK) return 0;
  if (check_dims(st->B, st->H, n, st->d, st->dv, chunk, st->dtype, true) != HLA_OK) return 0;
  if (chunk == 0) { fail(HLA_ERR_INVALID, "chunk must be set"); return 0; }
  return prefill_ws(st->B * st->H, n, st->d, st->dv, chunk);
}

int hla2_prefill(hla2_state* st, const void* q, const void* k, const void* v, int n, int chunk, float* out,
                 void* workspace, size_t workspace_bytes, void* stream) {
  int rc;
  if ((rc = check_state(st)) != HLA_OK) return rc;
  const int B = st->B, H = st->H, d = st->d, dv = st->dv, dtype = st->dtype;
  const int masked = st->masked, normalized = st->normalized;
  const float eps = st->eps;
  float* state = st->data;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v"))) return rc;
  if (out && !aligned16(out)) return fail(HLA_ERR_INVALID, "out is not 16-byte aligned");
  const int BH = B * H;
  const size_t cws = chunked_ws(BH, n, d, dv, chunk);
  const size_t fws = align256(hla::fused_workspace_bytes(BH, n, d, dv, chunk));
  const size_t need = prefill_ws(BH, n, d, dv, chunk);
  if (!workspace || workspace_bytes < need)
    return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(workspace);
  float* states = reinterpret_cast<float*>(base);
  float* prefix = reinterpret_cast<float*>(base + cws / 2);
  char* tail = base + (cws > fws ? cws : fws);
  float* total = reinterpret_cast<float*>(tail);
  float* init = reinterpret_cast<float*>(tail + align256(sizeof(float) * (size_t)BH * hla::state_floats(d, dv)));
  // the state's packed records to full ones, the forward from them, the new
  // total packed back into the state
  hipError_t e = hla::launch_state_unpack(state, init, BH, d, dv, s);
  if (e != hipSuccess) return hip_fail(e, "state unpack");
  if (hla::fused_supported(n, d, dv, chunk, dtype, out ? masked : 1)) {
    hla::Fwd f{q, k, v, out, BH, n, d, dv, chunk, masked, normalized, dtype, eps};
    e = hla::launch_fused(f, init, total, workspace, s);
    if (e != hipSuccess) return hip_fail(e, "fused prefill");
  } else {
    const int cc = path_chunk(chunk), Mc = (n + cc - 1) / cc;
    e = hla::launch_chunk_summaries(q, k, v, states, BH, n, d, dv, cc, dtype, s);
    if (e != hipSuccess) return hip_fail(e, "chunk summaries");
    e = hla::launch_scan(states, init, prefix, total, BH, Mc, d, dv, s);
    if (e != hipSuccess) return hip_fail(e, "scan");
    if (out) {
      hla::Fwd f{q, k, v, out, BH, n, d, dv, cc, masked, normalized, dtype, eps};
      e = hla::launch_readout(f, prefix, s);
      if (e != hipSuccess) return hip_fail(e, "readout");
    }
  }
  e = hla::launch_state_pack(total, state, BH, d, dv, s);
  if (e != hipSuccess) return hip_fail(e, "state pack");
  return ok();
}

int hla2_state_export(const hla2_state* st, float* full, void* stream) {
  int rc;
  if ((rc = check_state(st)) != HLA_OK) return rc;
  if ((rc = check_ptr(full, "full")) != HLA_OK) return rc;
  const hipError_t e = hla::launch_state_unpack(st->data, full, st->B * st->H, st->d, st->dv,
                                                reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "state export");
  return ok();
}

int hla2_step(hla2_state* st, const void* q_t, const void* k_t, const void* v_t, float* out_t, void* stream) {
  int rc;
  if ((rc = check_state(st)) != HLA_OK) return rc;
  if ((rc = check_ptr(q_t, "q_t")) || (rc = check_ptr(k_t, "k_t")) || (rc = check_ptr(v_t, "v_t")) ||
      (rc = check_ptr(out_t, "out_t")))
    return rc;
  hipError_t e = hla::launch_step(st->data, q_t, k_t, v_t, out_t, st->B * st->H, st->d, st->dv, st->masked,
                                  st->normalized, st->eps, st->dtype, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "step");
  return ok();
}

size_t hla3_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype) {
  if (check_dims(B, H, n, d, dv, chunk, dtype, true) != HLA_OK) return 0;
  if (chunk == 0) { fail(HLA_ERR_INVALID, "chunk must be set"); return 0; }
  if (!hla::hla3_supported(d, dv, chunk, 1)) {
    fail(HLA_ERR_UNSUPPORTED, "hla3_forward needs d, dv in {16, 32} (got d=%d dv=%d)", d, dv);
    return 0;
  }
  return hla::hla3_workspace(B * H, n, d, dv, chunk);
}

int hla3_forward(const void* q, const void* k, const void* v, float* out, int B, int H, int n, int d, int dv,
                 int chunk, int masked, int normalized, float eps, int dtype, void* workspace, size_t workspace_bytes,
                 void* stream) {
  int rc;
  if ((rc = check_dims(B, H, n, d, dv, chunk, dtype, true)) != HLA_OK) return rc;
  if (chunk == 0) return fail(HLA_ERR_INVALID, "chunk must be set");
  if ((rc = check_flags(masked, normalized, eps)) != HLA_OK) return rc;
  if ((rc = check_ptr(q, "q")) || (rc = check_ptr(k, "k")) || (rc = check_ptr(v, "v")) ||
      (rc = check_ptr(out, "out")))
    return rc;
  if (!hla::hla3_supported(d, dv, chunk, masked))
    return fail(HLA_ERR_UNSUPPORTED, "hla3_forward needs d, dv in {16, 32} (got masked=%d d=%d dv=%d)",
                masked, d, dv);
  const int BH = B * H;
  const size_t need = hla::hla3_workspace(BH, n, d, dv, chunk);
  if (!workspace || workspace_bytes < need)
    return fail(HLA_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  hla::Fwd f{q, k, v, out, BH, n, d, dv, chunk, masked, normalized, dtype, eps};
  hipError_t e = hla::launch_hla3(f, workspace, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hla3 forward");
  return ok();
}

}  // extern "C"
