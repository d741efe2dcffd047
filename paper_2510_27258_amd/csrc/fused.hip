// Fused masked second-order HLA forward for bf16 inputs on gfx950 MFMA.
//
// Algorithm (Sec. 4, two-level scan, Rem. scan-modes; Thm. 1 readout): the
// sequence of every head is cut into P segments of whole chunks, and the
// carries are kept as (S, Phi, eta) with Phi = S C - G and eta = S m - h (an
// exact change of variables of the 5-tuple).  In those variables Eq.
// (semidirect) reads Phi_{A(+)B} = Phi_A + Phi_B + S_A C_B: a segment's
// bracket Phi_s + S_{<s} C_s depends on the earlier segments only through
// the additive S prefix.  So
//   1. k_moments: S = K^T K of every segment;
//   2. k_walk_rs / k_walk<OUTPUT>: every segment walks its chunks from the
//      true S prefix with Phi0 = eta0 = 0, writes its outputs without the Phi
//      carry, and ends holding its bracket (Phi0, eta0), which it writes to
//      its record;
//   3. k_carry / k_fix: running sums of the brackets are the carries;
//      out_t += q_t^T Phi_c (and the division when normalised).
// With an initial state, k_init_convert converts it to the (S, C, m, Phi, eta)
// form first; k_total sums all records into the final state when a caller
// asks for it.  k_moments, k_carry and k_fix live in fused_tiles.h.
// At d = dv = 128 without states the forward takes the two-pass plan of
// fused_ws.h instead (run_ws): segment 0's output walk beside the summary
// walks of the later segments, the brackets, then the other segments' output
// walks from their true carries, so that every output row is written once.
//
// Per chunk (tokens of the chunk as the rows of Q, K, V; S0, Phi0, eta0 the
// carry of the chunk), with r_j = S_j q_j (the proof of Thm. 1 sums
// S_j q_j v_j^T):
//   W   = L (.) Q K^T                      (C x C, diagonal included)
//   R   = W K + Q S0                        (C x D, row j is r_j)
//   T   = L (.) Q R^T                       (C x C)
//   O   = T V + Q Phi0,   den = T 1 + Q eta0          (Thm. 1)
//   Phi0 += R^T V,  eta0 += R^T 1,  S0 += K^T K       (carry advance)
// This is Thm. 1 on the inclusive state (carry) (+) (local prefix): o_t =
// q_t^T Phi_t with Phi_t = sum_{j<=t} S_j q_j v_j^T.
//
// Numerics: q, k, v are exact in bf16.  Every computed operand that feeds an
// MFMA (W, R, T, S0, Phi0) is split as x = hi + lo with hi = bf16(x) and
// lo = bf16(x - hi); the product with an exact bf16 partner is taken as two
// MFMAs, so the operand keeps ~16 significant bits.  Accumulation is fp32.
//
// Layout: 256 threads = 4 waves on v_mfma_f32_32x32x16_bf16; a chunk has at
// most 2 row tiles of 32 tokens.  With d, dv <= 64 wave w owns output tile
// (row w/2, column w%2); with d or dv = 128 wave w owns column tile w over
// all row tiles.  The wave owning column c of R (or O) keeps the whole column
// c of S0 (or Phi0) in MFMA accumulators for the whole walk and feeds it back
// as the B operand straight from registers (with two row waves per column
// both keep a copy).  Q, K, K^T, V^T, W/T, R and R^T are staged in LDS as
// bf16.
#include <cmath>

#include "fused.h"
#include "fused_tiles.h"
#include "fused_ws.h"
#include "profile.h"

namespace hla {
namespace {

template <int C, int D, int DV, bool SUMMARY>
struct Cfg {
  // Q, K, V row-major (the transposed operands are read through the LDS
  // transpose unit).  Two reused buffers: B1 holds W, then R^T (after a
  // barrier); B2 holds T.  SUMMARY walks use only B1.
  static constexpr int CD = C > D ? C : D;
  static constexpr int ldQ = D + kPad, ldK = D + kPad, ldV = DV + kPad;
  static constexpr int ld1 = C + kPad, ld2 = CD + kPad, ldQt = C + kPad;
  static constexpr int ldW = ld1, ldRt = ld1, ldT = ld2;
  static constexpr int oQ = 0;
  static constexpr int oK = oQ + C * ldQ;
  static constexpr int oVt = oK + C * ldK;                       // V
  static constexpr int oB1h = oVt + C * ldV;
  static constexpr int oB1l = oB1h + CD * ld1;
  static constexpr int oB2h = oB1l + CD * ld1;
  static constexpr int oB2l = oB2h + (SUMMARY ? 0 : C * ld2);
  static constexpr int oQt = oB2l + (SUMMARY ? 0 : C * ld2);
  // bf16 elements of the tile region; at least D*D floats, where the walk's
  // prologue stages the S carry before the first tile
  static constexpr int n16 = oQt > 2 * D * D ? oQt : 2 * D * D;
  static constexpr int RT = C / 32, DT = D / 32, VT = DV / 32;       // 32-wide tiles
  static constexpr int KC = C / 16, KD = D / 16;                     // 16-deep k steps
  // Wave w owns column tile ct = w % NCT of R, O, S0 and Phi0 and the row
  // tiles rg, rg + NRG, ... (rg = w / NCT).  With four column tiles (d = 128)
  // every wave covers all row tiles and no state column is held twice.
  static constexpr int NCT = (DT > 2 || VT > 2) ? 4 : 2;
  static constexpr int NRG = kWaves / NCT;
  static constexpr int RPW = (RT + NRG - 1) / NRG;                   // row tiles per wave
  static constexpr int f_eta = 0, f_cs = D, f_den = D + RT * D, f_denp = f_den + C;   // fp32 region
  static constexpr int nf32 = f_denp + RT * C;
  static constexpr size_t bytes = (size_t)((n16 + 7) & ~7) * 2 + (size_t)nf32 * 4;
  // workgroups per CU: two when LDS allows and the state columns (d, dv <= 64) leave
  // registers for a second workgroup
  static constexpr int kBlocks = (2 * bytes <= 160 * 1024 && NCT == 2) ? 2 : 1;
  // global->LDS staging: 16-byte segments per operand
  static constexpr int segQ = C * D / 8, segV = C * DV / 8;
  static constexpr int pfQ = (segQ + kThreads - 1) / kThreads, pfV = (segV + kThreads - 1) / kThreads;
  static_assert(C % 32 == 0 && D % 32 == 0 && DV % 32 == 0 && C <= 64 && D <= 128 && DV <= 128, "tile shape");
  static_assert(DT <= NCT && VT <= NCT && RT <= 2, "wave layout");
  static_assert(bytes <= 160 * 1024, "LDS budget");
};

// Records: [BH][nseg + 1][F] in the S|C|m|G|h layout with Phi in the G slot
// and eta in the h slot.  Slot s < nseg: the segment's moments (S; C and m
// when a final state is wanted) and, after its walk, its bracket.  Slot nseg
// holds the initial state converted to this form (written only when there is
// one).  Carries and the total are plain sums of these records (the Phi form
// of Eq. (semidirect)); the total is converted back to G, h once (k_total).

// out[a][b] = z * Z[a][b] + sum_a' X[a][a'] Y[a'][b] for the thread's TI x TI
// register blocks; XT = X^T ([D][D+4]) and Y ([D][DV]) in LDS, Z and out in
// global memory with row stride DV (out may alias Z).
template <int D, int DV>
__device__ __forceinline__ void xy_plus(const float* XT, const float* Y, const float* Z, float z, float* out) {
  constexpr int TI = (D >= 128 || DV >= 128) ? 8 : 4, ldT = D + 4;
  constexpr int NBJ = DV / TI, NB = (D / TI) * NBJ;
  for (int blk = threadIdx.x; blk < NB; blk += blockDim.x) {
    const int a0 = TI * (blk / NBJ), b0 = TI * (blk % NBJ);
    float o[TI][TI] = {};
#pragma unroll 4
    for (int ap = 0; ap < D; ++ap) {
      float xv[TI], yv[TI];
#pragma unroll
      for (int i = 0; i < TI; i += 4) {
        const float4 x4 = *reinterpret_cast<const float4*>(&XT[ap * ldT + a0 + i]);
        const float4 y4 = *reinterpret_cast<const float4*>(&Y[ap * DV + b0 + i]);
        xv[i] = x4.x; xv[i + 1] = x4.y; xv[i + 2] = x4.z; xv[i + 3] = x4.w;
        yv[i] = y4.x; yv[i + 1] = y4.y; yv[i + 2] = y4.z; yv[i + 3] = y4.w;
      }
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TI; ++j) o[i][j] += xv[i] * yv[j];
    }
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TI; j += 4) {
        const size_t off = (size_t)(a0 + i) * DV + b0 + j;
        const float4 z4 = *reinterpret_cast<const float4*>(Z + off);
        *reinterpret_cast<float4*>(out + off) =
            make_float4(o[i][j] + z * z4.x, o[i][j + 1] + z * z4.y, o[i][j + 2] + z * z4.z, o[i][j + 3] + z * z4.w);
      }
  }
}

// out[a] = z * zv[a] + sum_a' X[a][a'] y[a'] for a = threadIdx.x < D.
template <int D>
__device__ __forceinline__ void xv_plus(const float* XT, const float* y, const float* zv, float z, float* out) {
  const int a = threadIdx.x;
  if (a >= D) return;
  float acc = 0.f;
#pragma unroll 8
  for (int ap = 0; ap < D; ++ap) acc += XT[ap * (D + 4) + a] * y[ap];
  out[a] = acc + z * zv[a];
}

// Stage X^T (X from float4 registers, row-major [D][D] split as element
// 4 * (tid + 256 r)), Y ([D][DV] float4 registers) and y into LDS.
template <int D, int DV>
__device__ __forceinline__ void stage_xy(float* XT, float* Y, float* y, const float4* xs, const float4* ys, float yv) {
  constexpr int nS4 = D * D / 4 / 256, nC4 = D * DV / 4 / 256, ldT = D + 4;
  const int tid = threadIdx.x;
#pragma unroll
  for (int r = 0; r < nS4; ++r) {
    const int e4 = tid + 256 * r, a = (4 * e4) / D, ap = (4 * e4) % D;
    XT[(ap + 0) * ldT + a] = xs[r].x;
    XT[(ap + 1) * ldT + a] = xs[r].y;
    XT[(ap + 2) * ldT + a] = xs[r].z;
    XT[(ap + 3) * ldT + a] = xs[r].w;
  }
#pragma unroll
  for (int r = 0; r < nC4; ++r) reinterpret_cast<float4*>(Y)[tid + 256 * r] = ys[r];
  if (tid < D) y[tid] = yv;
}

__device__ __forceinline__ void add4(float4& a, const float4& b) {
  a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
}

// k_init_convert: grid (1, BH), 256 threads.  Writes the initial state of
// every head into slot nseg of its records in the (S, C, m, Phi, eta) form:
// (S, C, m, S C - G, S m - h).
template <int D, int DV>
__global__ __launch_bounds__(256) void k_init_convert(float* __restrict__ segs, const float* __restrict__ init,
                                                      int nseg) {
  constexpr int nS4 = D * D / 4 / 256, nC4 = D * DV / 4 / 256;
  static_assert(D * D % 1024 == 0 && D * DV % 1024 == 0, "thread split");
  extern __shared__ float sm[];
  float* XT = sm;                 // [D][D+4]  S^T
  float* Y = XT + D * (D + 4);    // [D][DV]   C
  float* y = Y + D * DV;          // [D]       m
  const int bh = blockIdx.y, tid = threadIdx.x;
  const size_t F = state_floats(D, DV);
  const float* src = init + (size_t)bh * F;
  float* dst = segs + ((size_t)bh * (nseg + 1) + nseg) * F;
  float4 xs[nS4], ys[nC4];
#pragma unroll
  for (int r = 0; r < nS4; ++r) xs[r] = reinterpret_cast<const float4*>(src)[tid + 256 * r];
#pragma unroll
  for (int r = 0; r < nC4; ++r) ys[r] = reinterpret_cast<const float4*>(src + off_C(D, DV))[tid + 256 * r];
  const float yv = tid < D ? src[off_m(D, DV) + tid] : 0.f;
  stage_xy<D, DV>(XT, Y, y, xs, ys, yv);
#pragma unroll
  for (int r = 0; r < nS4; ++r) reinterpret_cast<float4*>(dst)[tid + 256 * r] = xs[r];
#pragma unroll
  for (int r = 0; r < nC4; ++r) reinterpret_cast<float4*>(dst + off_C(D, DV))[tid + 256 * r] = ys[r];
  if (tid < D) dst[off_m(D, DV) + tid] = yv;
  __syncthreads();
  xy_plus<D, DV>(XT, Y, src + off_G(D, DV), -1.f, dst + off_G(D, DV));
  xv_plus<D>(XT, y, src + off_h(D, DV), -1.f, dst + off_h(D, DV));
}

// k_total: grid (BH), 256 threads.  The state after all nsum segments in the
// S|C|m|G|h form: S, C, m, Phi, eta are sums over the converted initial state
// and the brackets; then G = S C - Phi and h = S m - eta.
template <int D, int DV>
__global__ __launch_bounds__(256) void k_total(const float* __restrict__ segs, const float* __restrict__ init,
                                               float* __restrict__ fin, int nseg, int nsum) {
  constexpr int nS4 = D * D / 4 / 256, nC4 = D * DV / 4 / 256, ldT = D + 4;
  extern __shared__ float sm[];
  float* XT = sm;
  float* Y = XT + D * ldT;
  float* y = Y + D * DV;
  const int bh = blockIdx.x, tid = threadIdx.x;
  const size_t F = state_floats(D, DV);
  const float* base = segs + (size_t)bh * (nseg + 1) * F;
  float* out = fin + (size_t)bh * F;
  float4 xs[nS4], ys[nC4];
  float yv = 0.f, ev = 0.f;
  const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int r = 0; r < nS4; ++r) xs[r] = z4;
#pragma unroll
  for (int r = 0; r < nC4; ++r) ys[r] = z4;
  for (int sp = init ? -1 : 0; sp < nsum; ++sp) {
    const float* x = base + (size_t)(sp < 0 ? nseg : sp) * F;
#pragma unroll
    for (int r = 0; r < nS4; ++r) add4(xs[r], reinterpret_cast<const float4*>(x)[tid + 256 * r]);
#pragma unroll
    for (int r = 0; r < nC4; ++r) add4(ys[r], reinterpret_cast<const float4*>(x + off_C(D, DV))[tid + 256 * r]);
    if (tid < D) {
      yv += x[off_m(D, DV) + tid];
      ev += x[off_h(D, DV) + tid];
    }
  }
  stage_xy<D, DV>(XT, Y, y, xs, ys, yv);
#pragma unroll
  for (int r = 0; r < nS4; ++r) reinterpret_cast<float4*>(out)[tid + 256 * r] = xs[r];
#pragma unroll
  for (int r = 0; r < nC4; ++r) reinterpret_cast<float4*>(out + off_C(D, DV))[tid + 256 * r] = ys[r];
  if (tid < D) {
    out[off_m(D, DV) + tid] = yv;
    out[off_h(D, DV) + tid] = ev;      // eta, replaced by h below
  }
  // Phi sum into the G slot of the output, then G = S C - Phi in place
  float* Gout = out + off_G(D, DV);
  for (int e4 = tid; e4 < D * DV / 4; e4 += 256) {
    float4 acc = z4;
    for (int sp = init ? -1 : 0; sp < nsum; ++sp)
      add4(acc, reinterpret_cast<const float4*>(base + (size_t)(sp < 0 ? nseg : sp) * F + off_G(D, DV))[e4]);
    reinterpret_cast<float4*>(Gout)[e4] = acc;
  }
  __syncthreads();
  xy_plus<D, DV>(XT, Y, Gout, -1.f, Gout);
  xv_plus<D>(XT, y, out + off_h(D, DV), -1.f, out + off_h(D, DV));
}


// One segment walk.  grid = (segments, BH), 4 waves.  Wave w owns column tile
// ct = w % NCT of R and of O and keeps column ct of S0 and of Phi0 (all their
// rows) in accumulators; it works on the row tiles rg, rg + NRG, ...
// The walk starts from S0 = the S prefix before the segment (the moments of
// the converted initial state and of the earlier segments) and Phi0 = eta0 = 0,
// and ends by writing the segment's bracket (its Phi0, eta0) into the Phi/eta
// slots of its record.  !SUMMARY also writes num (without the Phi carry of
// earlier segments) to out and, when normalised, den to den_out; k_fix adds
// the carry and divides.  SUMMARY skips T and O.
template <int C, int D, int DV, bool SUMMARY>
__global__ __launch_bounds__(kThreads, (Cfg<C, D, DV, SUMMARY>::kBlocks)) void k_walk(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, float* __restrict__ rec, const float* __restrict__ spre,
    int n, int cps, int nseg, int normalized, float eps, float lg2g) {
  using G = Cfg<C, D, DV, SUMMARY>;
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* Qs = lds + G::oQ;
  uint16_t* Ks = lds + G::oK;
  uint16_t* Vs = lds + G::oVt;    // V row-major
  uint16_t* Wh = lds + G::oB1h;   // W, then R^T
  uint16_t* Wl = lds + G::oB1l;
  uint16_t* Rth = Wh;
  uint16_t* Rtl = Wl;
  uint16_t* Th = lds + G::oB2h;   // T
  uint16_t* Tl = lds + G::oB2l;
  float* fl = reinterpret_cast<float*>(lds + ((G::n16 + 7) & ~7));
  float* eta = fl + G::f_eta;
  float* colsum = fl + G::f_cs;       // [RT][D]
  float* denp = fl + G::f_denp;       // [RT][C]

  int seg, bh;
  seg_head(seg, bh);
  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: per-wave branches stay scalar
  const int ct = w % G::NCT, rg = G::NRG == 1 ? 0 : w / G::NCT;
  // owns R column tile ct and S0 column ct / O column tile ct and Phi0 column ct
  const bool has_r = (G::DT == G::NCT || ct < G::DT) && (G::NRG == 1 || rg < G::RT);
  const bool has_o = (G::VT == G::NCT || ct < G::VT) && (G::NRG == 1 || rg < G::RT);
  const bool upd_p = SUMMARY ? (has_o && rg == 0) : has_o;
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t F = state_floats(D, DV);
  float* rc = rec + ((size_t)bh * (nseg + 1) + seg) * F;
  const rsrc_t ro = make_rsrc(SUMMARY ? nullptr : out + (size_t)bh * n * DV, SUMMARY ? 0u : (uint32_t)n * DV * 4);

  // ---- carry in (fp32 accumulators, column ct, all rows) ----
  f32x16 S0[G::DT], P0[G::DT];
#pragma unroll
  for (int i = 0; i < G::DT; ++i) {
    S0[i] = zero16();
    P0[i] = zero16();
  }
  for (int a = tid; a < D; a += kThreads) eta[a] = 0.f;
  if (spre) {
    // S0 = the S prefix of this segment (the converted initial state and the
    // earlier segments), staged through the (still free) tile region of LDS;
    // every wave picks up its columns
    constexpr int nS4 = D * D / 4 / kThreads;
    static_assert(D * D % (4 * kThreads) == 0 && D * D * 4 <= G::n16 * 2, "carry staging");
    const float4* x = reinterpret_cast<const float4*>(spre + ((size_t)bh * nseg + seg) * D * D);
    float4 sa[nS4];
#pragma unroll
    for (int r = 0; r < nS4; ++r) sa[r] = x[tid + kThreads * r];
    float* st = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int r = 0; r < nS4; ++r) reinterpret_cast<float4*>(st)[tid + kThreads * r] = sa[r];
    __syncthreads();
    if (has_r)
#pragma unroll
      for (int i = 0; i < G::DT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) S0[i][e] = st[(i * 32 + acc_row(e, lg)) * D + ct * 32 + lr];
    __syncthreads();
  }

  // ---- prefetch registers for the next chunk (buffer loads: the tail past n reads zero) ----
  const rsrc_t rq = make_rsrc(q + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rk = make_rsrc(k + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rv = make_rsrc(v + (size_t)bh * n * DV, (uint32_t)n * DV * 2);
  uint4 pq[G::pfQ], pk[G::pfQ], pv[G::pfV];
  auto fetch = [&](int c) {
    const uint32_t t0 = (uint32_t)c * C;
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + kThreads * i;        // consecutive lanes take consecutive pieces of a token row
      if (G::segQ % kThreads == 0 || e < G::segQ) {
        const uint32_t off = ((t0 + e / (D / 8)) * D + (e % (D / 8)) * 8) * 2;
        pq[i] = buf_load16(rq, off);
        pk[i] = buf_load16(rk, off);
      }
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + kThreads * i;
      if (G::segV % kThreads == 0 || e < G::segV) pv[i] = buf_load16(rv, ((t0 + e / (DV / 8)) * DV + (e % (DV / 8)) * 8) * 2);
    }
  };
  if (c_begin < c_end) fetch(c_begin);

  for (int c = c_begin; c < c_end; ++c) {
    const int t0 = c * C;
    // ---- stage 0: registers -> LDS (Q, K, V row-major) ----
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + kThreads * i;
      if (e < G::segQ) {
        const int t = e / (D / 8), a8 = (e % (D / 8)) * 8;
        *reinterpret_cast<uint4*>(Qs + t * G::ldQ + a8) = pq[i];
        *reinterpret_cast<uint4*>(Ks + t * G::ldK + a8) = pk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + kThreads * i;
      if (e < G::segV) {
        const int t = e / (DV / 8), b8 = (e % (DV / 8)) * 8;
        *reinterpret_cast<uint4*>(Vs + t * G::ldV + b8) = pv[i];
      }
    }
    lds_barrier();
    if (c + 1 < c_end) fetch(c + 1);

    // ---- stage 1: W = L (.) Q K^T, computed as W^T = K Q^T and stored transposed ----
    {
      const int it = w >> 1, jt = w & 1;       // key tile, query tile
      if (it < G::RT && jt < G::RT) {
        f32x16 acc = zero16();
        if (it <= jt) {
#pragma unroll
          for (int s = 0; s < G::KD; ++s)
            acc = mfma(frag(Ks, G::ldK, it * 32, s * 16), frag(Qs, G::ldQ, jt * 32, s * 16), acc);
#pragma unroll
          for (int e = 0; e < 16; ++e)   // keep key i <= query t
            if (it * 32 + acc_row(e, lg) > jt * 32 + lr) acc[e] = 0.f;
        }
        store_T(acc, Wh, Wl, G::ldW, it * 32, jt * 32);
      }
    }
    lds_barrier();

    // ---- stage 2: R = W K + Q S0 (old S0) on column tile ct; S0 += K^T K on column ct ----
    f32x16 racc[G::RPW];
#pragma unroll
    for (int i = 0; i < G::RPW; ++i) racc[i] = zero16();
    if (has_r) {
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag_tr(Ks, G::ldK, ct * 32, s * 16);
#pragma unroll
        for (int i = 0; i < G::RPW; ++i) {
          const int rt = rg + G::NRG * i;
          if (rt < G::RT && s * 16 <= rt * 32 + 31) {     // keys past the row tile: W is zero
            racc[i] = mfma(frag(Wh, G::ldW, rt * 32, s * 16), bK, racc[i]);
            racc[i] = mfma(frag(Wl, G::ldW, rt * 32, s * 16), bK, racc[i]);
          }
        }
      }
#pragma unroll
      for (int s = 0; s < G::KD; ++s) {
        bf16x8 bh, bl;
        frag_from_acc(S0[s >> 1], s & 1, bh, bl);
#pragma unroll
        for (int i = 0; i < G::RPW; ++i) {
          const int rt = rg + G::NRG * i;
          if (rt < G::RT) {
            const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, rt * 32, s * 16);
            racc[i] = mfma(aQ, bh, racc[i]);
            racc[i] = mfma(aQ, bl, racc[i]);
          }
        }
      }
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag_tr(Ks, G::ldK, ct * 32, s * 16);
#pragma unroll
        for (int i = 0; i < G::DT; ++i) S0[i] = mfma(frag_tr(Ks, G::ldK, i * 32, s * 16), bK, S0[i]);
      }
      // eta advance: column sums of R over each row tile
#pragma unroll
      for (int i = 0; i < G::RPW; ++i) {
        const int rt = rg + G::NRG * i;
        if (rt < G::RT) {
          float cs = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) cs += racc[i][e];
          cs += __shfl_xor(cs, 32);
          if (lg == 0) colsum[rt * D + ct * 32 + lr] = cs;
        }
      }
    }
    lds_barrier();     // every wave is done reading W: B1 takes R^T
    if (has_r)
#pragma unroll
      for (int i = 0; i < G::RPW; ++i) {
        const int rt = rg + G::NRG * i;
        if (rt < G::RT) {
          store_T(racc[i], Rth, Rtl, G::ldRt, rt * 32, ct * 32);
        }
      }
    lds_barrier();
    float eta_add = 0.f;
    if (tid < D)
#pragma unroll
      for (int i = 0; i < G::RT; ++i) eta_add += colsum[i * D + tid];

    if (!SUMMARY) {
      // ---- stage 3: T = L (.) Q R^T, computed as T^T = R Q^T, stored transposed into the W buffers ----
      {
        const int it = w >> 1, jt = w & 1;     // j tile, t tile
        const bool tile = it < G::RT && jt < G::RT;
        f32x16 acc = zero16();
        if (tile && it <= jt) {
#pragma unroll
          for (int s = 0; s < G::KD; ++s) {
            const bf16x8 b = frag(Qs, G::ldQ, jt * 32, s * 16);
            acc = mfma(frag_tr(Rth, G::ldRt, it * 32, s * 16), b, acc);
            acc = mfma(frag_tr(Rtl, G::ldRt, it * 32, s * 16), b, acc);
          }
#pragma unroll
          for (int e = 0; e < 16; ++e)     // keep j <= t
            if (it * 32 + acc_row(e, lg) > jt * 32 + lr) acc[e] = 0.f;
        }
        if (tile) {
          float ps = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) ps += acc[e];
          ps += __shfl_xor(ps, 32);
          if (lg == 0) denp[it * C + jt * 32 + lr] = ps;
        }
        if (tile) store_T(acc, Th, Tl, G::ldT, it * 32, jt * 32);   // B2: the last tile's T readers are done
      }
      lds_barrier();
      // den_t = sum_j T[t][j] + q_t . eta0: the row sums here, and eta0 of this
      // tile (before its advance) for k_fix, which adds q_t . (eta0 + eta_c)
      if (normalized) {
        if (tid < C && t0 + tid < n) {
          float s = 0.f;
#pragma unroll
          for (int i = 0; i < G::RT; ++i) s += denp[i * C + tid];
          den_out[(size_t)bh * n + t0 + tid] = s;
        }
        if (tid < D) den_out[(size_t)gridDim.y * n + ((size_t)bh * ((n + C - 1) / C) + c) * D + tid] = eta[tid];
      }
      lds_barrier();
      // ---- stage 4: O = T V + Q Phi0 (old Phi0) on column tile ct; stage 5: Phi0 += R^T V ----
      if (has_o) {
        f32x16 oacc[G::RPW];
#pragma unroll
        for (int i = 0; i < G::RPW; ++i) oacc[i] = zero16();
#pragma unroll
        for (int s = 0; s < G::KC; ++s) {
          const bf16x8 bV = frag_tr(Vs, G::ldV, ct * 32, s * 16);
#pragma unroll
          for (int i = 0; i < G::RPW; ++i) {
            const int rt = rg + G::NRG * i;
            if (rt < G::RT && s * 16 <= rt * 32 + 31) {   // j past the row tile: T is zero
              oacc[i] = mfma(frag(Th, G::ldT, rt * 32, s * 16), bV, oacc[i]);
              oacc[i] = mfma(frag(Tl, G::ldT, rt * 32, s * 16), bV, oacc[i]);
            }
          }
        }
#pragma unroll
        for (int s = 0; s < G::KD; ++s) {
          bf16x8 bh, bl;
          frag_from_acc(P0[s >> 1], s & 1, bh, bl);
#pragma unroll
          for (int i = 0; i < G::RPW; ++i) {
            const int rt = rg + G::NRG * i;
            if (rt < G::RT) {
              const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, rt * 32, s * 16);
              oacc[i] = mfma(aQ, bh, oacc[i]);
              oacc[i] = mfma(aQ, bl, oacc[i]);
            }
          }
        }
#pragma unroll
        for (int i = 0; i < G::RPW; ++i) {
          const int rt = rg + G::NRG * i;
          if (rt < G::RT)
#pragma unroll
            for (int e = 0; e < 16; ++e) {      // rows past n fall outside the buffer and are dropped
              const int t = rt * 32 + acc_row(e, lg);
              buf_store4(ro, (((uint32_t)t0 + t) * DV + ct * 32 + lr) * 4, oacc[i][e]);
            }
        }
      }
    }
    if (upd_p) {
      // Phi0 += R^T V on column ct
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bV = frag_tr(Vs, G::ldV, ct * 32, s * 16);
#pragma unroll
        for (int i = 0; i < G::DT; ++i) {
          P0[i] = mfma(frag(Rth, G::ldRt, i * 32, s * 16), bV, P0[i]);
          P0[i] = mfma(frag(Rtl, G::ldRt, i * 32, s * 16), bV, P0[i]);
        }
      }
    }
    lds_barrier();   // LDS tiles and den/eta are rewritten by the next chunk
    if (tid < D) eta[tid] += eta_add;
  }

  // the segment's bracket: Phi0 into the G slot, eta0 into the h slot (the
  // opaque lane index keeps the store addresses out of the walk's live range)
  int col = ct * 32 + lr;
  asm volatile("" : "+v"(col));
  if (has_o && rg == 0)
#pragma unroll
    for (int i = 0; i < G::DT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) rc[off_G(D, DV) + (size_t)(i * 32 + acc_row(e, lg)) * DV + col] = P0[i][e];
  if (tid < D) rc[off_h(D, DV) + tid] = eta[tid];
}

// ---------------------------------------------------------------------------
// Row-split walk (C = 64, D = DV): 2 x NCT waves.  Wave (h, ct) keeps rows
// [h D/2, (h+1) D/2) of column tile ct of S0 and of Phi0, so every state
// element is held, advanced and split by exactly one wave.  R = W K + Q S0
// and O = T V + Q Phi0 contract over the state rows: each wave forms the
// partial over its half for both row tiles, hands the partial of the other
// row tile to its partner (h' = 1 - h, same ct) through LDS in fp32, and
// finishes row tile rt = h with the partner's half and the W K (or T V)
// term.  The exchange slots reuse K | K^T (for R; K is dead after the S0
// advance) and the R buffer (for O; R is dead after T).
template <int D, bool SUMMARY>
struct CfgRS {
  static constexpr int C = 64, DV = D;
  static constexpr int NCT = D / 32, NW = 2 * NCT, NT = 64 * NW;
  static constexpr int HT = NCT / 2, HALF = D / 2;             // 32-row state tiles per half
  static constexpr int RT = 2, KC = C / 16, KH = D / 32;        // k-steps over tokens / over a half
  static constexpr int ldQ = D + kPad, ldK = D + kPad, ldKt = C + kPad, ldV = DV + kPad;
  static constexpr int ld1 = C + kPad, ld2 = D + kPad, ldT = C + kPad;
  static constexpr int oQ = 0;
  static constexpr int oK = oQ + C * ldQ;
  static constexpr int oKt = oK + C * ldK;                     // (room for the R exchange and T)
  static constexpr int oVt = oKt + D * ldKt;                   // V, row-major
  static constexpr int oB1h = oVt + DV * (C + kPad);           // W, then R^T
  static constexpr int oB1l = oB1h + D * ld1;
  static constexpr int oB2h = oB1l + D * ld1;                  // the O exchange; absent in summaries
  static constexpr int oB2l = oB2h + C * ld2;
  static constexpr int n16 = SUMMARY ? oB2h : oB2l + C * ld2;
  static constexpr int oX = oK;                                // R exchange, then T (hi | lo)
  static constexpr int oTh = oK, oTl = oK + C * ldT;
  static constexpr int xfl = 2 * NCT * 1024;                   // exchange floats
  static_assert(2 * xfl <= oVt - oK && 2 * C * ldT <= oVt - oK, "exchange and T fit K | K^T");
  static_assert(SUMMARY || 2 * xfl <= 2 * C * ld2, "O exchange fits its buffer");
  static_assert(C * ldV <= DV * (C + kPad), "V fits its buffer");
  static constexpr int f_eta = 0, f_cs = D, f_den = D + RT * D, f_denp = f_den + C;
  static constexpr int f_tab = f_denp + RT * C;                // decay tables, 4 x C
  static constexpr int nf32 = f_tab + 4 * C;
  static constexpr size_t bytes = (size_t)((n16 + 7) & ~7) * 2 + (size_t)nf32 * 4;
  static constexpr int kBlocks = 2 * bytes <= 160 * 1024 && NW <= 4 ? 2 : 1;
  static constexpr int segQ = C * D / 8, pfQ = segQ / NT, pfV = C * DV / 8 / NT;
  static_assert(segQ % NT == 0 && pfQ >= 1 && (C * D / NT) == 16, "staging and den split");
  static_assert(D == 64 || D == 128, "row-split shapes");
  static_assert(bytes <= 160 * 1024, "LDS budget");
};

// Exchange slot of (column tile ct, row tile rt): 32 x 32 fp32 in MFMA
// accumulator order, element 4q + j of lane l at [(slot * 4 + q) * 64 + l] * 4 + j.
template <bool O = false>
__device__ __forceinline__ void xch_put(float* X, int slot, const f32x16& a, int l = lane64<O>()) {
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<float4*>(X + ((slot * 4 + q) * 64 + l) * 4) = make_float4(a[4 * q], a[4 * q + 1], a[4 * q + 2], a[4 * q + 3]);
}
template <bool O = false>
__device__ __forceinline__ void xch_add(const float* X, int slot, f32x16& a, int l = lane64<O>()) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 u = *reinterpret_cast<const float4*>(X + ((slot * 4 + q) * 64 + l) * 4);
    a[4 * q] += u.x; a[4 * q + 1] += u.y; a[4 * q + 2] += u.z; a[4 * q + 3] += u.w;
  }
}

//
// DEC: the decayed operator (decay gamma = 2^lg2g).  With a the token's index
// in its tile, S_j = gamma^(a_j+1) S0 + sum_{i<=j} gamma^(a_j-a_i) k_i k_i^T and
// Phi_t = gamma^(2(a_t+1)) Phi0 + sum_{j<=t} gamma^(2(a_t-a_j)) r_j v_j^T, so
//   R   = diag(gamma^(a+1)) Q S0 + (W (.) gamma^(a_j-a_i)) K,
//   O   = diag(gamma^(2(a+1))) Q Phi0 + (T (.) gamma^(2(a_t-a_j))) V,
//   S0 <- gamma^C S0 + K^T diag(gamma^(C-1-a)) K,
//   Phi0 <- gamma^(2C) Phi0 + R^T diag(gamma^(2(C-1-a))) V  (eta0 likewise),
// and the segment prefix of S weighs segment s' by gamma^(L (s-1-s')), L its
// length.  The token weights of the state advances go on the B fragment in
// registers (scaled in fp32, split hi/lo).  Every factor is at most 1.
template <int D, bool SUMMARY, bool DEC = false>
__global__ __launch_bounds__((CfgRS<D, SUMMARY>::NT), (CfgRS<D, SUMMARY>::kBlocks)) void k_walk_rs(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, float* __restrict__ rec, const float* __restrict__ spre,
    int n, int cps, int nseg, int normalized, float eps, float lg2g) {
  using G = CfgRS<D, SUMMARY>;
  constexpr bool kO = D == 128;     // at 512 threads the hoisted LDS addresses would spill
  constexpr int C = G::C, DV = G::DV, NT = G::NT;
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* Qs = lds + G::oQ;
  uint16_t* Ks = lds + G::oK;
  uint16_t* Vs = lds + G::oVt;    // V row-major
  uint16_t* Wh = lds + G::oB1h;   // W, then R^T
  uint16_t* Wl = lds + G::oB1l;
  uint16_t* Th = lds + G::oTh;
  uint16_t* Tl = lds + G::oTl;
  float* XR = reinterpret_cast<float*>(lds + G::oX);     // R exchange
  float* XO = reinterpret_cast<float*>(lds + G::oB2h);   // O exchange
  float* fl = reinterpret_cast<float*>(lds + ((G::n16 + 7) & ~7));
  float* eta = fl + G::f_eta;
  float* colsum = fl + G::f_cs;       // [RT][D]
  float* denp = fl + G::f_denp;       // [RT][C]
  float* g1 = fl + G::f_tab;          // decay tables over the tile index a: gamma^(a+1),
  float* g2 = g1 + C;                 // gamma^(2(a+1)),
  float* w1 = g2 + C;                 // gamma^(C-1-a),
  float* w2 = w1 + C;                 // gamma^(2(C-1-a))

  int seg, bh;
  seg_head(seg, bh);
  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = w / G::NCT, ct = w % G::NCT;          // state row half, column tile
  if (DEC && tid < C) {
    g1[tid] = exp2f(lg2g * (float)(tid + 1));
    g2[tid] = exp2f(2.f * lg2g * (float)(tid + 1));
    w1[tid] = exp2f(lg2g * (float)(C - 1 - tid));
    w2[tid] = exp2f(2.f * lg2g * (float)(C - 1 - tid));
  }
  const int r0 = h * G::HALF;                         // first state row of this wave
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t F = state_floats(D, DV);
  float* rc = rec + ((size_t)bh * (nseg + 1) + seg) * F;
  const rsrc_t ro = make_rsrc(SUMMARY ? nullptr : out + (size_t)bh * n * DV, SUMMARY ? 0u : (uint32_t)n * DV * 4);

  // ---- carry in: rows r0 .. r0 + D/2 of column tile ct ----
  f32x16 S0[G::HT], P0[G::HT];
#pragma unroll
  for (int i = 0; i < G::HT; ++i) {
    S0[i] = zero16();
    P0[i] = zero16();
  }
  for (int a = tid; a < D; a += NT) eta[a] = 0.f;
  if (spre || nseg > 1) {
    // S0 = the S prefix of this segment (the converted initial state and the
    // earlier segments; decayed: each aged to this segment's start), staged
    // through the (still free) tile region of LDS.  Without spre (no initial
    // state, few segments) it is summed here from the S slots of the earlier
    // segments' records, which the moments launch wrote (walks write only G
    // and h), four records' loads in flight at a time; decayed, segment sp
    // is aged by gamma^(C cps (seg - 1 - sp)), as the prefix launch ages it.
    constexpr int nS4 = D * D / 4 / NT, SB = 4;
    static_assert(D * D % (4 * NT) == 0 && D * D * 4 <= G::n16 * 2, "carry staging");
    float4 sa[nS4];
    if (spre) {
      const float4* x = reinterpret_cast<const float4*>(spre + ((size_t)bh * nseg + seg) * D * D);
#pragma unroll
      for (int r = 0; r < nS4; ++r) sa[r] = x[tid + NT * r];
    } else {
#pragma unroll
      for (int r = 0; r < nS4; ++r) sa[r] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int sp = 0; sp < seg; sp += SB) {
        float4 u[SB][nS4];
#pragma unroll
        for (int j = 0; j < SB; ++j)
#pragma unroll
          for (int r = 0; r < nS4; ++r)
            u[j][r] = sp + j < seg
                          ? reinterpret_cast<const float4*>(rec + ((size_t)bh * (nseg + 1) + sp + j) * F)[tid + NT * r]
                          : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < SB; ++j) {
          // (entries past the last record hold zeros; their would-be age is
          // negative, so they take weight 0, not an overflowing power)
          const float a = !DEC ? 1.f : sp + j < seg ? exp2f(lg2g * (float)(C * cps) * (float)(seg - 1 - sp - j)) : 0.f;
#pragma unroll
          for (int r = 0; r < nS4; ++r) {
            sa[r].x += a * u[j][r].x; sa[r].y += a * u[j][r].y; sa[r].z += a * u[j][r].z; sa[r].w += a * u[j][r].w;
          }
        }
      }
    }
    float* st = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int r = 0; r < nS4; ++r) reinterpret_cast<float4*>(st)[tid + NT * r] = sa[r];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < G::HT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) S0[i][e] = st[(r0 + i * 32 + acc_row(e, lg)) * D + ct * 32 + lr];
    __syncthreads();
  }

  // ---- prefetch registers for the next chunk (buffer loads: the tail past n reads zero) ----
  const rsrc_t rq = make_rsrc(q + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rk = make_rsrc(k + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rv = make_rsrc(v + (size_t)bh * n * DV, (uint32_t)n * DV * 2);
  uint4 pq[G::pfQ], pk[G::pfQ], pv[G::pfV];
  auto fetch = [&](int c) {
    const uint32_t t0 = (uint32_t)c * C;
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + NT * i;        // consecutive lanes take consecutive pieces of a token row
      const uint32_t off = ((t0 + e / (D / 8)) * D + (e % (D / 8)) * 8) * 2;
      pq[i] = buf_load16(rq, off);
      pk[i] = buf_load16(rk, off);
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + NT * i;
      pv[i] = buf_load16(rv, ((t0 + e / (DV / 8)) * DV + (e % (DV / 8)) * 8) * 2);
    }
  };
  if (c_begin < c_end) fetch(c_begin);

  for (int c = c_begin; c < c_end; ++c) {
    const int t0 = c * C;
    // lane index for the fragment helpers: at d = 128 it is made opaque once
    // per tile, so the lane-dependent offsets are computed once per tile and
    // every access adds only a constant, while none is hoisted out of the
    // walk (held live through it, they would spill)
    int ln = tid & 63;
    if constexpr (kO) asm volatile("" : "+v"(ln));
    // ---- stage 0: registers -> LDS (Q, K, V row-major; the transposed operands are read through the
    // LDS transpose unit) ----
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + NT * i;
      const int t = e / (D / 8), a8 = (e % (D / 8)) * 8;
      *reinterpret_cast<uint4*>(Qs + t * G::ldQ + a8) = pq[i];
      *reinterpret_cast<uint4*>(Ks + t * G::ldK + a8) = pk[i];
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + NT * i;
      const int t = e / (DV / 8), b8 = (e % (DV / 8)) * 8;
      *reinterpret_cast<uint4*>(Vs + t * G::ldV + b8) = pv[i];
    }
    lds_barrier();
    if (c + 1 < c_end) fetch(c + 1);

    // ---- stage 1: W = L (.) Q K^T on tiles (key it <= query jt), stored transposed ----
    if (w < 4) {
      const int it = w >> 1, jt = w & 1;
      if (it <= jt) {
        f32x16 acc = zero16();
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          acc = mfma(frag<kO>(Ks, G::ldK, it * 32, s * 16, ln), frag<kO>(Qs, G::ldQ, jt * 32, s * 16, ln), acc);
#pragma unroll
        for (int e = 0; e < 16; ++e)   // keep key i <= query t
          if (it * 32 + acc_row(e, lg) > jt * 32 + lr) acc[e] = 0.f;
        if constexpr (DEC) {           // W (.) gamma^(t - i)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[e] *= exp2f(lg2g * (float)max(jt * 32 + lr - it * 32 - acc_row(e, lg), 0));
        }
        store_T<kO>(acc, Wh, Wl, G::ld1, it * 32, jt * 32, ln);
      }
    }
    lds_barrier();

    // ---- stage 2: R partials over this wave's state rows (both row tiles), then W K on row tile h ----
    f32x16 part[2];
    part[0] = zero16();
    part[1] = zero16();
#pragma unroll
    for (int j = 0; j < G::KH; ++j) {
      bf16x8 bh_, bl_;
      frag_from_acc(S0[j >> 1], j & 1, bh_, bl_);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        const bf16x8 aQ = frag_acc_order<kO>(Qs, G::ldQ, rt * 32, r0 + j * 16, ln);
        part[rt] = mfma(aQ, bh_, part[rt]);
        part[rt] = mfma(aQ, bl_, part[rt]);
      }
    }
    if constexpr (DEC) {               // Q S0 rows age by gamma^(a+1); S0 by gamma^C before its advance
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int e = 0; e < 16; ++e) part[rt][e] *= g1[rt * 32 + acc_row(e, lg)];
      const float gC = exp2f(lg2g * (float)C);
#pragma unroll
      for (int i = 0; i < G::HT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) S0[i][e] *= gC;
    }
#pragma unroll
    for (int s = 0; s < G::KC; ++s) {
      const bf16x8 bK = frag_tr<kO>(Ks, G::ldK, ct * 32, s * 16, ln);
      if (h == 0) {
        if (s < 2) {
          part[0] = mfma(frag<kO>(Wh, G::ld1, 0, s * 16, ln), bK, part[0]);
          part[0] = mfma(frag<kO>(Wl, G::ld1, 0, s * 16, ln), bK, part[0]);
        }
      } else {
        part[1] = mfma(frag<kO>(Wh, G::ld1, 32, s * 16, ln), bK, part[1]);
        part[1] = mfma(frag<kO>(Wl, G::ld1, 32, s * 16, ln), bK, part[1]);
      }
      // S0 += K^T K on this wave's rows (decayed: K^T diag(gamma^(C-1-a)) K)
      if constexpr (DEC) {
        bf16x8 kh, kl;
        scale_split(bK, w1 + s * 16 + 8 * lg, kh, kl);
#pragma unroll
        for (int i = 0; i < G::HT; ++i) {
          const bf16x8 aK = frag_tr<kO>(Ks, G::ldK, r0 + i * 32, s * 16, ln);
          S0[i] = mfma(aK, kh, S0[i]);
          S0[i] = mfma(aK, kl, S0[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < G::HT; ++i) S0[i] = mfma(frag_tr<kO>(Ks, G::ldK, r0 + i * 32, s * 16, ln), bK, S0[i]);
      }
    }
    lds_barrier();                      // K, K^T and W are dead: K | K^T takes the exchange
    xch_put<kO>(XR, ct * 2 + (1 - h), h == 0 ? part[1] : part[0], ln);
    lds_barrier();
    f32x16 racc = h == 0 ? part[0] : part[1];
    xch_add<kO>(XR, ct * 2 + h, racc, ln);
    {
      float cs = 0.f;                  // eta0 advance: R^T 1 (decayed: R^T gamma^(2(C-1-a)))
#pragma unroll
      for (int e = 0; e < 16; ++e) cs += DEC ? racc[e] * w2[h * 32 + acc_row(e, lg)] : racc[e];
      cs += __shfl_xor(cs, 32);
      if (lg == 0) colsum[h * D + ct * 32 + lr] = cs;
    }
    store_T<kO>(racc, Wh, Wl, G::ld1, h * 32, ct * 32, ln);     // R^T
    lds_barrier();
    float eta_add = 0.f;
    if (tid < D) eta_add = colsum[tid] + colsum[D + tid];

    f32x16 oacc[2];
    if (!SUMMARY) {
      // ---- stage 3: T = L (.) Q R^T (as T^T = R Q^T) on tiles j it <= t jt; stored transposed in K | K^T ----
      if (w < 4) {
        const int it = w >> 1, jt = w & 1;
        if (it <= jt) {
          f32x16 acc = zero16();
#pragma unroll
          for (int s = 0; s < D / 16; ++s) {
            const bf16x8 b = frag<kO>(Qs, G::ldQ, jt * 32, s * 16, ln);
            acc = mfma(frag_tr<kO>(Wh, G::ld1, it * 32, s * 16, ln), b, acc);
            acc = mfma(frag_tr<kO>(Wl, G::ld1, it * 32, s * 16, ln), b, acc);
          }
#pragma unroll
          for (int e = 0; e < 16; ++e)     // keep j <= t
            if (it * 32 + acc_row(e, lg) > jt * 32 + lr) acc[e] = 0.f;
          if constexpr (DEC) {             // T (.) gamma^(2(t - j))
#pragma unroll
            for (int e = 0; e < 16; ++e)
              acc[e] *= exp2f(2.f * lg2g * (float)max(jt * 32 + lr - it * 32 - acc_row(e, lg), 0));
          }
          float ps = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) ps += acc[e];
          ps += __shfl_xor(ps, 32);
          if (lg == 0) denp[it * C + jt * 32 + lr] = ps;
          store_T<kO>(acc, Th, Tl, G::ldT, it * 32, jt * 32, ln);
        } else if (lg == 0) {
          denp[it * C + jt * 32 + lr] = 0.f;
        }
      }
      // ---- stage 4a: O partials Q Phi0 (old Phi0) over this wave's rows ----
      oacc[0] = zero16();
      oacc[1] = zero16();
#pragma unroll
      for (int j = 0; j < G::KH; ++j) {
        bf16x8 bh_, bl_;
        frag_from_acc(P0[j >> 1], j & 1, bh_, bl_);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          const bf16x8 aQ = frag_acc_order<kO>(Qs, G::ldQ, rt * 32, r0 + j * 16, ln);
          oacc[rt] = mfma(aQ, bh_, oacc[rt]);
          oacc[rt] = mfma(aQ, bl_, oacc[rt]);
        }
      }
      if constexpr (DEC) {             // Q Phi0 rows age by gamma^(2(a+1))
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[rt][e] *= g2[rt * 32 + acc_row(e, lg)];
      }
    }
    // ---- stage 5: Phi0 += R^T V on this wave's rows (decayed: gamma^(2C) Phi0 + R^T diag(gamma^(2(C-1-a))) V) ----
    if constexpr (DEC) {
      const float g2C = exp2f(2.f * lg2g * (float)C);
#pragma unroll
      for (int i = 0; i < G::HT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) P0[i][e] *= g2C;
    }
#pragma unroll
    for (int s = 0; s < G::KC; ++s) {
      const bf16x8 bV = frag_tr<kO>(Vs, G::ldV, ct * 32, s * 16, ln);
      if constexpr (DEC) {
        bf16x8 vh, vl;
        scale_split(bV, w2 + s * 16 + 8 * lg, vh, vl);
#pragma unroll
        for (int i = 0; i < G::HT; ++i) {
          const bf16x8 ah = frag<kO>(Wh, G::ld1, r0 + i * 32, s * 16, ln);
          P0[i] = mfma(ah, vh, P0[i]);
          P0[i] = mfma(ah, vl, P0[i]);
          P0[i] = mfma(frag<kO>(Wl, G::ld1, r0 + i * 32, s * 16, ln), vh, P0[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < G::HT; ++i) {
          P0[i] = mfma(frag<kO>(Wh, G::ld1, r0 + i * 32, s * 16, ln), bV, P0[i]);
          P0[i] = mfma(frag<kO>(Wl, G::ld1, r0 + i * 32, s * 16, ln), bV, P0[i]);
        }
      }
    }
    if (!SUMMARY) {
      lds_barrier();                    // T and denp visible; R and R^T are dead
      xch_put<kO>(XO, ct * 2 + (1 - h), h == 0 ? oacc[1] : oacc[0], ln);
      // den_t = sum_j T[t][j] + q_t . eta0: the row sums here, and eta0 of this
      // tile (before its advance) for k_fix, which adds q_t . (eta0 + eta_c)
      if (normalized) {
        if (tid < C && t0 + tid < n) den_out[(size_t)bh * n + t0 + tid] = denp[tid] + denp[C + tid];
        if (tid < D) den_out[(size_t)gridDim.y * n + ((size_t)bh * ((n + C - 1) / C) + c) * D + tid] = eta[tid];
      }
      lds_barrier();
      f32x16 o = h == 0 ? oacc[0] : oacc[1];
      xch_add<kO>(XO, ct * 2 + h, o, ln);
      // ---- stage 4b: O (row tile h) += T V ----
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        if (h == 0 && s >= 2) break;      // j past row tile 0: T is zero
        const bf16x8 bV = frag_tr<kO>(Vs, G::ldV, ct * 32, s * 16, ln);
        o = mfma(frag<kO>(Th, G::ldT, h * 32, s * 16, ln), bV, o);
        o = mfma(frag<kO>(Tl, G::ldT, h * 32, s * 16, ln), bV, o);
      }
      // the output tile goes through this wave's own exchange slot (its last
      // reader was this wave's xch_add) so that each lane stores 16 bytes:
      // four stores per lane instead of sixteen
      float* ob = XO + (ct * 2 + h) * 1024;
#pragma unroll
      for (int e = 0; e < 16; ++e) ob[acc_row(e, lg) * 32 + lr] = o[e];
#pragma unroll
      for (int j = 0; j < 4; ++j) {       // rows past n fall outside the buffer and are dropped
        const int p = l + 64 * j, row = p >> 3, c4 = (p & 7) * 4;
        buf_store16(ro, (((uint32_t)t0 + h * 32 + row) * DV + ct * 32 + c4) * 4,
                    *reinterpret_cast<const float4*>(ob + row * 32 + c4));
      }
    }
    lds_barrier();   // LDS tiles and den/eta are rewritten by the next chunk
    if (tid < D) {
      if constexpr (DEC)
        eta[tid] = exp2f(2.f * lg2g * (float)C) * eta[tid] + eta_add;
      else
        eta[tid] += eta_add;
    }
  }

  // the segment's bracket: Phi0 into the G slot, eta0 into the h slot.  The
  // opaque copies of the lane coordinates keep the store addresses from being
  // computed before the walk (they would stay live through it).
  int col = ct * 32 + lr, lgo = lg;
  asm volatile("" : "+v"(col), "+v"(lgo));
#pragma unroll
  for (int i = 0; i < G::HT; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      rc[off_G(D, DV) + (size_t)(r0 + i * 32 + acc_row(e, lgo)) * DV + col] = P0[i][e];
  if (tid < D) rc[off_h(D, DV) + tid] = eta[tid];
}

struct Shape {
  int C, D, DV, blocks;   // blocks: output-walk workgroups per CU (column layout)
};
#define HLA_SHAPE_ROW(C_, D_, DV_) {C_, D_, DV_, Cfg<C_, D_, DV_, false>::kBlocks}
constexpr Shape kShapes[] = {HLA_SHAPE_ROW(64, 64, 64),  HLA_SHAPE_ROW(32, 32, 32),   HLA_SHAPE_ROW(64, 32, 32),
                             HLA_SHAPE_ROW(32, 64, 64),  HLA_SHAPE_ROW(64, 64, 32),   HLA_SHAPE_ROW(64, 32, 64),
                             HLA_SHAPE_ROW(64, 128, 128), HLA_SHAPE_ROW(32, 128, 128)};
#undef HLA_SHAPE_ROW

// The walk's tile: chunk 32 and 64 are walked as given; chunk 128 is walked
// in 64-token tiles.  The scan is exact for every chunking (Thm. 2), so the
// tile changes only the rounding order.
int fused_tile(int chunk) { return chunk == 32 ? 32 : (chunk == 64 || chunk == 128) ? 64 : 0; }

const Shape* find_shape(int chunk, int d, int dv) {
  const int C = fused_tile(chunk);
  for (const Shape& sh : kShapes)
    if (sh.C == C && sh.D == d && sh.DV == dv) return &sh;
  return nullptr;
}

template <int D, int DV>
hipError_t set_cross_lds(const void* kern, size_t* lds) {
  *lds = sizeof(float) * ((size_t)D * (D + 4) + (size_t)D * DV + D);
  return hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)*lds);
}

// Launch configuration of one walk kernel (function, threads, LDS bytes).
struct WalkK {
  const void* fn;
  int threads;
  size_t lds;
};

template <int C, int D, int DV, bool SUMMARY, bool RS, bool DEC = false>
WalkK walk_kernel() {
  if constexpr (RS) {
    return {(const void*)k_walk_rs<D, SUMMARY, DEC>, CfgRS<D, SUMMARY>::NT, CfgRS<D, SUMMARY>::bytes};
  } else {
    return {(const void*)k_walk<C, D, DV, SUMMARY>, kThreads, Cfg<C, D, DV, SUMMARY>::bytes};
  }
}

hipError_t launch_walk(const WalkK& kk, dim3 grid, hipStream_t s, const uint16_t* q, const uint16_t* k,
                       const uint16_t* v, float* out, float* den_out, float* rec, const float* spre, int n, int cps,
                       int nseg, int normalized, float eps, float lg2g) {
  hipError_t e = hipFuncSetAttribute(kk.fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kk.lds);
  if (e != hipSuccess) return e;
  void* args[] = {&q, &k, &v, &out, &den_out, &rec, &spre, &n, &cps, &nseg, &normalized, &eps, &lg2g};
  return prof_launch(kk.fn, grid, dim3(kk.threads), args, kk.lds, s);
}

size_t records_bytes(int BH, int P, int d, int dv) {
  return (sizeof(float) * (size_t)BH * (P + 1) * state_floats(d, dv) + 255) & ~size_t(255);
}

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

// Workspace of the walk + carry fix-up pipeline: records [BH][P + 1][F] |
// walk denominators [BH][n] and per-tile eta [BH][M][d] | carries
// [BH][P][d dv + d] | S prefixes [BH][P][d d].
size_t legacy_spre_offset(int BH, int n, int P, int C, int d, int dv) {
  const size_t den = sizeof(float) * (((size_t)BH * n + (size_t)BH * ((n + C - 1) / C) * d + 63) & ~size_t(63));
  const size_t carry = sizeof(float) * (size_t)BH * P * ((size_t)d * dv + d);
  return al256(records_bytes(BH, P, d, dv) + den + carry);
}
size_t legacy_ws_bytes(int BH, int n, int P, int C, int d, int dv) {
  return legacy_spre_offset(BH, n, P, C, d, dv) + sizeof(float) * (size_t)BH * P * d * d + 256;
}

// Workspace of the two-pass pipeline (d = dv = 128, no initial or final
// state): records [BH][P + 1][F] | S prefixes [BH][P][d d] | Phi, eta carries
// [BH][P][d dv + d].
size_t ws_pipeline_bytes(int BH, int P) {
  constexpr int D = CfgWS::D, DV = CfgWS::DV;
  return records_bytes(BH, P, D, DV) + al256(sizeof(float) * (size_t)BH * P * D * D) +
         al256(sizeof(float) * (size_t)BH * P * ((size_t)D * DV + D));
}

bool legacy_pipeline() {
  const char* e = getenv("HLA_FUSED_LEGACY");
  return e && e[0] == '1';
}

// Per-tile time of the summary walk over that of the output walk (both at
// one workgroup per CU, d = dv = 128: about 3.9 and 6.6 us per tile).
constexpr double kWsSummaryRatio = 0.65;

// Segments per head up to which the row-split walk (no initial state) sums
// its S prefix from the moments itself instead of reading it from a prefix
// launch.
constexpr int kWalkSumMax = 8;

// Segments of the two-pass plan: with Q = 256 / BH walks per head in each
// launch (one workgroup per CU), segments 1 .. P-1 get x tiles each (the
// last the rest) and segment 0 about r x, r the ratio above, so that segment
// 0's output walk and the summary walks beside it end together.  With fewer
// than two later segments the plan is a single output walk per head.
void ws_plan(int BH, int n, int* P, int* cps, int* c0) {
  const int M = (n + CfgWS::C - 1) / CfgWS::C;
  int Q = 256 / BH;
  if (const char* e = getenv("HLA_FUSED_SEGMENTS")) Q = atoi(e) - 1;
  double r = kWsSummaryRatio;
  if (const char* e = getenv("HLA_WS_RATIO")) r = atof(e);
  if (Q >= 2 && M >= 3 && r > 0.0) {
    int x = (int)ceil(M / (Q + r));
    const int l0 = std::max(1, (int)lround(r * x));
    if (l0 < M) {
      const int rest = M - l0;
      if ((rest + x - 1) / x > Q) x = (rest + Q - 1) / Q;
      const int p1 = (rest + x - 1) / x;
      if (p1 >= 2) {
        *P = 1 + p1;
        *cps = x;
        *c0 = l0;
        return;
      }
    }
  }
  *P = 1;
  *cps = M;
  *c0 = M;
}

hipError_t launch_ws(const void* fn, dim3 grid, hipStream_t s, void** args) {
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)CfgWS::bytes);
  if (e != hipSuccess) return e;
  return prof_launch(fn, grid, dim3(CfgWS::NT), args, CfgWS::bytes, s);
}

// The forward at d = dv = 128 (64-token tiles) without states, every output
// row written once (plan in ws_plan):
//   1. k_walk_ws_first: segment 0's output walk, and the summary walks of
//      segments 1 .. P-2 from a zero state (S, C, m, Phi, eta records);
//   2. k_ws_bracket: the S prefixes, summed from the records, and each
//      record's bracket (Phi_s + S_{<s} C_s, eta_s + S_{<s} m_s) in place;
//      k_seg_prefix: the running sums of the brackets, the Phi, eta carries;
//   3. k_walk_ws_out over segments 1 .. P-1 from their true carries.
// With P = 1, step 3 alone over whole heads.
hipError_t run_ws(const Fwd& f, char* ws, hipStream_t s) {
  constexpr int D = CfgWS::D, DV = CfgWS::DV;
  const int BH = f.BH;
  int P, cps, c0;
  ws_plan(BH, f.n, &P, &cps, &c0);
  const size_t F = state_floats(D, DV);
  float* segs = reinterpret_cast<float*>(ws);
  float* spre = reinterpret_cast<float*>(ws + records_bytes(BH, P, D, DV));
  float* carry = reinterpret_cast<float*>(reinterpret_cast<char*>(spre) + al256(sizeof(float) * (size_t)BH * P * D * D));
  const uint16_t* q = static_cast<const uint16_t*>(f.q);
  const uint16_t* k = static_cast<const uint16_t*>(f.k);
  const uint16_t* v = static_cast<const uint16_t*>(f.v);
  float* out = f.out;
  float* den = f.normalized ? f.den_out : nullptr;
  int n = f.n, normalized = f.normalized;
  float eps = f.eps;
  hipError_t e;
  if (P > 1) {
    prof_start("walk_first", s);
    void* a1[] = {&q, &k, &v, &out, &den, &segs, &n, &c0, &cps, &P, &normalized, &eps};
    e = launch_ws((const void*)k_walk_ws_first, dim3(P - 1, BH), s, a1);
    prof_stop(s);
    if (e != hipSuccess || (e = hipGetLastError()) != hipSuccess) return e;
    // the S prefixes of segments 1 .. P-1 and the brackets of 1 .. P-2 (no
    // walk writes record P - 1: the sums that include it are never stored)
    prof_start("bracket", s);
    HLA_LAUNCH((k_ws_bracket<D, DV>), dim3(P - 1, BH), dim3(1024), 0, s, segs, spre, P);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    prof_start("seg_prefix", s);
    HLA_LAUNCH(k_seg_prefix, dim3((D * DV + D + 1023) / 1024, BH), dim3(256), 0, s, segs, F, (int)off_G(D, DV),
               D * DV + D, 0, carry, P, 1.f);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const float* sp = P > 1 ? spre : nullptr;
  const float* cp = P > 1 ? carry : nullptr;
  int seg0 = P > 1 ? 1 : 0;
  prof_start("walk", s);
  void* a2[] = {&q, &k, &v, &out, &den, &sp, &cp, &n, &c0, &cps, &P, &seg0, &normalized, &eps};
  e = launch_ws((const void*)k_walk_ws_out, dim3(P > 1 ? P - 1 : 1, BH), s, a2);
  prof_stop(s);
  if (e != hipSuccess || (e = hipGetLastError()) != hipSuccess) return e;
  return hipSuccess;
}

// DEC: the decayed operator (row-split shapes, no initial or final state).
template <int C, int D, int DV, bool RS, bool DEC = false>
hipError_t run_shape(const Fwd& f, const float* init, float* final_state, char* ws, int P, int cps,
                     hipStream_t s) {
  static_assert(!DEC || RS, "the decayed walk is row-split only");
  const float lg2g = DEC ? (float)std::log2((double)f.gamma) : 0.f;
  const float rho2 = DEC ? (float)std::exp2(2.0 * std::log2((double)f.gamma) * (double)C * (double)cps) : 1.f;
  const int BH = f.BH;
  float* segs = reinterpret_cast<float*>(ws);                                  // [BH][P + 1][F] records
  float* den = reinterpret_cast<float*>(ws + records_bytes(BH, P, D, DV));    // [BH][n] walk denominators
  const uint16_t* q = static_cast<const uint16_t*>(f.q);
  const uint16_t* k = static_cast<const uint16_t*>(f.k);
  const uint16_t* v = static_cast<const uint16_t*>(f.v);
  const dim3 grid(P, BH);
  hipError_t e;
  if (init) {      // slot P <- the initial state in the (S, C, m, Phi, eta) form
    size_t lds;
    if ((e = set_cross_lds<D, DV>((const void*)k_init_convert<D, DV>, &lds)) != hipSuccess) return e;
    prof_start("init_convert", s);
    HLA_LAUNCH((k_init_convert<D, DV>), dim3(1, BH), dim3(256), lds, s, segs, init, P);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  prof_start("moments", s);
  if (final_state)
    HLA_LAUNCH((k_moments<C, D, DV, false, DEC>), grid, dim3(kThreads), 0, s, q, k, v, segs, f.n, cps, P, 1, lg2g);
  else
    HLA_LAUNCH((k_moments<C, D, DV, false, DEC, false>), grid, dim3(kThreads), 0, s, q, k, v, segs, f.n, cps, P, 0,
               lg2g);
  prof_stop(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // S prefix of every segment (the walks each read one): init + the earlier
  // segments' moments, each aged to the segment's start when decayed.  The
  // row-split walk without an initial state sums up to kWalkSumMax - 1
  // earlier moments itself, which saves this launch.
  float* spre = nullptr;
  const bool walk_sums = RS && !init && P <= kWalkSumMax;
  if ((P > 1 || init) && !walk_sums) {
    spre = reinterpret_cast<float*>(ws + legacy_spre_offset(BH, f.n, P, C, D, DV));
    const float rhoS = DEC ? (float)std::exp2((double)lg2g * (double)C * (double)cps) : 1.f;
    prof_start("seg_prefix", s);
    HLA_LAUNCH(k_seg_prefix, dim3((D * D + 1023) / 1024, BH), dim3(256), 0, s, segs, state_floats(D, DV), 0, D * D,
               init ? 1 : 0, spre, P, rhoS);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  prof_start(f.out ? "walk" : "walk_summary", s);
  e = f.out ? launch_walk(walk_kernel<C, D, DV, false, RS, DEC>(), grid, s, q, k, v, f.out, den, segs, spre, f.n,
                          cps, P, f.normalized, f.eps, lg2g)
            : launch_walk(walk_kernel<C, D, DV, true, RS, DEC>(), grid, s, q, k, v, nullptr, nullptr, segs, spre, f.n,
                          cps, P, 0, 0.f, lg2g);
  prof_stop(s);
  if (e != hipSuccess || (e = hipGetLastError()) != hipSuccess) return e;
  if (final_state) {
    size_t lds;
    if ((e = set_cross_lds<D, DV>((const void*)k_total<D, DV>, &lds)) != hipSuccess) return e;
    prof_start("total", s);
    HLA_LAUNCH((k_total<D, DV>), dim3(BH), dim3(256), lds, s, segs, init, final_state, P, P);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (f.out && (P > 1 || init || f.normalized)) {
    float* carry = den + (((size_t)BH * f.n + (size_t)BH * ((f.n + C - 1) / C) * D + 63) & ~size_t(63));
    prof_start("carry", s);
    HLA_LAUNCH((k_carry<D, DV>), dim3((D * DV / 8 + D + 255) / 256, BH), dim3(256), 0, s, segs, init, carry, P,
               rho2);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    using FC = FixCfg<C, D, DV>;
    static_assert(FC::lds <= 64 * 1024, "fix LDS");
    if ((e = hipFuncSetAttribute((const void*)k_fix<C, D, DV, DEC>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)FC::lds)) != hipSuccess)
      return e;
    const int M = (f.n + C - 1) / C, tpw = fix_tpw(M, BH);
    prof_start("fix", s);
    HLA_LAUNCH((k_fix<C, D, DV, DEC>), dim3((M + tpw - 1) / tpw, BH), dim3(FC::NT), FC::lds, s, q, f.out, den,
               carry, f.normalized ? f.den_out : nullptr, init ? 1 : 0, f.n, cps, P, f.normalized, f.eps, tpw,
               lg2g);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

// (64, 64, 64) and (64, 128, 128) walk in the row-split layout; the other
// shapes in the column layout.
bool row_split_shape(const Shape& sh) { return sh.C == 64 && sh.D == sh.DV && (sh.D == 64 || sh.D == 128); }

// The wave-specialised walk covers (64, 128, 128).
bool ws_shape(const Shape& sh) { return sh.C == CfgWS::C && sh.D == CfgWS::D && sh.DV == CfgWS::DV; }

int plan_blocks(const Shape& sh) {
  if (row_split_shape(sh)) return sh.D == 64 ? CfgRS<64, false>::kBlocks : CfgRS<128, false>::kBlocks;
  return sh.blocks;
}

void fused_plan(const Shape& sh, int BH, int n, int* P, int* cps) {
  const int M = (n + sh.C - 1) / sh.C;
  int p = 256 * plan_blocks(sh) / BH;
  if (const char* e = getenv("HLA_FUSED_SEGMENTS")) p = atoi(e);
  if (p < 1) p = 1;
  if (p > M) p = M;
  *cps = (M + p - 1) / p;
  *P = (M + *cps - 1) / *cps;             // every segment non-empty
}

}  // namespace

bool fused_plan_query(int BH, int n, int d, int dv, int chunk, int* P, int* tile, int* first, int* per) {
  const Shape* sh = find_shape(chunk, d, dv);
  if (!sh) return false;
  int cps, c0;
  if (ws_shape(*sh) && !legacy_pipeline()) {
    ws_plan(BH, n, P, &cps, &c0);   // the plan of the forward without states
  } else {
    fused_plan(*sh, BH, n, P, &cps);
    c0 = cps;
  }
  *tile = sh->C;
  if (first) *first = c0;
  if (per) *per = cps;
  return true;
}

bool fused_supported(int n, int d, int dv, int chunk, int dtype, int masked) {
  // per-head byte offsets of q/k/v and of the output stay below 2^31
  const long long span = (long long)n * (d > dv ? d : dv) * 4;
  return dtype == 1 && masked == 1 && n >= 1 && span < (1LL << 31) && find_shape(chunk, d, dv) != nullptr;
}

bool fused_decay_supported(int n, int d, int dv, int chunk, int dtype, int masked) {
  const Shape* sh = find_shape(chunk, d, dv);
  return fused_supported(n, d, dv, chunk, dtype, masked) && sh && row_split_shape(*sh);
}

size_t fused_workspace_bytes(int BH, int n, int d, int dv, int chunk) {
  const Shape* sh = find_shape(chunk, d, dv);
  if (!sh) return 0;
  int P, cps;
  fused_plan(*sh, BH, n, &P, &cps);
  const size_t legacy = legacy_ws_bytes(BH, n, P, sh->C, d, dv);
  if (ws_shape(*sh)) {
    int Pw, cw, c0;
    ws_plan(BH, n, &Pw, &cw, &c0);
    const size_t w = ws_pipeline_bytes(BH, Pw);
    return w > legacy ? w : legacy;
  }
  return legacy;
}

hipError_t launch_fused(const Fwd& f, const float* init, float* final_state, void* workspace, hipStream_t s) {
  const Shape* sh = find_shape(f.chunk, f.d, f.dv);
  if (!sh) return hipErrorNotSupported;
  int P, cps;
  fused_plan(*sh, f.BH, f.n, &P, &cps);
  char* ws = static_cast<char*>(workspace);
  if (f.gamma == 1.f && !init && !final_state && ws_shape(*sh) && !legacy_pipeline()) return run_ws(f, ws, s);
  if (f.gamma != 1.f) {           // decayed: row-split shapes only, no states
    if (!row_split_shape(*sh) || init || final_state) return hipErrorNotSupported;
    if (sh->D == 64) return run_shape<64, 64, 64, true, true>(f, init, final_state, ws, P, cps, s);
    return run_shape<64, 128, 128, true, true>(f, init, final_state, ws, P, cps, s);
  }
  if (row_split_shape(*sh)) {
    if (sh->D == 64) return run_shape<64, 64, 64, true>(f, init, final_state, ws, P, cps, s);
    return run_shape<64, 128, 128, true>(f, init, final_state, ws, P, cps, s);
  }
#define HLA_SHAPE(C_, D_, DV_) \
  if (sh->C == C_ && sh->D == D_ && sh->DV == DV_) return run_shape<C_, D_, DV_, false>(f, init, final_state, ws, P, cps, s);
  HLA_SHAPE(64, 64, 64)
  HLA_SHAPE(32, 32, 32)
  HLA_SHAPE(64, 32, 32)
  HLA_SHAPE(32, 64, 64)
  HLA_SHAPE(64, 64, 32)
  HLA_SHAPE(64, 32, 64)
  HLA_SHAPE(64, 128, 128)
  HLA_SHAPE(32, 128, 128)
#undef HLA_SHAPE
  return hipErrorNotSupported;
}

}  // namespace hla
