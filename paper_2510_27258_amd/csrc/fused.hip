// Fused masked second-order HLA forward for bf16 inputs on gfx950 MFMA.
//
// Algorithm (Sec. 4, two-level scan, Rem. scan-modes; Thm. 1 readout):
// the sequence of every head is cut into P segments of whole chunks.
//   1. k_walk<SUMMARY>: each workgroup walks one segment from a zero carry and
//      produces its summary (S, C, m, Phi, eta) with Phi = S C - G and
//      eta = S m - h (an exact change of variables of the 5-tuple).
//   2. k_flip turns summaries into the paper's 5-tuples (G = S C - Phi,
//      h = S m - eta); k_scan (hla2_scan.hip) takes the exclusive
//      semidirect-product scan over segments, Eq. (semidirect); k_flip turns
//      the carries back (Phi0 = S0 C0 - G0, eta0 = S0 m0 - h0).
//   3. k_walk<OUTPUT>: each workgroup walks one segment again from its carry
//      and writes the outputs.
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
// Layout: 256 threads = 4 waves.  Wave w owns the 16-column tiles
// {w, w+4, ...} of S0, R (over d) and of Phi0, O (over dv); S0 and Phi0 stay
// in MFMA accumulators for the whole walk and are fed back as MFMA B
// operands straight from registers.  Q, K, K^T, V^T, W/T, R and R^T are
// staged in LDS as bf16.
#include "fused.h"
#include "profile.h"

namespace hla {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint16_t u16x4;

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kPad = 8;   // bf16 elements of padding per LDS row

__device__ __forceinline__ uint16_t bf16_bits(__bf16 x) { return __builtin_bit_cast(uint16_t, x); }
__device__ __forceinline__ float bf16_to_f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// x = hi + lo (both bf16, round to nearest even)
__device__ __forceinline__ void split(float x, uint16_t& hi, uint16_t& lo) {
  const __bf16 h = (__bf16)x;
  hi = bf16_bits(h);
  lo = bf16_bits((__bf16)(x - (float)h));
}

__device__ __forceinline__ f32x4 mfma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Operand fragment from a row-major bf16 LDS tile X[row][k]: lane (r = l%16,
// g = l/16) takes X[row0 + r][k0 + 8g .. 8g+7].  It is the A operand of X Y
// (rows of X = rows of the result) and the B operand of Z X^T (rows of X =
// columns of the result); both operands of a product use the same k order.
__device__ __forceinline__ bf16x8 frag(const uint16_t* X, int ld, int row0, int k0) {
  const int l = threadIdx.x & 63;
  const uint16_t* p = X + (row0 + (l & 15)) * ld + k0 + 8 * (l >> 4);
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// Same, with the k order of accumulator-fed operands: lane takes
// X[row0 + r][k0 + 4g .. 4g+3] and X[row0 + r][k0 + 16 + 4g .. +3].
__device__ __forceinline__ bf16x8 frag_acc_order(const uint16_t* X, int ld, int row0, int k0) {
  const int l = threadIdx.x & 63;
  const uint16_t* p = X + (row0 + (l & 15)) * ld + k0 + 4 * (l >> 4);
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  const uint2 b = *reinterpret_cast<const uint2*>(p + 16);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// B operand from two fp32 accumulator tiles holding Y[k0 .. k0+15][n0..] and
// Y[k0+16 .. k0+31][n0..] (lane holds rows 4g..4g+3 of column r of each),
// split into hi and lo parts.  Pairs with frag_acc_order.
__device__ __forceinline__ void frag_from_acc(const f32x4& t0, const f32x4& t1, bf16x8& hi, bf16x8& lo) {
  uint16_t h[8], o[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    split(t0[j], h[j], o[j]);
    split(t1[j], h[4 + j], o[4 + j]);
  }
  uint4 hv, ov;
  hv.x = h[0] | (uint32_t)h[1] << 16; hv.y = h[2] | (uint32_t)h[3] << 16;
  hv.z = h[4] | (uint32_t)h[5] << 16; hv.w = h[6] | (uint32_t)h[7] << 16;
  ov.x = o[0] | (uint32_t)o[1] << 16; ov.y = o[2] | (uint32_t)o[3] << 16;
  ov.z = o[4] | (uint32_t)o[5] << 16; ov.w = o[6] | (uint32_t)o[7] << 16;
  hi = __builtin_bit_cast(bf16x8, hv);
  lo = __builtin_bit_cast(bf16x8, ov);
}

// Store an accumulator tile D[row0 + 4g + j][col0 + r] transposed, as
// X[col0 + r][row0 + 4g + j], split into hi/lo tiles (8-byte stores).
__device__ __forceinline__ void store_T(const f32x4& acc, uint16_t* Xh, uint16_t* Xl, int ld, int row0, int col0) {
  const int l = threadIdx.x & 63;
  uint16_t h[4], o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) split(acc[j], h[j], o[j]);
  const int off = (col0 + (l & 15)) * ld + row0 + 4 * (l >> 4);
  *reinterpret_cast<uint2*>(Xh + off) = make_uint2(h[0] | (uint32_t)h[1] << 16, h[2] | (uint32_t)h[3] << 16);
  *reinterpret_cast<uint2*>(Xl + off) = make_uint2(o[0] | (uint32_t)o[1] << 16, o[2] | (uint32_t)o[3] << 16);
}

// Store an accumulator tile row-major as X[row0 + 4g + j][col0 + r], hi/lo.
__device__ __forceinline__ void store_N(const f32x4& acc, uint16_t* Xh, uint16_t* Xl, int ld, int row0, int col0) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint16_t h, o;
    split(acc[j], h, o);
    const int off = (row0 + 4 * (l >> 4) + j) * ld + col0 + (l & 15);
    Xh[off] = h;
    Xl[off] = o;
  }
}

template <int C, int D, int DV, bool SUMMARY>
struct Cfg {
  static constexpr int ldQ = D + kPad, ldK = D + kPad, ldKt = C + kPad, ldVt = C + kPad;
  static constexpr int ldW = C + kPad, ldR = D + kPad, ldRt = C + kPad, ldQt = C + kPad;
  static constexpr int oQ = 0;
  static constexpr int oK = oQ + C * ldQ;
  static constexpr int oKt = oK + C * ldK;
  static constexpr int oVt = oKt + D * ldKt;
  static constexpr int oWh = oVt + DV * ldVt;
  static constexpr int oWl = oWh + C * ldW;
  static constexpr int oRh = oWl + C * ldW;
  static constexpr int oRl = oRh + (SUMMARY ? 0 : C * ldR);
  static constexpr int oRth = oRl + (SUMMARY ? 0 : C * ldR);
  static constexpr int oRtl = oRth + D * ldRt;
  static constexpr int oQt = oRtl + D * ldRt;
  static constexpr int n16 = oQt + (SUMMARY ? D * ldQt : 0);          // bf16 elements
  static constexpr int f_eta = 0, f_cs = D, f_den = 2 * D, f_denp = 2 * D + C;   // fp32 region
  static constexpr int nf32 = 2 * D + C + (C / 16) * C;
  static constexpr size_t bytes = (size_t)n16 * 2 + (size_t)nf32 * 4 + 16;
  static constexpr int RT = C / 16;                  // token tiles
  static constexpr int SA = (D / 16 + kWaves - 1) / kWaves;   // column tiles of S0/R per wave
  static constexpr int SB = (DV / 16 + kWaves - 1) / kWaves;  // column tiles of Phi0/O per wave
  static constexpr int DT = D / 16;
  static constexpr int KC = C / 32, KD = D / 32;
  // global->LDS staging: 16-byte segments per operand
  static constexpr int segQ = C * D / 8, segV = C * DV / 8;
  static constexpr int pfQ = (segQ + kThreads - 1) / kThreads, pfV = (segV + kThreads - 1) / kThreads;
  static_assert(C % 32 == 0 && D % 32 == 0 && DV % 16 == 0, "tile shape");
  static_assert(bytes <= 160 * 1024, "LDS budget");
};

// k_flip: for each record, X <- S C - X and y <- S m - y (both directions of
// Phi = S C - G, eta = S m - h).  One workgroup per (record, 32 columns).
// Records: head h, record i < per_head at src[(h*src_hs + i)*F] and
// dst[(h*dst_hs + i)*F].  In place (src == dst) is allowed.
__global__ __launch_bounds__(256) void k_flip(const float* src, float* dst, int per_head, int src_hs, int dst_hs,
                                              int d, int dv) {
  extern __shared__ float sm[];
  const int rec = blockIdx.x, blk = blockIdx.y, tid = threadIdx.x;
  const size_t F = state_floats(d, dv);
  const int hh = rec / per_head, ii = rec % per_head;
  const float* s = src + ((size_t)hh * src_hs + ii) * F;
  float* o = dst + ((size_t)hh * dst_hs + ii) * F;
  const int c0 = blk * 32, nc = min(32, dv - c0);
  float* Cs = sm;                       // [d][32]
  for (int idx = tid; idx < d * 32; idx += 256) {
    const int a = idx / 32, j = idx % 32;
    Cs[idx] = j < nc ? s[off_C(d, dv) + (size_t)a * dv + c0 + j] : 0.f;
  }
  __syncthreads();
  for (int idx = tid; idx < d * nc; idx += 256) {
    const int a = idx / nc, j = idx % nc;
    float acc = 0.f;
    for (int b = 0; b < d; ++b) acc += s[(size_t)a * d + b] * Cs[b * 32 + j];
    o[off_G(d, dv) + (size_t)a * dv + c0 + j] = acc - s[off_G(d, dv) + (size_t)a * dv + c0 + j];
  }
  if (blk == 0) {
    for (int a = tid; a < d; a += 256) {
      float acc = 0.f;
      for (int b = 0; b < d; ++b) acc += s[(size_t)a * d + b] * s[off_m(d, dv) + b];
      o[off_h(d, dv) + a] = acc - s[off_h(d, dv) + a];
    }
    if (src != dst) {
      for (size_t idx = tid; idx < (size_t)d * d; idx += 256) o[idx] = s[idx];
      for (int idx = tid; idx < d; idx += 256) o[off_m(d, dv) + idx] = s[off_m(d, dv) + idx];
    }
  }
  if (src != dst)
    for (int idx = tid; idx < d * nc; idx += 256) {
      const int a = idx / nc, j = idx % nc;
      o[off_C(d, dv) + (size_t)a * dv + c0 + j] = s[off_C(d, dv) + (size_t)a * dv + c0 + j];
    }
}

// One segment walk.  grid = (segments, BH).  SUMMARY: zero carry, writes the
// segment summary (S, C, m, Phi, eta) to `rec`.  !SUMMARY: reads the carry
// (S0, ., ., Phi0, eta0) from `rec` (NULL = zero) and writes outputs.
template <int C, int D, int DV, bool SUMMARY>
__global__ __launch_bounds__(kThreads, 1) void k_walk(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v, float* __restrict__ out,
                                                      float* __restrict__ rec, int n, int cps, int nseg,
                                                      int normalized, float eps) {
  using G = Cfg<C, D, DV, SUMMARY>;
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* Qs = lds + G::oQ;
  uint16_t* Ks = lds + G::oK;
  uint16_t* Kt = lds + G::oKt;
  uint16_t* Vt = lds + G::oVt;
  uint16_t* Wh = lds + G::oWh;   // W, later T
  uint16_t* Wl = lds + G::oWl;
  uint16_t* Rh = lds + G::oRh;
  uint16_t* Rl = lds + G::oRl;
  uint16_t* Rth = lds + G::oRth;
  uint16_t* Rtl = lds + G::oRtl;
  uint16_t* Qt = lds + G::oQt;
  float* fl = reinterpret_cast<float*>(lds + ((G::n16 + 7) & ~7));
  float* eta = fl + G::f_eta;
  float* colsum = fl + G::f_cs;
  float* den = fl + G::f_den;
  float* denp = fl + G::f_denp;

  const int seg = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t F = state_floats(D, DV);
  float* rc = rec ? rec + ((size_t)bh * nseg + seg) * F : nullptr;

  // ---- carry in (fp32 accumulators) ----
  f32x4 S0[G::SA][G::DT];
  f32x4 P0[G::SB][G::DT];
  f32x4 Cs[SUMMARY ? G::SB : 1][G::DT];
#pragma unroll
  for (int sa = 0; sa < G::SA; ++sa)
#pragma unroll
    for (int rt = 0; rt < G::DT; ++rt) {
      const int at = w + kWaves * sa;
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      if (!SUMMARY && rc && at < G::DT)
        for (int j = 0; j < 4; ++j) x[j] = rc[(size_t)(rt * 16 + 4 * lg + j) * D + at * 16 + lr];
      S0[sa][rt] = x;
    }
#pragma unroll
  for (int sb = 0; sb < G::SB; ++sb)
#pragma unroll
    for (int rt = 0; rt < G::DT; ++rt) {
      const int bt = w + kWaves * sb;
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      if (!SUMMARY && rc && bt * 16 < DV)
        for (int j = 0; j < 4; ++j) x[j] = rc[off_G(D, DV) + (size_t)(rt * 16 + 4 * lg + j) * DV + bt * 16 + lr];
      P0[sb][rt] = x;
      if (SUMMARY) Cs[SUMMARY ? sb : 0][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  for (int a = tid; a < D; a += kThreads) eta[a] = (!SUMMARY && rc) ? rc[off_h(D, DV) + a] : 0.f;
  float m_acc = 0.f;   // SUMMARY: column sum of Q for column tid (< D)

  // ---- prefetch registers for the next chunk ----
  uint4 pq[G::pfQ], pk[G::pfQ], pv[G::pfV];
  auto fetch = [&](int c) {
    const int t0 = c * C;
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + kThreads * i;
      const int t = e / (D / 8), a8 = (e % (D / 8)) * 8;
      uint4 zq = make_uint4(0, 0, 0, 0), zk = zq;
      if (e < G::segQ && t0 + t < n) {
        const size_t off = ((size_t)bh * n + t0 + t) * D + a8;
        zq = *reinterpret_cast<const uint4*>(q + off);
        zk = *reinterpret_cast<const uint4*>(k + off);
      }
      pq[i] = zq;
      pk[i] = zk;
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + kThreads * i;
      const int t = e / (DV / 8), b8 = (e % (DV / 8)) * 8;
      uint4 zv = make_uint4(0, 0, 0, 0);
      if (e < G::segV && t0 + t < n) zv = *reinterpret_cast<const uint4*>(v + ((size_t)bh * n + t0 + t) * DV + b8);
      pv[i] = zv;
    }
  };
  if (c_begin < c_end) fetch(c_begin);

  for (int c = c_begin; c < c_end; ++c) {
    const int t0 = c * C;
    // ---- stage 0: registers -> LDS (Q, K row-major; K^T, V^T; Q^T for summaries) ----
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + kThreads * i;
      if (e < G::segQ) {
        const int t = e / (D / 8), a8 = (e % (D / 8)) * 8;
        *reinterpret_cast<uint4*>(Qs + t * G::ldQ + a8) = pq[i];
        *reinterpret_cast<uint4*>(Ks + t * G::ldK + a8) = pk[i];
        const uint16_t* kk = reinterpret_cast<const uint16_t*>(&pk[i]);
#pragma unroll
        for (int j = 0; j < 8; ++j) Kt[(a8 + j) * G::ldKt + t] = kk[j];
        if (SUMMARY) {
          const uint16_t* qq = reinterpret_cast<const uint16_t*>(&pq[i]);
#pragma unroll
          for (int j = 0; j < 8; ++j) Qt[(a8 + j) * G::ldQt + t] = qq[j];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + kThreads * i;
      if (e < G::segV) {
        const int t = e / (DV / 8), b8 = (e % (DV / 8)) * 8;
        const uint16_t* vv = reinterpret_cast<const uint16_t*>(&pv[i]);
#pragma unroll
        for (int j = 0; j < 8; ++j) Vt[(b8 + j) * G::ldVt + t] = vv[j];
      }
    }
    __syncthreads();
    if (c + 1 < c_end) fetch(c + 1);
    if (SUMMARY && tid < D)
      for (int t = 0; t < C; ++t) m_acc += bf16_to_f(Qs[t * G::ldQ + tid]);

    // ---- stage 1: W = L (.) Q K^T, computed as W^T = K Q^T and stored transposed ----
    for (int it = w; it < G::RT; it += kWaves) {
      f32x4 acc[G::RT];
#pragma unroll
      for (int jt = 0; jt < G::RT; ++jt) acc[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < G::KD; ++s) {
        const bf16x8 a = frag(Ks, G::ldK, it * 16, s * 32);
#pragma unroll
        for (int jt = 0; jt < G::RT; ++jt) acc[jt] = mfma(a, frag(Qs, G::ldQ, jt * 16, s * 32), acc[jt]);
      }
#pragma unroll
      for (int jt = 0; jt < G::RT; ++jt) {
#pragma unroll
        for (int j = 0; j < 4; ++j)   // keep key i <= query t
          if (it * 16 + 4 * lg + j > jt * 16 + lr) acc[jt][j] = 0.f;
        store_T(acc[jt], Wh, Wl, G::ldW, it * 16, jt * 16);
      }
    }
    __syncthreads();

    // ---- stage 2: R = W K + Q S0 (old S0), then S0 += K^T K ----
#pragma unroll
    for (int sa = 0; sa < G::SA; ++sa) {
      const int at = w + kWaves * sa;
      if (at >= G::DT) break;
      f32x4 racc[G::RT];
#pragma unroll
      for (int rt = 0; rt < G::RT; ++rt) racc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag(Kt, G::ldKt, at * 16, s * 32);
#pragma unroll
        for (int rt = 0; rt < G::RT; ++rt) {
          racc[rt] = mfma(frag(Wh, G::ldW, rt * 16, s * 32), bK, racc[rt]);
          racc[rt] = mfma(frag(Wl, G::ldW, rt * 16, s * 32), bK, racc[rt]);
        }
      }
#pragma unroll
      for (int s = 0; s < G::KD; ++s) {
        bf16x8 bh, bl;
        frag_from_acc(S0[sa][2 * s], S0[sa][2 * s + 1], bh, bl);
#pragma unroll
        for (int rt = 0; rt < G::RT; ++rt) {
          const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, rt * 16, s * 32);
          racc[rt] = mfma(aQ, bh, racc[rt]);
          racc[rt] = mfma(aQ, bl, racc[rt]);
        }
      }
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag(Kt, G::ldKt, at * 16, s * 32);
#pragma unroll
        for (int rt = 0; rt < G::DT; ++rt) S0[sa][rt] = mfma(frag(Kt, G::ldKt, rt * 16, s * 32), bK, S0[sa][rt]);
      }
      // eta advance: column sums of R (applied after the readout has used the old eta)
      float cs = 0.f;
#pragma unroll
      for (int rt = 0; rt < G::RT; ++rt) cs += racc[rt][0] + racc[rt][1] + racc[rt][2] + racc[rt][3];
      cs += __shfl_xor(cs, 16);
      cs += __shfl_xor(cs, 32);
      if (lg == 0) colsum[at * 16 + lr] = cs;
#pragma unroll
      for (int rt = 0; rt < G::RT; ++rt) {
        store_T(racc[rt], Rth, Rtl, G::ldRt, rt * 16, at * 16);
        if (!SUMMARY) store_N(racc[rt], Rh, Rl, G::ldR, rt * 16, at * 16);
      }
    }
    __syncthreads();
    float eta_add = (tid < D) ? colsum[tid] : 0.f;

    if (!SUMMARY) {
      // ---- stage 3: T = L (.) Q R^T, computed as T^T = R Q^T, stored transposed into the W buffers ----
      for (int it = w; it < G::RT; it += kWaves) {
        f32x4 acc[G::RT];
#pragma unroll
        for (int jt = 0; jt < G::RT; ++jt) acc[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < G::KD; ++s) {
          const bf16x8 ah = frag(Rh, G::ldR, it * 16, s * 32);
          const bf16x8 al = frag(Rl, G::ldR, it * 16, s * 32);
#pragma unroll
          for (int jt = 0; jt < G::RT; ++jt) {
            const bf16x8 b = frag(Qs, G::ldQ, jt * 16, s * 32);
            acc[jt] = mfma(ah, b, acc[jt]);
            acc[jt] = mfma(al, b, acc[jt]);
          }
        }
#pragma unroll
        for (int jt = 0; jt < G::RT; ++jt) {
          float ps = 0.f;
#pragma unroll
          for (int j = 0; j < 4; ++j) {     // keep j <= t
            if (it * 16 + 4 * lg + j > jt * 16 + lr) acc[jt][j] = 0.f;
            ps += acc[jt][j];
          }
          ps += __shfl_xor(ps, 16);
          ps += __shfl_xor(ps, 32);
          if (lg == 0) denp[it * C + jt * 16 + lr] = ps;
          store_T(acc[jt], Wh, Wl, G::ldW, it * 16, jt * 16);
        }
      }
      __syncthreads();
      // den_t = sum_j T[t][j] + q_t . eta0
      if (normalized && tid < C) {
        float s = 0.f;
        for (int it = 0; it < G::RT; ++it) s += denp[it * C + tid];
        for (int a = 0; a < D; ++a) s += bf16_to_f(Qs[tid * G::ldQ + a]) * eta[a];
        den[tid] = s;
      }
      __syncthreads();
      // ---- stage 4: O = T V + Q Phi0 (old Phi0); stage 5: Phi0 += R^T V ----
#pragma unroll
      for (int sb = 0; sb < G::SB; ++sb) {
        const int bt = w + kWaves * sb;
        if (bt * 16 >= DV) break;
        f32x4 oacc[G::RT];
#pragma unroll
        for (int rt = 0; rt < G::RT; ++rt) oacc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < G::KC; ++s) {
          const bf16x8 bV = frag(Vt, G::ldVt, bt * 16, s * 32);
#pragma unroll
          for (int rt = 0; rt < G::RT; ++rt) {
            oacc[rt] = mfma(frag(Wh, G::ldW, rt * 16, s * 32), bV, oacc[rt]);
            oacc[rt] = mfma(frag(Wl, G::ldW, rt * 16, s * 32), bV, oacc[rt]);
          }
        }
#pragma unroll
        for (int s = 0; s < G::KD; ++s) {
          bf16x8 bh, bl;
          frag_from_acc(P0[sb][2 * s], P0[sb][2 * s + 1], bh, bl);
#pragma unroll
          for (int rt = 0; rt < G::RT; ++rt) {
            const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, rt * 16, s * 32);
            oacc[rt] = mfma(aQ, bh, oacc[rt]);
            oacc[rt] = mfma(aQ, bl, oacc[rt]);
          }
        }
#pragma unroll
        for (int rt = 0; rt < G::RT; ++rt)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int t = rt * 16 + 4 * lg + j;
            if (t0 + t < n) {
              float o = oacc[rt][j];
              if (normalized) o = o / (den[t] + eps);
              out[((size_t)bh * n + t0 + t) * DV + bt * 16 + lr] = o;
            }
          }
#pragma unroll
        for (int s = 0; s < G::KC; ++s) {
          const bf16x8 bV = frag(Vt, G::ldVt, bt * 16, s * 32);
#pragma unroll
          for (int rt = 0; rt < G::DT; ++rt) {
            P0[sb][rt] = mfma(frag(Rth, G::ldRt, rt * 16, s * 32), bV, P0[sb][rt]);
            P0[sb][rt] = mfma(frag(Rtl, G::ldRt, rt * 16, s * 32), bV, P0[sb][rt]);
          }
        }
      }
    } else {
      // summaries: Phi += R^T V and C += Q^T V
#pragma unroll
      for (int sb = 0; sb < G::SB; ++sb) {
        const int bt = w + kWaves * sb;
        if (bt * 16 >= DV) break;
#pragma unroll
        for (int s = 0; s < G::KC; ++s) {
          const bf16x8 bV = frag(Vt, G::ldVt, bt * 16, s * 32);
#pragma unroll
          for (int rt = 0; rt < G::DT; ++rt) {
            P0[sb][rt] = mfma(frag(Rth, G::ldRt, rt * 16, s * 32), bV, P0[sb][rt]);
            P0[sb][rt] = mfma(frag(Rtl, G::ldRt, rt * 16, s * 32), bV, P0[sb][rt]);
            Cs[SUMMARY ? sb : 0][rt] = mfma(frag(Qt, G::ldQt, rt * 16, s * 32), bV, Cs[SUMMARY ? sb : 0][rt]);
          }
        }
      }
    }
    __syncthreads();   // LDS tiles and den/eta are rewritten by the next chunk
    if (tid < D) eta[tid] += eta_add;
  }

  if (SUMMARY) {
    // record (S, C, m, Phi, eta): Phi in the G slot, eta in the h slot
    __syncthreads();
#pragma unroll
    for (int sa = 0; sa < G::SA; ++sa) {
      const int at = w + kWaves * sa;
      if (at >= G::DT) break;
#pragma unroll
      for (int rt = 0; rt < G::DT; ++rt)
        for (int j = 0; j < 4; ++j) rc[(size_t)(rt * 16 + 4 * lg + j) * D + at * 16 + lr] = S0[sa][rt][j];
    }
#pragma unroll
    for (int sb = 0; sb < G::SB; ++sb) {
      const int bt = w + kWaves * sb;
      if (bt * 16 >= DV) break;
#pragma unroll
      for (int rt = 0; rt < G::DT; ++rt)
        for (int j = 0; j < 4; ++j) {
          const size_t e = (size_t)(rt * 16 + 4 * lg + j) * DV + bt * 16 + lr;
          rc[off_G(D, DV) + e] = P0[sb][rt][j];
          rc[off_C(D, DV) + e] = Cs[SUMMARY ? sb : 0][rt][j];
        }
    }
    if (tid < D) {
      rc[off_m(D, DV) + tid] = m_acc;
      rc[off_h(D, DV) + tid] = eta[tid];
    }
  }
}

struct Shape {
  int C, D, DV;
};
constexpr Shape kShapes[] = {{64, 64, 64}, {32, 32, 32}, {64, 32, 32}, {32, 64, 64}, {64, 64, 32}, {64, 32, 64}};

template <int C, int D, int DV>
hipError_t run_shape(const Fwd& f, const float* init, float* final_state, char* ws, int P, int cps,
                     hipStream_t s) {
  const size_t F = state_floats(D, DV);
  const int BH = f.BH;
  float* segs = reinterpret_cast<float*>(ws);                    // [BH][P][F] segment summaries
  float* car = segs + (size_t)BH * P * F;                        // [BH][P][F] carries
  const uint16_t* q = static_cast<const uint16_t*>(f.q);
  const uint16_t* k = static_cast<const uint16_t*>(f.k);
  const uint16_t* v = static_cast<const uint16_t*>(f.v);
  const int nsum = final_state ? P : P - 1;                      // segments whose summary is needed
  const dim3 fblk((DV + 31) / 32);
  const size_t flds = sizeof(float) * D * 32;
  hipError_t e;
  if (nsum > 0) {
    auto ks = k_walk<C, D, DV, true>;
    const size_t lb = Cfg<C, D, DV, true>::bytes;
    if ((e = hipFuncSetAttribute((const void*)ks, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lb)) != hipSuccess)
      return e;
    prof_start("walk_summary", s);
    hipLaunchKernelGGL(ks, dim3(nsum, BH), dim3(kThreads), lb, s, q, k, v, (float*)nullptr, segs, f.n, cps, P, 0,
                       0.f);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    prof_start("flip", s);
    hipLaunchKernelGGL(k_flip, dim3(BH * nsum, fblk.x), dim3(256), flds, s, segs, segs, nsum, P, P, D, DV);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // carries: prefix of segment c at car[c]; the total goes to the final
    // state, or (when only P-1 summaries exist) is the carry of segment P-1
    prof_start("scan", s);
    if (final_state)
      e = launch_scan_strided(segs, init, car, final_state, BH, nsum, D, DV, (size_t)P * F, (size_t)P * F, F, s);
    else
      e = launch_scan_strided(segs, init, car, car + (size_t)(P - 1) * F, BH, nsum, D, DV, (size_t)P * F,
                              (size_t)P * F, (size_t)P * F, s);
    prof_stop(s);
    if (e != hipSuccess) return e;
  }
  if (!f.out) return hipSuccess;
  if (nsum > 0) {
    prof_start("flip", s);
    hipLaunchKernelGGL(k_flip, dim3(BH * P, fblk.x), dim3(256), flds, s, car, car, P, P, P, D, DV);
    prof_stop(s);
  } else if (init) {
    prof_start("flip", s);
    hipLaunchKernelGGL(k_flip, dim3(BH, fblk.x), dim3(256), flds, s, init, car, 1, 1, P, D, DV);
    prof_stop(s);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  auto kw = k_walk<C, D, DV, false>;
  const size_t lb = Cfg<C, D, DV, false>::bytes;
  if ((e = hipFuncSetAttribute((const void*)kw, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lb)) != hipSuccess)
    return e;
  prof_start("walk", s);
  hipLaunchKernelGGL(kw, dim3(P, BH), dim3(kThreads), lb, s, q, k, v, f.out,
                     (nsum > 0 || init) ? car : (float*)nullptr, f.n, cps, P, f.normalized, f.eps);
  prof_stop(s);
  return hipGetLastError();
}

}  // namespace

void fused_plan(int BH, int n, int chunk, int* P, int* cps) {
  const int M = (n + chunk - 1) / chunk;
  int p = 256 / BH;                       // about one workgroup per CU
  if (const char* e = getenv("HLA_FUSED_SEGMENTS")) p = atoi(e);
  if (p < 1) p = 1;
  if (p > M) p = M;
  *cps = (M + p - 1) / p;
  *P = (M + *cps - 1) / *cps;             // every segment non-empty
}

bool fused_supported(int n, int d, int dv, int chunk, int dtype, int masked) {
  if (dtype != 1 || masked != 1 || n < 1) return false;
  for (const Shape& sh : kShapes)
    if (sh.C == chunk && sh.D == d && sh.DV == dv) return true;
  return false;
}

size_t fused_workspace_bytes(int BH, int n, int d, int dv, int chunk) {
  int P, cps;
  fused_plan(BH, n, chunk, &P, &cps);
  return 2 * sizeof(float) * (size_t)BH * P * state_floats(d, dv) + 256;
}

hipError_t launch_fused(const Fwd& f, const float* init, float* final_state, void* workspace, hipStream_t s) {
  int P, cps;
  fused_plan(f.BH, f.n, f.chunk, &P, &cps);
  char* ws = static_cast<char*>(workspace);
#define HLA_SHAPE(C_, D_, DV_) \
  if (f.chunk == C_ && f.d == D_ && f.dv == DV_) return run_shape<C_, D_, DV_>(f, init, final_state, ws, P, cps, s);
  HLA_SHAPE(64, 64, 64)
  HLA_SHAPE(32, 32, 32)
  HLA_SHAPE(64, 32, 32)
  HLA_SHAPE(32, 64, 64)
  HLA_SHAPE(64, 64, 32)
  HLA_SHAPE(64, 32, 64)
#undef HLA_SHAPE
  return hipErrorNotSupported;
}

}  // namespace hla
