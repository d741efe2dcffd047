// Fused masked second-order HLA forward for bf16 inputs on gfx950 MFMA.
//
// Algorithm (Sec. 4, two-level scan, Rem. scan-modes; Thm. 1 readout):
// the sequence of every head is cut into P segments of whole chunks.
//   1. k_walk<SUMMARY>: each workgroup walks one segment from a zero carry and
//      produces its summary (S, C, m, Phi, eta) with Phi = S C - G and
//      eta = S m - h (an exact change of variables of the 5-tuple).
//   2. k_carry takes the exclusive semidirect-product scan over the segments
//      of each head on the paper's 5-tuples, Eq. (semidirect), reading the
//      summaries through G = S C - Phi, h = S m - eta and writing each carry
//      back as (S0, Phi0 = S0 C0 - G0, eta0 = S0 m0 - h0).
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
// Layout: 512 threads = 8 waves.  Wave w owns the 16-column tiles
// {w%4, w%4+4, ...} of S0, R (over d) and of Phi0, O (over dv), and half of
// the token tiles of R and O; S0 and Phi0 stay in MFMA accumulators for the
// whole walk and are fed back as MFMA B operands straight from registers.  Q, K, K^T, V^T, W/T, R and R^T are
// staged in LDS as bf16.
#include "fused.h"
#include "profile.h"

namespace hla {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint16_t u16x4;

constexpr int kWaves = 8;
constexpr int kColWaves = 4;              // waves that split the state columns
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
  static constexpr int n16 = oQt + (SUMMARY ? D * ldQt : 0);          // bf16 elements of tiles
  // the output walk folds its carry in fp32 scratch that reuses the tile region
  static constexpr int fold_f = SUMMARY ? 0 : 2 * D * (D + 2) + 2 * D * DV + 2 * D;
  static constexpr int n16t = (n16 > 2 * fold_f ? n16 : 2 * fold_f);
  static constexpr int f_eta = 0, f_cs = D, f_den = 3 * D, f_denp = 3 * D + C;   // fp32 region
  static constexpr int nf32 = 3 * D + C + (C / 16) * C;
  static constexpr size_t bytes = (size_t)((n16t + 7) & ~7) * 2 + (size_t)nf32 * 4;
  static constexpr int RT = C / 16;                  // token tiles
  static constexpr int SA = (D / 16 + kColWaves - 1) / kColWaves;   // column tiles of S0/R per wave
  static constexpr int SB = (DV / 16 + kColWaves - 1) / kColWaves;  // column tiles of Phi0/O per wave
  static constexpr int DT = D / 16;
  static constexpr int KC = C / 32, KD = D / 32;
  // global->LDS staging: 16-byte segments per operand
  static constexpr int segQ = C * D / 8, segV = C * DV / 8;
  static constexpr int pfQ = (segQ + kThreads - 1) / kThreads, pfV = (segV + kThreads - 1) / kThreads;
  static_assert(C % 32 == 0 && D % 32 == 0 && DV % 16 == 0, "tile shape");
  static_assert(bytes <= 160 * 1024, "LDS budget");
};

// k_carry: the carries of all segments of a head, by the exclusive
// semidirect-product scan of Eq. (semidirect) over the paper's 5-tuples,
// with the conversions to and from the walk's (S, Phi, eta) form folded in.
//   acc = init (or E); for s < nsum:
//     car[s]  = (S_acc, C_acc, m_acc, S_acc C_acc - G_acc, S_acc m_acc - h_acc)
//     seg s arrives as (S_s, C_s, m_s, Phi_s, eta_s); its G_s = S_s C_s - Phi_s,
//     acc (+)= seg:  G_acc += G_s + S_s C_acc = S_s (C_s + C_acc) - Phi_s + G_acc
//                    h_acc += S_s (m_s + m_acc) - eta_s + ...,  S, C, m add.
//   after the loop: car[nsum] (when nsum < P) in walk form, or the total in
//   5-tuple form to `fin`.
// One workgroup per (head, block of CB value columns); a head's blocks share
// an XCD.  Every workgroup keeps its own S_acc (registers, 64 per thread at
// d = 128) because every column block needs all of it.
template <int d, int dv, int CB>
__global__ __launch_bounds__(256) void k_carry(const float* __restrict__ segs, const float* __restrict__ init,
                                               float* __restrict__ car, float* __restrict__ fin, int BH, int nsum,
                                               int P) {
  constexpr int nblk = (dv + CB - 1) / CB;
  extern __shared__ float sm[];
  const int ldS = d + 4;
  float* XT = sm;                 // [d][d+4]  transposed S_acc or S_s
  float* Cacc = XT + d * ldS;     // [d][CB]
  float* Ybuf = Cacc + d * CB;    // [d][CB]
  float* macc = Ybuf + d * CB;    // [d]
  float* mbuf = macc + d;         // [d]
  const int tid = threadIdx.x;
  const int L = blockIdx.x;
  const int group = L / (8 * nblk), within = L % (8 * nblk);
  const int bh = group * 8 + within % 8, blk = within / 8;
  if (bh >= BH) return;
  const int c0 = blk * CB, ncol = min(CB, dv - c0);
  const size_t F = state_floats(d, dv);
  const size_t oC = off_C(d, dv), om = off_m(d, dv), oG = off_G(d, dv), oh = off_h(d, dv);
  const float* ini = init ? init + (size_t)bh * F : nullptr;
  const int nj4 = CB / 4, jq = tid % nj4, aq = tid / nj4;
  const bool active = (aq * 4 < d) && (jq * 4 < ncol);
  constexpr int nS = (d * d + 255) / 256;
  float sacc[nS];
  float gacc[4][4];
  float hacc = 0.f;
#pragma unroll
  for (int r = 0; r < nS; ++r) {
    const int idx = tid + 256 * r;
    sacc[r] = (ini && idx < d * d) ? ini[idx] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      gacc[i][j] = (ini && active) ? ini[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j] : 0.f;
#pragma unroll
  for (int idx = tid; idx < d * CB; idx += 256) {
    const int a = idx / CB, j = idx % CB;
    Cacc[idx] = (ini && j < ncol) ? ini[oC + (size_t)a * dv + c0 + j] : 0.f;
  }
  for (int a = tid; a < d; a += 256) macc[a] = ini ? ini[om + a] : 0.f;
  if (tid < d && ini) hacc = ini[oh + tid];

  // out[i][j] = sum_a' X[a0+i][a'] Y[a'][j0+j] with X staged transposed in XT
  auto product = [&](const float* Y, float acc[4][4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
#pragma unroll 8
    for (int ap = 0; ap < d; ++ap) {
      const float4 x4 = *reinterpret_cast<const float4*>(&XT[ap * ldS + aq * 4]);
      const float4 y4 = *reinterpret_cast<const float4*>(&Y[ap * CB + jq * 4]);
      const float xv[4] = {x4.x, x4.y, x4.z, x4.w}, yv[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += xv[i] * yv[j];
    }
  };
  auto stage_sacc = [&]() {
#pragma unroll
    for (int r = 0; r < nS; ++r) {
      const int idx = tid + 256 * r;
      if (idx < d * d) XT[(idx % d) * ldS + idx / d] = sacc[r];
    }
  };
  // write the acc state in walk form to dst (S, C, m copied; Phi, eta converted)
  auto write_walk_form = [&](float* dst) {
    __syncthreads();
    stage_sacc();
    __syncthreads();
    if (active) {
      float pr[4][4];
      product(Cacc, pr);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          dst[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j] = pr[i][j] - gacc[i][j];
    }
#pragma unroll
    for (int idx = tid; idx < d * CB; idx += 256) {
      const int a = idx / CB, j = idx % CB;
      if (j < ncol) dst[oC + (size_t)a * dv + c0 + j] = Cacc[idx];
    }
    if (blk == 0) {
#pragma unroll
      for (int r = 0; r < nS; ++r) {
        const int idx = tid + 256 * r;
        if (idx < d * d) dst[idx] = sacc[r];
      }
      if (tid < d) {
        float e = 0.f;
#pragma unroll 8
        for (int ap = 0; ap < d; ++ap) e += XT[ap * ldS + tid] * macc[ap];
        dst[om + tid] = macc[tid];
        dst[oh + tid] = e - hacc;
      }
    }
  };

  for (int sg = 0; sg < nsum; ++sg) {
    if (car) write_walk_form(car + ((size_t)bh * P + sg) * F);
    const float* x = segs + ((size_t)bh * P + sg) * F;
    __syncthreads();
    {
      // issue every global load of the segment before its first use
      constexpr int nSS = (d * d + 255) / 256, nCC = (d * CB + 255) / 256;
      float sv[nSS], cv[nCC];
#pragma unroll
      for (int r = 0; r < nSS; ++r) {
        const int idx = tid + 256 * r;
        sv[r] = idx < d * d ? x[idx] : 0.f;
      }
#pragma unroll
      for (int r = 0; r < nCC; ++r) {
        const int idx = tid + 256 * r, a = idx / CB, j = idx % CB;
        cv[r] = (idx < d * CB && j < ncol) ? x[oC + (size_t)a * dv + c0 + j] : 0.f;
      }
      const float mv = tid < d ? x[om + tid] : 0.f;
#pragma unroll
      for (int r = 0; r < nSS; ++r) {
        const int idx = tid + 256 * r;
        if (idx < d * d) XT[(idx % d) * ldS + idx / d] = sv[r];
      }
#pragma unroll
      for (int r = 0; r < nCC; ++r) {
        const int idx = tid + 256 * r;
        if (idx < d * CB) Ybuf[idx] = Cacc[idx] + cv[r];
      }
      if (tid < d) mbuf[tid] = macc[tid] + mv;
    }
    __syncthreads();
    if (active) {
      float phi[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) phi[i][j] = x[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j];
      float pr[4][4];
      product(Ybuf, pr);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) gacc[i][j] += pr[i][j] - phi[i][j];
    }
    if (tid < d) {
      const float eta_s = x[oh + tid];
      float e = 0.f;
#pragma unroll 8
      for (int ap = 0; ap < d; ++ap) e += XT[ap * ldS + tid] * mbuf[ap];
      hacc += e - eta_s;
    }
#pragma unroll
    for (int r = 0; r < nS; ++r) {
      const int idx = tid + 256 * r;
      if (idx < d * d) sacc[r] += XT[(idx % d) * ldS + idx / d];
    }
    __syncthreads();
#pragma unroll
    for (int idx = tid; idx < d * CB; idx += 256) Cacc[idx] = Ybuf[idx];
    if (tid < d) macc[tid] = mbuf[tid];
  }
  if (car && nsum < P) write_walk_form(car + ((size_t)bh * P + nsum) * F);
  if (fin) {
    float* dst = fin + (size_t)bh * F;
    __syncthreads();
    if (active)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) dst[oG + (size_t)(aq * 4 + i) * dv + c0 + jq * 4 + j] = gacc[i][j];
#pragma unroll
    for (int idx = tid; idx < d * CB; idx += 256) {
      const int a = idx / CB, j = idx % CB;
      if (j < ncol) dst[oC + (size_t)a * dv + c0 + j] = Cacc[idx];
    }
    if (blk == 0) {
#pragma unroll
      for (int r = 0; r < nS; ++r) {
        const int idx = tid + 256 * r;
        if (idx < d * d) dst[idx] = sacc[r];
      }
      if (tid < d) {
        dst[om + tid] = macc[tid];
        dst[oh + tid] = hacc;
      }
    }
  }
}

// Carry of segment `seg` of head bh, folded by the workgroup itself:
//   acc = init (+) seg_0 (+) ... (+) seg_{seg-1}     (Eq. (semidirect) on 5-tuples)
// where segment summaries arrive as (S, C, m, Phi, eta) and G_s = S_s C_s -
// Phi_s, h_s = S_s m_s - eta_s, so the cross term S_s C_acc and G_s combine
// into one product: G_acc += S_s (C_s + C_acc) - Phi_s.  The carry is then
// converted once: Phi0 = S_acc C_acc - G_acc, eta0 = S_acc m_acc - h_acc.
// S matrices are kept transposed in LDS ([a'][a], row length D+2) so a thread
// reads the two rows of its 2 x 4 output block as one 8-byte load.
// Results: S_acc^T in `Sout`, Phi0 in `Pout` [D][DV], eta0 in `eout`.
template <int D, int DV>
__device__ void fold_carry(const float* __restrict__ segs, const float* __restrict__ init, int bh, int seg,
                           int nseg, float* sc, float*& Sout, float*& Pout, float* eout) {
  constexpr int ldT = D + 2;
  constexpr int NB4 = DV / 4;                   // column quads
  constexpr int NT = (D / 2) * NB4;             // threads with a 2 x 4 output block
  static_assert(NT <= kThreads, "product split");
  const size_t F = state_floats(D, DV);
  float* SaccT = sc;                  // [D][D+2]
  float* SsT = SaccT + D * ldT;       // [D][D+2]
  float* Cacc = SsT + D * ldT;        // [D][DV]
  float* Y = Cacc + D * DV;           // [D][DV]
  float* macc = Y + D * DV;           // [D]
  float* y = macc + D;                // [D]
  const int tid = threadIdx.x;
  const bool act = tid < NT;
  const int a0 = act ? 2 * (tid / NB4) : 0, b0 = 4 * (tid % NB4);
  const float* ini = init ? init + (size_t)bh * F : nullptr;
  float g[2][4];
  float h = 0.f;
  for (int idx = tid; idx < D * D; idx += kThreads) SaccT[(idx % D) * ldT + idx / D] = ini ? ini[idx] : 0.f;
  for (int idx = tid; idx < D * DV; idx += kThreads) Cacc[idx] = ini ? ini[off_C(D, DV) + idx] : 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) g[i][j] = (ini && act) ? ini[off_G(D, DV) + (size_t)(a0 + i) * DV + b0 + j] : 0.f;
  if (tid < D) {
    macc[tid] = ini ? ini[off_m(D, DV) + tid] : 0.f;
    h = ini ? ini[off_h(D, DV) + tid] : 0.f;
  }
  // out[i][j] = sum_a' X[a0+i][a'] Z[a'][b0+j] with X^T in XT
  auto prod = [&](const float* XT, const float* Z, float o[2][4]) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) o[i][j] = 0.f;
#pragma unroll 8
    for (int ap = 0; ap < D; ++ap) {
      const float2 x2 = *reinterpret_cast<const float2*>(&XT[ap * ldT + a0]);
      const float4 z4 = *reinterpret_cast<const float4*>(&Z[ap * DV + b0]);
      const float xv[2] = {x2.x, x2.y}, zv[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[i][j] += xv[i] * zv[j];
    }
  };
  for (int sp = 0; sp < seg; ++sp) {
    const float* x = segs + ((size_t)bh * nseg + sp) * F;
    float phi[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) phi[i][j] = act ? x[off_G(D, DV) + (size_t)(a0 + i) * DV + b0 + j] : 0.f;
    const float eta_s = tid < D ? x[off_h(D, DV) + tid] : 0.f;
    __syncthreads();
    for (int idx = tid; idx < D * D; idx += kThreads) SsT[(idx % D) * ldT + idx / D] = x[idx];
    for (int idx = tid; idx < D * DV; idx += kThreads) Y[idx] = Cacc[idx] + x[off_C(D, DV) + idx];
    if (tid < D) y[tid] = macc[tid] + x[off_m(D, DV) + tid];
    __syncthreads();
    if (act) {
      float o[2][4];
      prod(SsT, Y, o);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) g[i][j] += o[i][j] - phi[i][j];
    }
    if (tid < D) {
      float acc = 0.f;
#pragma unroll 8
      for (int ap = 0; ap < D; ++ap) acc += SsT[ap * ldT + tid] * y[ap];
      h += acc - eta_s;
    }
    __syncthreads();
    for (int idx = tid; idx < D * D; idx += kThreads) {
      const int o = (idx / D) * ldT + idx % D;
      SaccT[o] += SsT[o];
    }
    for (int idx = tid; idx < D * DV; idx += kThreads) Cacc[idx] = Y[idx];
    if (tid < D) macc[tid] = y[tid];
  }
  __syncthreads();
  // Phi0 = S_acc C_acc - G_acc (into Y), eta0 = S_acc m_acc - h_acc
  if (act) {
    float o[2][4];
    prod(SaccT, Cacc, o);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Y[(a0 + i) * DV + b0 + j] = o[i][j] - g[i][j];
  }
  if (tid < D) {
    float acc = 0.f;
#pragma unroll 8
    for (int ap = 0; ap < D; ++ap) acc += SaccT[ap * ldT + tid] * macc[ap];
    eout[tid] = acc - h;
  }
  __syncthreads();
  Sout = SaccT;
  Pout = Y;
}

// One segment walk.  grid = (segments, BH), 8 waves.  Wave w owns column
// tile ct = w % 4 (+4, +8, ... when d or dv > 64) of S0/R and of Phi0/O, and
// the row half rh = w / 4 of the token tiles of R and O.  Both row halves keep
// a full copy of the S0/Phi0 columns they own (the carry updates are done by
// both), so every B operand taken from the carry stays in registers.
// SUMMARY: zero carry, writes the segment summary (S, C, m, Phi, eta) to
// `rec`.  !SUMMARY: reads the carry (S0, ., ., Phi0, eta0) from `rec` (NULL =
// zero) and writes outputs.
template <int C, int D, int DV, bool SUMMARY>
__global__ __launch_bounds__(kThreads, 1) void k_walk(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v, float* __restrict__ out,
                                                      float* __restrict__ rec, const float* __restrict__ init, int n,
                                                      int cps, int nseg, int normalized, float eps) {
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
  float* fl = reinterpret_cast<float*>(lds + ((G::n16t + 7) & ~7));
  float* eta = fl + G::f_eta;
  float* colsum = fl + G::f_cs;       // [2][D]: per row half
  float* den = fl + G::f_den;
  float* denp = fl + G::f_denp;

  const int seg = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const int ct = w % kColWaves, rh = w / kColWaves;
  constexpr int RH = G::RT / 2;                // token tiles per row half
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t F = state_floats(D, DV);
  float* rc = SUMMARY ? rec + ((size_t)bh * nseg + seg) * F : nullptr;

  // ---- carry in (fp32 accumulators) ----
  f32x4 S0[G::SA][G::DT];
  f32x4 P0[G::SB][G::DT];
  f32x4 Cs[SUMMARY ? G::SB : 1][G::DT];
#pragma unroll
  for (int sa = 0; sa < G::SA; ++sa)
#pragma unroll
    for (int rt = 0; rt < G::DT; ++rt) S0[sa][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int sb = 0; sb < G::SB; ++sb)
#pragma unroll
    for (int rt = 0; rt < G::DT; ++rt) {
      P0[sb][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (SUMMARY) Cs[SUMMARY ? sb : 0][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  for (int a = tid; a < D; a += kThreads) eta[a] = 0.f;
  if (!SUMMARY && (seg > 0 || init)) {
    // the tile region of LDS is free until the first chunk is staged
    float* Sc;
    float* Pc;
    fold_carry<D, DV>(rec, init, bh, seg, nseg, reinterpret_cast<float*>(lds), Sc, Pc, eta);
#pragma unroll
    for (int sa = 0; sa < G::SA; ++sa) {
      const int at = ct + kColWaves * sa;
      if (at >= G::DT) break;
#pragma unroll
      for (int rt = 0; rt < G::DT; ++rt)
#pragma unroll
        for (int j = 0; j < 4; ++j) S0[sa][rt][j] = Sc[(at * 16 + lr) * (D + 2) + rt * 16 + 4 * lg + j];
    }
#pragma unroll
    for (int sb = 0; sb < G::SB; ++sb) {
      const int bt = ct + kColWaves * sb;
      if (bt * 16 >= DV) break;
#pragma unroll
      for (int rt = 0; rt < G::DT; ++rt)
#pragma unroll
        for (int j = 0; j < 4; ++j) P0[sb][rt][j] = Pc[(rt * 16 + 4 * lg + j) * DV + bt * 16 + lr];
    }
    __syncthreads();
  }
  float m_acc = 0.f;   // SUMMARY: column sum of Q for column tid (< D)

  // ---- prefetch registers for the next chunk ----
  uint4 pq[G::pfQ], pk[G::pfQ], pv[G::pfV];
  auto fetch = [&](int c) {
    const int t0 = c * C;
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + kThreads * i;
      const int t = e % C, a8 = (e / C) * 8;     // consecutive lanes take consecutive tokens
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
      const int t = e % C, b8 = (e / C) * 8;
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
        const int t = e % C, a8 = (e / C) * 8;
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
        const int t = e % C, b8 = (e / C) * 8;
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
    for (int tile = w; tile < G::RT * G::RT; tile += kWaves) {
      const int it = tile % G::RT, jt = tile / G::RT;
      if (it > jt) {          // tile entirely above the diagonal of W^T (key after query): zero
        store_T(f32x4{0.f, 0.f, 0.f, 0.f}, Wh, Wl, G::ldW, it * 16, jt * 16);
        continue;
      }
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < G::KD; ++s) acc = mfma(frag(Ks, G::ldK, it * 16, s * 32), frag(Qs, G::ldQ, jt * 16, s * 32), acc);
#pragma unroll
      for (int j = 0; j < 4; ++j)   // keep key i <= query t
        if (it * 16 + 4 * lg + j > jt * 16 + lr) acc[j] = 0.f;
      store_T(acc, Wh, Wl, G::ldW, it * 16, jt * 16);
    }
    __syncthreads();

    // ---- stage 2: R = W K + Q S0 (old S0) on this wave's row half; S0 += K^T K ----
#pragma unroll
    for (int sa = 0; sa < G::SA; ++sa) {
      const int at = ct + kColWaves * sa;
      if (at >= G::DT) break;
      f32x4 racc[RH];
#pragma unroll
      for (int r = 0; r < RH; ++r) racc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag(Kt, G::ldKt, at * 16, s * 32);
#pragma unroll
        for (int r = 0; r < RH; ++r) {
          const int rt = rh * RH + r;
          if (s * 32 > rt * 16 + 15) continue;   // W row tile rt has no keys at or beyond s*32
          racc[r] = mfma(frag(Wh, G::ldW, rt * 16, s * 32), bK, racc[r]);
          racc[r] = mfma(frag(Wl, G::ldW, rt * 16, s * 32), bK, racc[r]);
        }
      }
#pragma unroll
      for (int s = 0; s < G::KD; ++s) {
        bf16x8 bh, bl;
        frag_from_acc(S0[sa][2 * s], S0[sa][2 * s + 1], bh, bl);
#pragma unroll
        for (int r = 0; r < RH; ++r) {
          const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, (rh * RH + r) * 16, s * 32);
          racc[r] = mfma(aQ, bh, racc[r]);
          racc[r] = mfma(aQ, bl, racc[r]);
        }
      }
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag(Kt, G::ldKt, at * 16, s * 32);
#pragma unroll
        for (int rt = 0; rt < G::DT; ++rt) S0[sa][rt] = mfma(frag(Kt, G::ldKt, rt * 16, s * 32), bK, S0[sa][rt]);
      }
      // eta advance: column sums of R over this row half
      float cs = 0.f;
#pragma unroll
      for (int r = 0; r < RH; ++r) cs += racc[r][0] + racc[r][1] + racc[r][2] + racc[r][3];
      cs += __shfl_xor(cs, 16);
      cs += __shfl_xor(cs, 32);
      if (lg == 0) colsum[rh * D + at * 16 + lr] = cs;
#pragma unroll
      for (int r = 0; r < RH; ++r) {
        const int rt = rh * RH + r;
        store_T(racc[r], Rth, Rtl, G::ldRt, rt * 16, at * 16);
        if (!SUMMARY) store_N(racc[r], Rh, Rl, G::ldR, rt * 16, at * 16);
      }
    }
    __syncthreads();
    const float eta_add = (tid < D) ? colsum[tid] + colsum[D + tid] : 0.f;

    if (!SUMMARY) {
      // ---- stage 3: T = L (.) Q R^T, computed as T^T = R Q^T, stored transposed into the W buffers ----
      for (int tile = w; tile < G::RT * G::RT; tile += kWaves) {
        const int it = tile % G::RT, jt = tile / G::RT;
        if (it > jt) {
          store_T(f32x4{0.f, 0.f, 0.f, 0.f}, Wh, Wl, G::ldW, it * 16, jt * 16);
          if (lg == 0) denp[it * C + jt * 16 + lr] = 0.f;
          continue;
        }
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < G::KD; ++s) {
          const bf16x8 b = frag(Qs, G::ldQ, jt * 16, s * 32);
          acc = mfma(frag(Rh, G::ldR, it * 16, s * 32), b, acc);
          acc = mfma(frag(Rl, G::ldR, it * 16, s * 32), b, acc);
        }
        float ps = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {     // keep j <= t
          if (it * 16 + 4 * lg + j > jt * 16 + lr) acc[j] = 0.f;
          ps += acc[j];
        }
        ps += __shfl_xor(ps, 16);
        ps += __shfl_xor(ps, 32);
        if (lg == 0) denp[it * C + jt * 16 + lr] = ps;
        store_T(acc, Wh, Wl, G::ldW, it * 16, jt * 16);
      }
      __syncthreads();
      // den_t = sum_j T[t][j] + q_t . eta0
      if (normalized && tid < C) {
        float s = 0.f;
        for (int it = 0; it < G::RT; ++it) s += denp[it * C + tid];
        for (int a = 0; a < D; ++a) s += bf16_to_f(Qs[tid * G::ldQ + a]) * eta[a];
        den[tid] = 1.f / (s + eps);
      }
      __syncthreads();
      // ---- stage 4: O = T V + Q Phi0 (old Phi0); stage 5: Phi0 += R^T V ----
#pragma unroll
      for (int sb = 0; sb < G::SB; ++sb) {
        const int bt = ct + kColWaves * sb;
        if (bt * 16 >= DV) break;
        f32x4 oacc[RH];
#pragma unroll
        for (int r = 0; r < RH; ++r) oacc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < G::KC; ++s) {
          const bf16x8 bV = frag(Vt, G::ldVt, bt * 16, s * 32);
#pragma unroll
          for (int r = 0; r < RH; ++r) {
            const int rt = rh * RH + r;
            if (s * 32 > rt * 16 + 15) continue;   // T row tile rt has no j at or beyond s*32
            oacc[r] = mfma(frag(Wh, G::ldW, rt * 16, s * 32), bV, oacc[r]);
            oacc[r] = mfma(frag(Wl, G::ldW, rt * 16, s * 32), bV, oacc[r]);
          }
        }
#pragma unroll
        for (int s = 0; s < G::KD; ++s) {
          bf16x8 bh, bl;
          frag_from_acc(P0[sb][2 * s], P0[sb][2 * s + 1], bh, bl);
#pragma unroll
          for (int r = 0; r < RH; ++r) {
            const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, (rh * RH + r) * 16, s * 32);
            oacc[r] = mfma(aQ, bh, oacc[r]);
            oacc[r] = mfma(aQ, bl, oacc[r]);
          }
        }
#pragma unroll
        for (int r = 0; r < RH; ++r)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int t = (rh * RH + r) * 16 + 4 * lg + j;
            if (t0 + t < n) {
              float o = oacc[r][j];
              if (normalized) o *= den[t];
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
        const int bt = ct + kColWaves * sb;
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

  if (SUMMARY && rh == 0) {
    // record (S, C, m, Phi, eta): Phi in the G slot, eta in the h slot
#pragma unroll
    for (int sa = 0; sa < G::SA; ++sa) {
      const int at = ct + kColWaves * sa;
      if (at >= G::DT) break;
#pragma unroll
      for (int rt = 0; rt < G::DT; ++rt)
        for (int j = 0; j < 4; ++j) rc[(size_t)(rt * 16 + 4 * lg + j) * D + at * 16 + lr] = S0[sa][rt][j];
    }
#pragma unroll
    for (int sb = 0; sb < G::SB; ++sb) {
      const int bt = ct + kColWaves * sb;
      if (bt * 16 >= DV) break;
#pragma unroll
      for (int rt = 0; rt < G::DT; ++rt)
        for (int j = 0; j < 4; ++j) {
          const size_t e = (size_t)(rt * 16 + 4 * lg + j) * DV + bt * 16 + lr;
          rc[off_G(D, DV) + e] = P0[sb][rt][j];
          rc[off_C(D, DV) + e] = Cs[SUMMARY ? sb : 0][rt][j];
        }
    }
  }
  if (SUMMARY) {
    __syncthreads();
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
  const uint16_t* q = static_cast<const uint16_t*>(f.q);
  const uint16_t* k = static_cast<const uint16_t*>(f.k);
  const uint16_t* v = static_cast<const uint16_t*>(f.v);
  const int nsum = final_state ? P : P - 1;                      // segments whose summary is needed
  hipError_t e;
  if (nsum > 0) {
    auto ks = k_walk<C, D, DV, true>;
    const size_t lb = Cfg<C, D, DV, true>::bytes;
    if ((e = hipFuncSetAttribute((const void*)ks, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lb)) != hipSuccess)
      return e;
    prof_start("walk_summary", s);
    hipLaunchKernelGGL(ks, dim3(nsum, BH), dim3(kThreads), lb, s, q, k, v, (float*)nullptr, segs,
                       (const float*)nullptr, f.n, cps, P, 0, 0.f);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const bool want_out = f.out != nullptr;
  if (final_state) {
    // total state after all P segments: the semidirect-product fold in k_carry
    constexpr int CB = (4096 / D < DV) ? 4096 / D : DV;
    constexpr int nblk = (DV + CB - 1) / CB;
    const size_t lds = sizeof(float) * ((size_t)D * (D + 4) + 2 * (size_t)D * CB + 2 * D);
    auto kc = k_carry<D, DV, CB>;
    if ((e = hipFuncSetAttribute((const void*)kc, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) !=
        hipSuccess)
      return e;
    prof_start("carry", s);
    hipLaunchKernelGGL(kc, dim3(((BH + 7) / 8) * 8 * nblk), dim3(256), lds, s, segs, init, (float*)nullptr,
                       final_state, BH, nsum, P);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (!want_out) return hipSuccess;
  auto kw = k_walk<C, D, DV, false>;
  const size_t lb = Cfg<C, D, DV, false>::bytes;
  if ((e = hipFuncSetAttribute((const void*)kw, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lb)) != hipSuccess)
    return e;
  prof_start("walk", s);
  hipLaunchKernelGGL(kw, dim3(P, BH), dim3(kThreads), lb, s, q, k, v, f.out, segs, init, f.n, cps, P,
                     f.normalized, f.eps);
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
  return sizeof(float) * (size_t)BH * P * state_floats(d, dv) + 256;
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
