// Fused masked second-order HLA forward for bf16 inputs on gfx950 MFMA.
//
// Algorithm (Sec. 4, two-level scan, Rem. scan-modes; Thm. 1 readout):
// the sequence of every head is cut into P segments of whole chunks.
//   1. k_walk<SUMMARY>: each workgroup walks one segment from a zero carry and
//      produces its summary (S, C, m, Phi, eta) with Phi = S C - G and
//      eta = S m - h (an exact change of variables of the 5-tuple).
//   2. k_seg_cross: the semidirect product of Eq. (semidirect) across
//      segments in reduce-then-scan form: each segment's contribution
//      G_s + S_s C_{<s} (and h_s + S_s m_{<s}) is computed in parallel.
//   3. k_walk<OUTPUT>: each workgroup sums the contributions before its
//      segment into its carry (fold_sum), converts it once to (S0, Phi0, eta0),
//      walks its chunks from that carry and writes the outputs.
//   k_total sums all contributions into the total state when a caller needs it.
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
// Layout: 256 threads = 4 waves on v_mfma_f32_32x32x16_bf16.  Every product
// of a chunk is at most 2 x 2 tiles of 32 x 32; wave w owns output tile
// (row w/2, column w%2).  The wave owning column c of R (or O) keeps the whole
// column c of S0 (or Phi0) in MFMA accumulators for the whole walk and feeds
// it back as the B operand straight from registers (both row waves of a
// column keep a copy).  Q, K, K^T, V^T, W/T, R and R^T are staged in LDS as
// bf16.
#include "fused.h"
#include "profile.h"

namespace hla {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

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
__device__ __forceinline__ uint32_t pack2(uint16_t a, uint16_t b) { return a | (uint32_t)b << 16; }

// Lane layout of v_mfma_f32_32x32x16_bf16 (l = lane, r = l % 32, g = l / 32):
//   A: row r, k = 8g .. 8g+7;  B: column r, the same k (any k order shared by
//   A and B gives the same product);  D: element e is D[8(e/4) + 4g + e%4][r].
__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int e = 0; e < 16; ++e) z[e] = 0.f;
  return z;
}
__device__ __forceinline__ int acc_row(int e, int g) { return 8 * (e >> 2) + 4 * g + (e & 3); }

// Operand fragment from a row-major bf16 LDS tile X[row][k]: lane takes
// X[row0 + r][k0 + 8g .. 8g+7].  A operand of X Y, or B operand of Z X^T.
__device__ __forceinline__ bf16x8 frag(const uint16_t* X, int ld, int row0, int k0) {
  const int l = threadIdx.x & 63;
  const uint16_t* p = X + (row0 + (l & 31)) * ld + k0 + 8 * (l >> 5);
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// Same, in the k order of an accumulator-fed partner: lane takes
// X[row0 + r][k0 + 4g .. 4g+3] and X[row0 + r][k0 + 8 + 4g .. 8+4g+3].
__device__ __forceinline__ bf16x8 frag_acc_order(const uint16_t* X, int ld, int row0, int k0) {
  const int l = threadIdx.x & 63;
  const uint16_t* p = X + (row0 + (l & 31)) * ld + k0 + 4 * (l >> 5);
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  const uint2 b = *reinterpret_cast<const uint2*>(p + 8);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// B operand for k rows 16h .. 16h+15 of an accumulator tile Y (32 rows): the
// lane's elements 8h .. 8h+7 are rows 16h + {4g..4g+3, 8+4g..8+4g+3} of its
// column, matching frag_acc_order.  Split into hi and lo parts.
__device__ __forceinline__ void frag_from_acc(const f32x16& t, int h, bf16x8& hi, bf16x8& lo) {
  uint16_t a[8], b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) split(t[8 * h + i], a[i], b[i]);
  hi = __builtin_bit_cast(bf16x8, make_uint4(pack2(a[0], a[1]), pack2(a[2], a[3]), pack2(a[4], a[5]), pack2(a[6], a[7])));
  lo = __builtin_bit_cast(bf16x8, make_uint4(pack2(b[0], b[1]), pack2(b[2], b[3]), pack2(b[4], b[5]), pack2(b[6], b[7])));
}

// Store an accumulator tile D[row0 + i][col0 + r] transposed as X[col0 + r][row0 + i],
// split into hi/lo tiles (four 8-byte stores each).
__device__ __forceinline__ void store_T(const f32x16& acc, uint16_t* Xh, uint16_t* Xl, int ld, int row0, int col0) {
  const int l = threadIdx.x & 63, g = l >> 5;
  const int base = (col0 + (l & 31)) * ld + row0 + 4 * g;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint16_t h[4], o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) split(acc[4 * q + j], h[j], o[j]);
    *reinterpret_cast<uint2*>(Xh + base + 8 * q) = make_uint2(pack2(h[0], h[1]), pack2(h[2], h[3]));
    *reinterpret_cast<uint2*>(Xl + base + 8 * q) = make_uint2(pack2(o[0], o[1]), pack2(o[2], o[3]));
  }
}

// Both layouts from one split: transposed into (Th, Tl) and row-major into (Nh, Nl).
__device__ __forceinline__ void store_TN(const f32x16& acc, uint16_t* Th, uint16_t* Tl, int ldT, uint16_t* Nh,
                                         uint16_t* Nl, int ldN, int row0, int col0) {
  const int l = threadIdx.x & 63, g = l >> 5;
  const int baseT = (col0 + (l & 31)) * ldT + row0 + 4 * g;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint16_t h[4], o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      split(acc[4 * q + j], h[j], o[j]);
      const int offN = (row0 + 8 * q + 4 * g + j) * ldN + col0 + (l & 31);
      Nh[offN] = h[j];
      Nl[offN] = o[j];
    }
    *reinterpret_cast<uint2*>(Th + baseT + 8 * q) = make_uint2(pack2(h[0], h[1]), pack2(h[2], h[3]));
    *reinterpret_cast<uint2*>(Tl + baseT + 8 * q) = make_uint2(pack2(o[0], o[1]), pack2(o[2], o[3]));
  }
}

// Store an accumulator tile row-major as X[row0 + i][col0 + r], hi/lo.
__device__ __forceinline__ void store_N(const f32x16& acc, uint16_t* Xh, uint16_t* Xl, int ld, int row0, int col0) {
  const int l = threadIdx.x & 63, g = l >> 5;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    uint16_t h, o;
    split(acc[e], h, o);
    const int off = (row0 + acc_row(e, g)) * ld + col0 + (l & 31);
    Xh[off] = h;
    Xl[off] = o;
  }
}

template <int C, int D, int DV, bool SUMMARY>
struct Cfg {
  // Two reused buffers: B1 holds W, then R^T (after a barrier); B2 holds R,
  // then T (after a barrier).  Summaries use only B1 and add Q^T.
  static constexpr int CD = C > D ? C : D;
  static constexpr int ldQ = D + kPad, ldK = D + kPad, ldKt = C + kPad, ldVt = C + kPad;
  static constexpr int ld1 = C + kPad, ld2 = CD + kPad, ldQt = C + kPad;
  static constexpr int ldW = ld1, ldRt = ld1, ldR = ld2, ldT = ld2;
  static constexpr int oQ = 0;
  static constexpr int oK = oQ + C * ldQ;
  static constexpr int oKt = oK + C * ldK;
  static constexpr int oVt = oKt + D * ldKt;
  static constexpr int oB1h = oVt + DV * ldVt;
  static constexpr int oB1l = oB1h + CD * ld1;
  static constexpr int oB2h = oB1l + CD * ld1;
  static constexpr int oB2l = oB2h + (SUMMARY ? 0 : C * ld2);
  static constexpr int oQt = oB2l + (SUMMARY ? 0 : C * ld2);
  static constexpr int n16 = oQt + (SUMMARY ? D * ldQt : 0);          // bf16 elements of tiles
  // the output walk folds its carry in fp32 scratch that reuses the tile region
  static constexpr int fold_f = SUMMARY ? 0 : D * (D + 4) + 2 * D * DV + D;   // fold_sum scratch
  static constexpr int n16t = (n16 > 2 * fold_f ? n16 : 2 * fold_f);
  static constexpr int RT = C / 32, DT = D / 32, VT = DV / 32;       // 32-wide tiles
  static constexpr int KC = C / 16, KD = D / 16;                     // 16-deep k steps
  static constexpr int f_eta = 0, f_cs = D, f_den = D + RT * D, f_denp = f_den + C;   // fp32 region
  static constexpr int nf32 = f_denp + RT * C;
  static constexpr size_t bytes = (size_t)((n16t + 7) & ~7) * 2 + (size_t)nf32 * 4;
  // global->LDS staging: 16-byte segments per operand
  static constexpr int segQ = C * D / 8, segV = C * DV / 8;
  static constexpr int pfQ = (segQ + kThreads - 1) / kThreads, pfV = (segV + kThreads - 1) / kThreads;
  static_assert(C % 32 == 0 && D % 32 == 0 && DV % 32 == 0 && C <= 64 && D <= 64 && DV <= 64, "tile shape");
  static_assert(bytes <= 160 * 1024, "LDS budget");
};

// The semidirect-product scan over segments, Eq. (semidirect), organised as
// reduce-then-scan.  For segments A (everything before s, including the
// initial state) and B = segment s:
//   G_{A(+)B} = G_A + [G_B + S_B C_A],   h_{A(+)B} = h_A + [h_B + S_B m_A]
// and S, C, m add.  The bracket depends on A only through the additive
// prefixes C_A and m_A, so every segment's bracket is computed in parallel
// (k_seg_cross); the carry of segment s is then a plain sum of the brackets
// and summaries before it (fold_sum, in the output walk's prologue), and the
// total state a plain sum of all of them (k_total).
//
// k_seg_cross: one workgroup per (segment s < nsum, head).  The summary of s
// arrives as (S, C, m, Phi, eta) with Phi = S C - G, eta = S m - h, so
//   G_s + S_s C_A = S_s (C_A + C_s) - Phi_s,  h_s + S_s m_A = S_s (m_A + m_s) - eta_s,
// with C_A = C_init + sum_{s'<s} C_s'.  The brackets replace Phi_s and eta_s
// in the record (in place; other workgroups read only S, C and m).
template <int D, int DV>
__global__ __launch_bounds__(256) void k_seg_cross(float* __restrict__ segs, const float* __restrict__ init,
                                                   int nseg) {
  constexpr int T = 256, ldT = D + 4, NB4 = DV / 4, NT = (D / 4) * NB4;
  constexpr int nS4 = D * D / 4 / T, nC4 = D * DV / 4 / T;
  static_assert(NT <= T && D * D % (4 * T) == 0 && D * DV % (4 * T) == 0, "thread split");
  extern __shared__ float sm[];
  float* XT = sm;                 // [D][D+4]  S_s^T
  float* Y = XT + D * ldT;        // [D][DV]   C_A + C_s
  float* y = Y + D * DV;          // [D]       m_A + m_s
  const int s = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const size_t F = state_floats(D, DV);
  float* x = segs + ((size_t)bh * nseg + s) * F;
  const float* ini = init ? init + (size_t)bh * F : nullptr;
  const bool act = tid < NT;
  const int a0 = act ? 4 * (tid / NB4) : 0, b0 = 4 * (tid % NB4);
  // issue every load first: S_s, Phi_s block, eta_s, then C and m of segments <= s
  float4 sv[nS4], pv[4], cs[nC4];
  float ev = 0.f, ms = 0.f;
#pragma unroll
  for (int r = 0; r < nS4; ++r) sv[r] = reinterpret_cast<const float4*>(x)[tid + T * r];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    pv[i] = act ? *reinterpret_cast<const float4*>(x + off_G(D, DV) + (size_t)(a0 + i) * DV + b0)
                : make_float4(0.f, 0.f, 0.f, 0.f);
  if (tid < D) ev = x[off_h(D, DV) + tid];
#pragma unroll
  for (int r = 0; r < nC4; ++r)
    cs[r] = ini ? reinterpret_cast<const float4*>(ini + off_C(D, DV))[tid + T * r] : make_float4(0.f, 0.f, 0.f, 0.f);
  if (tid < D && ini) ms = ini[off_m(D, DV) + tid];
  for (int sp = 0; sp <= s; ++sp) {
    const float* xp = segs + ((size_t)bh * nseg + sp) * F;
#pragma unroll
    for (int r = 0; r < nC4; ++r) {
      const float4 c4 = reinterpret_cast<const float4*>(xp + off_C(D, DV))[tid + T * r];
      cs[r].x += c4.x; cs[r].y += c4.y; cs[r].z += c4.z; cs[r].w += c4.w;
    }
    if (tid < D) ms += xp[off_m(D, DV) + tid];
  }
#pragma unroll
  for (int r = 0; r < nS4; ++r) {
    const int e4 = tid + T * r, a = (4 * e4) / D, ap = (4 * e4) % D;
    XT[(ap + 0) * ldT + a] = sv[r].x;
    XT[(ap + 1) * ldT + a] = sv[r].y;
    XT[(ap + 2) * ldT + a] = sv[r].z;
    XT[(ap + 3) * ldT + a] = sv[r].w;
  }
#pragma unroll
  for (int r = 0; r < nC4; ++r) reinterpret_cast<float4*>(Y)[tid + T * r] = cs[r];
  if (tid < D) y[tid] = ms;
  __syncthreads();
  if (act) {
    float o[4][4] = {};
#pragma unroll 8
    for (int ap = 0; ap < D; ++ap) {
      const float4 x4 = *reinterpret_cast<const float4*>(&XT[ap * ldT + a0]);
      const float4 z4 = *reinterpret_cast<const float4*>(&Y[ap * DV + b0]);
      const float xv[4] = {x4.x, x4.y, x4.z, x4.w}, zv[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[i][j] += xv[i] * zv[j];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<float4*>(x + off_G(D, DV) + (size_t)(a0 + i) * DV + b0) =
          make_float4(o[i][0] - pv[i].x, o[i][1] - pv[i].y, o[i][2] - pv[i].z, o[i][3] - pv[i].w);
  }
  if (tid < D) {
    float acc = 0.f;
#pragma unroll 8
    for (int ap = 0; ap < D; ++ap) acc += XT[ap * ldT + tid] * y[ap];
    x[off_h(D, DV) + tid] = acc - ev;
  }
}

// k_total: the state after all nsum segments, init (+) seg_0 (+) ... : S, C,
// m add; G and h add the brackets written by k_seg_cross.  Elementwise.
__global__ __launch_bounds__(256) void k_total(const float* __restrict__ segs, const float* __restrict__ init,
                                               float* __restrict__ fin, int nseg, int nsum, int F4) {
  const int bh = blockIdx.y;
  const size_t F = (size_t)F4 * 4;
  for (int e4 = blockIdx.x * 256 + threadIdx.x; e4 < F4; e4 += gridDim.x * 256) {
    float4 acc = init ? reinterpret_cast<const float4*>(init + bh * F)[e4] : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sp = 0; sp < nsum; ++sp) {
      const float4 v = reinterpret_cast<const float4*>(segs + ((size_t)bh * nseg + sp) * F)[e4];
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    reinterpret_cast<float4*>(fin + bh * F)[e4] = acc;
  }
}

// Carry of segment `seg` of head bh in the output walk's prologue: sum of the
// initial state and the records of segments < seg (after k_seg_cross), then
// Phi0 = S_acc C_acc - G_acc and eta0 = S_acc m_acc - h_acc.
// Results: S_acc^T in `Sout` ([D][D+4]), Phi0 in `Pout` ([D][DV]), eta0 in `eout`.
template <int D, int DV>
__device__ void fold_sum(const float* __restrict__ segs, const float* __restrict__ init, int bh, int seg,
                         int nseg, float* sc, float*& Sout, float*& Pout, float* eout) {
  constexpr int ldT = D + 4, NB4 = DV / 4, NT = (D / 4) * NB4;
  constexpr int nS4 = D * D / 4 / kThreads, nC4 = D * DV / 4 / kThreads;
  static_assert(NT <= kThreads && D * D % (4 * kThreads) == 0 && D * DV % (4 * kThreads) == 0, "thread split");
  const size_t F = state_floats(D, DV);
  float* XT = sc;                     // [D][D+4]  S_acc^T
  float* Y = XT + D * ldT;            // [D][DV]   Phi0
  float* Cs = Y + D * DV;             // [D][DV]   C_acc
  float* y = Cs + D * DV;             // [D]       m_acc
  const int tid = threadIdx.x;
  const bool act = tid < NT;
  const int a0 = act ? 4 * (tid / NB4) : 0, b0 = 4 * (tid % NB4);
  float4 sacc[nS4], cacc[nC4], gacc[4];
  float macc = 0.f, hacc = 0.f;
  auto add = [](float4& a, const float4& b) { a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w; };
  const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int r = 0; r < nS4; ++r) sacc[r] = z4;
#pragma unroll
  for (int r = 0; r < nC4; ++r) cacc[r] = z4;
#pragma unroll
  for (int i = 0; i < 4; ++i) gacc[i] = z4;
  for (int sp = -1; sp < seg; ++sp) {
    const float* x = sp < 0 ? (init ? init + (size_t)bh * F : nullptr) : segs + ((size_t)bh * nseg + sp) * F;
    if (!x) continue;
#pragma unroll
    for (int r = 0; r < nS4; ++r) add(sacc[r], reinterpret_cast<const float4*>(x)[tid + kThreads * r]);
#pragma unroll
    for (int r = 0; r < nC4; ++r) add(cacc[r], reinterpret_cast<const float4*>(x + off_C(D, DV))[tid + kThreads * r]);
    if (act)
#pragma unroll
      for (int i = 0; i < 4; ++i) add(gacc[i], *reinterpret_cast<const float4*>(x + off_G(D, DV) + (size_t)(a0 + i) * DV + b0));
    if (tid < D) {
      macc += x[off_m(D, DV) + tid];
      hacc += x[off_h(D, DV) + tid];
    }
  }
#pragma unroll
  for (int r = 0; r < nS4; ++r) {
    const int e4 = tid + kThreads * r, a = (4 * e4) / D, ap = (4 * e4) % D;
    XT[(ap + 0) * ldT + a] = sacc[r].x;
    XT[(ap + 1) * ldT + a] = sacc[r].y;
    XT[(ap + 2) * ldT + a] = sacc[r].z;
    XT[(ap + 3) * ldT + a] = sacc[r].w;
  }
#pragma unroll
  for (int r = 0; r < nC4; ++r) reinterpret_cast<float4*>(Cs)[tid + kThreads * r] = cacc[r];
  if (tid < D) y[tid] = macc;
  __syncthreads();
  if (act) {
    float o[4][4] = {};
#pragma unroll 8
    for (int ap = 0; ap < D; ++ap) {
      const float4 x4 = *reinterpret_cast<const float4*>(&XT[ap * ldT + a0]);
      const float4 c4 = *reinterpret_cast<const float4*>(&Cs[ap * DV + b0]);
      const float xv[4] = {x4.x, x4.y, x4.z, x4.w}, cv[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[i][j] += xv[i] * cv[j];
    }
    const float gv[4][4] = {{gacc[0].x, gacc[0].y, gacc[0].z, gacc[0].w}, {gacc[1].x, gacc[1].y, gacc[1].z, gacc[1].w},
                            {gacc[2].x, gacc[2].y, gacc[2].z, gacc[2].w}, {gacc[3].x, gacc[3].y, gacc[3].z, gacc[3].w}};
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Y[(a0 + i) * DV + b0 + j] = o[i][j] - gv[i][j];
  }
  if (tid < D) {
    float acc = 0.f;
#pragma unroll 8
    for (int ap = 0; ap < D; ++ap) acc += XT[ap * ldT + tid] * y[ap];
    eout[tid] = acc - hacc;
  }
  __syncthreads();
  Sout = XT;
  Pout = Y;
}

// One segment walk.  grid = (segments, BH), 4 waves.  Wave w works on output
// tile (rt = w/2, ct = w%2) of R and of O; it keeps columns ct of S0 and of
// Phi0 (all their rows) in accumulators.
// SUMMARY: zero carry, writes the segment summary (S, C, m, Phi, eta) to
// rec[bh][seg].  !SUMMARY: folds the carry from rec[bh][0..seg) and init,
// then writes outputs.
template <int C, int D, int DV, bool SUMMARY>
__global__ __launch_bounds__(kThreads, 2) void k_walk(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v, float* __restrict__ out,
                                                      float* __restrict__ rec, const float* __restrict__ init, int n,
                                                      int cps, int nseg, int normalized, float eps) {
  using G = Cfg<C, D, DV, SUMMARY>;
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* Qs = lds + G::oQ;
  uint16_t* Ks = lds + G::oK;
  uint16_t* Kt = lds + G::oKt;
  uint16_t* Vt = lds + G::oVt;
  uint16_t* Wh = lds + G::oB1h;   // W, then R^T
  uint16_t* Wl = lds + G::oB1l;
  uint16_t* Rth = Wh;
  uint16_t* Rtl = Wl;
  uint16_t* Rh = lds + G::oB2h;   // R, then T
  uint16_t* Rl = lds + G::oB2l;
  uint16_t* Th = Rh;
  uint16_t* Tl = Rl;
  uint16_t* Qt = lds + G::oQt;
  float* fl = reinterpret_cast<float*>(lds + ((G::n16t + 7) & ~7));
  float* eta = fl + G::f_eta;
  float* colsum = fl + G::f_cs;       // [RT][D]
  float* den = fl + G::f_den;         // [C]
  float* denp = fl + G::f_denp;       // [RT][C]

  const int seg = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int rt = w >> 1, ct = w & 1;
  const bool has_r = rt < G::RT && ct < G::DT;        // owns R tile (rt, ct) and S0 column ct
  const bool has_o = rt < G::RT && ct < G::VT;        // owns O tile (rt, ct) and Phi0 column ct
  const bool upd_p = SUMMARY ? (has_o && rt == 0) : has_o;
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t F = state_floats(D, DV);
  float* rc = SUMMARY ? rec + ((size_t)bh * nseg + seg) * F : nullptr;

  // ---- carry in (fp32 accumulators, column ct, all rows) ----
  f32x16 S0[G::DT], P0[G::DT], Cs[SUMMARY ? G::DT : 1];
#pragma unroll
  for (int i = 0; i < G::DT; ++i) {
    S0[i] = zero16();
    P0[i] = zero16();
    if (SUMMARY) Cs[SUMMARY ? i : 0] = zero16();
  }
  for (int a = tid; a < D; a += kThreads) eta[a] = 0.f;
  if (!SUMMARY && (seg > 0 || init)) {
    // the tile region of LDS is free until the first chunk is staged
    float* Sc;
    float* Pc;
    fold_sum<D, DV>(rec, init, bh, seg, nseg, reinterpret_cast<float*>(lds), Sc, Pc, eta);
#pragma unroll
    for (int i = 0; i < G::DT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = i * 32 + acc_row(e, lg);
        if (has_r) S0[i][e] = Sc[(ct * 32 + lr) * (D + 4) + row];
        if (has_o) P0[i][e] = Pc[row * DV + ct * 32 + lr];
      }
    __syncthreads();
  }
  float m_acc = 0.f;   // SUMMARY: column sum of Q for column tid (< D)

  // ---- prefetch registers for the next chunk ----
  uint4 pq[G::pfQ], pk[G::pfQ], pv[G::pfV];
  auto fetch = [&](int c) {
    const int t0 = c * C;
    if (t0 + C <= n && G::segQ % kThreads == 0 && G::segV % kThreads == 0) {   // full chunk: no guards
#pragma unroll
      for (int i = 0; i < G::pfQ; ++i) {
        const int e = tid + kThreads * i;
        const size_t off = ((size_t)bh * n + t0 + e % C) * D + (e / C) * 8;
        pq[i] = *reinterpret_cast<const uint4*>(q + off);
        pk[i] = *reinterpret_cast<const uint4*>(k + off);
      }
#pragma unroll
      for (int i = 0; i < G::pfV; ++i) {
        const int e = tid + kThreads * i;
        pv[i] = *reinterpret_cast<const uint4*>(v + ((size_t)bh * n + t0 + e % C) * DV + (e / C) * 8);
      }
      return;
    }
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
    if (SUMMARY && tid < D) {
      const uint16_t* row = Qt + tid * G::ldQt;
#pragma unroll
      for (int t8 = 0; t8 < C; t8 += 8) {
        const uint4 u = *reinterpret_cast<const uint4*>(row + t8);
        const uint16_t* e8 = reinterpret_cast<const uint16_t*>(&u);
#pragma unroll
        for (int j = 0; j < 8; ++j) m_acc += bf16_to_f(e8[j]);
      }
    }

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
    __syncthreads();

    // ---- stage 2: R = W K + Q S0 (old S0) on tile (rt, ct); S0 += K^T K on column ct ----
    f32x16 racc = zero16();
    if (has_r) {
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        if (s * 16 > rt * 32 + 31) break;         // keys past this row tile: W is zero
        const bf16x8 bK = frag(Kt, G::ldKt, ct * 32, s * 16);
        racc = mfma(frag(Wh, G::ldW, rt * 32, s * 16), bK, racc);
        racc = mfma(frag(Wl, G::ldW, rt * 32, s * 16), bK, racc);
      }
#pragma unroll
      for (int s = 0; s < G::KD; ++s) {
        bf16x8 bh, bl;
        frag_from_acc(S0[s >> 1], s & 1, bh, bl);
        const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, rt * 32, s * 16);
        racc = mfma(aQ, bh, racc);
        racc = mfma(aQ, bl, racc);
      }
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bK = frag(Kt, G::ldKt, ct * 32, s * 16);
#pragma unroll
        for (int i = 0; i < G::DT; ++i) S0[i] = mfma(frag(Kt, G::ldKt, i * 32, s * 16), bK, S0[i]);
      }
      // eta advance: column sums of R over this row tile
      float cs = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) cs += racc[e];
      cs += __shfl_xor(cs, 32);
      if (lg == 0) colsum[rt * D + ct * 32 + lr] = cs;
    }
    __syncthreads();     // every wave is done reading W: B1 takes R^T
    if (has_r) {
      if (SUMMARY)
        store_T(racc, Rth, Rtl, G::ldRt, rt * 32, ct * 32);
      else
        store_TN(racc, Rth, Rtl, G::ldRt, Rh, Rl, G::ldR, rt * 32, ct * 32);
    }
    __syncthreads();
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
            acc = mfma(frag(Rh, G::ldR, it * 32, s * 16), b, acc);
            acc = mfma(frag(Rl, G::ldR, it * 32, s * 16), b, acc);
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
        __syncthreads();     // every wave is done reading R: B2 takes T
        if (tile) store_T(acc, Th, Tl, G::ldT, it * 32, jt * 32);
      }
      __syncthreads();
      // den_t = sum_j T[t][j] + q_t . eta0, stored as 1 / (den_t + eps)
      if (normalized && tid < C) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < G::RT; ++i) s += denp[i * C + tid];
        const uint16_t* row = Qs + tid * G::ldQ;
#pragma unroll
        for (int a8 = 0; a8 < D; a8 += 8) {
          const uint4 u = *reinterpret_cast<const uint4*>(row + a8);
          const uint16_t* e8 = reinterpret_cast<const uint16_t*>(&u);
#pragma unroll
          for (int j = 0; j < 8; ++j) s += bf16_to_f(e8[j]) * eta[a8 + j];
        }
        den[tid] = 1.f / (s + eps);
      }
      __syncthreads();
      // ---- stage 4: O = T V + Q Phi0 (old Phi0) on tile (rt, ct); stage 5: Phi0 += R^T V ----
      if (has_o) {
        f32x16 oacc = zero16();
#pragma unroll
        for (int s = 0; s < G::KC; ++s) {
          if (s * 16 > rt * 32 + 31) break;       // j past this row tile: T is zero
          const bf16x8 bV = frag(Vt, G::ldVt, ct * 32, s * 16);
          oacc = mfma(frag(Th, G::ldT, rt * 32, s * 16), bV, oacc);
          oacc = mfma(frag(Tl, G::ldT, rt * 32, s * 16), bV, oacc);
        }
#pragma unroll
        for (int s = 0; s < G::KD; ++s) {
          bf16x8 bh, bl;
          frag_from_acc(P0[s >> 1], s & 1, bh, bl);
          const bf16x8 aQ = frag_acc_order(Qs, G::ldQ, rt * 32, s * 16);
          oacc = mfma(aQ, bh, oacc);
          oacc = mfma(aQ, bl, oacc);
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int t = rt * 32 + acc_row(e, lg);
          if (t0 + t < n) {
            float o = oacc[e];
            if (normalized) o *= den[t];
            out[((size_t)bh * n + t0 + t) * DV + ct * 32 + lr] = o;
          }
        }
      }
    }
    if (upd_p) {
      // Phi0 += R^T V (and, for summaries, C += Q^T V) on column ct
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        const bf16x8 bV = frag(Vt, G::ldVt, ct * 32, s * 16);
#pragma unroll
        for (int i = 0; i < G::DT; ++i) {
          P0[i] = mfma(frag(Rth, G::ldRt, i * 32, s * 16), bV, P0[i]);
          P0[i] = mfma(frag(Rtl, G::ldRt, i * 32, s * 16), bV, P0[i]);
          if (SUMMARY) Cs[SUMMARY ? i : 0] = mfma(frag(Qt, G::ldQt, i * 32, s * 16), bV, Cs[SUMMARY ? i : 0]);
        }
      }
    }
    __syncthreads();   // LDS tiles and den/eta are rewritten by the next chunk
    if (tid < D) eta[tid] += eta_add;
  }

  if (SUMMARY) {
    // record (S, C, m, Phi, eta): Phi in the G slot, eta in the h slot
    if (has_r && rt == 0)
#pragma unroll
      for (int i = 0; i < G::DT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) rc[(size_t)(i * 32 + acc_row(e, lg)) * D + ct * 32 + lr] = S0[i][e];
    if (upd_p)
#pragma unroll
      for (int i = 0; i < G::DT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const size_t o = (size_t)(i * 32 + acc_row(e, lg)) * DV + ct * 32 + lr;
          rc[off_G(D, DV) + o] = P0[i][e];
          rc[off_C(D, DV) + o] = Cs[SUMMARY ? i : 0][e];
        }
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
  if (nsum > 0) {
    const size_t lds = sizeof(float) * ((size_t)D * (D + 4) + (size_t)D * DV + D);
    auto kx = k_seg_cross<D, DV>;
    if ((e = hipFuncSetAttribute((const void*)kx, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) != hipSuccess)
      return e;
    prof_start("seg_cross", s);
    hipLaunchKernelGGL(kx, dim3(nsum, BH), dim3(256), lds, s, segs, init, P);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (final_state) {
    const int F4 = (int)(F / 4);
    prof_start("total", s);
    hipLaunchKernelGGL(k_total, dim3((F4 + 255) / 256, BH), dim3(256), 0, s, segs, init, final_state, P, nsum, F4);
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
  int p = 512 / BH;                       // about two workgroups per CU
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
