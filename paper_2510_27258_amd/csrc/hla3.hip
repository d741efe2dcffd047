// Masked third-order HLA forward (Sec. 7), fp32 arithmetic (dot products over
// d in fp64) on fp32 or bf16 inputs, by the chunk-parallel scan of Sec. 7.3 in
// a walk form; the walks' products run on 16 x 16 MFMA tiles.
//
// The corrected state F_t = S^K S^Q P - G1 - G2 - G3 (Eq. hla3-corrected-state)
// advances per token by (Eq. hla3-corrected-recurrence, with primes for the
// moments before token j, delta_j = q_j . k_j)
//   F += SK' q q^T k v^T + k k^T SQ' k v^T + k k^T q q^T P' + k k^T q q^T k v^T
//      = r_j delta_j v_j^T + k_j (sigma_j v_j + delta_j P'^T q_j + delta_j^2 v_j)^T,
// with r_j = SK'_j q_j and sigma_j = k_j^T SQ'_j k_j; num_t = q_t^T F_t and
// den_t = q_t^T eta_t (the same with v := 1).  Over a tile of tokens
// (Q, K, V as rows; A = Q K^T; L and Ls the causal masks with and without the
// diagonal) and moment carry (SK0, SQ0, P0, m0):
//   R  = Q SK0 + (A (.) Ls) K                      rows r_j
//   sigma_j = k_j^T SQ0 k_j + sum_{u<j} A_uj^2
//   Pq = Q P0 + (A (.) Ls) V,   pm = Q m0 + (A (.) Ls) 1
//   X  = (sigma + delta^2) (.) V + delta (.) Pq,   x = sigma + delta^2 + delta (.) pm
//   num = Q F0 + [(Q R^T) (.) L] (delta (.) V) + (A (.) L) X
//   den = Q eta0 + [(Q R^T) (.) L] delta + (A (.) L) x
//   F0 += R^T (delta (.) V) + K^T X,   eta0 += R^T delta + K^T x,
//   SK0 += K^T K, SQ0 += Q^T Q, P0 += K^T V, m0 += K^T 1.
// No increment depends on F, so F composes across segments as a plain sum of
// per-segment brackets (each computed with the true moment prefixes): these
// are exactly the carry terms of the operator (x)_3 (Eq. hla3-corrected-concat),
// S^K_A R_B + M_B[S^Q_A] + U_B P_A, applied from the segment's tokens
// without materialising the maps M.
//
// Launches (segments of whole tiles per head):
//   1. k3_moments: per segment, (SK, SQ, P, m) of its tokens.
//   2. k3_walk: per segment, moment carry = sum of the moments before it; walks
//      its tiles from F = 0, writes num (into out) and den (workspace) without
//      the F carry, and the segment's bracket (F, eta).
//   3. k3_fix: out_t += q_t^T F_c, den_t += q_t . eta_c with F_c the sum of the
//      brackets before the segment; normalises if asked.
#include <cstdlib>

#include "hla3.h"
#include "mfma16.h"
#include "profile.h"

namespace hla {
namespace {

constexpr int kT3 = 256;

template <int D, int DV>
struct Rec3 {   // per (head, segment): SK | SQ | P | m | F | eta
  static constexpr int oSK = 0, oSQ = D * D, oP = 2 * D * D, om = oP + D * DV, oF = om + D, oe = oF + D * DV;
  static constexpr int floats = oe + D;
};

template <typename T>
__device__ __forceinline__ float ld3(const T* p, size_t i) { return ldf(p, i); }

// Stage one tile of tokens (rows past n read as zero) into padded LDS rows.
template <typename T, int C, int D, int DV>
__device__ void stage_tile(const T* q, const T* k, const T* v, size_t head_tok, int t0, int n, float* Qs, float* Ks,
                           float* Vs) {
  for (int e = threadIdx.x; e < C * D; e += kT3) {
    const int t = e / D, a = e % D;
    const bool in = t0 + t < n;
    const size_t g = (head_tok + t0 + t) * D + a;
    Qs[t * (D + 1) + a] = in ? ld3(q, g) : 0.f;
    Ks[t * (D + 1) + a] = in ? ld3(k, g) : 0.f;
  }
  for (int e = threadIdx.x; e < C * DV; e += kT3) {
    const int t = e / DV, b = e % DV;
    Vs[t * (DV + 1) + b] = (t0 + t < n) ? ld3(v, (head_tok + t0 + t) * DV + b) : 0.f;
  }
}

// 1. Moments of each segment.  grid (nseg, BH).
template <typename T, int C, int D, int DV>
__global__ __launch_bounds__(kT3) void k3_moments(const T* __restrict__ q, const T* __restrict__ k,
                                                  const T* __restrict__ v, float* __restrict__ rec, int n, int cps,
                                                  int nseg) {
  using Rc = Rec3<D, DV>;
  constexpr int NO = 2 * D * D + D * DV + D;   // SK | SQ | P | m: the first NO floats of a record
  __shared__ float Qs[C * (D + 1)], Ks[C * (D + 1)], Vs[C * (DV + 1)], acc[NO];
  const int seg = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int M = (n + C - 1) / C, c0 = seg * cps, c1 = min(M, c0 + cps);
  for (int o = tid; o < NO; o += kT3) acc[o] = 0.f;     // each thread keeps its own slots
  for (int c = c0; c < c1; ++c) {
    stage_tile<T, C, D, DV>(q, k, v, (size_t)bh * n, c * C, n, Qs, Ks, Vs);
    __syncthreads();
    for (int o = tid; o < D * D; o += kT3) {            // K^T K and Q^T Q
      const int a = o / D, b = o % D;
      float sk = 0.f, sq = 0.f;
      for (int t = 0; t < C; ++t) {
        sk += Ks[t * (D + 1) + a] * Ks[t * (D + 1) + b];
        sq += Qs[t * (D + 1) + a] * Qs[t * (D + 1) + b];
      }
      acc[Rc::oSK + o] += sk;
      acc[Rc::oSQ + o] += sq;
    }
    for (int o = tid; o < D * DV; o += kT3) {           // K^T V
      const int a = o / DV, b = o % DV;
      float s = 0.f;
      for (int t = 0; t < C; ++t) s += Ks[t * (D + 1) + a] * Vs[t * (DV + 1) + b];
      acc[Rc::oP + o] += s;
    }
    for (int a = tid; a < D; a += kT3) {                 // K^T 1
      float s = 0.f;
      for (int t = 0; t < C; ++t) s += Ks[t * (D + 1) + a];
      acc[Rc::om + a] += s;
    }
    __syncthreads();
  }
  float* r = rec + ((size_t)bh * nseg + seg) * Rc::floats;
  for (int o = tid; o < NO; o += kT3) r[o] = acc[o];
}

// Exclusive running sums over the segments of a head, for the floats
// [off, off + len) of every record: pre[s] = sum_{s' < s} rec[s'].  grid
// (ceil(len / kT3), BH); each thread one float, reads and writes coalesced.
template <int D, int DV>
__global__ __launch_bounds__(kT3) void k3_prefix(const float* __restrict__ rec, float* __restrict__ pre, int nseg,
                                                 int off, int len) {
  using Rc = Rec3<D, DV>;
  const int e = blockIdx.x * kT3 + threadIdx.x;
  if (e >= len) return;
  const size_t base = (size_t)blockIdx.y * nseg * Rc::floats + off + e;
  float x = 0.f;
  for (int s0 = 0; s0 < nseg; s0 += 32) {    // 32 records' loads in flight at a time
    float r[32];
#pragma unroll
    for (int j = 0; j < 32; ++j) r[j] = s0 + j < nseg ? rec[base + (size_t)(s0 + j) * Rc::floats] : 0.f;
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      if (s0 + j < nseg) pre[base + (size_t)(s0 + j) * Rc::floats] = x;
      x += r[j];
    }
  }
}

// 2. The walk of one segment from its moment carry with F = 0.  grid (nseg, BH).
// Every product of a tile runs on 16 x 16 MFMA tiles, one per wave at a time:
// the dot products over d (Q K^T, Q SK0, Q P0, Q F0, Q R^T) in fp64
// (v_mfma_f64_16x16x4_f64, fp32 operands widened exactly), the products over
// the tile's tokens (the prefixes R and Pq, the outputs, the moment and F
// advances) in fp32 (v_mfma_f32_16x16x4_f32), as the arithmetic of the
// recurrence asks; products with a causal mask stop at the diagonal tile.
template <typename T, int C, int D, int DV>
__global__ __launch_bounds__(kT3) void k3_walk(const T* __restrict__ q, const T* __restrict__ k,
                                               const T* __restrict__ v, float* __restrict__ out,
                                               float* __restrict__ den_out, float* __restrict__ rec,
                                               const float* __restrict__ pre, int n, int cps, int nseg) {
  using Rc = Rec3<D, DV>;
  constexpr int lD = D + 1, lV = DV + 1, lC = C + 1, NW = kT3 / 64;
  constexpr int ct = C / 16, dt = D / 16, vt = DV / 16;
  __shared__ float Qs[C * lD], Ks[C * lD], Vs[C * lV];
  __shared__ float SK[D * lD], SQ[D * lD], Pm[D * lV], mv[D], F[D * lV], eta[D];
  __shared__ float A[C * lC], R[C * lD], Tm[C * lC], QSK[C * lD], QP[C * lV], QF[C * lV], Pq[C * lV], X[C * lV];
  __shared__ float sig[C], dl[C], pm[C], xv[C], qeta[C];
  const int seg = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, nn = tid & 15, g = (tid >> 4) & 3, pr = mfma_pr(nn);
  const int M = (n + C - 1) / C, c0 = seg * cps, c1 = min(M, c0 + cps);
  const size_t head_tok = (size_t)bh * n;
  float* recs = rec + (size_t)bh * nseg * Rc::floats;
  const f64x4c zd = {0.0, 0.0, 0.0, 0.0};

  // moment carry: the sum of the segments before this one (k3_prefix); F = eta = 0
  const float* prc = pre + ((size_t)bh * nseg + seg) * Rc::floats;
  for (int e = tid; e < D * D; e += kT3) {
    SK[(e / D) * lD + e % D] = prc[Rc::oSK + e];
    SQ[(e / D) * lD + e % D] = prc[Rc::oSQ + e];
  }
  for (int e = tid; e < D * DV; e += kT3) {
    Pm[(e / DV) * lV + e % DV] = prc[Rc::oP + e];
    F[(e / DV) * lV + e % DV] = 0.f;
  }
  for (int e = tid; e < D; e += kT3) {
    mv[e] = prc[Rc::om + e];
    eta[e] = 0.f;
  }

  for (int c = c0; c < c1; ++c) {
    const int t0 = c * C;
    stage_tile<T, C, D, DV>(q, k, v, head_tok, t0, n, Qs, Ks, Vs);
    __syncthreads();
    // s1: A = Q K^T (every tile: its upper part feeds sigma), Q SK0, Q P0, Q F0
    // in fp64 (a row such as o_1 = (q_1.k_1)^3 v_1 amplifies the cancellation
    // of q.k); q.m0, q.eta0 and k^T SQ0 k per token
    {
      constexpr int nA = ct * ct, nS = ct * dt, nP = ct * vt;
      for (int tile = w; tile < nA + nS + 2 * nP; tile += NW) {
        f64x4c acc = zd;
        float* dst;
        int ldd, mm, n0;
        auto aq = [&](int kk) { return (double)Qs[(mm + pr) * lD + kk]; };
        if (tile < nA) {
          mm = 16 * (tile / ct), n0 = 16 * (tile % ct), dst = A, ldd = lC;
          mma_lds<double>(acc, D, g, aq, [&](int kk) { return (double)Ks[(n0 + nn) * lD + kk]; });
        } else if (tile < nA + nS) {
          const int u = tile - nA;
          mm = 16 * (u / dt), n0 = 16 * (u % dt), dst = QSK, ldd = lD;
          mma_lds<double>(acc, D, g, aq, [&](int kk) { return (double)SK[kk * lD + n0 + nn]; });
        } else {
          const int u = tile - nA - nS, uu = u % nP;
          const float* B = u < nP ? Pm : F;
          mm = 16 * (uu / vt), n0 = 16 * (uu % vt), dst = u < nP ? QP : QF, ldd = lV;
          mma_lds<double>(acc, D, g, aq, [&](int kk) { return (double)B[kk * lV + n0 + nn]; });
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[(mm + 4 * g + i) * ldd + n0 + nn] = (float)acc[i];
      }
    }
    // per token t: q_t.m0, q_t.eta0 and k_t^T SQ0 k_t, one lane per (t, a) and
    // the sum over a across D consecutive lanes (D divides the wave)
    static_assert(64 % D == 0 && (C * D) % kT3 == 0, "token-row lanes");
    for (int e = tid; e < C * D; e += kT3) {
      const int t = e / D, a = e % D;
      double y = 0.0;
#pragma unroll
      for (int b = 0; b < D; ++b) y += (double)SQ[a * lD + b] * Ks[t * lD + b];
      double gq = (double)Ks[t * lD + a] * y, sm = (double)Qs[t * lD + a] * mv[a], wq = (double)Qs[t * lD + a] * eta[a];
#pragma unroll
      for (int o = 1; o < D; o <<= 1) {
        gq += __shfl_xor(gq, o);
        sm += __shfl_xor(sm, o);
        wq += __shfl_xor(wq, o);
      }
      if (a == 0) {
        pm[t] = (float)sm;
        qeta[t] = (float)wq;
        sig[t] = (float)gq;
      }
    }
    __syncthreads();
    // s2: prefixes inside the tile (strictly before j), in fp32:
    //   R = Q SK0 + (A (.) Ls) K,  Pq = Q P0 + (A (.) Ls) V,
    //   sigma_j += sum_{u<j} A_uj^2,  pm_j += sum_{u<j} A_ju,  delta_j = A_jj
    {
      constexpr int nS = ct * dt, nP = ct * vt;
      for (int tile = w; tile < nS + nP; tile += NW) {
        const bool isR = tile < nS;
        const int u = isR ? tile : tile - nS, cn = isR ? dt : vt, mm = 16 * (u / cn), n0 = 16 * (u % cn);
        const float* init = isR ? QSK : QP;
        const float* B = isR ? Ks : Vs;
        const int li = isR ? lD : lV;
        f32x4c acc;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = init[(mm + 4 * g + i) * li + n0 + nn];
        mma_lds<float>(acc, mm + 16, g, [&](int kk) { return kk < mm + nn ? A[(mm + nn) * lC + kk] : 0.f; },
                       [&](int kk) { return B[kk * li + n0 + nn]; });
        float* dst = isR ? R : Pq;
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[(mm + 4 * g + i) * li + n0 + nn] = acc[i];
      }
      const int j = tid >> 3, p = tid & 7;
      float s2 = 0.f, p2 = 0.f;
      if (j < C)
        for (int uu = p; uu < j; uu += 8) {
          const float a = A[uu * lC + j];
          s2 += a * a;
          p2 += A[j * lC + uu];
        }
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) {
        s2 += __shfl_xor(s2, o);
        p2 += __shfl_xor(p2, o);
      }
      if (p == 0 && j < C) {
        sig[j] += s2;
        pm[j] += p2;
        dl[j] = A[j * lC + j];
      }
    }
    __syncthreads();
    // s3: T = (Q R^T) (.) L in fp64 (tiles on or below the diagonal), X, x
    {
      constexpr int nT = ct * (ct + 1) / 2;
      for (int tile = w; tile < nT; tile += NW) {
        int mi = 0;
        while ((mi + 1) * (mi + 2) / 2 <= tile) ++mi;
        const int mm = 16 * mi, n0 = 16 * (tile - mi * (mi + 1) / 2);
        f64x4c acc = zd;
        mma_lds<double>(acc, D, g, [&](int kk) { return (double)Qs[(mm + pr) * lD + kk]; },
                        [&](int kk) { return (double)R[(n0 + nn) * lD + kk]; });
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = mm + 4 * g + i, j = n0 + nn;
          Tm[t * lC + j] = j <= t ? (float)acc[i] : 0.f;
        }
      }
    }
    for (int e = tid; e < C * DV; e += kT3) {
      const int j = e / DV, b = e % DV;
      const float d0 = dl[j];
      X[j * lV + b] = (sig[j] + d0 * d0) * Vs[j * lV + b] + d0 * Pq[j * lV + b];
    }
    for (int j = tid; j < C; j += kT3) {
      const float d0 = dl[j];
      xv[j] = sig[j] + d0 * d0 + d0 * pm[j];
    }
    __syncthreads();
    // s4: outputs without the F carry of earlier segments, then the advances,
    // all in fp32: num = Q F0 + (T diag(delta)) V + (A (.) L) X, and
    // F0 += R^T (delta (.) V) + K^T X, P0 += K^T V, SK0 += K^T K, SQ0 += Q^T Q
    {
      constexpr int nO = ct * vt, nF = dt * vt, nQ = dt * dt;
      for (int tile = w; tile < nO + 2 * nF + 2 * nQ; tile += NW) {
        f32x4c acc;
        if (tile < nO) {
          const int mm = 16 * (tile / vt), n0 = 16 * (tile % vt);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = QF[(mm + 4 * g + i) * lV + n0 + nn];
          mma_lds<float>(acc, mm + 16, g, [&](int kk) { return Tm[(mm + nn) * lC + kk] * dl[kk]; },
                         [&](int kk) { return Vs[kk * lV + n0 + nn]; });
          mma_lds<float>(acc, mm + 16, g, [&](int kk) { return kk <= mm + nn ? A[(mm + nn) * lC + kk] : 0.f; },
                         [&](int kk) { return X[kk * lV + n0 + nn]; });
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int t = mm + 4 * g + i;
            if (t0 + t < n) out[(head_tok + t0 + t) * DV + n0 + nn] = acc[i];
          }
        } else if (tile < nO + 2 * nF) {
          const bool isF = tile < nO + nF;
          const int u = isF ? tile - nO : tile - nO - nF, a0 = 16 * (u / vt), b0 = 16 * (u % vt);
          float* S = isF ? F : Pm;
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = S[(a0 + 4 * g + i) * lV + b0 + nn];
          if (isF) {
            mma_lds<float>(acc, C, g, [&](int kk) { return R[kk * lD + a0 + nn]; },
                           [&](int kk) { return dl[kk] * Vs[kk * lV + b0 + nn]; });
            mma_lds<float>(acc, C, g, [&](int kk) { return Ks[kk * lD + a0 + nn]; },
                           [&](int kk) { return X[kk * lV + b0 + nn]; });
          } else {
            mma_lds<float>(acc, C, g, [&](int kk) { return Ks[kk * lD + a0 + nn]; },
                           [&](int kk) { return Vs[kk * lV + b0 + nn]; });
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) S[(a0 + 4 * g + i) * lV + b0 + nn] = acc[i];
        } else {
          const bool isK = tile < nO + 2 * nF + nQ;
          const int u = isK ? tile - nO - 2 * nF : tile - nO - 2 * nF - nQ, a0 = 16 * (u / dt), b0 = 16 * (u % dt);
          float* S = isK ? SK : SQ;
          const float* Y = isK ? Ks : Qs;
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = S[(a0 + 4 * g + i) * lD + b0 + nn];
          mma_lds<float>(acc, C, g, [&](int kk) { return Y[kk * lD + a0 + nn]; },
                         [&](int kk) { return Y[kk * lD + b0 + nn]; });
#pragma unroll
          for (int i = 0; i < 4; ++i) S[(a0 + 4 * g + i) * lD + b0 + nn] = acc[i];
        }
      }
    }
    {  // den (eight lanes per token) and the eta0, m0 advances (eight lanes per dimension)
      const int r = tid >> 3, p = tid & 7;
      float sd = 0.f, e2 = 0.f, sm = 0.f;
      if (r < C)
        for (int j = p; j <= r; j += 8) sd += Tm[r * lC + j] * dl[j] + A[r * lC + j] * xv[j];
      if (r < D)
        for (int j = p; j < C; j += 8) {
          e2 += R[j * lD + r] * dl[j] + Ks[j * lD + r] * xv[j];
          sm += Ks[j * lD + r];
        }
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) {
        sd += __shfl_xor(sd, o);
        e2 += __shfl_xor(e2, o);
        sm += __shfl_xor(sm, o);
      }
      if (p == 0 && r < C && t0 + r < n) den_out[head_tok + t0 + r] = qeta[r] + sd;
      if (p == 0 && r < D) {
        eta[r] += e2;
        mv[r] += sm;
      }
    }
    __syncthreads();
  }
  // the segment's bracket (F, eta)
  float* r = recs + (size_t)seg * Rc::floats;
  for (int e = tid; e < D * DV; e += kT3) r[Rc::oF + e] = F[(e / DV) * lV + e % DV];
  for (int e = tid; e < D; e += kT3) r[Rc::oe + e] = eta[e];
}

// 3. Add the F carry of earlier segments and normalise.  grid (nseg, BH).
template <typename T, int C, int D, int DV>
__global__ __launch_bounds__(kT3) void k3_fix(const T* __restrict__ q, float* __restrict__ out,
                                              const float* __restrict__ den_in, const float* __restrict__ pre, int n,
                                              int cps, int nseg, int normalized, float eps) {
  using Rc = Rec3<D, DV>;
  __shared__ float Fc[D * (DV + 1)], ec[D], Qs[C * (D + 1)], inv[C];
  const int seg = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  if (seg == 0 && !normalized) return;          // nothing to add
  const int M = (n + C - 1) / C, c0 = seg * cps, c1 = min(M, c0 + cps);
  const size_t head_tok = (size_t)bh * n;
  const float* pr = pre + ((size_t)bh * nseg + seg) * Rc::floats;   // the brackets before this segment
  for (int e = tid; e < D * DV; e += kT3) Fc[(e / DV) * (DV + 1) + e % DV] = pr[Rc::oF + e];
  for (int e = tid; e < D; e += kT3) ec[e] = pr[Rc::oe + e];
  for (int c = c0; c < c1; ++c) {
    const int t0 = c * C;
    for (int e = tid; e < C * D; e += kT3) {
      const int t = e / D, a = e % D;
      Qs[t * (D + 1) + a] = (t0 + t < n) ? ld3(q, (head_tok + t0 + t) * D + a) : 0.f;
    }
    __syncthreads();
    if (normalized)
      for (int t = tid; t < C; t += kT3) {
        double s = 0.0;
        for (int a = 0; a < D; ++a) s += (double)Qs[t * (D + 1) + a] * ec[a];
        inv[t] = (t0 + t < n) ? 1.f / (den_in[head_tok + t0 + t] + (float)s + eps) : 0.f;
      }
    __syncthreads();
    for (int e = tid; e < C * DV; e += kT3) {
      const int t = e / DV, b = e % DV;
      if (t0 + t >= n) continue;
      double s = 0.0;
      for (int a = 0; a < D; ++a) s += (double)Qs[t * (D + 1) + a] * Fc[a * (DV + 1) + b];
      const size_t o = (head_tok + t0 + t) * DV + b;
      float y = out[o] + (float)s;
      if (normalized) y *= inv[t];
      out[o] = y;
    }
    __syncthreads();
  }
}

// The unmasked operator (Sec. 7.1): o_t = q_t^T S^K_t S^Q_t P_t, den_t =
// q_t^T S^K_t S^Q_t m^K_t, every summary inclusive.  With the moment carry
// (SK0, SQ0, P0, m0) of the tokens before the tile and W = L (.) Q K^T:
//   R   = Q SK0 + W K                         (row t: q_t^T S^K_t)
//   Sm  = R SQ0 + (L (.) R Q^T) Q             (row t: q_t^T S^K_t S^Q_t)
//   O   = Sm P0 + (L (.) Sm K^T) V,   den = Sm m0 + (L (.) Sm K^T) 1.
// The summaries only add, so a segment's walk from the moment prefix gives
// its outputs whole: no bracket and no fix-up.  The products of R, U, Sm,
// Tm and O run on fp64 MFMA tiles (fp32 operands widened exactly) and R, Sm
// are kept in fp64; the moment advances on fp32 MFMA.  grid (nseg, BH).
template <typename T, int C, int D, int DV>
__global__ __launch_bounds__(kT3) void k3u_walk(const T* __restrict__ q, const T* __restrict__ k,
                                                const T* __restrict__ v, float* __restrict__ out,
                                                const float* __restrict__ pre, int n, int cps, int nseg,
                                                int normalized, float eps) {
  using Rc = Rec3<D, DV>;
  constexpr int lD = D + 1, lV = DV + 1, lC = C + 1, NW = kT3 / 64;
  constexpr int ct = C / 16, dt = D / 16, vt = DV / 16, nW = ct * (ct + 1) / 2, nR = ct * dt, nO = ct * vt;
  __shared__ float Qs[C * lD], Ks[C * lD], Vs[C * lV];
  __shared__ float SK[D * lD], SQ[D * lD], Pm[D * lV], mv[D];
  __shared__ float W[C * lC], U[C * lC], Tm[C * lC];
  __shared__ double R[C * lD], Sm[C * lD], dn[C];
  const int seg = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, nn = tid & 15, g = (tid >> 4) & 3, pr = mfma_pr(nn);
  const int M = (n + C - 1) / C, c0 = seg * cps, c1 = min(M, c0 + cps);
  const size_t head_tok = (size_t)bh * n;
  const f64x4c zd = {0.0, 0.0, 0.0, 0.0};
  // tile `tile` of the lower triangle of C x C tiles: rows mm, columns n0
  auto lower = [&](int tile, int& mm, int& n0) {
    int mi = 0;
    while ((mi + 1) * (mi + 2) / 2 <= tile) ++mi;
    mm = 16 * mi;
    n0 = 16 * (tile - mi * (mi + 1) / 2);
  };

  const float* prc = pre + ((size_t)bh * nseg + seg) * Rc::floats;   // moments of the segments before
  for (int e = tid; e < D * D; e += kT3) {
    SK[(e / D) * lD + e % D] = prc[Rc::oSK + e];
    SQ[(e / D) * lD + e % D] = prc[Rc::oSQ + e];
  }
  for (int e = tid; e < D * DV; e += kT3) Pm[(e / DV) * lV + e % DV] = prc[Rc::oP + e];
  for (int e = tid; e < D; e += kT3) mv[e] = prc[Rc::om + e];

  for (int c = c0; c < c1; ++c) {
    const int t0 = c * C;
    stage_tile<T, C, D, DV>(q, k, v, head_tok, t0, n, Qs, Ks, Vs);
    __syncthreads();
    // W = L (.) Q K^T;  R = Q SK0 (first part)
    for (int tile = w; tile < nW + nR; tile += NW) {
      f64x4c acc = zd;
      int mm, n0;
      if (tile < nW) {
        lower(tile, mm, n0);
        mma_lds<double>(acc, D, g, [&](int kk) { return (double)Qs[(mm + pr) * lD + kk]; },
                        [&](int kk) { return (double)Ks[(n0 + nn) * lD + kk]; });
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = mm + 4 * g + i, j = n0 + nn;
          W[t * lC + j] = j <= t ? (float)acc[i] : 0.f;
        }
      } else {
        const int u = tile - nW;
        mm = 16 * (u / dt), n0 = 16 * (u % dt);
        mma_lds<double>(acc, D, g, [&](int kk) { return (double)Qs[(mm + pr) * lD + kk]; },
                        [&](int kk) { return (double)SK[kk * lD + n0 + nn]; });
#pragma unroll
        for (int i = 0; i < 4; ++i) R[(mm + 4 * g + i) * lD + n0 + nn] = acc[i];
      }
    }
    __syncthreads();
    // R += W K
    for (int tile = w; tile < nR; tile += NW) {
      const int mm = 16 * (tile / dt), n0 = 16 * (tile % dt);
      f64x4c acc;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = R[(mm + 4 * g + i) * lD + n0 + nn];
      mma_lds<double>(acc, mm + 16, g, [&](int kk) { return (double)W[(mm + pr) * lC + kk]; },
                      [&](int kk) { return (double)Ks[kk * lD + n0 + nn]; });
#pragma unroll
      for (int i = 0; i < 4; ++i) R[(mm + 4 * g + i) * lD + n0 + nn] = acc[i];
    }
    __syncthreads();
    // U = L (.) R Q^T
    for (int tile = w; tile < nW; tile += NW) {
      int mm, n0;
      lower(tile, mm, n0);
      f64x4c acc = zd;
      mma_lds<double>(acc, D, g, [&](int kk) { return R[(mm + pr) * lD + kk]; },
                      [&](int kk) { return (double)Qs[(n0 + nn) * lD + kk]; });
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = mm + 4 * g + i, u = n0 + nn;
        U[t * lC + u] = u <= t ? (float)acc[i] : 0.f;
      }
    }
    __syncthreads();
    // Sm = R SQ0 + U Q
    for (int tile = w; tile < nR; tile += NW) {
      const int mm = 16 * (tile / dt), n0 = 16 * (tile % dt);
      f64x4c acc = zd;
      mma_lds<double>(acc, D, g, [&](int kk) { return R[(mm + pr) * lD + kk]; },
                      [&](int kk) { return (double)SQ[kk * lD + n0 + nn]; });
      mma_lds<double>(acc, mm + 16, g, [&](int kk) { return (double)U[(mm + pr) * lC + kk]; },
                      [&](int kk) { return (double)Qs[kk * lD + n0 + nn]; });
#pragma unroll
      for (int i = 0; i < 4; ++i) Sm[(mm + 4 * g + i) * lD + n0 + nn] = acc[i];
    }
    __syncthreads();
    // Tm = L (.) Sm K^T;  the carry part of den (eight lanes per token)
    for (int tile = w; tile < nW; tile += NW) {
      int mm, n0;
      lower(tile, mm, n0);
      f64x4c acc = zd;
      mma_lds<double>(acc, D, g, [&](int kk) { return Sm[(mm + pr) * lD + kk]; },
                      [&](int kk) { return (double)Ks[(n0 + nn) * lD + kk]; });
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = mm + 4 * g + i, j = n0 + nn;
        Tm[t * lC + j] = j <= t ? (float)acc[i] : 0.f;
      }
    }
    {
      const int t = tid >> 3, p = tid & 7;
      double s = 0.0;
      if (t < C)
        for (int a = p; a < D; a += 8) s += Sm[t * lD + a] * mv[a];
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) s += __shfl_xor(s, o);
      if (p == 0 && t < C) dn[t] = s;
    }
    __syncthreads();
    if (normalized) {
      const int t = tid >> 3, p = tid & 7;
      double s = 0.0;
      if (t < C)
        for (int j = p; j <= t; j += 8) s += Tm[t * lC + j];
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) s += __shfl_xor(s, o);
      if (p == 0 && t < C) dn[t] += s;
      __syncthreads();
    }
    // O = Sm P0 + Tm V
    for (int tile = w; tile < nO; tile += NW) {
      const int mm = 16 * (tile / vt), n0 = 16 * (tile % vt);
      f64x4c acc = zd;
      mma_lds<double>(acc, D, g, [&](int kk) { return Sm[(mm + pr) * lD + kk]; },
                      [&](int kk) { return (double)Pm[kk * lV + n0 + nn]; });
      mma_lds<double>(acc, mm + 16, g, [&](int kk) { return (double)Tm[(mm + pr) * lC + kk]; },
                      [&](int kk) { return (double)Vs[kk * lV + n0 + nn]; });
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = mm + 4 * g + i;
        if (t0 + t < n)
          out[(head_tok + t0 + t) * DV + n0 + nn] = normalized ? (float)(acc[i] / (dn[t] + (double)eps)) : (float)acc[i];
      }
    }
    __syncthreads();
    // advance the moments past this tile: P0 += K^T V, SK0 += K^T K, SQ0 += Q^T Q (fp32), m0 += K^T 1
    {
      constexpr int nF = dt * vt, nQ = dt * dt;
      for (int tile = w; tile < nF + 2 * nQ; tile += NW) {
        f32x4c acc;
        if (tile < nF) {
          const int a0 = 16 * (tile / vt), b0 = 16 * (tile % vt);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = Pm[(a0 + 4 * g + i) * lV + b0 + nn];
          mma_lds<float>(acc, C, g, [&](int kk) { return Ks[kk * lD + a0 + nn]; },
                         [&](int kk) { return Vs[kk * lV + b0 + nn]; });
#pragma unroll
          for (int i = 0; i < 4; ++i) Pm[(a0 + 4 * g + i) * lV + b0 + nn] = acc[i];
        } else {
          const bool isK = tile < nF + nQ;
          const int u = isK ? tile - nF : tile - nF - nQ, a0 = 16 * (u / dt), b0 = 16 * (u % dt);
          float* S = isK ? SK : SQ;
          const float* Y = isK ? Ks : Qs;
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = S[(a0 + 4 * g + i) * lD + b0 + nn];
          mma_lds<float>(acc, C, g, [&](int kk) { return Y[kk * lD + a0 + nn]; },
                         [&](int kk) { return Y[kk * lD + b0 + nn]; });
#pragma unroll
          for (int i = 0; i < 4; ++i) S[(a0 + 4 * g + i) * lD + b0 + nn] = acc[i];
        }
      }
      const int a = tid >> 3, p = tid & 7;
      float sm = 0.f;
      if (a < D)
        for (int j = p; j < C; j += 8) sm += Ks[j * lD + a];
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) sm += __shfl_xor(sm, o);
      if (p == 0 && a < D) mv[a] += sm;
    }
    __syncthreads();
  }
}

template <typename T, int C, int D, int DV>
hipError_t run3(const Fwd& f, float* recs, float* pre, float* den, int P, int cps, hipStream_t s) {
  using Rc = Rec3<D, DV>;
  const T* q = static_cast<const T*>(f.q);
  const T* k = static_cast<const T*>(f.k);
  const T* v = static_cast<const T*>(f.v);
  const dim3 grid(P, f.BH);
  constexpr int nmom = Rc::oF, nbr = Rc::floats - Rc::oF;   // moments SK|SQ|P|m, brackets F|eta
  prof_start("hla3_moments", s);
  HLA_LAUNCH((k3_moments<T, C, D, DV>), grid, dim3(kT3), 0, s, q, k, v, recs, f.n, cps, P);
  prof_stop(s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  prof_start("hla3_prefix", s);
  HLA_LAUNCH((k3_prefix<D, DV>), dim3((nmom + kT3 - 1) / kT3, f.BH), dim3(kT3), 0, s, recs, pre, P, 0, nmom);
  prof_stop(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (!f.masked) {     // the unmasked operator: outputs whole from the moment prefix
    prof_start("hla3_walk", s);
    HLA_LAUNCH((k3u_walk<T, C, D, DV>), grid, dim3(kT3), 0, s, q, k, v, f.out, pre, f.n, cps, P, f.normalized,
               f.eps);
    prof_stop(s);
    return hipGetLastError();
  }
  prof_start("hla3_walk", s);
  HLA_LAUNCH((k3_walk<T, C, D, DV>), grid, dim3(kT3), 0, s, q, k, v, f.out, den, recs, pre, f.n, cps, P);
  prof_stop(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  prof_start("hla3_prefix", s);
  HLA_LAUNCH((k3_prefix<D, DV>), dim3((nbr + kT3 - 1) / kT3, f.BH), dim3(kT3), 0, s, recs, pre, P, (int)Rc::oF, nbr);
  prof_stop(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  prof_start("hla3_fix", s);
  HLA_LAUNCH((k3_fix<T, C, D, DV>), grid, dim3(kT3), 0, s, q, f.out, den, pre, f.n, cps, P, f.normalized, f.eps);
  prof_stop(s);
  return hipGetLastError();
}

int tile3(int chunk) { return chunk >= 32 ? 32 : chunk; }

void plan3(int BH, int n, int chunk, int* P, int* cps) {
  const int C = tile3(chunk);
  const int M = (n + C - 1) / C;
  int p = 512 / BH;
  if (const char* e = getenv("HLA_FUSED_SEGMENTS")) p = atoi(e);
  if (p < 1) p = 1;
  if (p > M) p = M;
  *cps = (M + p - 1) / p;
  *P = (M + *cps - 1) / *cps;
}

size_t rec_floats(int d, int dv) { return 2 * (size_t)d * d + 2 * (size_t)d * dv + 2 * (size_t)d; }

}  // namespace

bool hla3_supported(int d, int dv, int chunk, int masked) {
  return (masked == 0 || masked == 1) && (d == 16 || d == 32) && (dv == 16 || dv == 32) &&
         (chunk >= 16 && chunk <= 128);
}

size_t hla3_workspace(int BH, int n, int d, int dv, int chunk) {
  int P, cps;
  plan3(BH, n, chunk, &P, &cps);
  const size_t a = ((sizeof(float) * (size_t)BH * P * rec_floats(d, dv)) + 255) & ~size_t(255);
  return 2 * a + sizeof(float) * (size_t)BH * n + 256;
}

hipError_t launch_hla3(const Fwd& f, void* workspace, hipStream_t s) {
  int P, cps;
  plan3(f.BH, f.n, f.chunk, &P, &cps);
  char* base = static_cast<char*>(workspace);
  const size_t a = ((sizeof(float) * (size_t)f.BH * P * rec_floats(f.d, f.dv)) + 255) & ~size_t(255);
  float* recs = reinterpret_cast<float*>(base);         // [BH][P] records
  float* pre = reinterpret_cast<float*>(base + a);      // their exclusive running sums
  float* den = reinterpret_cast<float*>(base + 2 * a);
  const int C = tile3(f.chunk);
#define HLA3_CASE(T_, C_, D_, DV_) \
  if (C == C_ && f.d == D_ && f.dv == DV_) return run3<T_, C_, D_, DV_>(f, recs, pre, den, P, cps, s);
#define HLA3_DT(T_)                                                                                       \
  HLA3_CASE(T_, 16, 16, 16) HLA3_CASE(T_, 16, 16, 32) HLA3_CASE(T_, 16, 32, 16) HLA3_CASE(T_, 16, 32, 32) \
  HLA3_CASE(T_, 32, 16, 16) HLA3_CASE(T_, 32, 16, 32) HLA3_CASE(T_, 32, 32, 16) HLA3_CASE(T_, 32, 32, 32)
  if (f.dtype == 1) {
    HLA3_DT(uint16_t)
  } else {
    HLA3_DT(float)
  }
#undef HLA3_DT
#undef HLA3_CASE
  return hipErrorNotSupported;
}

}  // namespace hla
