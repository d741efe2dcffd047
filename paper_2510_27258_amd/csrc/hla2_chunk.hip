// Chunk-parallel second-order HLA, general path (fp32 SIMT arithmetic).
//
// Two kernels, one workgroup per (head, chunk):
//   k_chunk_summary  the chunk's masked summary (S, C, m, G, h) with zero
//                    carry-in, built from dense intra-chunk products
//                    (prefix summaries of Sec. 3 and the masking summaries G, h
//                    of Sec. 3.1, restricted to the chunk).
//   k_readout        per-token outputs of a chunk from its exclusive carry-in
//                    state (Thm. 1 applied to carry (+) local prefix, Eq.
//                    (semidirect); Rem. scan-modes, inter-chunk parallelism).
// Any d, dv <= 128 and chunk <= 128 are accepted; fp32 or bf16 inputs.
//
// Decay gamma in (0, 1] (decay section; decay-aware monoid): the pair (i, j)
// enters row t with weight gamma^{(t-i)+(t-j)}, the masked operator keeping
// i <= j.  A chunk's summary is then taken relative to its last token, and
// the scan composes chunks with attenuation rho = gamma^length (G and h by
// rho^2, the cross term by rho).  gamma = 1 is the undecayed operator: every
// power below is exp2(0) = 1 exactly.
#include "common.h"
#include "profile.h"

namespace hla {

// ----------------------------------------------------------------------------
// Chunk summary.  With A_s[i][j] = [j < i] k_i . q_j (strictly lower):
//   S = K^T K,  C = Q^T V,  m = Q^T 1,  G = K^T (A_s V),  h = K^T (A_s 1).
// G is sum_i k_i k_i^T C_{i-1} with C local to the chunk (Sec. 3.1).
// With decay every token t of a chunk of L tokens carries w_t = gamma^(L-1-t)
// in S, C and m and the pair (i, j) carries w_i w_j in G, h.
//
// The chunk is walked in blocks of TB = min(chunk, 32) tokens staged in LDS
// (fp32, zero rows past n), so any chunk up to 128 fits:
//   1. Y = A_s [V | 1] block row by block row: Y_ib = sum_{jb <= ib} A_s(ib, jb) [V_jb | 1];
//   2. S, C, m, G, h summed over the token blocks, S, C and G in 4 x 4
//      register tiles that each thread keeps for the whole chunk.
// fp32 arithmetic throughout.  LDS: K, Q [TB][d+1], V [TB][dv+1],
// A [TB][TB+1], Y [chunk][dv+1].
// ----------------------------------------------------------------------------
constexpr int kSumThreads = 512;
constexpr int kSumTiles = 2;    // 4 x 4 tiles of a d x d or d x dv product per thread (d, dv <= 128)

// acc[r] += the thread's r-th 4 x 4 tile of A B (M x N, K terms), tiles dealt
// round-robin over the workgroup; A(m, k) = al(m, k), B(k, n) = bl(k, n).
template <typename AL, typename BL>
__device__ __forceinline__ void tile_acc(float (&acc)[kSumTiles][16], int M, int N, int K, AL al, BL bl) {
  const int tn = N / 4, tiles = (M / 4) * tn;
#pragma unroll
  for (int r = 0; r < kSumTiles; ++r) {
    const int ti = threadIdx.x + kSumThreads * r;
    if (ti >= tiles) continue;
    const int m0 = (ti / tn) * 4, n0 = (ti % tn) * 4;
    for (int kk = 0; kk < K; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = al(m0 + i, kk);
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = bl(kk, n0 + j);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[r][i * 4 + j] += av[i] * bv[j];
    }
  }
}

template <typename F>
__device__ __forceinline__ void tile_put(const float (&acc)[kSumTiles][16], int M, int N, F put) {
  const int tn = N / 4, tiles = (M / 4) * tn;
#pragma unroll
  for (int r = 0; r < kSumTiles; ++r) {
    const int ti = threadIdx.x + kSumThreads * r;
    if (ti >= tiles) continue;
    const int m0 = (ti / tn) * 4, n0 = (ti % tn) * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) put(m0 + i, n0 + j, acc[r][i * 4 + j]);
  }
}

template <typename T>
__global__ __launch_bounds__(kSumThreads) void k_chunk_summary(const T* __restrict__ q, const T* __restrict__ k,
                                                               const T* __restrict__ v, float* __restrict__ states,
                                                               int n, int d, int dv, int chunk, int M, float lg2g) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0);
  const int TB = chunk < 32 ? chunk : 32, nb = chunk / TB;
  const int ld = d + 1, ldv = dv + 1, lda = TB + 1;
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  float* Kb = smem;                          // [TB][ld]
  float* Qb = Kb + TB * ld;                  // [TB][ld]
  float* Vb = Qb + TB * ld;                  // [TB][ldv]
  float* Ab = Vb + TB * ldv;                 // [TB][lda]
  float* Y = Ab + TB * lda;                  // [chunk][ldv]: A_s V | A_s 1
  float* st = states + ((size_t)bh * M + c) * state_floats(d, dv);
  auto w = [&](int t) { return exp2f(lg2g * (float)(L - 1 - t)); };   // gamma^(L-1-t)
  auto stage_qk = [&](float* dst, const T* src, int tb) {
    for (int idx = tid; idx < TB * d; idx += kSumThreads) {
      const int t = idx / d, a = idx % d, tt = tb * TB + t;
      dst[t * ld + a] = tt < L ? ldf(src, qk_base + (size_t)tt * d + a) : 0.f;
    }
  };
  auto stage_v = [&](int tb) {
    for (int idx = tid; idx < TB * dv; idx += kSumThreads) {
      const int t = idx / dv, b = idx % dv, tt = tb * TB + t;
      Vb[t * ldv + b] = tt < L ? ldf(v, v_base + (size_t)tt * dv + b) : 0.f;
    }
  };

  // 1. Y rows of block ib from the blocks jb <= ib
  for (int ib = 0; ib < nb; ++ib) {
    float accy[kSumTiles][16] = {};
    float ysum = 0.f;
    for (int jb = 0; jb <= ib; ++jb) {
      if (jb == 0) stage_qk(Kb, k, ib);
      stage_qk(Qb, q, jb);
      stage_v(jb);
      __syncthreads();
      // A_s(ib, jb): [j < i] gamma^(2L-2-i-j) k_i . q_j
      for (int idx = tid; idx < TB * TB; idx += kSumThreads) {
        const int i = idx / TB, j = idx % TB, gi = ib * TB + i, gj = jb * TB + j;
        float x = 0.f;
        if (gj < gi) {
          for (int a = 0; a < d; ++a) x += Kb[i * ld + a] * Qb[j * ld + a];
          x *= exp2f(lg2g * (float)(2 * L - 2 - gi - gj));
        }
        Ab[i * lda + j] = x;
      }
      __syncthreads();
      tile_acc(accy, TB, dv, TB, [&](int i, int j) { return Ab[i * lda + j]; },
               [&](int j, int b) { return Vb[j * ldv + b]; });
      if (tid < TB)
        for (int j = 0; j < TB; ++j) ysum += Ab[tid * lda + j];
      __syncthreads();             // Q, V and A are restaged for the next block
    }
    tile_put(accy, TB, dv, [&](int i, int b, float x) { Y[(ib * TB + i) * ldv + b] = x; });
    if (tid < TB) Y[(ib * TB + tid) * ldv + dv] = ysum;
  }

  // 2. S = K^T diag(w) K, C = Q^T diag(w) V, m = Q^T w, G = K^T Y, h = K^T (A_s 1)
  float accs[kSumTiles][16] = {}, accc[kSumTiles][16] = {}, accg[kSumTiles][16] = {};
  float am = 0.f, ah = 0.f;
  for (int tb = 0; tb < nb; ++tb) {
    stage_qk(Kb, k, tb);
    stage_qk(Qb, q, tb);
    stage_v(tb);
    if (tid < TB) Ab[tid] = tb * TB + tid < L ? w(tb * TB + tid) : 0.f;   // the block's token weights
    __syncthreads();               // also orders the Y writes of step 1 before their reads
    const float* Yb = Y + tb * TB * ldv;
    tile_acc(accs, d, d, TB, [&](int a, int t) { return Kb[t * ld + a]; },
             [&](int t, int b) { return Ab[t] * Kb[t * ld + b]; });
    tile_acc(accc, d, dv, TB, [&](int a, int t) { return Qb[t * ld + a]; },
             [&](int t, int b) { return Ab[t] * Vb[t * ldv + b]; });
    tile_acc(accg, d, dv, TB, [&](int a, int t) { return Kb[t * ld + a]; },
             [&](int t, int b) { return Yb[t * ldv + b]; });
    if (tid < d)
      for (int t = 0; t < TB; ++t) {
        am += Ab[t] * Qb[t * ld + tid];
        ah += Kb[t * ld + tid] * Yb[t * ldv + dv];
      }
    __syncthreads();
  }
  tile_put(accs, d, d, [&](int a, int b, float x) { st[(size_t)a * d + b] = x; });
  tile_put(accc, d, dv, [&](int a, int b, float x) { st[off_C(d, dv) + (size_t)a * dv + b] = x; });
  tile_put(accg, d, dv, [&](int a, int b, float x) { st[off_G(d, dv) + (size_t)a * dv + b] = x; });
  if (tid < d) {
    st[off_m(d, dv) + tid] = am;
    st[off_h(d, dv) + tid] = ah;
  }
}

// ----------------------------------------------------------------------------
// Readout of one chunk from its carry-in (S0, C0, m0, G0, h0).
// With p_t = S0 q_t and r_j = S_j q_j = p_j + sum_{i<=j, i in chunk} (k_i.q_j) k_i:
//   masked:   o_t = q_t^T (S0 C0 - G0) + sum_{j<=t} (q_t . r_j) v_j
//             den_t = q_t^T (S0 m0 - h0) + sum_{j<=t} (q_t . r_j)
//   unmasked: o_t = r_t^T C0 + sum_{j<=t} (r_t . q_j) v_j,   den_t = r_t . m0 + sum_{j<=t} r_t . q_j
// (q_t^T S_t = r_t^T since S is symmetric.)  These are Thm. 1 evaluated on
// the inclusive state carry (+) local prefix, grouped so that no d x dv
// product of states is formed.  With decay (local index a of token t, carry
// taken at the token before the chunk):
//   r_j = g^(a_j+1) S0 q_j + sum_{i<=j} g^(a_j-a_i) (k_i.q_j) k_i,
//   masked:   o_t = g^(2(a+1)) q_t^T (S0 C0 - G0) + sum_{j<=t} g^(2(a-a_j)) (q_t . r_j) v_j
//   unmasked: o_t = g^(a+1) r_t^T C0 + sum_{j<=t} g^(a-a_j) (r_t . q_j) v_j
// (the decayed inclusive state is g^(a+1) S0 + S_loc etc., and the S_loc C0
// terms of S C - G still cancel).
// ----------------------------------------------------------------------------
// The dot products over d accumulate in fp64 and R is held in fp64: a row
// whose value is far below the size of its terms (row 0 is (q_0.k_0)^2 v_0,
// with q_0.k_0 a cancelling dot product) keeps the fp32-input bar only when
// r_j and q_t . r_j are not rounded to fp32 on the way.  Chunks of up to 64
// tokens (the forward paths cut larger chunks, exact by Thm. 2).
//
// The chunk's q and k are staged in LDS (fp32, zero rows past n), and every
// product runs as register tiles: a thread owns 4 x 4 outputs at a time
// (512 threads, so two waves share each SIMD).
// LDS: R [chunk][d+1] fp64, Q and K [chunk][d+1] fp32, W/T [chunk][chunk+1]
// fp32, den [chunk] fp32 (149 KB at chunk 64, d 128).

// Out(m, n) = sum_k A(m, k) B(k, n) for m < M, n < N (multiples of 4), k < K,
// 4 x 4 outputs per thread and tile.  A(m, k) = a[m sam + k sak] (LDS);
// B(k, n) = bl(k, n).  lower: tiles wholly above the diagonal (n > m) are not
// computed; epi(m, n, 0) is called for their outputs.
template <typename Acc, typename TA, typename BL, typename EPI>
__device__ __forceinline__ void tgemm(int M, int N, int K, const TA* a, int sam, int sak, BL bl, EPI epi,
                                      bool lower) {
  const int tn = N / 4, tiles = (M / 4) * tn;
  for (int ti = threadIdx.x; ti < tiles; ti += blockDim.x) {
    const int m0 = (ti / tn) * 4, n0 = (ti % tn) * 4;
    Acc acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = Acc(0);
    if (!lower || n0 <= m0 + 3) {
      for (int kk = 0; kk < K; ++kk) {
        Acc av[4], bv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) av[i] = (Acc)a[(m0 + i) * sam + kk * sak];
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[j] = (Acc)bl(kk, n0 + j);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * bv[j];
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) epi(m0 + i, n0 + j, acc[i][j]);
  }
}

template <typename T>
__global__ __launch_bounds__(512) void k_readout(const T* __restrict__ q, const T* __restrict__ k,
                                                 const T* __restrict__ v, const float* __restrict__ prefix,
                                                 float* __restrict__ out, float* __restrict__ den_out, int n,
                                                 int d, int dv, int chunk, int M, int masked, int normalized,
                                                 float eps, float lg2g) {
  extern __shared__ double smemd[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0), Lp = chunk, ld = d + 1, ldw = chunk + 1;
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  double* R = smemd;                                           // [Lp][ld]
  float* Qs = reinterpret_cast<float*>(R + (size_t)Lp * ld);   // [Lp][ld]
  float* Ks = Qs + (size_t)Lp * ld;                            // [Lp][ld]
  float* W = Ks + (size_t)Lp * ld;                             // [Lp][ldw]
  float* dn = W + (size_t)Lp * ldw;                            // [Lp]
  const float* st = prefix + ((size_t)bh * M + c) * state_floats(d, dv);
  const float* S0 = st;
  const float* C0 = st + off_C(d, dv);
  const float* m0 = st + off_m(d, dv);
  const float* G0 = st + off_G(d, dv);
  const float* h0 = st + off_h(d, dv);
  float* o = out + v_base;
  auto g = [&](int e) { return exp2f(lg2g * (float)e); };      // gamma^e

  for (int idx = tid; idx < Lp * d; idx += blockDim.x) {
    const int t = idx / d, a = idx % d;
    Qs[t * ld + a] = t < L ? ldf(q, qk_base + (size_t)t * d + a) : 0.f;
    Ks[t * ld + a] = t < L ? ldf(k, qk_base + (size_t)t * d + a) : 0.f;
  }
  __syncthreads();

  // P = Q S0 into R;  W[t][i] = [i <= t] g^(t-i) q_t . k_i
  tgemm<double>(Lp, d, d, Qs, ld, 1, [&](int kk, int nn) { return S0[(size_t)kk * d + nn]; },
                [&](int m, int nn, double x) { R[m * ld + nn] = x; }, false);
  tgemm<double>(Lp, Lp, d, Qs, ld, 1, [&](int kk, int nn) { return Ks[nn * ld + kk]; },
                [&](int t, int i, double x) { W[t * ldw + i] = i <= t ? (float)(x * (double)g(t - i)) : 0.f; },
                true);
  __syncthreads();
  if (masked) {
    // carry term g^(2(a+1)) (q_t^T S0 C0 - q_t^T G0) (and its denominator)
    const int tn = dv / 4, tiles = (Lp / 4) * tn;
    for (int ti = tid; ti < tiles; ti += blockDim.x) {
      const int mm = (ti / tn) * 4, n0 = (ti % tn) * 4;
      double acc[4][4] = {};
      for (int a = 0; a < d; ++a) {
        double rc[4], qc[4], cb[4], gb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          rc[i] = R[(mm + i) * ld + a];
          qc[i] = Qs[(mm + i) * ld + a];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          cb[j] = C0[(size_t)a * dv + n0 + j];
          gb[j] = G0[(size_t)a * dv + n0 + j];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] += rc[i] * cb[j] - qc[i] * gb[j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (mm + i < L)
#pragma unroll
          for (int j = 0; j < 4; ++j) o[(size_t)(mm + i) * dv + n0 + j] = (float)acc[i][j] * g(2 * (mm + i) + 2);
    }
    for (int t = tid; t < L; t += blockDim.x) {
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += R[t * ld + a] * (double)m0[a] - (double)Qs[t * ld + a] * (double)h0[a];
      dn[t] = (float)s * g(2 * t + 2);
    }
  }
  __syncthreads();
  // the carry part of r_t decays by g^(a+1); then R += W K  (r_j = S_j q_j)
  tgemm<double>(Lp, d, Lp, W, ldw, 1, [&](int kk, int nn) { return Ks[kk * ld + nn]; },
                [&](int j, int a, double x) { R[j * ld + a] = R[j * ld + a] * (double)g(j + 1) + x; }, false);
  __syncthreads();
  // T[t][j] = [j <= t] g^(2(t-j)) (q_t . r_j)  (masked)  or  g^(t-j) (r_t . q_j)  (unmasked)
  if (masked)
    tgemm<double>(Lp, Lp, d, Qs, ld, 1, [&](int kk, int nn) { return R[nn * ld + kk]; },
                  [&](int t, int j, double x) { W[t * ldw + j] = j <= t ? (float)(x * (double)g(2 * (t - j))) : 0.f; },
                  true);
  else
    tgemm<double>(Lp, Lp, d, R, ld, 1, [&](int kk, int nn) { return (double)Qs[nn * ld + kk]; },
                  [&](int t, int j, double x) { W[t * ldw + j] = j <= t ? (float)(x * (double)g(t - j)) : 0.f; },
                  true);
  if (!masked) {
    tgemm<double>(Lp, dv, d, R, ld, 1, [&](int kk, int nn) { return C0[(size_t)kk * dv + nn]; },
                  [&](int t, int b, double x) {
                    if (t < L) o[(size_t)t * dv + b] = (float)x * g(t + 1);
                  },
                  false);
    for (int t = tid; t < L; t += blockDim.x) {
      double s = 0.0;
      for (int a = 0; a < d; ++a) s += R[t * ld + a] * (double)m0[a];
      dn[t] = (float)s * g(t + 1);
    }
  }
  __syncthreads();
  if (normalized) {
    for (int t = tid; t < L; t += blockDim.x) {
      float s = dn[t];
      for (int j = 0; j <= t; ++j) s += W[t * ldw + j];
      dn[t] = s;
      if (den_out) den_out[(size_t)bh * n + t0 + t] = s;
    }
    __syncthreads();
  }
  // o_t += sum_{j <= t} T[t][j] v_j (rows past the chunk's tokens read as zero)
  tgemm<float>(Lp, dv, Lp, W, ldw, 1,
               [&](int kk, int nn) { return kk < L ? ldf(v, v_base + (size_t)kk * dv + nn) : 0.f; },
               [&](int t, int b, float x) {
                 if (t < L) {
                   const float y = o[(size_t)t * dv + b] + x;
                   o[(size_t)t * dv + b] = normalized ? y / (dn[t] + eps) : y;
                 }
               },
               false);
}

// ----------------------------------------------------------------------------
static size_t summary_lds(int chunk, int d, int dv) {
  const size_t tb = chunk < 32 ? chunk : 32;
  return sizeof(float) * (2 * tb * (d + 1) + tb * (dv + 1) + tb * (tb + 1) + (size_t)chunk * (dv + 1));
}
static size_t readout_lds(int chunk, int d) {
  return sizeof(double) * (size_t)chunk * (d + 1) +
         sizeof(float) * (2 * (size_t)chunk * (d + 1) + (size_t)chunk * (chunk + 1) + chunk);
}

hipError_t launch_chunk_summaries(const void* q, const void* k, const void* v, float* states,
                                  int BH, int n, int d, int dv, int chunk, int dtype, hipStream_t s, float gamma) {
  const float lg2g = log2f(gamma);
  const int M = (n + chunk - 1) / chunk;
  const size_t lds = summary_lds(chunk, d, dv);
  dim3 grid(M, BH), block(kSumThreads);
  if (dtype == 1) {
    auto kern = k_chunk_summary<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const uint16_t*)q, (const uint16_t*)k,
                       (const uint16_t*)v, states, n, d, dv, chunk, M, lg2g);
  } else {
    auto kern = k_chunk_summary<float>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const float*)q, (const float*)k, (const float*)v,
                       states, n, d, dv, chunk, M, lg2g);
  }
  return hipGetLastError();
}

hipError_t launch_readout(const Fwd& f, const float* prefix, hipStream_t s) {
  if (f.chunk > kReadoutMaxChunk) return hipErrorInvalidValue;
  const float lg2g = log2f(f.gamma);
  const int M = (f.n + f.chunk - 1) / f.chunk;
  const size_t lds = readout_lds(f.chunk, f.d);
  dim3 grid(M, f.BH), block(512);
  if (f.dtype == 1) {
    auto kern = k_readout<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const uint16_t*)f.q, (const uint16_t*)f.k,
                       (const uint16_t*)f.v, prefix, f.out, f.den_out, f.n, f.d, f.dv, f.chunk, M, f.masked,
                       f.normalized, f.eps, lg2g);
  } else {
    auto kern = k_readout<float>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const float*)f.q, (const float*)f.k, (const float*)f.v,
                       prefix, f.out, f.den_out, f.n, f.d, f.dv, f.chunk, M, f.masked, f.normalized, f.eps, lg2g);
  }
  return hipGetLastError();
}

}  // namespace hla
