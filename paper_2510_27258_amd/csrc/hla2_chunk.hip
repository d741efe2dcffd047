// Chunk-parallel second-order HLA, general path (fp32 and fp64 arithmetic).
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
#include "mfma16.h"
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
//   2. S, C, m, G, h summed over the token blocks.
// Every product runs on fp32 MFMA (v_mfma_f32_16x16x4_f32: lane l = 16 g + n
// supplies A[n][k_g] and B[k_g][n] and holds D[4 g + i][n], i < 4): fp32
// products and sums, one 16 x 16 output tile per wave at a time; a wave keeps
// its tiles of Y (over the blocks jb) and of S, C, G (over the chunk) in its
// accumulators.  LDS rows are padded to 17 floats modulo 32, so that the
// reads along rows (k over tokens) and along columns (A_s = K Q^T, k over the
// dimensions) of a half-wave fall in distinct banks but one.
// LDS: K, Q [TB][ld], V [TB][ldv], A [TB][lda], Y [chunk][ldv], w [TB].
// ----------------------------------------------------------------------------
constexpr int kSumThreads = 512, kSumWaves = kSumThreads / 64;
constexpr int kSumTiles = 8;   // 16 x 16 tiles of S, C or G per wave: (128 / 16)^2 over 8 waves

__host__ __device__ constexpr int sum_ld(int x) { return (x + 31) / 32 * 32 + 17; }


__device__ __forceinline__ float4 ld4f(const float* p, size_t i) { return *reinterpret_cast<const float4*>(p + i); }
__device__ __forceinline__ float4 ld4f(const uint16_t* p, size_t i) {
  const uint2 x = *reinterpret_cast<const uint2*>(p + i);
  return make_float4(__uint_as_float(x.x << 16), __uint_as_float(x.x & 0xffff0000u), __uint_as_float(x.y << 16),
                     __uint_as_float(x.y & 0xffff0000u));
}

template <typename T>
__global__ __launch_bounds__(kSumThreads) void k_chunk_summary_blocks(const T* __restrict__ q, const T* __restrict__ k,
                                                               const T* __restrict__ v, float* __restrict__ states,
                                                               int n, int d, int dv, int chunk, int M, float lg2g) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, nn = tid & 15, g = (tid >> 4) & 3;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0);
  const int TB = chunk < 32 ? chunk : 32, nb = chunk / TB;
  const int ld = sum_ld(d), ldv = sum_ld(dv), lda = sum_ld(TB);
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  float* Kb = smem;                          // [TB][ld]
  float* Qb = Kb + TB * ld;                  // [TB][ld]
  float* Vb = Qb + TB * ld;                  // [TB][ldv]
  float* Ab = Vb + TB * ldv;                 // [TB][lda]
  float* Y = Ab + TB * lda;                  // [chunk][ldv]: A_s V | A_s 1
  float* wv = Y + chunk * ldv;               // [TB]: the block's token weights
  float* st = states + ((size_t)bh * M + c) * state_floats(d, dv);
  auto wt = [&](int t) { return exp2f(lg2g * (float)(L - 1 - t)); };   // gamma^(L-1-t)
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
  const f32x4c zero = {0.f, 0.f, 0.f, 0.f};

  // 1. Y rows of block ib from the blocks jb <= ib
  const int at = TB / 16, ytn = dv / 16, ytiles = at * ytn;   // ytiles <= 16: two per wave
  for (int ib = 0; ib < nb; ++ib) {
    f32x4c ya[2] = {zero, zero};
    float ysum = 0.f;
    for (int jb = 0; jb <= ib; ++jb) {
      if (jb == 0) stage_qk(Kb, k, ib);
      stage_qk(Qb, q, jb);
      stage_v(jb);
      __syncthreads();
      // A_s(ib, jb) = [j < i] gamma^(2L-2-i-j) k_i . q_j, one 16 x 16 tile per wave
      if (w < at * at) {
        const int i0 = (w / at) * 16, j0 = (w % at) * 16;
        f32x4c x = zero;
        if (jb < ib || j0 <= i0)
          for (int k0 = 0; k0 < d; k0 += 4) x = mfma4(Kb[(i0 + nn) * ld + k0 + g], Qb[(j0 + nn) * ld + k0 + g], x);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = i0 + 4 * g + e, j = j0 + nn, gi = ib * TB + i, gj = jb * TB + j;
          Ab[i * lda + j] = gj < gi ? x[e] * exp2f(lg2g * (float)(2 * L - 2 - gi - gj)) : 0.f;
        }
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int tile = w + kSumWaves * r;
        if (tile < ytiles) {
          const int i0 = (tile / ytn) * 16, b0 = (tile % ytn) * 16;
          for (int k0 = 0; k0 < TB; k0 += 4)
            ya[r] = mfma4(Ab[(i0 + nn) * lda + k0 + g], Vb[(k0 + g) * ldv + b0 + nn], ya[r]);
        }
      }
      if (tid < TB)
        for (int j = 0; j < TB; ++j) ysum += Ab[tid * lda + j];
      __syncthreads();             // Q, V and A are restaged for the next block
    }
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int tile = w + kSumWaves * r;
      if (tile < ytiles) {
        const int i0 = (tile / ytn) * 16, b0 = (tile % ytn) * 16;
#pragma unroll
        for (int e = 0; e < 4; ++e) Y[(ib * TB + i0 + 4 * g + e) * ldv + b0 + nn] = ya[r][e];
      }
    }
    if (tid < TB) Y[(ib * TB + tid) * ldv + dv] = ysum;
  }

  // 2. S = K^T diag(w) K, C = Q^T diag(w) V, m = Q^T w, G = K^T Y, h = K^T (A_s 1)
  const int stn = d / 16, sti = stn * stn, ctn = dv / 16, cti = stn * ctn;
  f32x4c as[kSumTiles], ac[kSumTiles], ag[kSumTiles];
#pragma unroll
  for (int r = 0; r < kSumTiles; ++r) as[r] = ac[r] = ag[r] = zero;
  float am = 0.f, ah = 0.f;
  for (int tb = 0; tb < nb; ++tb) {
    stage_qk(Kb, k, tb);
    stage_qk(Qb, q, tb);
    stage_v(tb);
    if (tid < TB) wv[tid] = tb * TB + tid < L ? wt(tb * TB + tid) : 0.f;
    __syncthreads();               // also orders the Y writes of step 1 before their reads
    const float* Yb = Y + tb * TB * ldv;
#pragma unroll
    for (int r = 0; r < kSumTiles; ++r) {
      const int tile = w + kSumWaves * r;
      if (tile < sti) {
        const int a0 = (tile / stn) * 16, b0 = (tile % stn) * 16;
        for (int k0 = 0; k0 < TB; k0 += 4) {
          const int t = k0 + g;
          as[r] = mfma4(Kb[t * ld + a0 + nn], wv[t] * Kb[t * ld + b0 + nn], as[r]);
        }
      }
      if (tile < cti) {
        const int a0 = (tile / ctn) * 16, b0 = (tile % ctn) * 16;
        for (int k0 = 0; k0 < TB; k0 += 4) {
          const int t = k0 + g;
          ac[r] = mfma4(Qb[t * ld + a0 + nn], wv[t] * Vb[t * ldv + b0 + nn], ac[r]);
          ag[r] = mfma4(Kb[t * ld + a0 + nn], Yb[t * ldv + b0 + nn], ag[r]);
        }
      }
    }
    if (tid < d)
      for (int t = 0; t < TB; ++t) {
        am += wv[t] * Qb[t * ld + tid];
        ah += Kb[t * ld + tid] * Yb[t * ldv + dv];
      }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < kSumTiles; ++r) {
    const int tile = w + kSumWaves * r;
    if (tile < sti) {
      const int a0 = (tile / stn) * 16, b0 = (tile % stn) * 16;
#pragma unroll
      for (int e = 0; e < 4; ++e) st[(size_t)(a0 + 4 * g + e) * d + b0 + nn] = as[r][e];
    }
    if (tile < cti) {
      const int a0 = (tile / ctn) * 16, b0 = (tile % ctn) * 16;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        st[off_C(d, dv) + (size_t)(a0 + 4 * g + e) * dv + b0 + nn] = ac[r][e];
        st[off_G(d, dv) + (size_t)(a0 + 4 * g + e) * dv + b0 + nn] = ag[r][e];
      }
    }
  }
  if (tid < d) {
    st[off_m(d, dv) + tid] = am;
    st[off_h(d, dv) + tid] = ah;
  }
}

// One pass over the blocks when the chunk's Q and V fit in LDS (the forward
// paths' chunks of up to 64 tokens): block tb is staged once (its Q and V
// kept for the later blocks, its K for this step only), with the next
// block's loads in flight meanwhile, and
//   A_row = A_s(tb, 0 .. tb),  Y_tb = A_row [V_{0..tb} | 1],
//   S += K_tb^T diag(w) K_tb,  C += Q_tb^T diag(w) V_tb,  G += K_tb^T Y_tb,
//   m += Q_tb^T w,  h += K_tb^T (A_row 1).
// LDS: Q, V [chunk][ld, ldv], K [TB][ld], A_row [TB][sum_ld(chunk)],
// Y [TB][ldv], w [TB]; the column sums of m and h are reduced through A_row.
template <typename T>
__global__ __launch_bounds__(kSumThreads) void k_chunk_summary(const T* __restrict__ q, const T* __restrict__ k,
                                                               const T* __restrict__ v, float* __restrict__ states,
                                                               int n, int d, int dv, int chunk, int M, float lg2g) {
  extern __shared__ float smem[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, nn = tid & 15, g = (tid >> 4) & 3;
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0);
  const int TB = chunk < 32 ? chunk : 32, nb = chunk / TB;
  const int ld = sum_ld(d), ldv = sum_ld(dv), lar = sum_ld(chunk);
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  float* Qa = smem;                          // [chunk][ld]
  float* Va = Qa + chunk * ld;               // [chunk][ldv]
  float* Kb = Va + chunk * ldv;              // [TB][ld]
  float* Ar = Kb + TB * ld;                  // [TB][lar]
  float* Yb = Ar + TB * lar;                 // [TB][ldv]: A_row V | A_row 1
  float* wv = Yb + TB * ldv;                 // [TB]
  float* st = states + ((size_t)bh * M + c) * state_floats(d, dv);
  const f32x4c zero = {0.f, 0.f, 0.f, 0.f};
  // staging: piece e = tid + 512 i of a block is row e / (width / 4), columns 4 (e % (width / 4)) ..
  const int nqk = TB * d / 4, nv = TB * dv / 4;
  float4 pk[2], pq[2], pv[2];
  auto fetch = [&](int tb) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int e = tid + kSumThreads * i;
      const int tq = tb * TB + e / (d / 4), tv = tb * TB + e / (dv / 4);
      const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
      const bool okq = e < nqk && tq < L, okv = e < nv && tv < L;
      pk[i] = okq ? ld4f(k, qk_base + (size_t)tq * d + (e % (d / 4)) * 4) : z;
      pq[i] = okq ? ld4f(q, qk_base + (size_t)tq * d + (e % (d / 4)) * 4) : z;
      pv[i] = okv ? ld4f(v, v_base + (size_t)tv * dv + (e % (dv / 4)) * 4) : z;
    }
  };
  auto put4 = [&](float* dst, const float4& x) { dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w; };
  const int at = TB / 16, stn = d / 16, sti = stn * stn, ctn = dv / 16, cti = stn * ctn, ytiles = at * ctn;
  f32x4c as[kSumTiles], ac[kSumTiles], ag[kSumTiles];
#pragma unroll
  for (int r = 0; r < kSumTiles; ++r) as[r] = ac[r] = ag[r] = zero;
  // m and h: thread (column a, part p) sums the block rows p, p + P, ...
  const int P = kSumThreads / d, ma = tid % d, mp = tid / d;
  float am = 0.f, ah = 0.f;
  fetch(0);
  for (int tb = 0; tb < nb; ++tb) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int e = tid + kSumThreads * i;
      if (e < nqk) {
        const int t = e / (d / 4), a = (e % (d / 4)) * 4;
        put4(Kb + t * ld + a, pk[i]);
        put4(Qa + (tb * TB + t) * ld + a, pq[i]);
      }
      if (e < nv) put4(Va + (tb * TB + e / (dv / 4)) * ldv + (e % (dv / 4)) * 4, pv[i]);
    }
    if (tid < TB) wv[tid] = tb * TB + tid < L ? exp2f(lg2g * (float)(L - 1 - tb * TB - tid)) : 0.f;
    if (tb + 1 < nb) fetch(tb + 1);
    __syncthreads();
    // A_row[i][j] = [j < tb TB + i] gamma^(2L-2-gi-j) k_i . q_j for the keys j of blocks 0 .. tb
    const int jn = (tb + 1) * TB / 16, atiles = at * jn;
    for (int tile = w; tile < atiles; tile += kSumWaves) {
      const int i0 = (tile / jn) * 16, j0 = (tile % jn) * 16;
      f32x4c x = zero;
      if (j0 < tb * TB + i0 + 15)
        mma_lds<float>(x, d, g, [&](int kk) { return Kb[(i0 + nn) * ld + kk]; },
                       [&](int kk) { return Qa[(j0 + nn) * ld + kk]; });
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = i0 + 4 * g + e, j = j0 + nn, gi = tb * TB + i;
        Ar[i * lar + j] = j < gi ? x[e] * exp2f(lg2g * (float)(2 * L - 2 - gi - j)) : 0.f;
      }
    }
    __syncthreads();
    // Y_tb = A_row V (the keys up to the row tile's last query) and A_row 1
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int tile = w + kSumWaves * r;
      if (tile < ytiles) {
        const int i0 = (tile / ctn) * 16, b0 = (tile % ctn) * 16;
        f32x4c y = zero;
        mma_lds<float>(y, tb * TB + i0 + 16, g, [&](int kk) { return Ar[(i0 + nn) * lar + kk]; },
                       [&](int kk) { return Va[kk * ldv + b0 + nn]; });
#pragma unroll
        for (int e = 0; e < 4; ++e) Yb[(i0 + 4 * g + e) * ldv + b0 + nn] = y[e];
      }
    }
    {
      const int row = tid >> 4, p = tid & 15;
      float x = 0.f;
      if (row < TB)
        for (int j = p; j < (tb + 1) * TB; j += 16) x += Ar[row * lar + j];
      x += __shfl_xor(x, 1);
      x += __shfl_xor(x, 2);
      x += __shfl_xor(x, 4);
      x += __shfl_xor(x, 8);
      if (p == 0 && row < TB) Yb[row * ldv + dv] = x;
    }
    __syncthreads();
    const float* Qt = Qa + tb * TB * ld;
    const float* Vt = Va + tb * TB * ldv;
// (a rolled loop: unrolled, the three products' operands of all eight tiles
    // would be scheduled together and spill)
#pragma unroll 1
    for (int r = 0; r < kSumTiles; ++r) {
      const int tile = w + kSumWaves * r;
      if (tile < sti) {
        const int a0 = (tile / stn) * 16, b0 = (tile % stn) * 16;
        mma_lds<float>(as[r], TB, g, [&](int t) { return Kb[t * ld + a0 + nn]; },
                       [&](int t) { return wv[t] * Kb[t * ld + b0 + nn]; });
      }
      if (tile < cti) {
        const int a0 = (tile / ctn) * 16, b0 = (tile % ctn) * 16;
        mma_lds<float>(ac[r], TB, g, [&](int t) { return Qt[t * ld + a0 + nn]; },
                       [&](int t) { return wv[t] * Vt[t * ldv + b0 + nn]; });
        mma_lds<float>(ag[r], TB, g, [&](int t) { return Kb[t * ld + a0 + nn]; },
                       [&](int t) { return Yb[t * ldv + b0 + nn]; });
      }
    }
    for (int t = mp; t < TB; t += P) {
      am += wv[t] * Qt[t * ld + ma];
      ah += Kb[t * ld + ma] * Yb[t * ldv + dv];
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < kSumTiles; ++r) {
    const int tile = w + kSumWaves * r;
    if (tile < sti) {
      const int a0 = (tile / stn) * 16, b0 = (tile % stn) * 16;
#pragma unroll
      for (int e = 0; e < 4; ++e) st[(size_t)(a0 + 4 * g + e) * d + b0 + nn] = as[r][e];
    }
    if (tile < cti) {
      const int a0 = (tile / ctn) * 16, b0 = (tile % ctn) * 16;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        st[off_C(d, dv) + (size_t)(a0 + 4 * g + e) * dv + b0 + nn] = ac[r][e];
        st[off_G(d, dv) + (size_t)(a0 + 4 * g + e) * dv + b0 + nn] = ag[r][e];
      }
    }
  }
  // m and h: the P partial sums of each column, through the A_row space
  Ar[tid] = am;
  Ar[kSumThreads + tid] = ah;
  __syncthreads();
  if (tid < d) {
    float xm = 0.f, xh = 0.f;
    for (int p = 0; p < P; ++p) {
      xm += Ar[p * d + tid];
      xh += Ar[kSumThreads + p * d + tid];
    }
    st[off_m(d, dv) + tid] = xm;
    st[off_h(d, dv) + tid] = xh;
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
// Every product runs on MFMA, one 16 x 16 output tile per wave at a time
// (lane l = 16 g + n supplies A[n][k_g] and B[k_g][n] and holds
// D[4 g + i][n]): the fp64 ones (Q S0, Q K^T, the carry term, W K, the T
// products) on v_mfma_f64_16x16x4_f64 with fp32 operands widened exactly,
// T V on v_mfma_f32_16x16x4_f32.  Triangular products stop at the
// diagonal tile.  A wave keeps the carry part of its output tiles in its
// accumulators until T V is added.
// LDS: R [chunk][d+1] fp64 (V [chunk][dv+1] fp32 in its place once R is
// dead), Q and K [chunk][d+1] fp32, W/T [chunk][chunk+1] fp32, den [chunk]
// fp32 (149 KB at chunk 64, d = dv = 128).
template <typename T>
__global__ __launch_bounds__(512) void k_readout(const T* __restrict__ q, const T* __restrict__ k,
                                                 const T* __restrict__ v, const float* __restrict__ prefix,
                                                 float* __restrict__ out, float* __restrict__ den_out, int n,
                                                 int d, int dv, int chunk, int M, int masked, int normalized,
                                                 float eps, float lg2g) {
  extern __shared__ double smemd[];
  const int c = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, nn = tid & 15, g = (tid >> 4) & 3;
  const int pr = mfma_pr(nn);        // fp64 A rows in the order that returns the fp32 layout
  const int t0 = c * chunk;
  const int L = min(chunk, n - t0), Lp = chunk, ld = d + 1, ldw = chunk + 1, ldv = dv + 1;
  const size_t qk_base = ((size_t)bh * n + t0) * d;
  const size_t v_base = ((size_t)bh * n + t0) * dv;
  double* R = smemd;                                           // [Lp][ld]
  float* Vs = reinterpret_cast<float*>(smemd);                 // [Lp][ldv], once R is dead
  const size_t rv = (size_t)Lp * ld * 2 > (size_t)Lp * ldv ? (size_t)Lp * ld * 2 : (size_t)Lp * ldv;
  float* Qs = reinterpret_cast<float*>(smemd) + ((rv + 3) & ~size_t(3));   // [Lp][ld]
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
  auto gp = [&](int e) { return exp2f(lg2g * (float)e); };     // gamma^e
  const int mt = Lp / 16, rn = d / 16, rtiles = mt * rn, on = dv / 16, otiles = mt * on;
  const int wtiles = mt * (mt + 1) / 2;                        // tiles on or below the diagonal
  auto lower_tile = [&](int tile, int& m0_, int& n0_) {
    int mi = 0;
    while ((mi + 1) * (mi + 2) / 2 <= tile) ++mi;
    m0_ = 16 * mi;
    n0_ = 16 * (tile - mi * (mi + 1) / 2);
  };
  const f64x4c zd = {0.0, 0.0, 0.0, 0.0};
  const f32x4c zf = {0.f, 0.f, 0.f, 0.f};

  // V's loads go out first; V is written to LDS only once R is dead
  float4 pvr[4];     // Lp dv / 4 <= 2048 pieces over 512 threads
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int idx = tid + 512 * i, t = idx / (dv / 4), b = (idx % (dv / 4)) * 4;
    pvr[i] = idx < Lp * dv / 4 && t < L ? ld4f(v, v_base + (size_t)t * dv + b) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  for (int idx = tid; idx < Lp * d / 4; idx += blockDim.x) {
    const int t = idx / (d / 4), a = (idx % (d / 4)) * 4;
    const float4 xq = t < L ? ld4f(q, qk_base + (size_t)t * d + a) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 xk = t < L ? ld4f(k, qk_base + (size_t)t * d + a) : make_float4(0.f, 0.f, 0.f, 0.f);
    float* pq = Qs + t * ld + a;
    float* pk = Ks + t * ld + a;
    pq[0] = xq.x; pq[1] = xq.y; pq[2] = xq.z; pq[3] = xq.w;
    pk[0] = xk.x; pk[1] = xk.y; pk[2] = xk.z; pk[3] = xk.w;
  }
  __syncthreads();

  // P = Q S0 into R;  W[t][i] = [i <= t] g^(t-i) q_t . k_i
  for (int tile = w; tile < rtiles; tile += kSumWaves) {
    const int mm = (tile / rn) * 16, n0 = (tile % rn) * 16;
    f64x4c acc = zd;
    mma_glb<double>(acc, d, g, [&](int kk) { return (double)Qs[(mm + pr) * ld + kk]; },
                    [&](int kk) { return S0[(size_t)kk * d + n0 + nn]; });
#pragma unroll
    for (int i = 0; i < 4; ++i) R[(mm + 4 * g + i) * ld + n0 + nn] = acc[i];
  }
  for (int tile = w; tile < wtiles; tile += kSumWaves) {
    int mm, n0;
    lower_tile(tile, mm, n0);
    f64x4c acc = zd;
    mma_lds<double>(acc, d, g, [&](int kk) { return (double)Qs[(mm + pr) * ld + kk]; },
                    [&](int kk) { return (double)Ks[(n0 + nn) * ld + kk]; });
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = mm + 4 * g + i, j = n0 + nn;
      W[t * ldw + j] = j <= t ? (float)(acc[i] * (double)gp(t - j)) : 0.f;
    }
  }
  __syncthreads();
  // eight lanes per token row: x(t) summed over the d dimensions, in fp64
  auto rowdot = [&](auto term) {
    const int t = tid >> 3, p = tid & 7;
    double s = 0.0;
    if (t < Lp)
      for (int a = p; a < d; a += 8) s += term(t, a);
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    return s;
  };
  f32x4c oc[4];      // carry part of this wave's output tiles w + 8 r
#pragma unroll
  for (int r = 0; r < 4; ++r) oc[r] = zf;
  if (masked) {
    // carry term g^(2(a+1)) (q_t^T S0 C0 - q_t^T G0) (and its denominator)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tile = w + kSumWaves * r;
      if (tile < otiles) {
        const int mm = (tile / on) * 16, n0 = (tile % on) * 16;
        f64x4c acc = zd;
        mma_glb<double>(acc, d, g, [&](int kk) { return R[(mm + pr) * ld + kk]; },
                        [&](int kk) { return C0[(size_t)kk * dv + n0 + nn]; });
        mma_glb<double>(acc, d, g, [&](int kk) { return -(double)Qs[(mm + pr) * ld + kk]; },
                        [&](int kk) { return G0[(size_t)kk * dv + n0 + nn]; });
#pragma unroll
        for (int i = 0; i < 4; ++i) oc[r][i] = (float)acc[i] * gp(2 * (mm + 4 * g + i) + 2);
      }
    }
    const double s = rowdot([&](int t, int a) { return R[t * ld + a] * (double)m0[a] - (double)Qs[t * ld + a] * (double)h0[a]; });
    if ((tid & 7) == 0 && (tid >> 3) < Lp) dn[tid >> 3] = (float)s * gp(2 * (tid >> 3) + 2);
  }
  __syncthreads();
  // the carry part of r_t decays by g^(a+1); then R += W K  (r_j = S_j q_j; W is zero past the diagonal)
  for (int tile = w; tile < rtiles; tile += kSumWaves) {
    const int mm = (tile / rn) * 16, n0 = (tile % rn) * 16;
    f64x4c acc = zd;
    mma_lds<double>(acc, mm + 16, g, [&](int kk) { return (double)W[(mm + pr) * ldw + kk]; },
                    [&](int kk) { return (double)Ks[kk * ld + n0 + nn]; });
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = mm + 4 * g + i;
      R[j * ld + n0 + nn] = R[j * ld + n0 + nn] * (double)gp(j + 1) + acc[i];
    }
  }
  __syncthreads();
  // T[t][j] = [j <= t] g^(2(t-j)) (q_t . r_j)  (masked)  or  g^(t-j) (r_t . q_j)  (unmasked)
  for (int tile = w; tile < wtiles; tile += kSumWaves) {
    int mm, n0;
    lower_tile(tile, mm, n0);
    f64x4c acc = zd;
    if (masked)
      mma_lds<double>(acc, d, g, [&](int kk) { return (double)Qs[(mm + pr) * ld + kk]; },
                      [&](int kk) { return R[(n0 + nn) * ld + kk]; });
    else
      mma_lds<double>(acc, d, g, [&](int kk) { return R[(mm + pr) * ld + kk]; },
                      [&](int kk) { return (double)Qs[(n0 + nn) * ld + kk]; });
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = mm + 4 * g + i, j = n0 + nn;
      W[t * ldw + j] = j <= t ? (float)(acc[i] * (double)gp(masked ? 2 * (t - j) : t - j)) : 0.f;
    }
  }
  if (!masked) {
    // carry term g^(a+1) r_t^T C0 (and its denominator)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tile = w + kSumWaves * r;
      if (tile < otiles) {
        const int mm = (tile / on) * 16, n0 = (tile % on) * 16;
        f64x4c acc = zd;
        mma_glb<double>(acc, d, g, [&](int kk) { return R[(mm + pr) * ld + kk]; },
                        [&](int kk) { return C0[(size_t)kk * dv + n0 + nn]; });
#pragma unroll
        for (int i = 0; i < 4; ++i) oc[r][i] = (float)acc[i] * gp(mm + 4 * g + i + 1);
      }
    }
    const double s = rowdot([&](int t, int a) { return R[t * ld + a] * (double)m0[a]; });
    if ((tid & 7) == 0 && (tid >> 3) < Lp) dn[tid >> 3] = (float)s * gp((tid >> 3) + 1);
  }
  __syncthreads();
  // V into the space of R (rows past the chunk's tokens zero); the rows' denominators
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int idx = tid + 512 * i;
    if (idx < Lp * dv / 4) {
      float* pv = Vs + (idx / (dv / 4)) * ldv + (idx % (dv / 4)) * 4;
      pv[0] = pvr[i].x; pv[1] = pvr[i].y; pv[2] = pvr[i].z; pv[3] = pvr[i].w;
    }
  }
  if (normalized) {
    const int t = tid >> 3, p = tid & 7;
    float s = 0.f;
    if (t < Lp)
      for (int j = p; j <= t; j += 8) s += W[t * ldw + j];
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    if (p == 0 && t < Lp) {
      s += dn[t];
      dn[t] = s;
      if (den_out && t < L) den_out[(size_t)bh * n + t0 + t] = s;
    }
  }
  __syncthreads();
  // o_t = carry + sum_{j <= t} T[t][j] v_j
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int tile = w + kSumWaves * r;
    if (tile < otiles) {
      const int mm = (tile / on) * 16, n0 = (tile % on) * 16;
      f32x4c acc = oc[r];
      mma_lds<float>(acc, mm + 16, g, [&](int kk) { return W[(mm + nn) * ldw + kk]; },
                     [&](int kk) { return Vs[kk * ldv + n0 + nn]; });
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = mm + 4 * g + i;
        if (t < L) o[(size_t)t * dv + n0 + nn] = normalized ? acc[i] / (dn[t] + eps) : acc[i];
      }
    }
  }
}

// ----------------------------------------------------------------------------
static size_t summary1_lds(int chunk, int d, int dv) {
  const size_t tb = chunk < 32 ? chunk : 32;
  return sizeof(float) * ((size_t)chunk * (sum_ld(d) + sum_ld(dv)) + tb * (sum_ld(d) + sum_ld(chunk) + sum_ld(dv)) + tb);
}
static size_t summary_lds(int chunk, int d, int dv) {
  const size_t tb = chunk < 32 ? chunk : 32;
  return sizeof(float) * (2 * tb * sum_ld(d) + tb * sum_ld(dv) + tb * sum_ld((int)tb) + (size_t)chunk * sum_ld(dv) + tb);
}
static size_t readout_lds(int chunk, int d, int dv) {
  const size_t r = 2 * (size_t)chunk * (d + 1), v = (size_t)chunk * (dv + 1);   // floats of R, or of V after it
  return sizeof(float) * (((r > v ? r : v) + 3) / 4 * 4 + 2 * (size_t)chunk * (d + 1) + (size_t)chunk * (chunk + 1) + chunk);
}

hipError_t launch_chunk_summaries(const void* q, const void* k, const void* v, float* states,
                                  int BH, int n, int d, int dv, int chunk, int dtype, hipStream_t s, float gamma) {
  const float lg2g = log2f(gamma);
  const int M = (n + chunk - 1) / chunk;
  // the one-pass kernel when the chunk's Q and V fit (and the m, h partials fit in A_row), else the block kernel
  const size_t l1 = summary1_lds(chunk, d, dv);
  const bool one = l1 <= 160 * 1024 && (size_t)(chunk < 32 ? chunk : 32) * sum_ld(chunk) >= 2 * kSumThreads;
  const size_t lds = one ? l1 : summary_lds(chunk, d, dv);
  dim3 grid(M, BH), block(kSumThreads);
  if (dtype == 1) {
    auto kern = one ? k_chunk_summary<uint16_t> : k_chunk_summary_blocks<uint16_t>;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    HLA_LAUNCH(kern, grid, block, lds, s, (const uint16_t*)q, (const uint16_t*)k,
                       (const uint16_t*)v, states, n, d, dv, chunk, M, lg2g);
  } else {
    auto kern = one ? k_chunk_summary<float> : k_chunk_summary_blocks<float>;
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
  const size_t lds = readout_lds(f.chunk, f.d, f.dv);
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
