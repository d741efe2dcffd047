// Asymmetric second-order HLA (AHLA, Sec. 6) forward for bf16 inputs on
// gfx950 MFMA.
//
// AHLA streams o_t = q_t^T E_t with P_t = sum_{j<=t} k_j v_j^T and
// E_t = sum_{i<=t} k_i (q_i^T P_i) (Thm. AHLA); normalised, den_t = q_t^T n_t
// with m_t = sum_{j<=t} k_j and n_t = sum_{i<=t} k_i (q_i^T m_i).
//
// Per chunk of C tokens (the rows of Q, K, V), with the carry P0, m0, E0, n0
// of everything before the chunk and A = L (.) Q K^T (diagonal kept):
//   R   = A V + Q P0          (C x dv, row t is q_t^T P_t)
//   s   = A 1 + Q m0          (C,      s_t = q_t^T m_t)
//   O   = A R + Q E0,   den = A s + Q n0
//   P0 += K^T V,  m0 += K^T 1,  E0 += K^T R,  n0 += K^T s
// which is the recurrence of Thm. AHLA summed over the chunk.
//
// Across segments the pipeline is the one of the fused second-order forward:
// the (+)_AHLA concatenation of Eq. (AHLA-semidirect) adds R_B P_A to E, and
// R_B P_A is exactly what a segment's walk accumulates when it starts from
// the true P prefix.  So
//   1. k_moments<KV>: P = K^T V and m = K^T 1 of every segment;
//   2. k_seg_prefix: the running sums of P and m^K over the segments;
//      k_ahla_walk: every segment walks from P0 = the P prefix of the
//      segments before it (m0 likewise) and E0 = n0 = 0, writes the partial
//      outputs (and, normalised, A s plus the n0 of every tile), and leaves
//      its bracket E0 (n0) in the G (h) slot of its record;
//   3. k_carry / k_fix: running sums of the brackets are the E and n carries
//      of the segments; out_t += q_t^T E_c, den_t += q_t . (n0 + n_c).
//
// Layout: wave w owns column tile ct = w % NCT of the output for RPW row
// tiles (from row tile (w / NCT) RPW), and keeps column ct of P0 and E0 (all
// d rows) in MFMA accumulators.  At d = 64 (RPW = 1) the two row waves of a
// column both keep it, so no partial sums are exchanged; at d = 128 (RPW = 2)
// four waves, one per SIMD, each keep one column (the state once, with up to
// 512 registers a wave: two row waves per column spilled 152 bytes a lane).
// Numerics as in the second-order walk: q, k, v exact in bf16; every computed
// operand (A, R, P0, E0) split into bf16 hi + lo, fp32 accumulation.
#include <cstdlib>

#include "ahla.h"
#include "fused_tiles.h"
#include "profile.h"

namespace hla {
namespace {

template <int D>
struct CfgAH {
  static constexpr int C = 64, DV = D;
  static constexpr int NCT = D / 32, RPW = D == 128 ? 2 : 1, NW = 2 * NCT / RPW, NT = 64 * NW;
  static constexpr int ST = D / 32, KC = C / 16, KD = D / 16;
  static constexpr int ldQ = D + kPad, ldK = D + kPad, ldV = DV + kPad, ldW = C + kPad, ldR = C + kPad;
  static constexpr int oQ = 0;
  static constexpr int oV = oQ + C * ldQ;
  static constexpr int oK = oV + C * ldV;
  static constexpr int oWh = oK + C * ldK;     // A, row-major (query, key)
  static constexpr int oWl = oWh + C * ldW;
  static constexpr int oRh = oWl + C * ldW;    // R^T (column, token)
  static constexpr int oRl = oRh + DV * ldR;
  static constexpr int n16 = oRl + DV * ldR;
  static constexpr int oX = oQ;                // output staging, over Q | V once both are dead
  static_assert(NW * RPW * 1024 * 2 <= oK - oQ, "output staging fits Q | V");
  static_assert(D * DV * 2 <= n16, "carry staging fits the tile region");
  static constexpr int f_m = 0, f_n = D, f_rs = 2 * D, f_s = 2 * D + 2 * C;
  static constexpr int nf32 = f_s + C;
  static constexpr size_t bytes = (size_t)((n16 + 7) & ~7) * 2 + (size_t)nf32 * 4;
  static constexpr int kBlocks = 2 * bytes <= 160 * 1024 && NW <= 4 ? 2 : 1;
  static constexpr int pfQ = C * D / 8 / NT, pfV = C * DV / 8 / NT;
  static_assert(C * D / 8 % NT == 0 && C * DV / 8 % NT == 0 && pfQ >= 1, "staging");
  static_assert(D == 64 || D == 128, "AHLA walk shapes");
  static_assert(bytes <= 160 * 1024, "LDS budget");
  static_assert(NT >= D + C, "den lanes and state lanes are distinct");
};

template <int D>
__global__ __launch_bounds__((CfgAH<D>::NT), (CfgAH<D>::kBlocks))
__attribute__((amdgpu_waves_per_eu(CfgAH<D>::RPW == 2 ? 1 : 2))) void k_ahla_walk(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, float* __restrict__ rec, const float* __restrict__ ppre,
    int n, int cps, int nseg, int normalized) {
  using G = CfgAH<D>;
  constexpr bool kO = D == 128;     // per-tile opaque lane index (registers)
  constexpr int C = G::C, DV = G::DV, NT = G::NT, ST = G::ST, RPW = G::RPW;
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* Qs = lds + G::oQ;
  uint16_t* Vs = lds + G::oV;
  uint16_t* Ks = lds + G::oK;
  uint16_t* Wh = lds + G::oWh;
  uint16_t* Wl = lds + G::oWl;
  uint16_t* Rh = lds + G::oRh;
  uint16_t* Rl = lds + G::oRl;
  float* XO = reinterpret_cast<float*>(lds + G::oX);
  float* fl = reinterpret_cast<float*>(lds + ((G::n16 + 7) & ~7));
  float* m0 = fl + G::f_m;    // m prefix at the tile start
  float* n0 = fl + G::f_n;    // n of the segment so far
  float* rs = fl + G::f_rs;   // [2][C] row sums of A per key row tile
  float* sv = fl + G::f_s;    // s_t

  int seg, bh;
  seg_head(seg, bh);
  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rtb = (w / G::NCT) * RPW, ct = w % G::NCT;   // row tiles rtb .. rtb + RPW - 1
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t F = state_floats(D, DV);
  float* rc = rec + ((size_t)bh * (nseg + 1) + seg) * F;
  const rsrc_t ro = make_rsrc(out + (size_t)bh * n * DV, (uint32_t)n * DV * 4);
  const int ta = tid - (NT - D);    // the last D lanes keep m0[ta] and n0[ta]

  // ---- carry in: P0 and m0 are the sums of the moments of the earlier segments ----
  f32x16 P0[ST], E0[ST];
#pragma unroll
  for (int i = 0; i < ST; ++i) {
    P0[i] = zero16();
    E0[i] = zero16();
  }
  if (ta >= 0) {
    m0[ta] = 0.f;
    n0[ta] = 0.f;
  }
  if (seg > 0) {
    // P0, m0 = the prefix of the earlier segments' moments: one record
    // [D * DV | D] per segment (k_seg_prefix), or without ppre (few
    // segments) the sum of the earlier records' C | m slots, which the
    // moments launch wrote (walks write only G and h), four records' loads
    // in flight at a time
    constexpr int nP4 = D * DV / 4 / NT, SB = 4;
    static_assert(D * DV % (4 * NT) == 0, "carry staging split");
    float4 pa[nP4];
    float ma = 0.f;
    if (ppre) {
      const float* x = ppre + ((size_t)bh * nseg + seg) * ((size_t)D * DV + D);
#pragma unroll
      for (int r = 0; r < nP4; ++r) pa[r] = reinterpret_cast<const float4*>(x)[tid + NT * r];
      if (ta >= 0) ma = x[D * DV + ta];
    } else {
      const float* base = rec + (size_t)bh * (nseg + 1) * F + off_C(D, DV);
#pragma unroll
      for (int r = 0; r < nP4; ++r) pa[r] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int sp = 0; sp < seg; sp += SB) {
        float4 u[SB][nP4];
        float um[SB];
#pragma unroll
        for (int j = 0; j < SB; ++j) {
          const float* x = base + (size_t)(sp + j) * F;
#pragma unroll
          for (int r = 0; r < nP4; ++r)
            u[j][r] = sp + j < seg ? reinterpret_cast<const float4*>(x)[tid + NT * r] : make_float4(0.f, 0.f, 0.f, 0.f);
          um[j] = sp + j < seg && ta >= 0 ? x[D * DV + ta] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < SB; ++j) {
#pragma unroll
          for (int r = 0; r < nP4; ++r) {
            pa[r].x += u[j][r].x; pa[r].y += u[j][r].y; pa[r].z += u[j][r].z; pa[r].w += u[j][r].w;
          }
          ma += um[j];
        }
      }
    }
    float* st = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int r = 0; r < nP4; ++r) reinterpret_cast<float4*>(st)[tid + NT * r] = pa[r];
    if (ta >= 0) m0[ta] = ma;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < ST; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) P0[i][e] = st[(i * 32 + acc_row(e, lg)) * DV + ct * 32 + lr];
    __syncthreads();
  }

  // ---- prefetch registers for the next chunk (buffer loads: the tail past n reads zero) ----
  const rsrc_t rq = make_rsrc(q + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rk = make_rsrc(k + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rv = make_rsrc(v + (size_t)bh * n * DV, (uint32_t)n * DV * 2);
  uint4 pq[G::pfQ], pk[G::pfQ], pv[G::pfV];
  // 16-byte piece e of a C x W tile: token pt, first column pc.  At d = 64
  // consecutive lanes take consecutive pieces of a token row (coalesced
  // loads, contiguous LDS stores); at d = 128 consecutive tokens, which
  // measured faster for this walk there.
  constexpr bool RP = D <= 64;
  auto pt = [](int e, int W) { return RP ? e / (W / 8) : e % C; };
  auto pc = [](int e, int W) { return RP ? (e % (W / 8)) * 8 : (e / C) * 8; };
  auto fetch = [&](int c) {
    const uint32_t t0 = (uint32_t)c * C;
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + NT * i;
      const uint32_t off = ((t0 + pt(e, D)) * D + pc(e, D)) * 2;
      pq[i] = buf_load16(rq, off);
      pk[i] = buf_load16(rk, off);
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + NT * i;
      pv[i] = buf_load16(rv, ((t0 + pt(e, DV)) * DV + pc(e, DV)) * 2);
    }
  };
  if (c_begin < c_end) fetch(c_begin);

  for (int c = c_begin; c < c_end; ++c) {
    const int t0 = c * C;
    // lane index for the fragment helpers, opaque once per tile at d = 128:
    // lane offsets are formed once per tile and no address is hoisted out of
    // the walk
    int ln = tid & 63;
    if constexpr (kO) asm volatile("" : "+v"(ln));
    // ---- stage 0: registers -> LDS, row-major (transposed operands go through the transpose unit) ----
#pragma unroll
    for (int i = 0; i < G::pfQ; ++i) {
      const int e = tid + NT * i;
      const int t = pt(e, D), a8 = pc(e, D);
      *reinterpret_cast<uint4*>(Qs + t * G::ldQ + a8) = pq[i];
      *reinterpret_cast<uint4*>(Ks + t * G::ldK + a8) = pk[i];
    }
#pragma unroll
    for (int i = 0; i < G::pfV; ++i) {
      const int e = tid + NT * i;
      const int t = pt(e, DV), b8 = pc(e, DV);
      *reinterpret_cast<uint4*>(Vs + t * G::ldV + b8) = pv[i];
    }
    lds_barrier();
    if (c + 1 < c_end) fetch(c + 1);

    // ---- stage 1: A = L (.) Q K^T on tiles (key it <= query jt), as A^T = K Q^T, stored row-major ----
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
        if (normalized) {              // row sums of A (over the keys of this tile)
          float ps = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) ps += acc[e];
          ps += __shfl_xor(ps, 32);
          if (lg == 0) rs[it * C + jt * 32 + lr] = ps;
        }
        store_T<kO>(acc, Wh, Wl, G::ldW, it * 32, jt * 32, ln);
      } else if (normalized && lg == 0) {
        rs[it * C + jt * 32 + lr] = 0.f;
      }
    }
    lds_barrier();

    // s_t = (A 1)_t + q_t . m0
    if (normalized && tid < C) {
      float a = rs[tid] + rs[C + tid];
      const uint16_t* row = Qs + tid * G::ldQ;
#pragma unroll
      for (int a8 = 0; a8 < D; a8 += 8) {
        const uint4 x = *reinterpret_cast<const uint4*>(row + a8);
        const uint32_t u[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          a += __uint_as_float(u[j] << 16) * m0[a8 + 2 * j];
          a += __uint_as_float(u[j] & 0xffff0000u) * m0[a8 + 2 * j + 1];
        }
      }
      sv[tid] = a;
    }

    // ---- stage 2: R = Q P0 + A V and the O partial Q E0 (old carries); P0 += K^T V ----
    f32x16 racc[RPW], oacc[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      racc[r] = zero16();
      oacc[r] = zero16();
    }
#pragma unroll
    for (int j = 0; j < G::KD; ++j) {
      bf16x8 ph, pl, eh, el;
      frag_from_acc(P0[j >> 1], j & 1, ph, pl);
      frag_from_acc(E0[j >> 1], j & 1, eh, el);
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const bf16x8 aQ = frag_acc_order<kO>(Qs, G::ldQ, (rtb + r) * 32, j * 16, ln);
        racc[r] = mfma(aQ, ph, racc[r]);
        racc[r] = mfma(aQ, pl, racc[r]);
        oacc[r] = mfma(aQ, eh, oacc[r]);
        oacc[r] = mfma(aQ, el, oacc[r]);
      }
    }
#pragma unroll
    for (int s = 0; s < G::KC; ++s) {
      const bf16x8 bV = frag_tr<kO>(Vs, G::ldV, ct * 32, s * 16, ln);
#pragma unroll
      for (int r = 0; r < RPW; ++r)
        if (s < 2 * (rtb + r + 1)) {    // keys past the row tile: A is zero
          racc[r] = mfma(frag<kO>(Wh, G::ldW, (rtb + r) * 32, s * 16, ln), bV, racc[r]);
          racc[r] = mfma(frag<kO>(Wl, G::ldW, (rtb + r) * 32, s * 16, ln), bV, racc[r]);
        }
#pragma unroll
      for (int i = 0; i < ST; ++i) P0[i] = mfma(frag_tr<kO>(Ks, G::ldK, i * 32, s * 16, ln), bV, P0[i]);
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r) store_T<kO>(racc[r], Rh, Rl, G::ldR, (rtb + r) * 32, ct * 32, ln);   // R^T
    lds_barrier();                      // R^T and s visible; Q and V are dead

    // ---- normalised: den partial (A s)_t, the tile's n0, then m0 and n0 advance ----
    if (normalized) {
      if (tid < C) {
        const int t = tid, iend = t < 32 ? 32 : 64;   // A[t][i] = 0 for i > t; key tile 1 unwritten for t < 32
        const uint16_t* wh = Wh + t * G::ldW;
        const uint16_t* wl = Wl + t * G::ldW;
        float a = 0.f;
        for (int i8 = 0; i8 < iend; i8 += 8) {
          const uint4 xh = *reinterpret_cast<const uint4*>(wh + i8);
          const uint4 xl = *reinterpret_cast<const uint4*>(wl + i8);
          const uint32_t uh[4] = {xh.x, xh.y, xh.z, xh.w}, ul[4] = {xl.x, xl.y, xl.z, xl.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            a += (__uint_as_float(uh[j] << 16) + __uint_as_float(ul[j] << 16)) * sv[i8 + 2 * j];
            a += (__uint_as_float(uh[j] & 0xffff0000u) + __uint_as_float(ul[j] & 0xffff0000u)) * sv[i8 + 2 * j + 1];
          }
        }
        if (t0 + t < n) den_out[(size_t)bh * n + t0 + t] = a;
      }
      if (ta >= 0) {
        den_out[(size_t)gridDim.y * n + ((size_t)bh * M + c) * D + ta] = n0[ta];
        float sn = 0.f, sm = 0.f;
#pragma unroll 8
        for (int t = 0; t < C; ++t) {
          const float kv = bf16_to_f(Ks[t * G::ldK + ta]);
          sn += kv * sv[t];
          sm += kv;
        }
        n0[ta] += sn;
        m0[ta] += sm;
      }
    }

    // ---- stage 3: E0 += K^T R;  O += A R (A and R both split: hi hi, hi lo, lo hi) ----
#pragma unroll
    for (int s = 0; s < G::KC; ++s) {
      const bf16x8 brh = frag<kO>(Rh, G::ldR, ct * 32, s * 16, ln);
      const bf16x8 brl = frag<kO>(Rl, G::ldR, ct * 32, s * 16, ln);
#pragma unroll
      for (int i = 0; i < ST; ++i) {
        const bf16x8 aK = frag_tr<kO>(Ks, G::ldK, i * 32, s * 16, ln);
        E0[i] = mfma(aK, brh, E0[i]);
        E0[i] = mfma(aK, brl, E0[i]);
      }
#pragma unroll
      for (int r = 0; r < RPW; ++r)
        if (s < 2 * (rtb + r + 1)) {
          const bf16x8 awh = frag<kO>(Wh, G::ldW, (rtb + r) * 32, s * 16, ln);
          const bf16x8 awl = frag<kO>(Wl, G::ldW, (rtb + r) * 32, s * 16, ln);
          oacc[r] = mfma(awh, brh, oacc[r]);
          oacc[r] = mfma(awh, brl, oacc[r]);
          oacc[r] = mfma(awl, brh, oacc[r]);
        }
    }
    // the output tiles go through this wave's staging slots so that each lane
    // stores 16 bytes; rows past n fall outside the buffer and are dropped
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      float* ob = XO + (w * RPW + r) * 1024;
#pragma unroll
      for (int e = 0; e < 16; ++e) ob[acc_row(e, lg) * 32 + lr] = oacc[r][e];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int p = l + 64 * j, row = p >> 3, c4 = (p & 7) * 4;
        buf_store16(ro, (((uint32_t)t0 + (rtb + r) * 32 + row) * DV + ct * 32 + c4) * 4,
                    *reinterpret_cast<const float4*>(ob + row * 32 + c4));
      }
    }
    lds_barrier();   // every LDS tile is rewritten by the next chunk
  }

  // the segment's bracket: E0 into the G slot (the waves of row tile 0; any
  // other row waves hold the same columns), n0 into the h slot
  int col = ct * 32 + lr;
  asm volatile("" : "+v"(col));
  if (rtb == 0) {
#pragma unroll
    for (int i = 0; i < ST; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) rc[off_G(D, DV) + (size_t)(i * 32 + acc_row(e, lg)) * DV + col] = E0[i][e];
  }
  if (ta >= 0) rc[off_h(D, DV) + ta] = n0[ta];
}

// Segments: enough walks to fill the chip (workgroups per CU times 256 CUs).
void ahla_plan(int D, int BH, int n, int* P, int* cps) {
  const int M = (n + 63) / 64;
  const int blocks = D == 64 ? CfgAH<64>::kBlocks : CfgAH<128>::kBlocks;
  int p = 256 * blocks / BH;
  if (const char* e = getenv("HLA_FUSED_SEGMENTS")) p = atoi(e);
  if (p < 1) p = 1;
  if (p > M) p = M;
  *cps = (M + p - 1) / p;
  *P = (M + *cps - 1) / *cps;
}

size_t records_bytes_ah(int BH, int P, int d) {
  return (sizeof(float) * (size_t)BH * (P + 1) * state_floats(d, d) + 255) & ~size_t(255);
}
size_t den_bytes_ah(int BH, int n, int d) {
  return sizeof(float) * (((size_t)BH * n + (size_t)BH * ((n + 63) / 64) * d + 63) & ~size_t(63));
}
// carries [BH][P][d d + d] (k_carry), then the moment prefixes [BH][P][d d + d]
size_t carry_bytes_ah(int BH, int P, int d) { return sizeof(float) * (size_t)BH * P * ((size_t)d * d + d); }

// Segments per head up to which an AHLA walk sums its P and m^K prefixes
// from the moment records itself instead of reading them from a prefix launch.
constexpr int kAhlaWalkSumMax = 8;

template <int D>
hipError_t run_ahla(const Fwd& f, char* ws, int P, int cps, hipStream_t s) {
  constexpr int C = 64;
  using G = CfgAH<D>;
  const int BH = f.BH;
  float* segs = reinterpret_cast<float*>(ws);
  float* den = reinterpret_cast<float*>(ws + records_bytes_ah(BH, P, D));
  float* carry = reinterpret_cast<float*>(ws + records_bytes_ah(BH, P, D) + den_bytes_ah(BH, f.n, D));
  float* ppre = reinterpret_cast<float*>(reinterpret_cast<char*>(carry) + carry_bytes_ah(BH, P, D));
  const uint16_t* q = static_cast<const uint16_t*>(f.q);
  const uint16_t* k = static_cast<const uint16_t*>(f.k);
  const uint16_t* v = static_cast<const uint16_t*>(f.v);
  const dim3 grid(P, BH);
  hipError_t e;
  if (P > 1) {
    prof_start("ahla_moments", s);
    HLA_LAUNCH((k_moments<C, D, D, true>), grid, dim3(kThreads), 0, s, q, k, v, segs, f.n, cps, P, 1, 0.f);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (P > kAhlaWalkSumMax) {
      prof_start("ahla_prefix", s);     // the P and m^K slots are adjacent (C | m)
      HLA_LAUNCH(k_seg_prefix, dim3((D * D + D + 1023) / 1024, BH), dim3(256), 0, s, segs, state_floats(D, D),
                 (int)off_C(D, D), D * D + D, 0, ppre, P, 1.f);
      prof_stop(s);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  // up to kAhlaWalkSumMax segments per head each walk sums the earlier moments itself
  const float* ppre_walk = P > kAhlaWalkSumMax ? ppre : nullptr;
  if ((e = hipFuncSetAttribute((const void*)k_ahla_walk<D>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)G::bytes)) != hipSuccess)
    return e;
  prof_start("ahla_walk", s);
  HLA_LAUNCH((k_ahla_walk<D>), grid, dim3(G::NT), G::bytes, s, q, k, v, f.out, den, segs, ppre_walk, f.n,
             cps, P, f.normalized);
  prof_stop(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (P > 1 || f.normalized) {
    prof_start("ahla_carry", s);
    HLA_LAUNCH((k_carry<D, D>), dim3((D * D / 8 + D + 255) / 256, BH), dim3(256), 0, s, segs,
                       (const float*)nullptr, carry, P, 1.f);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    using FC = FixCfg<C, D, D>;
    if ((e = hipFuncSetAttribute((const void*)k_fix<C, D, D>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)FC::lds)) != hipSuccess)
      return e;
    const int M = (f.n + C - 1) / C, tpw = fix_tpw(M, BH);
    prof_start("ahla_fix", s);
    HLA_LAUNCH((k_fix<C, D, D>), dim3((M + tpw - 1) / tpw, BH), dim3(FC::NT), FC::lds, s, q, f.out, den,
                       carry, (float*)nullptr, 0, f.n, cps, P, f.normalized, f.eps, tpw, 0.f);
    prof_stop(s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

bool ahla_supported(int n, int d, int dv, int chunk, int dtype) {
  const long long span = (long long)n * d * 4;   // per-head byte offsets stay below 2^31
  return dtype == 1 && n >= 1 && d == dv && (d == 64 || d == 128) && (chunk == 64 || chunk == 128) &&
         span < (1LL << 31);
}

size_t ahla_workspace_bytes(int BH, int n, int d) {
  int P, cps;
  ahla_plan(d, BH, n, &P, &cps);
  return records_bytes_ah(BH, P, d) + den_bytes_ah(BH, n, d) + 2 * carry_bytes_ah(BH, P, d) + 256;
}

hipError_t launch_ahla(const Fwd& f, void* workspace, hipStream_t s) {
  if (!ahla_supported(f.n, f.d, f.dv, f.chunk, f.dtype)) return hipErrorNotSupported;
  int P, cps;
  ahla_plan(f.d, f.BH, f.n, &P, &cps);
  char* ws = static_cast<char*>(workspace);
  return f.d == 64 ? run_ahla<64>(f, ws, P, cps, s) : run_ahla<128>(f, ws, P, cps, s);
}

}  // namespace hla
