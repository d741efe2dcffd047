// Wave-specialised segment walk for d = dv = 128 on 64-token tiles (the
// masked second-order forward of Sec. 4 with the Thm. 1 readout), and the
// segment prefix sums that feed it.  Included by fused.hip only.
//
// Per tile (rows = the tile's tokens; S0, Phi0, eta0 the carry before it):
//   W = L (.) Q K^T,  R = W K + Q S0,  S0 += K^T K               (key side)
//   T = L (.) Q R^T,  O = T V + Q Phi0,  den = T 1 + Q eta0,
//   Phi0 += R^T V,  eta0 += R^T 1                                (value side)
// The key side of tile c + 1 does not depend on the value side of tile c
// (only on S0), and the value side of tile c needs R_c only.  So waves 0-3
// hold S0 (wave w: columns 32w .. 32w + 31, all 128 rows) and run the key
// side one tile ahead, while waves 4-7 hold Phi0 the same way and run the
// value side: in each step the two halves work on different tiles at once,
// one wave of each on every SIMD, and meet at three barriers:
//   phase 1: key side W_{c+1}, Q S0;     value side T_c, Q Phi0, q . eta0
//   phase 2: key side W K, S0 adv.;      value side T V, Phi0 adv., 1/(den+eps)
//   phase 3: key side stores R_{c+1} (and its column sums); value side stores
//            O_c (16-byte stores through LDS); next tiles staged.
// A state column tile is held, split and advanced by one wave; R and T are
// formed once and shared through LDS.  Numerics as the other walks: every
// computed operand is split into bf16 hi + lo, q/k/v are exact, fp32
// accumulation.
//
// Two-pass plan (no initial or final state).  Segment 0 holds c0 tiles and
// every later segment cps tiles (the last the rest); the first launch runs,
// side by side, the output walk of segment 0 (its carry is zero) and the
// summary walks of segments 1 .. P-2 from a zero state, the latter also
// forming C = Q^T V and m = Q^T 1 of their tiles; the S prefixes, the
// brackets (Eq. semidirect in the Phi form: the bracket of segment s is
// Phi_s + S_{<s} C_s, k_ws_bracket) and their running sums turn these
// records into the true carries; the second launch runs the output
// walks of segments 1 .. P-1 from their carries, so every output row is
// final when written (division included).  Segment 0 is shorter than the
// others by about the ratio of the two walks' per-tile times, so that both
// launches fill every CU for the same time.
#pragma once
#include "fused_tiles.h"

namespace hla {
namespace {

struct CfgWS {
  static constexpr int C = 64, D = 128, DV = 128;
  static constexpr int NT = 512;                                 // 8 waves
  // V is read only through the transpose unit: a row stride of 8 banks
  // modulo 32 keeps the four rows of each 16-lane read in different banks
  static constexpr int ldQ = D + kPad, ldK = D + kPad, ldV = DV + 16;
  static constexpr int ldW = C + kPad, ldT = C + kPad, ldR = C + kPad;
  static constexpr int oQ0 = 0;                                  // Q of even tiles
  static constexpr int oQ1 = oQ0 + C * ldQ;                      // Q of odd tiles
  static constexpr int oK = oQ1 + C * ldQ;
  static constexpr int oV = oK + C * ldK;
  static constexpr int oWh = oV + C * ldV, oWl = oWh + C * ldW;  // W[query][key]
  static constexpr int oTh = oWl + C * ldW, oTl = oTh + C * ldT; // T[query][key]
  static constexpr int oRh = oTl + C * ldT, oRl = oRh + D * ldR; // R^T[d][token]
  static constexpr int n16 = oRl + D * ldR;
  static constexpr int f_eta = 0, f_inc = D, f_denp = 2 * D, f_qeta = 2 * D + 2 * C, f_inv = f_qeta + C;
  static constexpr int nf32 = f_inv + C;
  static constexpr size_t bytes = (size_t)n16 * 2 + (size_t)nf32 * 4;
  static constexpr int PF = C * D / 8 / NT;                      // 16-byte pieces per thread per operand
  static_assert(PF * NT * 8 == C * D && (n16 * 2) % 16 == 0, "staging split");
  static_assert(bytes <= 160 * 1024, "LDS budget");
  static_assert(4 * C * 32 * 4 <= (oRh - oWh) * 2, "output staging fits the W | T region");
};

// Tile range of segment seg: segment 0 holds tiles [0, c0), segment s >= 1
// tiles [c0 + (s - 1) cps, c0 + s cps), cut at M.
__device__ __forceinline__ void ws_range(int seg, int c0, int cps, int M, int& c_begin, int& nt) {
  c_begin = seg == 0 ? 0 : c0 + (seg - 1) * cps;
  nt = min(M, seg == 0 ? c0 : c_begin + cps) - c_begin;
}

// Instruction order for one block of LDS-fed products: PRE LDS reads first,
// then the NM MFMAs with the remaining NR - PRE reads spread evenly between
// them, so each wave keeps several fragment reads in flight instead of
// waiting on the read that feeds the very next MFMA (mask 0x100: LDS reads,
// 0x008: MFMAs).  It only orders; data dependences still hold.
template <int PRE, int NM, int NR, int I = 0>
__device__ __forceinline__ void read_ahead() {
  if constexpr (I == 0) __builtin_amdgcn_sched_group_barrier(0x100, PRE, 0);
  if constexpr (I < NM) {
    constexpr int c = ((I + 1) * (NR - PRE)) / NM - (I * (NR - PRE)) / NM;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (c > 0) __builtin_amdgcn_sched_group_barrier(0x100, c, 0);
    read_ahead<PRE, NM, NR, I + 1>();
  }
}

// One segment's walk over tiles [c_begin, c_begin + nt) of head bh.
// s_in: S0 at the start (D x D, row-major; null: zero); c_in: Phi0 (D x DV)
// then eta0 (D) at the start (null: zero; unused by SUMMARY); rec: this
// segment's record (null: none), which receives the ending S0, Phi0 and eta0
// in its S, G and h slots, and with SUMMARY also the segment's C = Q^T V and
// m = Q^T 1 in its C and m slots.  Each block of products is ordered with
// read_ahead.
template <bool SUMMARY>
__device__ __forceinline__ void walk_ws(uint16_t* lds,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, const float* __restrict__ s_in,
    const float* __restrict__ c_in, float* __restrict__ rec, int bh, int n, int c_begin, int nt, int normalized,
    float eps) {
  using G = CfgWS;
  constexpr int C = G::C, D = G::D, DV = G::DV, NT = G::NT;
  static_assert(D == DV, "S0 and Phi0 share the column-tile layout");
  uint16_t* Ks = lds + G::oK;
  uint16_t* Vs = lds + G::oV;
  uint16_t* Wh = lds + G::oWh;
  uint16_t* Wl = lds + G::oWl;
  uint16_t* Th = lds + G::oTh;
  uint16_t* Tl = lds + G::oTl;
  uint16_t* Rh = lds + G::oRh;
  uint16_t* Rl = lds + G::oRl;
  float* fl = reinterpret_cast<float*>(lds + G::n16);
  float* eta = fl + G::f_eta;      // eta0 of the value side's current tile
  float* inc = fl + G::f_inc;      // R^T 1 of the tile the key side formed last
  float* denp = fl + G::f_denp;    // [2][C]: row sums of T over key tiles 0 and 1
  float* qeta = fl + G::f_qeta;    // [C]: q_t . eta0
  float* inv = fl + G::f_inv;      // [C]: 1 / (den_t + eps)

  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool keyside = w < 4;        // waves 0-3: S0 and R; waves 4-7: Phi0, T and O
  const int cw = w & 3;              // this wave's state column tile

  // ---- carry in: column tile cw of S0 (key side) or Phi0 (value side), all rows ----
  f32x16 st[4];      // rows 32i .. 32i + 31
  {
    const float* src = keyside ? s_in : (SUMMARY ? nullptr : c_in);
    if (src) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) st[i][e] = src[(size_t)(32 * i + acc_row(e, lg)) * D + cw * 32 + lr];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) st[i] = zero16();
    }
  }
  f32x16 cacc[4];    // SUMMARY, value side: column tile cw of C = Q^T V
  float macc[8];     // SUMMARY, value side: partial column sums of Q
  if (SUMMARY) {
#pragma unroll
    for (int i = 0; i < 4; ++i) cacc[i] = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) macc[j] = 0.f;
  }
  if (tid < D) {
    eta[tid] = (!SUMMARY && c_in) ? c_in[D * DV + tid] : 0.f;
    inc[tid] = 0.f;
  }
  if (tid < C) denp[C + tid] = 0.f;  // key tile 1 adds nothing to query rows 0 .. 31

  const rsrc_t rq = make_rsrc(q + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rk = make_rsrc(k + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rv = make_rsrc(v + (size_t)bh * n * DV, (uint32_t)n * DV * 2);
  // staging registers: consecutive lanes take consecutive 16-byte pieces of a token row
  uint4 pq[G::PF], pk[G::PF], pv[G::PF];
  auto piece = [&](int i) { return tid + NT * i; };
  auto fetch_qk = [&](int c) {
#pragma unroll
    for (int i = 0; i < G::PF; ++i) {
      const int e = piece(i);
      const uint32_t off = (((uint32_t)c * C + e / (D / 8)) * D + (e % (D / 8)) * 8) * 2;
      pq[i] = buf_load16(rq, off);
      pk[i] = buf_load16(rk, off);
    }
  };
  auto fetch_v = [&](int c) {
#pragma unroll
    for (int i = 0; i < G::PF; ++i) {
      const int e = piece(i);
      pv[i] = buf_load16(rv, (((uint32_t)c * C + e / (DV / 8)) * DV + (e % (DV / 8)) * 8) * 2);
    }
  };
  auto stage = [&](uint16_t* dst, int ld, int width, const uint4* p) {
#pragma unroll
    for (int i = 0; i < G::PF; ++i) {
      const int e = piece(i);
      *reinterpret_cast<uint4*>(dst + (e / (width / 8)) * ld + (e % (width / 8)) * 8) = p[i];
    }
  };
  // Loads of Q, K of tile t + 2 and V of tile t + 1 are issued at the end of
  // phase 1 of step t (after the phase's products, so the staging registers
  // are not live through them) and staged in phase 3 (both sides): the value
  // side is done with Q of tile t, the key side with K of tile t + 1, the
  // value side with V of tile t.
  auto prefetch = [&](int t) {
    if (t + 2 < nt) fetch_qk(c_begin + t + 2);
    if (t + 1 < nt) fetch_v(c_begin + t + 1);
  };
  auto restage = [&](int t) {
    if (t + 2 < nt) {
      stage(lds + ((t & 1) ? G::oQ1 : G::oQ0), G::ldQ, D, pq);
      stage(Ks, G::ldK, D, pk);
    }
    if (t + 1 < nt) stage(Vs, G::ldV, DV, pv);
  };

  // prologue: Q, K of the first tile in LDS
  fetch_qk(c_begin);
  stage(lds + G::oQ0, G::ldQ, D, pq);
  stage(Ks, G::ldK, D, pk);
  __syncthreads();

  // The two sides run separate loops with the same three barriers per step,
  // so each keeps its own registers (no copies where the paths would merge).
  if (keyside) {
    for (int t = -1; t < nt; ++t) {
      const bool hasX = t + 1 < nt;  // key side on tile t + 1
      const uint16_t* Qx = lds + (((t + 1) & 1) ? G::oQ1 : G::oQ0);
      // the lane index made opaque once per step: offsets are formed here and
      // every access adds a constant, none hoisted out of the loop
      int ln = tid & 63;
      asm volatile("" : "+v"(ln));
      const int lr = ln & 31, lg = ln >> 5;
      // phase 1: W^T tile (keys it, queries jt) = K Q^T, it <= jt; R = Q S0
      // on column tile cw (S0 before tile t + 1)
      f32x16 acc[2];
      if (hasX && cw < 3) {
        const int it = cw == 2 ? 1 : 0, jt = cw == 0 ? 0 : 1;
        f32x16 a = zero16();
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          a = mfma(frag<true>(Ks, G::ldK, it * 32, s * 16, ln), frag<true>(Qx, G::ldQ, jt * 32, s * 16, ln), a);
        read_ahead<6, 8, 16>();      // W: 8 MFMAs, 16 reads
        if (it == jt)
#pragma unroll
          for (int e = 0; e < 16; ++e)   // keep key <= query
            if (acc_row(e, lg) > lr) a[e] = 0.f;
        store_T<true>(a, Wh, Wl, G::ldW, it * 32, jt * 32, ln);
      }
      if (hasX) {
        acc[0] = zero16();
        acc[1] = zero16();
#pragma unroll
        for (int j = 0; j < D / 16; ++j) {
          bf16x8 bh_, bl_;
          frag_from_acc(st[j >> 1], j & 1, bh_, bl_);
#pragma unroll
          for (int rt = 0; rt < 2; ++rt) {
            const bf16x8 aQ = frag_acc_order<true>(Qx, G::ldQ, rt * 32, j * 16, ln);
            acc[rt] = mfma(aQ, bh_, acc[rt]);
            acc[rt] = mfma(aQ, bl_, acc[rt]);
          }
        }
        read_ahead<6, 32, 16>();     // Q S0: 32 MFMAs, 16 reads
      }
      prefetch(t);
      lds_barrier();
      // phase 2: R += W K, then S0 += K^T K
      if (hasX) {
        bf16x8 bK[C / 16];             // K column tile cw: B operand of W K and of the S0 advance
#pragma unroll
        for (int s = 0; s < C / 16; ++s) {
          bK[s] = frag_tr<true>(Ks, G::ldK, cw * 32, s * 16, ln);
#pragma unroll
          for (int rt = 0; rt < 2; ++rt)
            if (s < 2 || rt == 1) {    // keys past the query tile: W is zero
              acc[rt] = mfma(frag<true>(Wh, G::ldW, rt * 32, s * 16, ln), bK[s], acc[rt]);
              acc[rt] = mfma(frag<true>(Wl, G::ldW, rt * 32, s * 16, ln), bK[s], acc[rt]);
            }
        }
#pragma unroll
        for (int s = 0; s < C / 16; ++s)
#pragma unroll
          for (int i = 0; i < 4; ++i) st[i] = mfma(frag_tr<true>(Ks, G::ldK, i * 32, s * 16, ln), bK[s], st[i]);
        read_ahead<16, 28, 52>();    // W K, S0 advance: 28 MFMAs, 52 reads
      }
      lds_barrier();
      // phase 3: R^T of tile t + 1 for the value side, and its column sums
      if (hasX) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) store_T<true>(acc[rt], Rh, Rl, G::ldR, rt * 32, cw * 32, ln);
        float cs = 0.f;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int e = 0; e < 16; ++e) cs += acc[rt][e];
        cs += __shfl_xor(cs, 32);
        if (lg == 0) inc[cw * 32 + lr] = cs;
      }
      restage(t);
      lds_barrier();
    }
  } else {
    const rsrc_t ro = make_rsrc(SUMMARY ? nullptr : out + (size_t)bh * n * DV, SUMMARY ? 0u : (uint32_t)n * DV * 4);
    for (int t = -1; t < nt; ++t) {
      const bool hasY = t >= 0;      // value side on tile t
      const uint16_t* Qy = lds + ((t & 1) ? G::oQ1 : G::oQ0);
      // the lane index made opaque once per step (as on the key side), and the
      // lane coordinates and thread index taken from it, so no lane-dependent
      // address or mask is hoisted out of the loop
      int ln = tid & 63;
      asm volatile("" : "+v"(ln));
      const int lr = ln & 31, lg = ln >> 5, u = ln + 64 * (w - 4);
      f32x16 acc[2];
      // phase 1 (SUMMARY): C += Q^T V on column tile cw, and this thread's
      // share of m: columns 8 (u % 16) .. + 7 over tokens 4 (u / 16) .. + 3
      // (rows past n were loaded as zeros)
      if (SUMMARY && hasY) {
#pragma unroll
        for (int s = 0; s < C / 16; ++s) {
          const bf16x8 bV = frag_tr<true>(Vs, G::ldV, cw * 32, s * 16, ln);
#pragma unroll
          for (int i = 0; i < 4; ++i) cacc[i] = mfma(frag_tr<true>(Qy, G::ldQ, i * 32, s * 16, ln), bV, cacc[i]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint4 x = *reinterpret_cast<const uint4*>(Qy + (4 * (u >> 4) + r) * G::ldQ + (u & 15) * 8);
          macc[0] += __uint_as_float(x.x << 16); macc[1] += __uint_as_float(x.x & 0xffff0000u);
          macc[2] += __uint_as_float(x.y << 16); macc[3] += __uint_as_float(x.y & 0xffff0000u);
          macc[4] += __uint_as_float(x.z << 16); macc[5] += __uint_as_float(x.z & 0xffff0000u);
          macc[6] += __uint_as_float(x.w << 16); macc[7] += __uint_as_float(x.w & 0xffff0000u);
        }
      }
      // phase 1: T^T tile (keys it, queries jt) = R Q^T, it <= jt; O = Q Phi0; q . eta0
      if (!SUMMARY && hasY) {
        if (cw < 3) {
          const int it = cw == 2 ? 1 : 0, jt = cw == 0 ? 0 : 1;
          f32x16 a = zero16();
#pragma unroll
          for (int s = 0; s < D / 16; ++s) {
            const bf16x8 b = frag<true>(Qy, G::ldQ, jt * 32, s * 16, ln);
            a = mfma(frag_tr<true>(Rh, G::ldR, it * 32, s * 16, ln), b, a);
            a = mfma(frag_tr<true>(Rl, G::ldR, it * 32, s * 16, ln), b, a);
          }
          read_ahead<10, 16, 40>();    // T: 16 MFMAs, 40 reads
          if (it == jt)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (acc_row(e, lg) > lr) a[e] = 0.f;
          float ps = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) ps += a[e];
          ps += __shfl_xor(ps, 32);
          if (lg == 0) denp[it * C + jt * 32 + lr] = ps;
          store_T<true>(a, Th, Tl, G::ldT, it * 32, jt * 32, ln);
        }
        acc[0] = zero16();
        acc[1] = zero16();
#pragma unroll
        for (int j = 0; j < D / 16; ++j) {
          bf16x8 bh_, bl_;
          frag_from_acc(st[j >> 1], j & 1, bh_, bl_);
#pragma unroll
          for (int rt = 0; rt < 2; ++rt) {
            const bf16x8 aQ = frag_acc_order<true>(Qy, G::ldQ, rt * 32, j * 16, ln);
            acc[rt] = mfma(aQ, bh_, acc[rt]);
            acc[rt] = mfma(aQ, bl_, acc[rt]);
          }
        }
        read_ahead<6, 32, 16>();     // Q Phi0
        if (normalized) {            // four lanes per token, 32 dimensions each
          const int tok = u >> 2, p0 = (u & 3) * 32;
          const uint16_t* row = Qy + tok * G::ldQ + p0;
          float sd = 0.f;
#pragma unroll
          for (int a = 0; a < 32; a += 8) {
            const uint4 x = *reinterpret_cast<const uint4*>(row + a);
            const float4 e0 = *reinterpret_cast<const float4*>(eta + p0 + a);
            const float4 e1 = *reinterpret_cast<const float4*>(eta + p0 + a + 4);
            sd += __uint_as_float(x.x << 16) * e0.x + __uint_as_float(x.x & 0xffff0000u) * e0.y;
            sd += __uint_as_float(x.y << 16) * e0.z + __uint_as_float(x.y & 0xffff0000u) * e0.w;
            sd += __uint_as_float(x.z << 16) * e1.x + __uint_as_float(x.z & 0xffff0000u) * e1.y;
            sd += __uint_as_float(x.w << 16) * e1.z + __uint_as_float(x.w & 0xffff0000u) * e1.w;
          }
          sd += __shfl_xor(sd, 1);
          sd += __shfl_xor(sd, 2);
          if ((u & 3) == 0) qeta[tok] = sd;
        }
      }
      prefetch(t);
      lds_barrier();
      // phase 2: O += T V and Phi0 += R^T V on column tile cw (one read of V
      // for both), eta0 += R^T 1, and the rows' 1 / (den + eps)
      if (hasY) {
#pragma unroll
        for (int s = 0; s < C / 16; ++s) {
          const bf16x8 bV = frag_tr<true>(Vs, G::ldV, cw * 32, s * 16, ln);
          if (!SUMMARY)
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
              if (s < 2 || rt == 1) {
                acc[rt] = mfma(frag<true>(Th, G::ldT, rt * 32, s * 16, ln), bV, acc[rt]);
                acc[rt] = mfma(frag<true>(Tl, G::ldT, rt * 32, s * 16, ln), bV, acc[rt]);
              }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            st[i] = mfma(frag<true>(Rh, G::ldR, i * 32, s * 16, ln), bV, st[i]);
            st[i] = mfma(frag<true>(Rl, G::ldR, i * 32, s * 16, ln), bV, st[i]);
          }
        }
        if constexpr (SUMMARY) read_ahead<12, 32, 40>();   // Phi0 advance: 32 MFMAs, 40 reads
        else read_ahead<12, 44, 52>();                    // T V, Phi0 advance: 44 MFMAs, 52 reads
        if (u < D) eta[u] += inc[u];
        if (!SUMMARY && normalized && u < C) {
          const float den = denp[u] + denp[C + u] + qeta[u];
          inv[u] = __builtin_amdgcn_rcpf(den + eps);
          const uint32_t tok = (uint32_t)(c_begin + t) * C + u;
          if (den_out && tok < (uint32_t)n) den_out[(size_t)bh * n + tok] = den;
        }
      }
      lds_barrier();
      // phase 3: next tiles staged and their successors' loads issued first,
      // so that waiting for those loads later never waits for the output
      // stores (one in-order counter covers both); then the output rows
      // (scaled by 1 / (den + eps) when normalised), staged through this
      // wave's slot of the dead W | T region so that every lane stores 16
      // bytes (8 stores a lane instead of 32)
      restage(t);
      if (!SUMMARY && hasY) {
        const uint32_t t0 = (uint32_t)(c_begin + t) * C;
        float* ob = reinterpret_cast<float*>(lds + G::oWh) + cw * (C * 32);   // [C][32] fp32
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            // element 4 qd + j of a row tile is row 8 qd + 4 lg + j: four
            // consecutive rows, whose scales are one float4
            const int r0 = rt * 32 + 8 * qd + 4 * lg;
            const float4 sc = normalized ? *reinterpret_cast<const float4*>(inv + r0) : make_float4(1.f, 1.f, 1.f, 1.f);
            ob[(r0 + 0) * 32 + lr] = acc[rt][4 * qd + 0] * sc.x;
            ob[(r0 + 1) * 32 + lr] = acc[rt][4 * qd + 1] * sc.y;
            ob[(r0 + 2) * 32 + lr] = acc[rt][4 * qd + 2] * sc.z;
            ob[(r0 + 3) * 32 + lr] = acc[rt][4 * qd + 3] * sc.w;
          }
#pragma unroll
        for (int j = 0; j < C / 8; ++j) {     // rows past n fall outside the buffer and are dropped
          const int row = 8 * j + (ln >> 3), c4 = (ln & 7) * 4;
          buf_store16(ro, ((t0 + row) * DV + cw * 32 + c4) * 4, *reinterpret_cast<const float4*>(ob + row * 32 + c4));
        }
      }
      lds_barrier();
    }
  }
  // ending state into the record: S0 (key side), Phi0 and eta0 (value side),
  // and with SUMMARY the segment's C and m
  if (rec) {
    int col = cw * 32 + lr;
    asm volatile("" : "+v"(col));
    float* dst = rec + (keyside ? 0 : off_G(D, DV));
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) dst[(size_t)(32 * i + acc_row(e, lg)) * D + col] = st[i][e];
    const int u = tid - 256;
    float* red = reinterpret_cast<float*>(lds + G::oWh);   // [16][D] partial sums of m (dead W | T region)
    if (!keyside) {
      if (u < D) rec[off_h(D, DV) + u] = eta[u];
      if (SUMMARY) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e) rec[off_C(D, DV) + (size_t)(32 * i + acc_row(e, lg)) * DV + col] = cacc[i][e];
#pragma unroll
        for (int j = 0; j < 8; ++j) red[(u >> 4) * D + (u & 15) * 8 + j] = macc[j];
      }
    }
    if (SUMMARY) {
      lds_barrier();
      if (!keyside && u < D) {
        float m = 0.f;
#pragma unroll
        for (int g = 0; g < 16; ++g) m += red[g * D + u];
        rec[off_m(D, DV) + u] = m;
      }
    }
  }
}

// First launch of the two-pass plan, grid (P - 1, BH): segment 0's output
// walk (zero carry) and the summary walks of segments 1 .. P-2 (zero state),
// each writing its record rec[bh][seg].
__global__ __launch_bounds__(CfgWS::NT, 1) void k_walk_ws_first(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, float* __restrict__ rec, int n, int c0, int cps,
    int nseg, int normalized, float eps) {
  extern __shared__ __align__(16) uint16_t lds[];
  int seg, bh;
  seg_head(seg, bh);
  int cb, nt;
  ws_range(seg, c0, cps, (n + CfgWS::C - 1) / CfgWS::C, cb, nt);
  float* r = rec + ((size_t)bh * (nseg + 1) + seg) * state_floats(CfgWS::D, CfgWS::DV);
  if (seg == 0)
    walk_ws<false>(lds, q, k, v, out, den_out, nullptr, nullptr, r, bh, n, cb, nt, normalized, eps);
  else
    walk_ws<true>(lds, q, k, v, nullptr, nullptr, nullptr, nullptr, r, bh, n, cb, nt, 0, 0.f);
}

// Output walks from the true carries, grid (walks, BH): grid column x walks
// segment seg0 + x.  spre: [BH][nseg][D*D] S prefixes and carry:
// [BH][nseg][D*DV + D] Phi, eta carries (both null for a single segment: zero).
__global__ __launch_bounds__(CfgWS::NT, 1) void k_walk_ws_out(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, const float* __restrict__ spre,
    const float* __restrict__ carry, int n, int c0, int cps, int nseg, int seg0, int normalized, float eps) {
  constexpr int D = CfgWS::D, DV = CfgWS::DV;
  extern __shared__ __align__(16) uint16_t lds[];
  int seg, bh;
  seg_head(seg, bh);
  seg += seg0;
  int cb, nt;
  ws_range(seg, c0, cps, (n + CfgWS::C - 1) / CfgWS::C, cb, nt);
  const float* si = spre ? spre + ((size_t)bh * nseg + seg) * D * D : nullptr;
  const float* ci = carry ? carry + ((size_t)bh * nseg + seg) * (D * DV + D) : nullptr;
  walk_ws<false>(lds, q, k, v, out, den_out, si, ci, nullptr, bh, n, cb, nt, normalized, eps);
}

// The S prefixes and the brackets of the two-pass plan (Eq. semidirect in
// the Phi form).  For segment s = 1 .. nseg-1: S_{<s}, the sum of the S
// slots of records 0 .. s-1 (record 0 holds the ending state of segment 0's
// output walk, records 1 .. nseg-2 the summaries), into spre[s] for the
// output walks.  For s <= nseg-2, whose record holds its S, C, m, Phi, eta
// from a zero start, also b_s = (Phi_s + S_{<s} C_s, eta_s + S_{<s} m_s),
// written in place of (Phi_s, eta_s); record 0 already holds b_0.
// grid (nseg - 1, BH), 1024 threads, one workgroup per (segment, head), a
// head's workgroups on one XCD.  S_{<s} and C_s are split into bf16 hi + lo
// in LDS, as every computed operand of the walks, and wave w forms the
// 32 x 32 tile (w / 4, w % 4) of S_{<s} C_s in three passes (hi hi, hi lo,
// lo hi) with fp32 accumulation.
template <int D, int DV>
__global__ __launch_bounds__(1024) void k_ws_bracket(float* __restrict__ rec, float* __restrict__ spre, int nseg) {
  constexpr int ldS = D + kPad, ldC = DV + 16, NT = 1024;   // ldC: C is read through the transpose unit
  static_assert(D == 128 && DV == 128, "16 waves of 32 x 32 output tiles");
  __shared__ __align__(16) uint16_t Sh[D * ldS], Sl[D * ldS], Ch[D * ldC], Cl[D * ldC];
  __shared__ float mv[D], ep[8 * D];
  int s, bh;
  seg_head(s, bh);
  s += 1;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int r0 = 32 * (w >> 2), c0 = 32 * (w & 3);
  const size_t F = state_floats(D, DV);
  float* r = rec + ((size_t)bh * (nseg + 1) + s) * F;
  constexpr int NS4 = D * D / 4 / NT;
  // S_{<s}: the earlier records' S slots, two records' loads in flight at a time
  float4 sx[NS4];
#pragma unroll
  for (int i = 0; i < NS4; ++i) sx[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  const float* r0s = rec + (size_t)bh * (nseg + 1) * F;
  for (int sp = 0; sp < s; sp += 2) {
    float4 u[2][NS4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < NS4; ++i)
        u[j][i] = sp + j < s ? reinterpret_cast<const float4*>(r0s + (size_t)(sp + j) * F)[tid + NT * i]
                             : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < NS4; ++i) {
        sx[i].x += u[j][i].x; sx[i].y += u[j][i].y; sx[i].z += u[j][i].z; sx[i].w += u[j][i].w;
      }
  }
  float4* spw = reinterpret_cast<float4*>(spre + ((size_t)bh * nseg + s) * D * D);
#pragma unroll
  for (int i = 0; i < NS4; ++i) spw[tid + NT * i] = sx[i];
  if (s == nseg - 1) return;   // the last segment has no summary, so no bracket
#pragma unroll
  for (int i = 0; i < NS4; ++i) {
    const int e = tid + NT * i, row = e / (D / 4), c4 = e % (D / 4);
    const float4 x = sx[i];
    const float4 y = *reinterpret_cast<const float4*>(r + off_C(D, DV) + (size_t)row * DV + 4 * c4);
    uint32_t h0, h1, l0, l1;
    split2(x.x, x.y, h0, l0);
    split2(x.z, x.w, h1, l1);
    *reinterpret_cast<uint2*>(Sh + row * ldS + 4 * c4) = make_uint2(h0, h1);
    *reinterpret_cast<uint2*>(Sl + row * ldS + 4 * c4) = make_uint2(l0, l1);
    split2(y.x, y.y, h0, l0);
    split2(y.z, y.w, h1, l1);
    *reinterpret_cast<uint2*>(Ch + row * ldC + 4 * c4) = make_uint2(h0, h1);
    *reinterpret_cast<uint2*>(Cl + row * ldC + 4 * c4) = make_uint2(l0, l1);
  }
  if (tid < D) mv[tid] = r[off_m(D, DV) + tid];
  f32x16 acc;        // b_s: element e is row r0 + acc_row(e, lg), column c0 + lr
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = r[off_G(D, DV) + (size_t)(r0 + acc_row(e, lg)) * DV + c0 + lr];
  const float eta = tid < D ? r[off_h(D, DV) + tid] : 0.f;
  __syncthreads();
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const bf16x8 ah = frag(Sh, ldS, r0, 16 * ks), al = frag(Sl, ldS, r0, 16 * ks);
    const bf16x8 bh_ = frag_tr(Ch, ldC, c0, 16 * ks), bl_ = frag_tr(Cl, ldC, c0, 16 * ks);
    acc = mfma(ah, bh_, acc);
    acc = mfma(ah, bl_, acc);
    acc = mfma(al, bh_, acc);
  }
  {  // S_{<s} m_s: eight partial sums of 16 k per row, then their total
    const int row = tid % D, part = tid / D;
    float x = 0.f;
#pragma unroll
    for (int j = 0; j < D / 8; ++j) {
      const int kk = part * (D / 8) + j;
      x += (bf16_to_f(Sh[row * ldS + kk]) + bf16_to_f(Sl[row * ldS + kk])) * mv[kk];
    }
    ep[part * D + row] = x;
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) r[off_G(D, DV) + (size_t)(r0 + acc_row(e, lg)) * DV + c0 + lr] = acc[e];
  __syncthreads();
  if (tid < D) {
    float e = eta;
#pragma unroll
    for (int p = 0; p < 8; ++p) e += ep[p * D + tid];
    r[off_h(D, DV) + tid] = e;
  }
}

}  // namespace
}  // namespace hla
