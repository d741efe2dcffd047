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
// The walk starts from the true carry of its segment: S0 = S prefix, and
// (output walk) Phi0, eta0 = the running sums of the earlier segments'
// brackets, so every output row is final when written (division included).
// The SUMMARY form starts from Phi0 = eta0 = 0, skips T and O, and writes its
// ending (Phi0, eta0), the segment's bracket, into its record.
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

// grid (segments walked, BH), 512 threads.  spre: [BH][nseg][D*D] S prefixes
// (null: zero); carry: [BH][nseg][D*DV + D] Phi, eta carries (null: zero;
// unused by SUMMARY); rec: [BH][nseg + 1][F] records (SUMMARY writes the
// bracket into the G and h slots of its segment).
template <bool SUMMARY>
__global__ __launch_bounds__(CfgWS::NT, 1) void k_walk_ws(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    float* __restrict__ out, float* __restrict__ den_out, const float* __restrict__ spre,
    const float* __restrict__ carry, float* __restrict__ rec, int n, int cps, int nseg, int normalized,
    float eps) {
  using G = CfgWS;
  constexpr int C = G::C, D = G::D, DV = G::DV, NT = G::NT;
  extern __shared__ __align__(16) uint16_t lds[];
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

  int seg, bh;
  seg_head(seg, bh);
  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool keyside = w < 4;        // waves 0-3: S0 and R; waves 4-7: Phi0, T and O
  const int cw = w & 3;              // this wave's state column tile
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, nt = min(M, c_begin + cps) - c_begin;
  const size_t F = state_floats(D, DV);

  // ---- carry in: column tile cw of S0 (key side) or Phi0 (value side), all rows ----
  f32x16 st[4];      // rows 32i .. 32i + 31
  {
    const float* src = keyside ? (spre ? spre + ((size_t)bh * nseg + seg) * D * D : nullptr)
                               : ((!SUMMARY && carry) ? carry + ((size_t)bh * nseg + seg) * (D * DV + D) : nullptr);
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
  if (tid < D) {
    eta[tid] = (!SUMMARY && carry) ? carry[((size_t)bh * nseg + seg) * (D * DV + D) + D * DV + tid] : 0.f;
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
    if (SUMMARY) {                   // the bracket: Phi0 into the G slot, eta0 into the h slot
      const int u = tid - 256;
      float* rc = rec + ((size_t)bh * (nseg + 1) + seg) * F;
      int col = cw * 32 + lr;
      asm volatile("" : "+v"(col));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) rc[off_G(D, DV) + (size_t)(32 * i + acc_row(e, lg)) * DV + col] = st[i][e];
      if (u < D) rc[off_h(D, DV) + u] = eta[u];
    }
  }
}

}  // namespace
}  // namespace hla
