// Gradients of the masked second-order HLA (the reverse scan of Sec. 4.2)
// for bf16 inputs on gfx950 MFMA.
//
// With S_j = sum_{i<=j} k_i k_i^T, r_j = S_j q_j, Phi_j = sum_{j'<=j} r_j' v_j'^T
// (the forward prefixes of Thm. 1's proof), the upstream gradient g_t and the
// reverse prefixes U_j = sum_{t>=j} q_t g_t^T, u_j = U_j v_j and
// Z_i = sum_{j>=i} u_j q_j^T, the vector-Jacobian product of the masked
// operator is
//   dq_j = Phi_j g_j + S_j u_j,   dv_j = U_j^T r_j,   dk_i = (Z_i + Z_i^T) k_i.
// Every term is a first-order (linear) attention read causally or
// anti-causally.  Writing LA+(x, y, z)_j = sum_{i<=j} (x_j.y_i) z_i and
// LA-(x, y, z)_j = sum_{i>=j} (x_j.y_i) z_i:
//   r  = LA+(q, k, k)                       u  = LA-(v, g, q)
//   dq = LA+(g, v, r) + LA+(u, k, k)        dv = LA-(r, q, g)
//   dk = LA-(k, q, u) + LA-(k, u, q).
// The two dk passes share x and swap y and z; they run as one paired walk.
// Each pass is the first-order chunk scan: the state sum y z^T of a segment
// does not depend on anything before it, so every segment's walk starts from
// the exact prefix (suffix) of the segment moments and no fix-up follows.
//
// A moments pass (la_pass<..., MOM = true>) writes the moments
// M_s = sum_{i in s} y_i z_i^T of every segment; k_la_scan replaces them in
// place by their exclusive prefix (suffix) sums; a walk pass (MOM = false;
// k_la runs one pass or up to three side by side) walks a segment's 64-token tiles in
// time order (causal) or in reverse (anti-causal) from
// S0 = sum of the moments of the segments before (after) it, one record:
//   A = Q K^T masked (key <= query, or key >= query), O = A Z + X S0,
//   S0 += Y^T Z,
// and writes (or adds) O.  Operands that are exact in bf16 (q, k, v) take
// one MFMA pass; fp32 operands (g, r, u) and every computed operand (A, S0)
// are split into bf16 hi + lo, and a product of two split operands takes
// three passes (hi hi, hi lo, lo hi).  Accumulation is fp32.
#include <cstdlib>
#include <type_traits>

#include "backward.h"
#include "fused_tiles.h"
#include "profile.h"

namespace hla {
namespace {

template <int D>
struct CfgLA {
  static constexpr int C = 64;
  static constexpr int NCT = D / 32, NW = 2 * NCT, NT = 64 * NW;   // wave: row tile w / NCT, column tile w % NCT
  static constexpr int ST = D / 32, KC = C / 16, KD = D / 16;
  static constexpr int ld = D + kPad, ldA = C + kPad;
  // row-major bf16 tiles: X, Y, Z each hi | lo, then A hi | lo
  static constexpr int oXh = 0, oXl = oXh + C * ld, oYh = oXl + C * ld, oYl = oYh + C * ld;
  static constexpr int oZh = oYl + C * ld, oZl = oZh + C * ld, oAh = oZl + C * ld, oAl = oAh + C * ldA;
  static constexpr int n16 = oAl + C * ldA;
  static constexpr size_t bytes = (size_t)n16 * 2;
  static_assert(D * D * 2 <= n16, "state staging fits the tile region");
  static constexpr int kBlocks = 2 * bytes <= 160 * 1024 && NW <= 4 ? 2 : 1;
  static_assert(bytes <= 160 * 1024, "LDS budget");
  static_assert(D == 64 || D == 128, "linear-attention pass shapes");
};

// One 64 x D operand tile, rows t0 .. t0+63 of a [n][D] array, staged into
// LDS as bf16 (hi, and lo for fp32 inputs).  Rows past n read zero.
template <int D, int NT, bool F32>
struct Stage {
  static constexpr int EP = F32 ? 4 : 8;                     // elements per 16-byte piece
  static constexpr int NPC = 64 * D / EP;                    // pieces per tile
  static constexpr int NV = NPC / NT;                        // pieces per thread
  static_assert(NPC % NT == 0, "staging split");
  uint4 p[NV];
  __device__ __forceinline__ void fetch(rsrc_t r, int c, int tid) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e = tid + NT * i, t = e / (D / EP), a = (e % (D / EP)) * EP;   // consecutive lanes along a row
      p[i] = buf_load16(r, (((uint32_t)c * 64 + t) * D + a) * (F32 ? 4 : 2));
    }
  }
  __device__ __forceinline__ void store(uint16_t* hi, uint16_t* lo, int ld, int tid) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e = tid + NT * i, t = e / (D / EP), a = (e % (D / EP)) * EP;
      if constexpr (F32) {
        uint32_t h0, l0, h1, l1;
        split2(__uint_as_float(p[i].x), __uint_as_float(p[i].y), h0, l0);
        split2(__uint_as_float(p[i].z), __uint_as_float(p[i].w), h1, l1);
        *reinterpret_cast<uint2*>(hi + t * ld + a) = make_uint2(h0, h1);
        *reinterpret_cast<uint2*>(lo + t * ld + a) = make_uint2(l0, l1);
      } else {
        *reinterpret_cast<uint4*>(hi + t * ld + a) = p[i];
      }
    }
  }
};

// grid (nseg, BH), NT threads.  rev: anti-causal (keys at or after the
// query; tiles walked from the last).  acc_out: add to out instead of writing
// it.  tr: the records hold the transposed moments (sum z y^T of another pass).
// TWO: two passes that share x and swap y and z, LA(x, y, z) + LA(x, z, y),
// in one walk: A2 = X Z^T masked adds A2 Y, and the state is
// sum (y z^T + z y^T), staged from the moments of (y, z) plus their transpose
// (x and y exact in bf16: A2 takes the lo regions of X and Y).
template <int D, bool XF, bool YF, bool ZF, bool MOM, bool TWO = false, int MO = 0>
__device__ __forceinline__ void la_pass(
    const void* __restrict__ xp, const void* __restrict__ yp, const void* __restrict__ zp, float* __restrict__ out,
    float* __restrict__ rec, int n, int cps, int nseg, int rev, int acc_out, int tr, int scanned,
    const void* __restrict__ wp, float* __restrict__ rec2, int seg, int bh) {
  using G = CfgLA<D>;
  static_assert(!TWO || (!XF && !YF && !MOM), "the paired pass keeps A2 in the lo tiles of x and y");
  // MO: the walk also forms its segment's moments sum w o^T of its own output
  // o with w (MO = 1: a further bf16 input wp, staged in the lo tile of z;
  // MO = 2: w = z), into rec2; o goes through the lo tiles of x and y (MO = 1)
  // or x and z (MO = 2), which exact bf16 operands leave free
  static_assert(MO == 0 || (!MOM && !TWO && !XF && !ZF && (MO == 2 || !YF)), "free lo tiles for o and w");
  constexpr bool kO = D == 128;
  constexpr int C = G::C, NT = G::NT, ST = G::ST, ld = G::ld, ldA = G::ldA;
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* Xh = lds + G::oXh;
  uint16_t* Xl = lds + G::oXl;
  uint16_t* Yh = lds + G::oYh;
  uint16_t* Yl = lds + G::oYl;
  uint16_t* Zh = lds + G::oZh;
  uint16_t* Zl = lds + G::oZl;
  uint16_t* Ah = lds + G::oAh;
  uint16_t* Al = lds + G::oAl;
  uint16_t* A2h = Xl;             // TWO: A2 = X Z^T masked, in the (unused) lo tiles of x and y
  uint16_t* A2l = Yl;

  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rt = w / G::NCT, ct = w % G::NCT;
  const int M = (n + C - 1) / C;
  const int c_begin = seg * cps, c_end = min(M, c_begin + cps);
  const size_t DD = (size_t)D * D;

  // ---- state: zero for the moments; else the moments of the segments
  // before (after) this one, which k_la_scan has summed into this segment's
  // record ----
  f32x16 S0[ST];
#pragma unroll
  for (int i = 0; i < ST; ++i) S0[i] = zero16();
  const size_t eX = (XF ? 4 : 2), eY = (YF ? 4 : 2), eZ = (ZF ? 4 : 2);
  const rsrc_t rx = make_rsrc(static_cast<const char*>(xp) + (size_t)bh * n * D * eX, (uint32_t)(n * D * eX));
  const rsrc_t ry = make_rsrc(static_cast<const char*>(yp) + (size_t)bh * n * D * eY, (uint32_t)(n * D * eY));
  const rsrc_t rz = make_rsrc(static_cast<const char*>(zp) + (size_t)bh * n * D * eZ, (uint32_t)(n * D * eZ));
  const rsrc_t ro = make_rsrc(MOM ? nullptr : out + (size_t)bh * n * D, MOM ? 0u : (uint32_t)n * D * 4);
  Stage<D, NT, XF> sx;
  Stage<D, NT, YF> sy;
  Stage<D, NT, ZF> sz;
  Stage<D, NT, false> sw;
  const rsrc_t rw = make_rsrc(MO == 1 ? static_cast<const char*>(wp) + (size_t)bh * n * D * 2 : nullptr,
                              MO == 1 ? (uint32_t)(n * D * 2) : 0u);
  const int nt = c_end - c_begin;
  auto tile_of = [&](int i) { return rev ? c_end - 1 - i : c_begin + i; };
  // the first tile's loads go out before the state record's, so the two wait together
  if (nt > 0) {
    if (!MOM) sx.fetch(rx, tile_of(0), tid);
    sy.fetch(ry, tile_of(0), tid);
    sz.fetch(rz, tile_of(0), tid);
    if (MO == 1) sw.fetch(rw, tile_of(0), tid);
  }
  // MO: column ct of w o^T, all rows, over this wave's row tile of tokens
  // (the two waves of a column tile add their halves at the end)
  constexpr int SH = MO ? ST : 1;
  f32x16 M2[SH];
#pragma unroll
  for (int i = 0; i < SH; ++i) M2[i] = zero16();
  if (!MOM && nseg > 1) {
    // the records to sum: this segment's alone once k_la_scan has run
    // (scanned), else those of every segment before (after) it
    const int s_lo = scanned ? seg : rev ? seg + 1 : 0, s_hi = scanned ? seg + 1 : rev ? nseg : seg;
    if (s_lo < s_hi) {
      constexpr int nP4 = D * D / 4 / NT, RB = D == 64 ? 8 : 4, lds_ = D + 1;
      static_assert(D * D % (4 * NT) == 0 && D * lds_ * 4 <= 2 * G::n16, "state staging split");
      float4 pa[nP4];
#pragma unroll
      for (int r = 0; r < nP4; ++r) pa[r] = make_float4(0.f, 0.f, 0.f, 0.f);
      // RB records at a time, all their loads issued before the sums
      for (int sp = s_lo; sp < s_hi; sp += RB) {
        float4 u[RB][nP4];
#pragma unroll
        for (int j = 0; j < RB; ++j)
#pragma unroll
          for (int r = 0; r < nP4; ++r)
            u[j][r] = sp + j < s_hi
                          ? reinterpret_cast<const float4*>(rec + ((size_t)bh * nseg + sp + j) * DD)[tid + NT * r]
                          : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < RB; ++j)
#pragma unroll
          for (int r = 0; r < nP4; ++r) {
            pa[r].x += u[j][r].x; pa[r].y += u[j][r].y; pa[r].z += u[j][r].z; pa[r].w += u[j][r].w;
          }
      }
      // staged row-major with an odd row stride, so the transposed reads
      // (tr, TWO) fall in different banks
      float* st = reinterpret_cast<float*>(lds);
#pragma unroll
      for (int r = 0; r < nP4; ++r) {
        const int e = 4 * (tid + NT * r), row = e / D, col = e % D;
        st[row * lds_ + col] = pa[r].x;
        st[row * lds_ + col + 1] = pa[r].y;
        st[row * lds_ + col + 2] = pa[r].z;
        st[row * lds_ + col + 3] = pa[r].w;
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < ST; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int ra = i * 32 + acc_row(e, lg), cb = ct * 32 + lr;
          if constexpr (TWO)
            S0[i][e] = st[ra * lds_ + cb] + st[cb * lds_ + ra];
          else
            S0[i][e] = tr ? st[cb * lds_ + ra] : st[ra * lds_ + cb];
        }
      __syncthreads();
    }
  }

  for (int it = 0; it < nt; ++it) {
    const int c = tile_of(it);
    // ---- stage 0: operands into LDS (fp32 ones split into hi | lo) ----
    if (!MOM) sx.store(Xh, Xl, ld, tid);
    sy.store(Yh, Yl, ld, tid);
    sz.store(Zh, Zl, ld, tid);
    if (MO == 1) sw.store(Zl, nullptr, ld, tid);
    lds_barrier();
    if (it + 1 < nt) {
      if (!MOM) sx.fetch(rx, tile_of(it + 1), tid);
      sy.fetch(ry, tile_of(it + 1), tid);
      sz.fetch(rz, tile_of(it + 1), tid);
      if (MO == 1) sw.fetch(rw, tile_of(it + 1), tid);
    }

    f32x16 o = zero16();
    if (!MOM) {
      // ---- stage 1: A = X Y^T masked, as A^T = Y X^T on tiles (key kt, query qt), stored row-major ----
      if (w < 4) {
        const int kt = w >> 1, qt = w & 1;
        if (rev ? kt >= qt : kt <= qt) {
          f32x16 a = zero16();
#pragma unroll
          for (int s = 0; s < D / 16; ++s) {
            const bf16x8 yh = frag<kO>(Yh, ld, kt * 32, s * 16), xh = frag<kO>(Xh, ld, qt * 32, s * 16);
            a = mfma(yh, xh, a);
            if (XF) a = mfma(yh, frag<kO>(Xl, ld, qt * 32, s * 16), a);
            if (YF) a = mfma(frag<kO>(Yl, ld, kt * 32, s * 16), xh, a);
          }
#pragma unroll
          for (int e = 0; e < 16; ++e) {   // keep key <= query (causal) or key >= query (anti-causal)
            const int key = kt * 32 + acc_row(e, lg), qry = qt * 32 + lr;
            if (rev ? key < qry : key > qry) a[e] = 0.f;
          }
          store_T<kO>(a, Ah, Al, ldA, kt * 32, qt * 32);
          if constexpr (TWO) {            // A2 = X Z^T on the same tile, z split
            f32x16 a2 = zero16();
#pragma unroll
            for (int s = 0; s < D / 16; ++s) {
              const bf16x8 xh = frag<kO>(Xh, ld, qt * 32, s * 16);
              a2 = mfma(frag<kO>(Zh, ld, kt * 32, s * 16), xh, a2);
              a2 = mfma(frag<kO>(Zl, ld, kt * 32, s * 16), xh, a2);
            }
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int key = kt * 32 + acc_row(e, lg), qry = qt * 32 + lr;
              if (rev ? key < qry : key > qry) a2[e] = 0.f;
            }
            store_T<kO>(a2, A2h, A2l, ldA, kt * 32, qt * 32);
          }
        }
      }
      lds_barrier();
      // ---- stage 2: O = X S0 (state before this tile) + A Z ----
#pragma unroll
      for (int j = 0; j < G::KD; ++j) {
        bf16x8 sh, sl;
        frag_from_acc(S0[j >> 1], j & 1, sh, sl);
        const bf16x8 ah = frag_acc_order<kO>(Xh, ld, rt * 32, j * 16);
        o = mfma(ah, sh, o);
        o = mfma(ah, sl, o);
        if (XF) o = mfma(frag_acc_order<kO>(Xl, ld, rt * 32, j * 16), sh, o);
      }
#pragma unroll
      for (int s = 0; s < G::KC; ++s) {
        // keys of this k step against the row tile's queries: causal needs s < 2 (rt + 1), anti-causal s >= 2 rt
        if (rev ? s >= 2 * rt : s < 2 * (rt + 1)) {
          const bf16x8 zh = frag_tr<kO>(Zh, ld, ct * 32, s * 16);
          const bf16x8 ah = frag<kO>(Ah, ldA, rt * 32, s * 16), al = frag<kO>(Al, ldA, rt * 32, s * 16);
          o = mfma(ah, zh, o);
          o = mfma(al, zh, o);
          if (ZF) o = mfma(ah, frag_tr<kO>(Zl, ld, ct * 32, s * 16), o);
          if constexpr (TWO) {            // + A2 Y
            const bf16x8 yh = frag_tr<kO>(Yh, ld, ct * 32, s * 16);
            o = mfma(frag<kO>(A2h, ldA, rt * 32, s * 16), yh, o);
            o = mfma(frag<kO>(A2l, ldA, rt * 32, s * 16), yh, o);
          }
        }
      }
    }
    uint16_t* Oh = Xl;                       // MO: this tile's o, hi | lo
    uint16_t* Ol = MO == 1 ? Yl : Zl;
    if constexpr (MO != 0) store_N<kO>(o, Oh, Ol, ld, rt * 32, ct * 32);
    // ---- state advance: S0 += Y^T Z (column ct, all rows) ----
#pragma unroll
    for (int s = 0; s < G::KC; ++s) {
      const bf16x8 zh = frag_tr<kO>(Zh, ld, ct * 32, s * 16);
      bf16x8 zl;
      if (ZF) zl = frag_tr<kO>(Zl, ld, ct * 32, s * 16);
#pragma unroll
      for (int i = 0; i < ST; ++i) {
        const bf16x8 yh = frag_tr<kO>(Yh, ld, i * 32, s * 16);
        S0[i] = mfma(yh, zh, S0[i]);
        if (ZF) S0[i] = mfma(yh, zl, S0[i]);
        if (YF) S0[i] = mfma(frag_tr<kO>(Yl, ld, i * 32, s * 16), zh, S0[i]);
      }
      if constexpr (TWO) {                // + Z^T Y
        const bf16x8 yb = frag_tr<kO>(Yh, ld, ct * 32, s * 16);
#pragma unroll
        for (int i = 0; i < ST; ++i) {
          S0[i] = mfma(frag_tr<kO>(Zh, ld, i * 32, s * 16), yb, S0[i]);
          S0[i] = mfma(frag_tr<kO>(Zl, ld, i * 32, s * 16), yb, S0[i]);
        }
      }
    }
    if (!MOM) {
      // rows past n fall outside the buffer: loads read 0, stores drop
      const uint32_t ob = (((uint32_t)c * C + rt * 32 + 4 * lg) * D + ct * 32 + lr) * 4;
      float prev[16];
#pragma unroll
      for (int e = 0; e < 16; ++e)
        prev[e] = acc_out ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                                ro, (int)(ob + (8 * (e >> 2) + (e & 3)) * D * 4), 0, 0))
                          : 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) buf_store4(ro, ob + (8 * (e >> 2) + (e & 3)) * D * 4, prev[e] + o[e]);
    }
    if constexpr (MO != 0) {
      // M2 += w^T o over this wave's 32 tokens: the o piece read back is the
      // one this wave stored (a wave's LDS accesses complete in order), and w
      // was staged before the first barrier of the tile
      const uint16_t* Wt = MO == 1 ? Zl : Zh;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int k0 = rt * 32 + s * 16;
        const bf16x8 oh = frag_tr<kO>(Oh, ld, ct * 32, k0), ol = frag_tr<kO>(Ol, ld, ct * 32, k0);
#pragma unroll
        for (int i = 0; i < SH; ++i) {
          const bf16x8 a = frag_tr<kO>(Wt, ld, i * 32, k0);
          M2[i] = mfma(a, oh, M2[i]);
          M2[i] = mfma(a, ol, M2[i]);
        }
      }
    }
    lds_barrier();   // the next tile rewrites every LDS tile
  }

  if (MO != 0 && nseg > 1) {   // this segment's w o^T (no walk reads it with one segment)
    // the second token half's sums through LDS ([ct][row][32], free after the
    // loop's last barrier), added by the first half's waves, which write
    float* part = reinterpret_cast<float*>(lds) + ct * (D * 32);
    if (rt == 1)
#pragma unroll
      for (int i = 0; i < SH; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) part[(i * 32 + acc_row(e, lg)) * 32 + lr] = M2[i][e];
    lds_barrier();
    if (rt == 0) {
      int col = ct * 32 + lr;
      asm volatile("" : "+v"(col));
      float* r2 = rec2 + ((size_t)bh * nseg + seg) * DD;
#pragma unroll
      for (int i = 0; i < SH; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = i * 32 + acc_row(e, lg);
          r2[(size_t)row * D + col] = M2[i][e] + part[row * 32 + lr];
        }
    }
  }
  if (MOM && rt == 0) {   // both row waves hold the column; row tile 0's write it
    int col = ct * 32 + lr;
    asm volatile("" : "+v"(col));
    float* r = rec + ((size_t)bh * nseg + seg) * DD;
#pragma unroll
    for (int i = 0; i < ST; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) r[(size_t)(i * 32 + acc_row(e, lg)) * D + col] = S0[i][e];
  }
}

// The arguments of one pass, and a pass as a type (its template arguments).
struct LaArgs {
  const void* xp;
  const void* yp;
  const void* zp;
  float* out;
  float* rec;
  int n, cps, nseg, rev, acc_out, tr, scanned;
  const void* wp;
  float* rec2;
};
template <int D, bool XF, bool YF, bool ZF, bool MOM, bool TWO = false, int MO = 0>
struct LaPass {
  static __device__ __forceinline__ void run(const LaArgs& a, int seg, int bh) {
    la_pass<D, XF, YF, ZF, MOM, TWO, MO>(a.xp, a.yp, a.zp, a.out, a.rec, a.n, a.cps, a.nseg, a.rev, a.acc_out, a.tr,
                                         a.scanned, a.wp, a.rec2, seg, bh);
  }
};

// grid (segments, heads, passes): pass A, or up to three independent passes
// of the same shape in one launch, pass z on blockIdx.z (NP passes).
template <int D, int NP, class A, class B = A, class C = A>
__global__ __launch_bounds__((CfgLA<D>::NT), (CfgLA<D>::kBlocks)) void k_la(LaArgs a0, LaArgs a1, LaArgs a2) {
  int seg, bh;
  seg_head(seg, bh);
  if constexpr (NP == 1) {
    A::run(a0, seg, bh);
  } else if constexpr (NP == 2) {
    if (blockIdx.z == 0)
      A::run(a0, seg, bh);
    else
      B::run(a1, seg, bh);
  } else {
    if (blockIdx.z == 0)
      A::run(a0, seg, bh);
    else if (blockIdx.z == 1)
      B::run(a1, seg, bh);
    else
      C::run(a2, seg, bh);
  }
}

// The segment moments of one set turned in place into their exclusive
// prefix (rev = 0: the sum over the segments before each one, for causal
// walks) or suffix (rev = 1: over the segments after it, for anti-causal
// walks), so that a walk reads one record.  grid (D*D/256, BH), 64 * NPG
// threads (NPG <= 16): a block owns 64 consecutive float4 of the records of
// one head, and thread group g of it the g-th run of ceil(P / NPG)
// consecutive segments.  The groups sum their runs, take the exclusive sum
// of the groups before them from LDS, then rewrite their runs.
__global__ __launch_bounds__(1024) void k_la_scan(float* __restrict__ rec, int rev, int P, int DD) {
  __shared__ float4 part[16][64];
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6, npg = blockDim.x >> 6;
  const int per = (P + npg - 1) / npg, p0 = min(P, grp * per), p1 = min(P, p0 + per);
  float4* base = reinterpret_cast<float4*>(rec + (size_t)blockIdx.y * P * DD) + blockIdx.x * 64 + lane;
  const size_t stride = DD / 4;
  auto at = [&](int p) { return base + (size_t)(rev ? P - 1 - p : p) * stride; };
  float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int p = p0; p < p1; ++p) {
    const float4 u = *at(p);
    sum.x += u.x; sum.y += u.y; sum.z += u.z; sum.w += u.w;
  }
  part[grp][lane] = sum;
  __syncthreads();
  float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int g = 0; g < grp; ++g) {
    const float4 u = part[g][lane];
    x.x += u.x; x.y += u.y; x.z += u.z; x.w += u.w;
  }
#pragma unroll 4
  for (int p = p0; p < p1; ++p) {
    float4* a = at(p);
    const float4 u = *a;
    *a = x;
    x.x += u.x; x.y += u.y; x.z += u.z; x.w += u.w;
  }
}

// Segments per head above which the moments are scanned first: a walk sums
// at most this many records itself (in one or two batches of loads).
constexpr int kScanAbove = 8;

void la_plan(int D, int BH, int n, int* P, int* cps) {
  const int M = (n + 63) / 64;
  const int blocks = D == 64 ? CfgLA<64>::kBlocks : CfgLA<128>::kBlocks;
  int p = 256 * blocks / BH;
  if (const char* e = getenv("HLA_FUSED_SEGMENTS")) p = atoi(e);
  if (p < 1) p = 1;
  if (p > M) p = M;
  *cps = (M + p - 1) / p;
  *P = (M + *cps - 1) / *cps;
}

// Prefix (rev: suffix) sums of one moment set, in place, when P > kScanAbove.
hipError_t la_scan(float* rec, int rev, int BH, int P, int D, hipStream_t s) {
  if (P <= kScanAbove) return hipSuccess;
  int npg = 1;
  while (npg < 16 && npg < P) npg *= 2;
  prof_start("bwd_scan", s);
  HLA_LAUNCH(k_la_scan, dim3(D * D / 256, BH), dim3(64 * npg), 0, s, rec, rev, P, D * D);
  prof_stop(s);
  return hipGetLastError();
}

// One launch of pass A, or of passes A and B side by side (grid z = 2), over
// every (segment, head).  A pass's moments (MOM) are the sums y z^T of each
// segment; a walk (TWO: the paired walk LA(x, y, z) + LA(x, z, y); MO: also
// the moments w o^T of its output into rec2, with w = wp (MO = 1) or z
// (MO = 2)) starts every segment from the moments of the others on its side.
template <int D, int NP, class A, class B = A, class C = A>
hipError_t la_launch(const char* name, const LaArgs& a0, const LaArgs& a1, const LaArgs& a2, int BH, int P,
                     hipStream_t s) {
  using G = CfgLA<D>;
  const void* kf = (const void*)k_la<D, NP, A, B, C>;
  hipError_t e;
  if ((e = hipFuncSetAttribute(kf, hipFuncAttributeMaxDynamicSharedMemorySize, (int)G::bytes)) != hipSuccess) return e;
  prof_start(name, s);
  HLA_LAUNCH((k_la<D, NP, A, B, C>), dim3(P, BH, NP), dim3(G::NT), G::bytes, s, a0, a1, a2);
  prof_stop(s);
  return hipGetLastError();
}

// The arguments of a pass LA(x, y, z) (rev: anti-causal; acc: add to out;
// tr: the records hold the transposed moments).
LaArgs la_args(const void* x, const void* y, const void* z, float* out, float* rec, int n, int cps, int P, int rev,
               int acc, int tr, const void* wp = nullptr, float* rec2 = nullptr) {
  return LaArgs{x, y, z, out, rec, n, cps, P, rev, acc, tr, P > kScanAbove ? 1 : 0, wp, rec2};
}

size_t rec_bytes(int BH, int P, int d) {
  return (sizeof(float) * (size_t)BH * P * d * d + 255) & ~size_t(255);
}
size_t vec_bytes(int BH, int n, int d) { return (sizeof(float) * (size_t)BH * n * d + 255) & ~size_t(255); }

template <int D>
hipError_t run_backward(const Bwd& b, char* ws, hipStream_t s) {
  int P, cps;
  la_plan(D, b.BH, b.n, &P, &cps);
  const int BH = b.BH, n = b.n;
  const size_t rb = rec_bytes(BH, P, D);
  // four moment sets serve the seven passes: k^T k (r and the second dq
  // term), g^T q (u; transposed for dv), v^T r (the first dq term) and
  // q^T u (the first dk term; transposed for the second)
  float* kk = reinterpret_cast<float*>(ws);
  float* gq = reinterpret_cast<float*>(ws + rb);
  float* vr = reinterpret_cast<float*>(ws + 2 * rb);
  float* qu = reinterpret_cast<float*>(ws + 3 * rb);
  float* r = reinterpret_cast<float*>(ws + 4 * rb);
  float* u = reinterpret_cast<float*>(ws + 4 * rb + vec_bytes(BH, n, D));
  hipError_t e;
#define HLA_TRY(x) if ((e = (x)) != hipSuccess) return e
  // Each moment set serves walks of one direction only, so with many
  // segments the scan turns it in place into the prefixes (k^T k, v^T r:
  // causal) or suffixes (g^T q, q^T u: anti-causal) the walks start from.
  // Passes that do not depend on each other share a launch.
  using MomKK = LaPass<D, false, false, false, true>;
  using MomGQ = LaPass<D, false, true, false, true>;
  using WalkR = LaPass<D, false, false, false, false, false, 1>;    // also v^T r
  using WalkU = LaPass<D, false, true, false, false, false, 2>;     // also q^T u
  using WalkG = LaPass<D, true, false, true, false>;                       // x, z fp32: dq (first term), dv
  using WalkU2 = LaPass<D, true, false, false, false>;                     // x fp32: dq (second term)
  using WalkK = LaPass<D, false, false, true, false, true>;          // paired dk
  const LaArgs none{};
  // the moments k^T k (r, the second dq term) and g^T q (u; transposed for dv)
  if (P > 1)
    HLA_TRY((la_launch<D, 2, MomKK, MomGQ>("bwd_moments", la_args(b.k, b.k, b.k, nullptr, kk, n, cps, P, 0, 0, 0),
                                           la_args(b.g, b.g, b.q, nullptr, gq, n, cps, P, 0, 0, 0), none, BH, P,
                                           s)));
  HLA_TRY(la_scan(kk, 0, BH, P, D, s));
  HLA_TRY(la_scan(gq, 1, BH, P, D, s));
  // r = LA+(q, k, k) with the v^T r moments, beside u = LA-(v, g, q) with the q^T u moments
  HLA_TRY((la_launch<D, 2, WalkR, WalkU>("bwd_ru", la_args(b.q, b.k, b.k, r, kk, n, cps, P, 0, 0, 0, b.v, vr),
                                         la_args(b.v, b.g, b.q, u, gq, n, cps, P, 1, 0, 0, nullptr, qu), none, BH,
                                         P, s)));
  HLA_TRY(la_scan(vr, 0, BH, P, D, s));
  HLA_TRY(la_scan(qu, 1, BH, P, D, s));
  // the first dq term LA+(g, v, r), beside dv = LA-(r, q, g) (moments q^T g =
  // (g^T q)^T) and dk = LA-(k, q, u) + LA-(k, u, q) in one paired walk (state
  // sum q u^T + u q^T); then the second dq term LA+(u, k, k), added
  HLA_TRY((la_launch<D, 3, WalkG, WalkG, WalkK>("bwd_dq_dv_dk", la_args(b.g, b.v, r, b.dq, vr, n, cps, P, 0, 0, 0),
                                                la_args(r, b.q, b.g, b.dv, gq, n, cps, P, 1, 0, 1),
                                                la_args(b.k, b.q, u, b.dk, qu, n, cps, P, 1, 0, 0), BH, P, s)));
  HLA_TRY((la_launch<D, 1, WalkU2>("bwd_dq", la_args(u, b.k, b.k, b.dq, kk, n, cps, P, 0, 1, 0), none, none, BH, P,
                                   s)));
#undef HLA_TRY
  return hipSuccess;
}

}  // namespace

bool backward_supported(int n, int d, int dv, int dtype) {
  const long long span = (long long)n * d * 4;   // per-head byte offsets stay below 2^31
  return dtype == 1 && n >= 1 && d == dv && (d == 64 || d == 128) && span < (1LL << 31);
}

size_t backward_workspace_bytes(int BH, int n, int d) {
  int P, cps;
  la_plan(d, BH, n, &P, &cps);
  return 4 * rec_bytes(BH, P, d) + 2 * vec_bytes(BH, n, d) + 256;
}

hipError_t launch_backward(const Bwd& b, void* workspace, hipStream_t s) {
  if (!backward_supported(b.n, b.d, b.dvd, b.dtype)) return hipErrorNotSupported;
  char* ws = static_cast<char*>(workspace);
  return b.d == 64 ? run_backward<64>(b, ws, s) : run_backward<128>(b, ws, s);
}

}  // namespace hla
