// Device building blocks shared by the fused second-order walks (Sec. 4
// two-level scan) and the AHLA walk (Sec. 6): bf16 MFMA tile fragments on
// v_mfma_f32_32x32x16_bf16, hi/lo splitting of computed operands, buffer
// resources, the segment moments, and the carry fix-up that adds the prefix
// of the earlier segments to every output.  Included by the .hip files only
// (everything lives in an anonymous namespace).
#pragma once
#include <type_traits>

#include "common.h"

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

// The same for a pair: hi = (hi(x0), hi(x1)) and lo likewise, packed low
// half first.  One packed conversion gives both high parts, so a pair costs
// two conversions, two unpacks and two subtractions.
__device__ __forceinline__ void split2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  hi = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){x0, x1}, b2));
  const float h0 = __uint_as_float(hi << 16), h1 = __uint_as_float(hi & 0xffff0000u);
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){x0 - h0, x1 - h1}, b2));
}

// Buffer resource over [p, p + bytes): loads past the end return zero and
// stores past the end are dropped, which zero-fills the ragged last chunk and
// clips its outputs.  Offsets are 32-bit bytes from p.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(rsrc_t r, uint32_t off) {
  const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(x[0], x[1], x[2], x[3]);
}
__device__ __forceinline__ void buf_store4(rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, 0);
}
__device__ __forceinline__ void buf_store16(rsrc_t r, uint32_t off, const float4& v) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                                               __float_as_uint(v.w)},
                                         r, (int)off, 0, 0);
}

// Workgroup -> (segment, head) for the walks, grid (segments, heads): a
// walk's prologue reads the moment records of the segments before it, so the
// segments of one head go to one XCD and share those reads through its L2
// (the fix-up uses it for its tile groups, which share carry reads).
// Workgroups are dealt to the 8 XCDs round-robin by linear index, so the k-th
// workgroup on XCD x takes pair x * (total / 8) + k.
__device__ __forceinline__ void seg_head(int& seg, int& bh) {
  const int P = gridDim.x, total = gridDim.x * gridDim.y, L = blockIdx.x + gridDim.x * blockIdx.y;
  if (total % 8) {
    seg = blockIdx.x;
    bh = blockIdx.y;
    return;
  }
  const int idx = (L % 8) * (total / 8) + L / 8;
  seg = idx % P;
  bh = idx / P;
}

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

// Lane index.  With O set it passes through an empty asm statement, so each
// fragment access computes its LDS address next to the access instead of the
// compiler hoisting every distinct address out of a walk loop and keeping them
// live (or spilled) through it; worth it only where registers run out.
template <bool O = false>
__device__ __forceinline__ int lane64() {
  int l = threadIdx.x & 63;
  if constexpr (O) asm volatile("" : "+v"(l));
  return l;
}

// Operand fragment from a row-major bf16 LDS tile X[row][k]: lane takes
// X[row0 + r][k0 + 8g .. 8g+7].  A operand of X Y, or B operand of Z X^T.
template <bool O = false>
__device__ __forceinline__ bf16x8 frag(const uint16_t* X, int ld, int row0, int k0, int l = lane64<O>()) {
  const uint16_t* p = X + (row0 + (l & 31)) * ld + k0 + 8 * (l >> 5);
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// Same, in the k order of an accumulator-fed partner: lane takes
// X[row0 + r][k0 + 4g .. 4g+3] and X[row0 + r][k0 + 8 + 4g .. 8+4g+3].
template <bool O = false>
__device__ __forceinline__ bf16x8 frag_acc_order(const uint16_t* X, int ld, int row0, int k0, int l = lane64<O>()) {
  const uint16_t* p = X + (row0 + (l & 31)) * ld + k0 + 4 * (l >> 5);
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  const uint2 b = *reinterpret_cast<const uint2*>(p + 8);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// Operand fragment read through the LDS transpose unit from a row-major bf16
// tile Y[k][n]: lane takes Y[k0 + 8g .. 8g+7][n0 + r], the fragment frag()
// would take from Y^T.  ds_read_b64_tr_b16 works in groups of 16 lanes:
// element m of lane j's result is element j % 4 of the 8 bytes read by lane
// 4m + j / 4 of its group.  So lane j of a group reads row k + j / 4 at
// columns 4 (j % 4) .. + 3, and receives rows k .. k+3 of column j; two reads
// give the 8 rows of a fragment.  (Layout checked on the device by an
// in-bounds probe.)  Y and ld must keep 8-byte alignment (ld % 4 == 0).
template <bool O = false>
__device__ __forceinline__ bf16x8 frag_tr(const uint16_t* Y, int ld, int n0, int k0, int l = lane64<O>()) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
  const int grp = l >> 4, j = l & 15;
  const uint16_t* p = Y + (k0 + 8 * (grp >> 1) + (j >> 2)) * ld + n0 + 16 * (grp & 1) + 4 * (j & 3);
  const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
  const v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p + 4 * ld));
  const uint2 ua = __builtin_bit_cast(uint2, a), ub = __builtin_bit_cast(uint2, b);
  return __builtin_bit_cast(bf16x8, make_uint4(ua.x, ua.y, ub.x, ub.y));
}

// B operand for k rows 16h .. 16h+15 of an accumulator tile Y (32 rows): the
// lane's elements 8h .. 8h+7 are rows 16h + {4g..4g+3, 8+4g..8+4g+3} of its
// column, matching frag_acc_order.  Split into hi and lo parts.
__device__ __forceinline__ void frag_from_acc(const f32x16& t, int h, bf16x8& hi, bf16x8& lo) {
  uint32_t a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) split2(t[8 * h + 2 * i], t[8 * h + 2 * i + 1], a[i], b[i]);
  hi = __builtin_bit_cast(bf16x8, make_uint4(a[0], a[1], a[2], a[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(b[0], b[1], b[2], b[3]));
}

// Decay (the decayed second-order operator): a bf16 operand fragment whose 8
// elements are the tokens t0 .. t0+7 of one column, scaled per token by
// w[t0 + m] (fp32, from an LDS table) and split into bf16 hi + lo.
__device__ __forceinline__ void scale_split(const bf16x8& x, const float* w, bf16x8& hi, bf16x8& lo) {
  const float4 w0 = *reinterpret_cast<const float4*>(w), w1 = *reinterpret_cast<const float4*>(w + 4);
  const float wm[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
  uint32_t a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) split2((float)x[2 * i] * wm[2 * i], (float)x[2 * i + 1] * wm[2 * i + 1], a[i], b[i]);
  hi = __builtin_bit_cast(bf16x8, make_uint4(a[0], a[1], a[2], a[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(b[0], b[1], b[2], b[3]));
}

// Store an accumulator tile D[row0 + i][col0 + r] transposed as X[col0 + r][row0 + i],
// split into hi/lo tiles (four 8-byte stores each).
template <bool O = false>
__device__ __forceinline__ void store_T(const f32x16& acc, uint16_t* Xh, uint16_t* Xl, int ld, int row0, int col0, int l = lane64<O>()) {
  const int g = l >> 5;
  const int base = (col0 + (l & 31)) * ld + row0 + 4 * g;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t h[2], o[2];
    split2(acc[4 * q], acc[4 * q + 1], h[0], o[0]);
    split2(acc[4 * q + 2], acc[4 * q + 3], h[1], o[1]);
    *reinterpret_cast<uint2*>(Xh + base + 8 * q) = make_uint2(h[0], h[1]);
    *reinterpret_cast<uint2*>(Xl + base + 8 * q) = make_uint2(o[0], o[1]);
  }
}

// Store an accumulator tile row-major as X[row0 + i][col0 + r], hi/lo.
template <bool O = false>
__device__ __forceinline__ void store_N(const f32x16& acc, uint16_t* Xh, uint16_t* Xl, int ld, int row0, int col0, int l = lane64<O>()) {
  const int g = l >> 5;
#pragma unroll
  for (int e = 0; e < 16; e += 2) {
    uint32_t h, o;
    split2(acc[e], acc[e + 1], h, o);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int off = (row0 + acc_row(e + j, g)) * ld + col0 + (l & 31);
      Xh[off] = (uint16_t)(h >> (16 * j));
      Xl[off] = (uint16_t)(o >> (16 * j));
    }
  }
}

// ---------------------------------------------------------------------------
// Segment moments.  The walks start from the true S prefix, so every segment
// needs S of the segments before it; with a final state also C and m.  grid
// (nseg, BH), 4 waves: S = K^T K and C = Q^T V over the segment's tiles on
// MFMA (q/k/v are exact in bf16, one pass), m = Q^T 1.  Written to the S, C
// and m slots of the segment's record.
//
// KV (the AHLA walk, Sec. 6): P = K^T V into the C slot and m^K = K^T 1 into
// the m slot; no S, and q is not read (want_cm is ignored).
// DEC (decay gamma = 2^lg2g; S only): S = sum_t gamma^(e - t) k_t k_t^T with e
// the segment's last token, the weight applied to one factor per token in
// fp32 and split hi/lo.
// CM = false compiles the S-only form alone (want_cm is ignored): without the
// C and m registers and buffers it runs at a higher occupancy.
template <int C, int D, int DV, bool KV = false, bool DEC = false, bool CM = true>
__global__ __launch_bounds__(kThreads) void k_moments(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                      const uint16_t* __restrict__ v, float* __restrict__ rec, int n,
                                                      int cps, int nseg, int want_cm, float lg2g) {
  constexpr int DT = D / 32, VT = DV / 32, KC = C / 16;
  constexpr int nS = (DT * DT + kWaves - 1) / kWaves, nC = (DT * VT + kWaves - 1) / kWaves;
  constexpr int segQ = C * D / 8, segV = C * DV / 8;
  // Kt: K^T (C and m path) or a row-major k tile (S-only path)
  constexpr int nKt = C * (D + 16);                       // a row-major k tile
  constexpr int nV = C * (DV + 16) > kWaves * D * 2 ? C * (DV + 16) : kWaves * D * 2;   // also m's partials
  __shared__ __align__(16) uint16_t Kt[nKt], Qs_[(KV || !CM) ? 8 : C * (D + 16)], Vt[CM ? nV : 8];
  __shared__ __align__(16) float wtab[DEC ? C : 4];   // decay weights of the current tile's tokens
  static_assert(CM || !KV, "the AHLA moments form K^T V");
  if (KV) want_cm = 1;
  if (!CM) want_cm = 0;
  const int seg = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int M = (n + C - 1) / C, c0 = seg * cps, c1 = min(M, c0 + cps);
  const rsrc_t rq = make_rsrc(q + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rk = make_rsrc(k + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t rv = make_rsrc(v + (size_t)bh * n * DV, (uint32_t)n * DV * 2);
  f32x16 sacc[nS], cacc[nC];
#pragma unroll
  for (int i = 0; i < nS; ++i) sacc[i] = zero16();
#pragma unroll
  for (int i = 0; i < nC; ++i) cacc[i] = zero16();
  float macc = 0.f;
  if (!want_cm) {
    // S only: K tiles streamed through a ring of PF register slots (loads are
    // unconditional; the tile index is clamped to the segment), so PF tiles
    // are in flight while one is multiplied.  A tile sits row-major in LDS
    // (16-byte stores) and the K^T fragments are read through the transpose
    // unit; a row stride of 8 banks modulo 32 keeps the four rows of each
    // 16-lane transposed read in different banks.
    constexpr int PF = 4, NL = (segQ + kThreads - 1) / kThreads, ldk = D + 16;
    uint16_t* Ks = Kt;
    uint4 kb[PF][NL];
    auto load = [&](int c, auto slot_tag) {
      constexpr int sl = decltype(slot_tag)::value;
      const uint32_t t0 = (uint32_t)min(c, c1 - 1) * C;
#pragma unroll
      for (int i = 0; i < NL; ++i) {      // consecutive lanes take consecutive pieces of a token row
        const int e = min(tid + kThreads * i, segQ - 1);
        kb[sl][i] = buf_load16(rk, ((t0 + e / (D / 8)) * D + (e % (D / 8)) * 8) * 2);
      }
    };
    auto step = [&](int c, auto slot_tag) {
      constexpr int sl = decltype(slot_tag)::value;
      if (DEC && tid < C) wtab[tid] = exp2f(lg2g * (float)((c0 + cps - 1 - c) * C + C - 1 - tid));
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int e = tid + kThreads * i;
        if (e < segQ) *reinterpret_cast<uint4*>(Ks + (e / (D / 8)) * ldk + (e % (D / 8)) * 8) = kb[sl][i];
      }
      lds_barrier();
      load(c + PF, slot_tag);
#pragma unroll
      for (int i = 0; i < nS; ++i) {
        const int ti = w + kWaves * i;
        if (ti < DT * DT) {
          const int it = ti / DT, jt = ti % DT;
#pragma unroll
          for (int s = 0; s < KC; ++s) {
            const bf16x8 a = frag_tr(Ks, ldk, it * 32, s * 16);
            if constexpr (DEC) {
              bf16x8 bh, bl;
              scale_split(frag_tr(Ks, ldk, jt * 32, s * 16), wtab + s * 16 + 8 * lg, bh, bl);
              sacc[i] = mfma(a, bh, sacc[i]);
              sacc[i] = mfma(a, bl, sacc[i]);
            } else {
              sacc[i] = mfma(a, frag_tr(Ks, ldk, jt * 32, s * 16), sacc[i]);
            }
          }
        }
      }
      lds_barrier();
    };
    if (c0 < c1) {
      load(c0, std::integral_constant<int, 0>());
      load(c0 + 1, std::integral_constant<int, 1>());
      load(c0 + 2, std::integral_constant<int, 2>());
      load(c0 + 3, std::integral_constant<int, 3>());
    }
    for (int c = c0; c < c1; c += PF) {
      step(c, std::integral_constant<int, 0>());
      if (c + 1 < c1) step(c + 1, std::integral_constant<int, 1>());
      if (c + 2 < c1) step(c + 2, std::integral_constant<int, 2>());
      if (c + 3 < c1) step(c + 3, std::integral_constant<int, 3>());
    }
  }
  // with C (and m): the next tile's k, q, v pieces are loaded into registers
  // while the current one is multiplied (loads unconditional: piece and tile
  // indices are clamped, only owners store).  Tiles sit row-major in LDS
  // (16-byte stores, row stride d + 16 as in the S-only path) and every
  // transposed operand is read through the transpose unit.  m = Q^T 1 is
  // summed from the staged pieces: a thread's pieces always cover the same
  // eight columns a8 .. a8+7.
  constexpr int NLK = (segQ + kThreads - 1) / kThreads, NLV = (segV + kThreads - 1) / kThreads;
  constexpr int ldk = D + 16, ldv = DV + 16;
  static_assert(kThreads % (D / 8) == 0 && kThreads % (DV / 8) == 0, "fixed columns per thread");
  uint16_t* Qr = KV ? Kt : Qs_;           // row-major q (k for the K^T V form)
  uint4 pk_[NLK], pq_[NLK], pv_[NLV];
  float m8[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) m8[j] = 0.f;
  auto fetch_cm = [&](int c) {
    const uint32_t t0 = (uint32_t)min(c, c1 - 1) * C;
#pragma unroll
    for (int i = 0; i < NLK; ++i) {     // consecutive lanes take consecutive pieces of a token row
      const int e = min(tid + kThreads * i, segQ - 1);
      const uint32_t off = ((t0 + e / (D / 8)) * D + (e % (D / 8)) * 8) * 2;
      if (!KV) pk_[i] = buf_load16(rk, off);
      pq_[i] = buf_load16(KV ? rk : rq, off);
    }
#pragma unroll
    for (int i = 0; i < NLV; ++i) {
      const int e = min(tid + kThreads * i, segV - 1);
      pv_[i] = buf_load16(rv, ((t0 + e / (DV / 8)) * DV + (e % (DV / 8)) * 8) * 2);
    }
  };
  if (want_cm && c0 < c1) fetch_cm(c0);
  for (int c = want_cm ? c0 : c1; c < c1; ++c) {
#pragma unroll
    for (int i = 0; i < NLK; ++i) {
      const int e = tid + kThreads * i;
      if (e < segQ) {
        const int o = (e / (D / 8)) * ldk + (e % (D / 8)) * 8;
        if (!KV) *reinterpret_cast<uint4*>(Kt + o) = pk_[i];
        *reinterpret_cast<uint4*>(Qr + o) = pq_[i];
        const uint32_t u[4] = {pq_[i].x, pq_[i].y, pq_[i].z, pq_[i].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          m8[2 * j] += __uint_as_float(u[j] << 16);
          m8[2 * j + 1] += __uint_as_float(u[j] & 0xffff0000u);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NLV; ++i) {
      const int e = tid + kThreads * i;
      if (e < segV) *reinterpret_cast<uint4*>(Vt + (e / (DV / 8)) * ldv + (e % (DV / 8)) * 8) = pv_[i];
    }
    lds_barrier();
    if (c + 1 < c1) fetch_cm(c + 1);
#pragma unroll
    for (int i = 0; i < nS; ++i) {
      const int ti = w + kWaves * i;
      if (!KV && ti < DT * DT) {
        const int it = ti / DT, jt = ti % DT;
#pragma unroll
        for (int s = 0; s < KC; ++s)
          sacc[i] = mfma(frag_tr(Kt, ldk, it * 32, s * 16), frag_tr(Kt, ldk, jt * 32, s * 16), sacc[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < nC; ++i) {
      const int ti = w + kWaves * i;
      if (ti < DT * VT) {
        const int it = ti / VT, jt = ti % VT;
#pragma unroll
        for (int s = 0; s < KC; ++s)
          cacc[i] = mfma(frag_tr(Qr, ldk, it * 32, s * 16), frag_tr(Vt, ldv, jt * 32, s * 16), cacc[i]);
      }
    }
    lds_barrier();
  }
  if (want_cm) {      // m: sum the partial column sums over the lanes, then the waves, that share columns
#pragma unroll
    for (int o = D / 8; o < 64; o <<= 1)
#pragma unroll
      for (int j = 0; j < 8; ++j) m8[j] += __shfl_xor(m8[j], o);
    float* part = reinterpret_cast<float*>(Vt);          // [kWaves][D]; the tiles are dead
    if (l < D / 8)
#pragma unroll
      for (int j = 0; j < 8; ++j) part[w * D + l * 8 + j] = m8[j];
    lds_barrier();
    if (tid < D) {
      macc = 0.f;
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww) macc += part[ww * D + tid];
    }
  }
  float* r = rec + ((size_t)bh * (nseg + 1) + seg) * state_floats(D, DV);
#pragma unroll
  for (int i = 0; i < nS; ++i) {
    const int ti = w + kWaves * i;
    if (!KV && ti < DT * DT) {
      const int it = ti / DT, jt = ti % DT;
#pragma unroll
      for (int e = 0; e < 16; ++e) r[(size_t)(it * 32 + acc_row(e, lg)) * D + jt * 32 + lr] = sacc[i][e];
    }
  }
  if (want_cm) {
#pragma unroll
    for (int i = 0; i < nC; ++i) {
      const int ti = w + kWaves * i;
      if (ti < DT * VT) {
        const int it = ti / VT, jt = ti % VT;
#pragma unroll
        for (int e = 0; e < 16; ++e)
          r[off_C(D, DV) + (size_t)(it * 32 + acc_row(e, lg)) * DV + jt * 32 + lr] = cacc[i][e];
      }
    }
    if (tid < D) r[off_m(D, DV) + tid] = macc;
  }
}

// dst[bh][s][0 .. len): the exclusive running sums over a head's segments of
// one part of the records rec[bh][0 .. nseg] (F floats each, from float `off`
// on): x_0 = (use_init ? slot nseg : 0), x_{s+1} = rho x_s + slot s (rho: the
// decay of one segment's moments over the next, 1 without decay).  Each walk
// then reads its segment's prefix as one record.  grid (ceil(len / 1024), BH).
__global__ __launch_bounds__(256) void k_seg_prefix(const float* __restrict__ rec, size_t F, int off, int len,
                                                    int use_init, float* __restrict__ dst, int nseg, float rho) {
  const int bh = blockIdx.y, p = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (p >= len) return;
  const float* base = rec + (size_t)bh * (nseg + 1) * F + off + p;
  float4 x = use_init ? *reinterpret_cast<const float4*>(base + (size_t)nseg * F) : make_float4(0.f, 0.f, 0.f, 0.f);
  float* out = dst + (size_t)bh * nseg * len + p;
  for (int s = 0; s < nseg; ++s) {
    *reinterpret_cast<float4*>(out + (size_t)s * len) = x;
    const float4 u = *reinterpret_cast<const float4*>(base + (size_t)s * F);
    x.x = rho * x.x + u.x; x.y = rho * x.y + u.y; x.z = rho * x.z + u.z; x.w = rho * x.w + u.w;
  }
}

// The carry fix-up.  The walks run every segment with Phi0 = eta0 = 0, so
// their outputs miss q_t^T Phi_c and q_t . eta_c, where (Phi_c, eta_c) is the
// sum of the converted initial state and the brackets of the segments before
// this one (the Phi form of Eq. (semidirect)).
//
// k_carry: (Phi_c, eta_c) of every segment, as running sums over the records.
// Per segment, NC floats: Phi_c split into bf16 hi and lo in the B-fragment
// order of k_fix (piece p = (ct * D/16 + s) * 64 + lane holds the 8 values
// Phi_c[16s + 8(lane/32) + j][32ct + lane%32], j = 0..7: D*DV/8 pieces of
// 16 bytes, all hi pieces then all lo pieces), then eta_c in fp32 [D].
// grid (ceil((D*DV/8 + D) / 256), BH); reads and writes coalesced.
// rho2: attenuation of a carry over one segment (gamma^(2L) with decay, else 1):
// carry_{s+1} = rho2 carry_s + bracket_s.
template <int D, int DV>
__global__ __launch_bounds__(256) void k_carry(const float* __restrict__ rec, const float* __restrict__ init,
                                               float* __restrict__ carry, int nseg, float rho2) {
  constexpr int NC = D * DV + D, NP = D * DV / 8, KD = D / 16;
  const int bh = blockIdx.y, p = blockIdx.x * 256 + threadIdx.x;
  if (p >= NP + D) return;
  const size_t F = state_floats(D, DV);
  const float* base = rec + (size_t)bh * (nseg + 1) * F;
  if (p >= NP) {                     // eta_c[a]
    const int a = p - NP;
    const float* src = base + off_h(D, DV) + a;
    float x = init ? src[(size_t)nseg * F] : 0.f;
    for (int sp = 0; sp < nseg; ++sp) {
      carry[((size_t)bh * nseg + sp) * NC + D * DV + a] = x;
      x = rho2 * x + src[(size_t)sp * F];
    }
    return;
  }
  const int ct = p / (KD * 64), s = (p / 64) % KD, lane = p % 64;
  const float* src = base + off_G(D, DV) + (size_t)(16 * s + 8 * (lane >> 5)) * DV + 32 * ct + (lane & 31);
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = init ? src[(size_t)nseg * F + j * DV] : 0.f;
  for (int sp = 0; sp < nseg; ++sp) {
    uint16_t h8[8], o8[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) split(x[j], h8[j], o8[j]);
    uint4* dst = reinterpret_cast<uint4*>(carry + ((size_t)bh * nseg + sp) * NC);
    dst[p] = make_uint4(pack2(h8[0], h8[1]), pack2(h8[2], h8[3]), pack2(h8[4], h8[5]), pack2(h8[6], h8[7]));
    dst[NP + p] = make_uint4(pack2(o8[0], o8[1]), pack2(o8[2], o8[3]), pack2(o8[4], o8[5]), pack2(o8[6], o8[7]));
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = rho2 * x[j] + src[(size_t)sp * F + j * DV];
  }
}

// k_fix: one workgroup per (tpw consecutive tiles, head), one wave per (row
// tile, value column tile): out_t += q_t^T Phi_c on MFMA, then out_t /= den_t
// + eps when normalised, with den_t = (row sum of the walk) + q_t . (eta0 of
// the tile + eta_c).  A wave keeps the B fragments of its column of Phi_c
// (split hi/lo) in registers, reloaded when a tile starts a new segment; q is
// exact in bf16 and goes through LDS, the next tile's q and this tile's
// earlier outputs in flight during the products.  Tiles of segment 0 have
// nothing to add unless there is an initial state or a division.
template <int C, int D, int DV>
struct FixCfg {
  static constexpr int VT = DV / 32, RT = C / 32, NT = 64 * VT * RT, KD = D / 16, ldQ = D + kPad;
  static constexpr int QE = C * D / 8, QV = (QE + NT - 1) / NT;       // 16-byte pieces of a q tile
  static constexpr size_t lds = 2 * (size_t)C * ldQ + 4 * ((size_t)D + C);
  static_assert(NT >= D && NT <= 1024, "fix workgroup");
};

// DEC (decay gamma = 2^lg2g): the carry of a segment reaches token t aged by
// gamma^(2(p+1)), p = t - (first token of the segment); the tile's eta0 by
// gamma^(2(a+1)), a = t - (first token of the tile).
template <int C, int D, int DV, bool DEC = false>
__global__ __launch_bounds__((FixCfg<C, D, DV>::NT)) void k_fix(
    const uint16_t* __restrict__ q, float* __restrict__ out, const float* __restrict__ den_in,
    const float* __restrict__ carry, float* __restrict__ den_out, int has_init, int n, int cps, int nseg,
    int normalized, float eps, int tpw, float lg2g) {
  using F = FixCfg<C, D, DV>;
  constexpr int NT = F::NT, KD = F::KD, ldQ = F::ldQ, QE = F::QE, QV = F::QV, NC = D * DV + D;
  extern __shared__ __align__(16) uint16_t lds[];      // q tile | fp32 eta | 1/den
  uint16_t* Qs = lds;
  float* es = reinterpret_cast<float*>(Qs + C * ldQ);
  float* inv = es + D;
  // d <= 64: a head's tile groups on one XCD, where they share the reads of
  // their segments' carries (at d = 128 the spread placement measured faster)
  int grp = blockIdx.x, bh = blockIdx.y;
  if constexpr (D <= 64) seg_head(grp, bh);
  const int tid = threadIdx.x, l = tid & 63, lr = l & 31, lg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), ct = w % F::VT, rt = w / F::VT;
  const int M = (n + C - 1) / C;
  int c0 = grp * tpw;
  const int c1 = min(M, c0 + tpw);
  if (!has_init && !normalized) c0 = max(c0, cps);
  if (c0 >= c1) return;
  const rsrc_t rq = make_rsrc(q + (size_t)bh * n * D, (uint32_t)n * D * 2);
  const rsrc_t ro = make_rsrc(out + (size_t)bh * n * DV, (uint32_t)n * DV * 4);
  uint4 qp[QV];
  auto load_q = [&](int c) {          // clamped piece index: every lane loads, only owners store
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int e = min(tid + NT * i, QE - 1), t = e / (D / 8), a8 = (e % (D / 8)) * 8;
      qp[i] = buf_load16(rq, (((uint32_t)c * C + t) * D + a8) * 2);
    }
  };
  load_q(c0);
  bf16x8 bhi[KD], blo[KD];
  int loaded = -1;
  for (int c = c0; c < c1; ++c) {
    const int seg = c / cps;
    const float* cb = carry + ((size_t)bh * nseg + seg) * NC;
    if (seg != loaded) {              // uniform: B fragments of Phi_c, column ct * 32 + lr
      const uint4* pc = reinterpret_cast<const uint4*>(cb) + ct * KD * 64 + l;
#pragma unroll
      for (int s = 0; s < KD; ++s) {
        bhi[s] = __builtin_bit_cast(bf16x8, pc[s * 64]);
        blo[s] = __builtin_bit_cast(bf16x8, pc[D * DV / 8 + s * 64]);
      }
      loaded = seg;
    }
    const uint32_t t0 = (uint32_t)c * C;
    lds_barrier();                  // the previous tile's readers of Qs are done
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int e = tid + NT * i;
      if (e < QE) *reinterpret_cast<uint4*>(Qs + (e / (D / 8)) * ldQ + (e % (D / 8)) * 8) = qp[i];
    }
    if (normalized && tid < D) {      // eta at the tile start: the walk's eta0 + eta_c
      const float ec = DEC ? cb[D * DV + tid] * exp2f(2.f * lg2g * (float)(C * (c - seg * cps))) : cb[D * DV + tid];
      es[tid] = ec + den_in[(size_t)gridDim.y * n + ((size_t)bh * M + c) * D + tid];
    }
    lds_barrier();
    // rows past n fall outside the buffer: loads read 0, stores drop
    const uint32_t ob = ((t0 + rt * 32 + 4 * lg) * DV + ct * 32 + lr) * 4;
    float prev[16];
#pragma unroll
    for (int e = 0; e < 16; ++e)
      prev[e] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(ro, (int)(ob + (8 * (e >> 2) + (e & 3)) * DV * 4), 0, 0));
    load_q(c + 1 < c1 ? c + 1 : c);
    if (normalized) {                 // den_t = rowsum_t + q_t . es, TPR lanes per row
      constexpr int TPR = NT / C < D / 8 ? NT / C : D / 8, PER = D / TPR;
      static_assert(PER % 8 == 0 && TPR * C <= NT, "den lanes");
      const int t = tid / TPR, p0 = (tid % TPR) * PER;
      const uint16_t* row = Qs + (t < C ? t : C - 1) * ldQ + p0;
      float sd = 0.f;
#pragma unroll
      for (int a = 0; a < PER; a += 8) {
        const uint4 x = *reinterpret_cast<const uint4*>(row + a);
        const uint32_t u[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sd += __uint_as_float(u[j] << 16) * es[p0 + a + 2 * j];
          sd += __uint_as_float(u[j] & 0xffff0000u) * es[p0 + a + 2 * j + 1];
        }
      }
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) sd += __shfl_xor(sd, o);
      if (DEC) sd *= exp2f(2.f * lg2g * (float)(t + 1));
      if (tid % TPR == 0 && t < C) {
        const bool in = t0 + t < (uint32_t)n;
        const float den = in ? den_in[(size_t)bh * n + t0 + t] + sd : 0.f;
        inv[t] = in ? 1.f / (den + eps) : 0.f;
        if (den_out && in) den_out[(size_t)bh * n + t0 + t] = den;
      }
      lds_barrier();
    }
    f32x16 acc = zero16();
#pragma unroll
    for (int s = 0; s < KD; ++s) {
      const bf16x8 aQ = frag(Qs, ldQ, rt * 32, s * 16);
      acc = mfma(aQ, bhi[s], acc);
      acc = mfma(aQ, blo[s], acc);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float y = DEC ? prev[e] + acc[e] * exp2f(2.f * lg2g * (float)(C * (c - seg * cps) + rt * 32 + acc_row(e, lg) + 1))
                    : prev[e] + acc[e];
      if (normalized) y *= inv[rt * 32 + acc_row(e, lg)];
      buf_store4(ro, ob + (8 * (e >> 2) + (e & 3)) * DV * 4, y);
    }
  }
}

// Tiles per k_fix workgroup: about 2048 workgroups over all heads, 1 to 16 tiles each.
inline int fix_tpw(int M, int BH) {
  const long t = (long)M * BH / 2048;
  return t < 1 ? 1 : (t > 16 ? 16 : (int)t);
}

}  // namespace
}  // namespace hla
