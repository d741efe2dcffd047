// Exclusive scan of second-order segment states under the masked semidirect
// product, Eq. (semidirect):
//   (S_A+S_B, C_A+C_B, m_A+m_B, G_A+G_B+S_B C_A, h_A+h_B+S_B m_A).
// For each head the input is a sequence of M segment states (chunk or segment
// summaries, record layout S|C|m|G|h); the output holds, for every segment,
// E (+) init (+) x_0 (+) ... (+) x_{c-1} (Rem. scan-modes), and optionally the
// inclusive total.  With decay the concatenation of the decay-aware monoid is
// used (rho = gamma^length of the later segment, read with rho^2 on G and h):
//   (rho S_A + S_B, rho C_A + C_B, rho m_A + m_B, rho^2 G_A + G_B + rho S_B C_A,
//    rho^2 h_A + h_B + rho S_B m_A);
// every segment has attenuation rho except the last (rho_last).
//
// The only cross-segment product is S_c C_acc, where C_acc is an additive
// prefix, so the work splits over column blocks of C and G.  One workgroup
// owns (head, column block) and streams the head's segments in order; the
// blocks also share out the rows of S and h, and block 0 carries m.  The
// column blocks of one head are placed on the same XCD so the segment's S
// tile, read by each of them, is served from that XCD's L2.  Waves share
// only LDS, so the barriers order LDS alone: the next segment's loads and
// this segment's prefix stores stay in flight across them.
#include <type_traits>

#include "common.h"
#include "profile.h"

namespace hla {

// Columns of C and G per workgroup.  Narrow blocks give more workgroups per
// head (more loads in flight) but every block re-reads S_c (from L2 after the
// first) and moves C/G in short row pieces; measured best: 4 columns at
// d = 64, 16 at d = 128.
constexpr int scan_cols(int d) { return d == 16 ? 16 : d == 32 ? 8 : d == 64 ? 4 : 16; }

// Scan geometry for key dimension d: the product S_c C_acc of a workgroup
// (d x d times d x CB) gives each of the 256 threads one row a and NB
// adjacent columns; S_c and C_acc are double-buffered in LDS when both
// copies fit, so a step needs one barrier.
template <int d>
struct ScanCfg {
  static constexpr int CB = scan_cols(d), NB = d * CB / 256, TPR = CB / NB;
  static constexpr int ldS = d + 4;
  static constexpr int NBUF = 2 * d * ldS * 4 <= 80 * 1024 ? 2 : 1;
  static constexpr int nS4 = d * d / 4 / 256 > 0 ? d * d / 4 / 256 : 1;   // float4 of S_c per thread
  static constexpr int nC4 = (d * CB / 4 + 255) / 256;                    // float4 of a C or G block
  static constexpr int PF = d <= 64 ? 2 : 1;                              // segments loaded ahead
  static constexpr size_t lds_floats = (size_t)NBUF * (d * ldS + d * CB) + d;
  static_assert(NB >= 1 && CB % NB == 0 && 256 / TPR == d && CB % 4 == 0 && PF <= 4, "one row per thread group");
};

// One workgroup per (head, CB columns of C/G); NBLK = dv / CB blocks per
// head.  Block blk also owns rows [r0, r1) of S and h (S_acc and h_acc of
// those rows), and block 0 owns m.
template <int d, int NBLK>
__global__ __launch_bounds__(256) void k_scan(const float* __restrict__ states, const float* __restrict__ init,
                                              float* __restrict__ prefix, float* __restrict__ total,
                                              int BH, int M, int dv, int nblk, size_t in_stride,
                                              size_t pre_stride, size_t tot_stride, float rho_full,
                                              float rho_last) {
  using K = ScanCfg<d>;
  constexpr int CB = K::CB, NB = K::NB, ldS = K::ldS, nC4 = K::nC4;
  extern __shared__ float smem[];
  float* Sbuf = smem;                              // [NBUF][d][ldS]   S_c
  float* Cbuf = Sbuf + K::NBUF * d * ldS;          // [NBUF][d][CB]    C_acc before segment c
  float* macc = Cbuf + K::NBUF * d * CB;           // [d]
  const int tid = threadIdx.x;
  const int L = blockIdx.x;
  const int group = L / (8 * NBLK), within = L % (8 * NBLK);
  const int bh = group * 8 + within % 8;          // one head's blocks share an XCD (and its L2)
  const int blk = within / 8;
  if (bh >= BH) return;
  const int c0 = blk * CB;
  constexpr int rows = (d + NBLK - 1) / NBLK;
  const int r0 = min(d, blk * rows), r1 = min(d, r0 + rows);
  const size_t F = state_floats(d, dv);
  const size_t oC = off_C(d, dv), om = off_m(d, dv), oG = off_G(d, dv), oh = off_h(d, dv);
  const float* in = states + (size_t)bh * in_stride;
  float* pre = prefix + (size_t)bh * pre_stride;
  const float* ini = init ? init + (size_t)bh * F : nullptr;
  const int a = tid / K::TPR, j0 = (tid % K::TPR) * NB;     // product: row a, columns c0 + j0 ..
  const int nown = (r1 - r0) * d;                            // S elements owned by this block
  // float4 e of a C or G block: row e / (CB/4), columns c0 + 4 (e % (CB/4)) ..
  auto blk_off = [&](int e) { return (size_t)(e / (CB / 4)) * dv + c0 + 4 * (e % (CB / 4)); };
  auto ld4 = [](const float* p) { return *reinterpret_cast<const float4*>(p); };
  auto st4 = [](float* p, const float4& v) { *reinterpret_cast<float4*>(p) = v; };

  // carried state: S_acc (own rows; element e = tid + 256 i), G_acc row a, h_acc (own rows)
  constexpr int nSO = (rows * d + 255) / 256;
  float sacc[nSO], gacc[NB], hacc = 0.f;
#pragma unroll
  for (int i = 0; i < nSO; ++i) {
    const int e = tid + 256 * i;
    sacc[i] = (ini && e < nown) ? ini[(size_t)r0 * d + e] : 0.f;
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) gacc[j] = ini ? ini[oG + (size_t)a * dv + c0 + j0 + j] : 0.f;
  if (tid < r1 - r0 && ini) hacc = ini[oh + r0 + tid];
  for (int e = tid; e < d * CB; e += 256) Cbuf[e] = ini ? ini[oC + (size_t)(e / CB) * dv + c0 + e % CB] : 0.f;
  if (tid < d) macc[tid] = ini ? ini[om + tid] : 0.f;

  // registers holding segments c .. c + PF - 1 (slot c % PF), loaded PF steps ahead
  constexpr int PF = K::PF;
  float4 sv[PF][K::nS4], cv[PF][nC4];
  float gv[PF][NB], mv[PF], hv[PF];
  auto load = [&](int c, auto slot_tag) {
    constexpr int sl = decltype(slot_tag)::value;
    const float* x = in + (size_t)min(c, M - 1) * F;
    // every lane loads (indices clamped into the record) so no load sits under
    // a branch and the wait counts stay exact across steps; out-of-range
    // lanes are masked where the values are used
#pragma unroll
    for (int r = 0; r < K::nS4; ++r) sv[sl][r] = ld4(x + 4 * min(tid + 256 * r, d * d / 4 - 1));
#pragma unroll
    for (int r = 0; r < nC4; ++r) cv[sl][r] = ld4(x + oC + blk_off(min(tid + 256 * r, d * CB / 4 - 1)));
    if constexpr (NB % 4 == 0) {
#pragma unroll
      for (int j = 0; j < NB; j += 4) {
        const float4 g = ld4(x + oG + (size_t)a * dv + c0 + j0 + j);
        gv[sl][j] = g.x; gv[sl][j + 1] = g.y; gv[sl][j + 2] = g.z; gv[sl][j + 3] = g.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < NB; ++j) gv[sl][j] = x[oG + (size_t)a * dv + c0 + j0 + j];
    }
    mv[sl] = x[om + min(tid, d - 1)];
    hv[sl] = x[oh + r0 + min(tid, rows - 1)];
  };
  if (M > 0) load(0, std::integral_constant<int, 0>());
  if constexpr (PF > 1)
    if (M > 1) load(1, std::integral_constant<int, 1>());
  lds_barrier();

  // one step: write the prefix of segment c, then consume slot sl and refill it with segment c + PF
  auto step = [&](int c, auto slot_tag) -> bool {
    constexpr int sl = decltype(slot_tag)::value;
    const int p = K::NBUF == 2 ? (c & 1) : 0;   // LDS buffer (c parity)
    float* Sc = Sbuf + p * d * ldS;
    float* Cacc = Cbuf + p * d * CB;        // C before segment c
    float* Cnext = Cbuf + (K::NBUF == 2 ? (1 - p) : 0) * d * CB;
    float* dst = (c < M) ? pre + (size_t)c * F : (total ? total + (size_t)bh * tot_stride : nullptr);
    // the exclusive prefix of segment c (or the total after the last)
    if (dst) {
#pragma unroll
      for (int i = 0; i < nSO; ++i) {
        const int e = tid + 256 * i;
        if (e < nown) dst[(size_t)r0 * d + e] = sacc[i];
      }
#pragma unroll
      for (int r = 0; r < nC4; ++r) {
        const int e = tid + 256 * r;
        if (e < d * CB / 4) st4(dst + oC + blk_off(e), ld4(Cacc + 4 * e));
      }
      if constexpr (NB % 4 == 0) {
#pragma unroll
        for (int j = 0; j < NB; j += 4)
          st4(dst + oG + (size_t)a * dv + c0 + j0 + j, make_float4(gacc[j], gacc[j + 1], gacc[j + 2], gacc[j + 3]));
      } else {
#pragma unroll
        for (int j = 0; j < NB; ++j) dst[oG + (size_t)a * dv + c0 + j0 + j] = gacc[j];
      }
      if (blk == 0 && tid < d) dst[om + tid] = macc[tid];
      if (tid < r1 - r0) dst[oh + r0 + tid] = hacc;
    }
    if (c == M) return false;
    const float rho = c == M - 1 ? rho_last : rho_full, rho2 = rho * rho;
    // stage segment c: S_c, and rho C_acc + C_c for the next step
#pragma unroll
    for (int r = 0; r < K::nS4; ++r) {
      const int e4 = tid + 256 * r;
      if (e4 * 4 < d * d) {
        const int row = (4 * e4) / d, col = (4 * e4) % d;
        st4(&Sc[row * ldS + col], sv[sl][r]);
      }
    }
    float4 cn[nC4];
#pragma unroll
    for (int r = 0; r < nC4; ++r) {
      const int e = tid + 256 * r;
      if (e < d * CB / 4) {
        const float4 o = ld4(Cacc + 4 * e);
        cn[r] = make_float4(rho * o.x + cv[sl][r].x, rho * o.y + cv[sl][r].y, rho * o.z + cv[sl][r].z,
                            rho * o.w + cv[sl][r].w);
        if (K::NBUF == 2) st4(Cnext + 4 * e, cn[r]);
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) gacc[j] = rho2 * gacc[j] + gv[sl][j];
    const float m_c = mv[sl];
    if (tid < r1 - r0) hacc = rho2 * hacc + hv[sl];
    lds_barrier();
    if (c + PF < M) load(c + PF, slot_tag);
    // G_acc += S_c C_acc (segment A = accumulated prefix, B = segment c)
    {
      float acc[NB];
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[j] = 0.f;
      const float* srow = Sc + a * ldS;
#pragma unroll 4
      for (int ap = 0; ap < d; ap += 4) {
        const float4 s4 = ld4(srow + ap);
        const float sv4[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float* crow = Cacc + (ap + u) * CB + j0;
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[j] += sv4[u] * crow[j];
        }
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) gacc[j] += rho * acc[j];
    }
    // h_acc += S_c m_acc and S_acc += S_c on the owned rows
    if (tid < r1 - r0) {
      const float* srow = Sc + (r0 + tid) * ldS;
      float e = 0.f;
#pragma unroll 8
      for (int ap = 0; ap < d; ++ap) e += srow[ap] * macc[ap];
      hacc += rho * e;
    }
#pragma unroll
    for (int i = 0; i < nSO; ++i) {
      const int e = tid + 256 * i;
      if (e < nown) sacc[i] = rho * sacc[i] + Sc[(r0 + e / d) * ldS + e % d];
    }
    if (K::NBUF == 1) {
      lds_barrier();   // everyone is done with Sc and Cacc
#pragma unroll
      for (int r = 0; r < nC4; ++r) {
        const int e = tid + 256 * r;
        if (e < d * CB / 4) st4(Cacc + 4 * e, cn[r]);
      }
    }
    lds_barrier();   // macc readers are done; NBUF == 2: the other buffers are free
    if (tid < d) macc[tid] = rho * macc[tid] + m_c;
    return true;
  };
  for (int c = 0;; c += PF) {
    if (!step(c, std::integral_constant<int, 0>())) break;
    if constexpr (PF > 1)
      if (!step(c + 1, std::integral_constant<int, 1>())) break;
  }
}

// ---------------------------------------------------------------------------
// Row-block scan for d == dv.  One workgroup per (head, block of RPB rows),
// one wave per 16-column tile.  The product of a block is computed transposed,
// G_acc[rows]^T += C_acc^T S_c[rows]^T, on fp32 MFMA
// (v_mfma_f32_16x16x4_f32: lane l = 16g + n supplies A[n][k_g] and B[k_g][n]
// and holds D[4g + i][n], i < 4): A is wave w's column tile of C_acc, B the
// block's S_c rows, so a lane holds G_acc[row n][4 adjacent columns].  The
// contraction index of step s for lane group g is k = (d/4) g + s.  At
// d = 128 the same product runs on bf16 MFMA (v_mfma_f32_16x16x32_bf16, the
// same output layout; lane group g supplies 8 consecutive k of its range)
// over exact three-piece splits of both operands.
//   * every workgroup keeps all of C_acc, as A fragments in registers (wave
//     w: columns 16w .. 16w+15), and its own RPB rows of C_acc and S_acc in
//     row-major 16-byte pieces; C_c is read by each row block of the head,
//     and the blocks of one head share an XCD so the re-reads hit its L2;
//   * G_acc (the block's rows, wave w's columns) stays in the accumulator
//     layout and is staged through LDS for the prefix stores, so that every
//     store of the block's rows (S, C, G) is a contiguous row-major piece
//     (the accumulator layout would write 64-byte halves of 128-byte lines);
//   * wave t forms h_acc of row tile t (rows 16t .. 16t+15 of the block)
//     from m_acc, which sits in LDS, double-buffered by segment parity;
//   * the block's S_c rows and all of C_c go through LDS in 16-byte pieces
//     (C with its 16-column tiles XOR-swizzled by row group, so the column
//     reads of the four lane groups fall in different banks);
//   * loads run ahead in register slots, one slot per segment ahead, each
//     slot refilled as soon as its segment is consumed: the block's own rows
//     (S_c, G_c, h_c) and m_c PF segments ahead, C_c PFC ahead.  No load or
//     store of the steady-state loop sits under a branch (lanes that own
//     nothing store past the end of the record, which the buffer drops), so
//     the compiler's wait counts stay partial and the prefetch stays deep.
// Each block writes its rows of S, C, G, h, and block 0 writes m.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;

// Exact three-piece bf16 split of fp32 values: hi keeps the top 8 significand
// bits (truncation), mid the next 8 bits of the remainder, lo the rest, which
// then spans at most 8 bit positions; so x = hi + mid + lo exactly for every
// normal x whose pieces stay normal.  Products of two such splits keep the six
// cross terms down to 2^-24 relative (the three dropped terms are below it),
// the rounding level of an fp32 product.  Pieces are returned packed, two
// bf16 per word, in the order of the inputs.
__device__ __forceinline__ uint32_t bf16_hi_pair(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }
__device__ __forceinline__ void split3_pair(float x0, float x1, uint32_t& h, uint32_t& m, uint32_t& l) {
  const uint32_t u0 = __float_as_uint(x0), u1 = __float_as_uint(x1);
  const float r0 = x0 - __uint_as_float(u0 & 0xffff0000u), r1 = x1 - __uint_as_float(u1 & 0xffff0000u);
  const uint32_t v0 = __float_as_uint(r0), v1 = __float_as_uint(r1);
  const float s0 = r0 - __uint_as_float(v0 & 0xffff0000u), s1 = r1 - __uint_as_float(v1 & 0xffff0000u);
  h = bf16_hi_pair(u0, u1);
  m = bf16_hi_pair(v0, v1);
  l = bf16_hi_pair(__float_as_uint(s0), __float_as_uint(s1));
}

// Buffer resource over one record; loads and stores then take a 32-bit lane
// offset plus a uniform offset, which keeps per-load addresses out of VGPRs.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rec_rsrc(const float* p, uint32_t floats) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, (int)(floats * 4), 0x00020000);
}
__device__ __forceinline__ float rld(__amdgpu_buffer_rsrc_t r, uint32_t vf, uint32_t sf) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)(vf * 4), (int)(sf * 4), 0));
}
__device__ __forceinline__ f32x4_t rld4(__amdgpu_buffer_rsrc_t r, uint32_t vf, uint32_t sf) {
  return __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, (int)(vf * 4), (int)(sf * 4), 0));
}
__device__ __forceinline__ void rst(__amdgpu_buffer_rsrc_t r, uint32_t vf, uint32_t sf, float x) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), r, (int)(vf * 4), (int)(sf * 4), 2);
}
// The 16-byte store takes its uniform offset in the lane offset, with a zero
// soffset: with an SGPR soffset the compiler may place a VALU write of the
// store's data registers right after the store, and on gfx950 such a write
// was seen to reach memory in place of the data.
__device__ __forceinline__ void rst4(__amdgpu_buffer_rsrc_t r, uint32_t vf, uint32_t sf, f32x4_t x) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) uint32_t, x), r,
                                         (int)((vf + sf) * 4), 0, 2);
}

template <int d>
struct RbCfg {
  static constexpr int RPB = d == 128 ? 32 : 16;       // rows per workgroup
  // 16-column tiles per wave (two, at four waves of up to 512 registers,
  // measured slower at d = 128 than one at eight waves)
  static constexpr int CT = 1;
  static constexpr int NW = d / 16 / CT, NT = 64 * NW, RT = RPB / 16, KS = d / 4, RB = d / RPB;
  static constexpr int ldS = d + 4;
  static constexpr int NSP = RPB * d / 4 / NT;         // 16-byte pieces of the block's S rows per thread
  static constexpr int NC4 = d * d / 4 / NT;           // 16-byte pieces of C_c per thread
  static constexpr int NCO = RPB * d / 4 / NT;         // 16-byte pieces of the block's C rows per thread
  static constexpr int NM = (d + 63) / 64;             // m values per lane
  static constexpr int CBUF = d == 128 ? 1 : 2;        // C_c buffers in LDS
  // segments loaded ahead, one register slot each (a slot is refilled as
  // soon as its segment's data is consumed): the block's S, G, h rows and m
  // (read by this workgroup only) PF ahead; C_c (read by each row block of
  // the head, the later ones from L2) PFC ahead
  static constexpr int PF = d == 128 ? 2 : 4;
  static constexpr int PFC = d == 128 ? 1 : 4;
  static constexpr int GRP = PF == PFC ? PF : PF * PFC;   // steps per unrolled group
  // LDS: the block's S_c rows and the G_acc rows staged for row-major
  // prefix stores (two each, by segment parity), C_c (CBUF) and m_acc (two)
  static constexpr size_t lds_floats = 4 * (size_t)RPB * ldS + (size_t)CBUF * d * d + 2 * d;
  // d = 128: the product runs on bf16 MFMA (16x16x32) over exact three-piece
  // splits of both operands (six cross products), 2.7x the fp32 MFMA rate.
  // The block's S_c rows are split once, when staged, into three bf16 planes
  // (one per piece; by segment parity where C_c is double-buffered, else one
  // set, which the step's first barrier protects); each wave splits its own
  // column tile of C_acc.
  static constexpr bool SPL = d == 128;
  static constexpr int ldB = d + 8;                    // plane row stride (bf16): 16-byte reads of rows n, n+1 in different banks
  static constexpr int NPB = CBUF == 1 ? 1 : 2;
  static constexpr size_t plane = (size_t)RPB * ldB;   // bf16 per plane
  static constexpr size_t lds_bytes = lds_floats * 4 + (SPL ? (size_t)NPB * 3 * plane * 2 : 0);
  static_assert(lds_floats % 4 == 0 && ldB % 8 == 0 && lds_bytes <= 160 * 1024, "LDS layout");
  static_assert(GRP <= 4 && PF <= 4 && PFC <= 4 && GRP % PF == 0 && GRP % PFC == 0, "unrolled slots");
  static_assert(NSP * NT * 4 == RPB * d && KS % 4 == 0 && NC4 * NT * 4 == d * d && NCO * NT * 4 == RPB * d &&
                    NW * CT * 16 == d && NW >= RT,
                "row-block geometry");
};

// Column of C_c element (k, j) in LDS: 16-column tiles XOR-swizzled by the row group k / (d/4).
template <int d>
__device__ __forceinline__ int cswz(int k, int j) {
  return j ^ ((((k / (d / 4)) % (d / 16))) << 4);
}

template <int d>
__global__ __launch_bounds__((RbCfg<d>::NT)) void k_scan_rb(const float* __restrict__ states, const float* __restrict__ init, float* __restrict__ prefix,
               float* __restrict__ total, int BH, int M, size_t in_stride, size_t pre_stride, size_t tot_stride,
               float rho_full, float rho_last) {
  using K = RbCfg<d>;
  constexpr int RT = K::RT, KS = K::KS, NT = K::NT, ldS = K::ldS, PF = K::PF, PFC = K::PFC, GRP = K::GRP, NM = K::NM, NC4 = K::NC4, NCO = K::NCO, NSP = K::NSP, CT = K::CT;
  using std::integral_constant;
  constexpr size_t F = (size_t)d * d + 2 * (size_t)d * d + 2 * d;
  constexpr uint32_t oC = d * d, om = 2 * d * d, oG = 2 * d * d + d, oh = 3 * d * d + d;
  extern __shared__ float smem[];
  float* Sbuf = smem;                                  // [2][RPB][ldS]  the block's S_c rows
  float* Gst = Sbuf + 2 * K::RPB * ldS;                // [2][RPB][ldS]  G_acc rows for the prefix stores
  float* Cbuf = Gst + 2 * K::RPB * ldS;                // [CBUF][d][d]   C_c, swizzled
  float* macc = Cbuf + K::CBUF * d * d;                // [2][d]         m_acc by segment parity
  uint16_t* Bpl = reinterpret_cast<uint16_t*>(smem + K::lds_floats);   // [NPB][3][RPB][ldB] S_c row pieces
  const int tid = threadIdx.x, l = tid & 63, g = l >> 4, n = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int L = blockIdx.x, group = L / (8 * K::RB), within = L % (8 * K::RB);
  const int bh = group * 8 + within % 8;               // a head's row blocks share an XCD (and its L2)
  const int rb = within / 8;
  if (bh >= BH) return;
  const int r0 = rb * K::RPB, cw = 16 * CT * w;        // the wave's first column
  const float* in = states + (size_t)bh * in_stride;
  float* pre = prefix + (size_t)bh * pre_stride;

  // carried state: C_acc column pieces (A fragments; tile ct = columns cw + 16 ct ..), G_acc
  // [row 16t + n][cw + 16 ct + 4g + i], h_acc, and the block's rows of S_acc and C_acc row-major:
  // piece j of a thread is row r0 + e / d, columns e % d .. + 3, e = 4 (tid + NT j)
  float cacc[CT][KS], hacc[RT];
  f32x4_t gacc[CT][RT], sown[NCO], cown[NCO];
  if (init) {
    const auto x = rec_rsrc(init + (size_t)bh * F, (uint32_t)F);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int s = 0; s < KS; ++s) cacc[ct][s] = rld(x, KS * g * d + cw + 16 * ct + n, oC + s * d);
#pragma unroll
    for (int j = 0; j < NCO; ++j) {
      cown[j] = rld4(x, 4 * (tid + NT * j), oC + r0 * d);
      sown[j] = rld4(x, 4 * (tid + NT * j), r0 * d);
    }
#pragma unroll
    for (int t = 0; t < RT; ++t) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) gacc[ct][t] = rld4(x, (r0 + n) * d + cw + 16 * ct + 4 * g, oG + 16 * t * d);
      hacc[t] = rld(x, r0 + n, oh + 16 * t);
    }
    if (w == 0)
      for (int a = l; a < d; a += 64) macc[a] = rld(x, a, om);   // parity 0
  } else {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int s = 0; s < KS; ++s) cacc[ct][s] = 0.f;
#pragma unroll
    for (int j = 0; j < NCO; ++j) {
      cown[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      sown[j] = cown[j];
    }
#pragma unroll
    for (int t = 0; t < RT; ++t) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) gacc[ct][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      hacc[t] = 0.f;
    }
    if (w == 0)
      for (int a = l; a < d; a += 64) macc[a] = 0.f;
  }

  // segment data in register slots
  f32x4_t sp[PF][NSP], cp[PFC][NC4], gc[PF][CT][RT];
  float hc[PF][RT], mc[PF][NM];
  auto load_c = [&](int c, auto slot_tag) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_tag)::value;
    const auto x = rec_rsrc(in + (size_t)min(c, M - 1) * F, (uint32_t)F);
#pragma unroll
    for (int j = 0; j < NC4; ++j) cp[sl][j] = rld4(x, 4 * tid, oC + 4 * NT * j);
  };
  auto load_s = [&](int c, auto slot_tag) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_tag)::value;
    const auto x = rec_rsrc(in + (size_t)min(c, M - 1) * F, (uint32_t)F);
#pragma unroll
    for (int j = 0; j < NSP; ++j) {
      const int e = tid + NT * j, row = e / (d / 4), c4 = (e % (d / 4)) * 4;
      sp[sl][j] = rld4(x, (r0 + row) * d + c4, 0);
    }
  };
  auto load_g = [&](int c, auto slot_tag) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_tag)::value;
    const auto x = rec_rsrc(in + (size_t)min(c, M - 1) * F, (uint32_t)F);
#pragma unroll
    for (int t = 0; t < RT; ++t) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) gc[sl][ct][t] = rld4(x, (r0 + n) * d + cw + 16 * ct + 4 * g, oG + 16 * t * d);
      hc[sl][t] = rld(x, r0 + n, oh + 16 * t);
    }
#pragma unroll
    for (int j = 0; j < NM; ++j) mc[sl][j] = rld(x, min(l + 64 * j, d - 1), om);
  };
  // the exclusive prefix held now (m_acc in buffer mb), into record dst.  G_acc
  // goes through LDS (Gst, buffer par) so that every store of the block's
  // rows is a contiguous row-major piece; the caller has a barrier between
  // gst_write and put, and the two buffers alternate by segment parity, so a
  // buffer is rewritten only after a later barrier.
  constexpr uint32_t kDrop = 0x10000000u;   // a lane offset (floats) past any record: the store is dropped
  auto gst_write = [&](int par) __attribute__((always_inline)) {
    float* gs = Gst + par * K::RPB * ldS;
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
        *reinterpret_cast<f32x4_t*>(gs + (16 * t + n) * ldS + cw + 16 * ct + 4 * g) = gacc[ct][t];
  };
  auto put = [&](float* dst, const float* mb, int par) __attribute__((always_inline)) {
    const auto y = rec_rsrc(dst, (uint32_t)F);
    const float* gs = Gst + par * K::RPB * ldS;
#pragma unroll
    for (int j = 0; j < NCO; ++j) {
      const int e = 4 * (tid + NT * j);
      rst4(y, e, r0 * d, sown[j]);
      rst4(y, e, oC + r0 * d, cown[j]);
      rst4(y, e, oG + r0 * d, *reinterpret_cast<const f32x4_t*>(gs + (e / d) * ldS + e % d));
    }
    const bool mown = w == 0 && rb == 0;
#pragma unroll
    for (int t = 0; t < RT; ++t) rst(y, w == t && g == 0 ? r0 + n : kDrop, oh + 16 * t, hacc[t]);
#pragma unroll
    for (int j = 0; j < NM; ++j) {
      const int a = min(l + 64 * j, d - 1);
      rst(y, mown && l + 64 * j < d ? a : kDrop, om, mb[a]);
    }
  };
  // segment c from slots sl (rows, m) and slc (C_c): write its prefix, then fold it in
  auto step = [&](int c, auto slot_tag, auto cslot_tag) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_tag)::value, slc = decltype(cslot_tag)::value;
    float* Sc = Sbuf + (c & 1) * K::RPB * ldS;
    float* Cc = Cbuf + (K::CBUF == 2 ? (c & 1) : 0) * d * d;
    if (K::CBUF == 1) lds_barrier();   // the previous segment's readers of Cc are done
#pragma unroll
    for (int j = 0; j < NSP; ++j) {
      const int e = tid + NT * j, row = e / (d / 4), c4 = (e % (d / 4)) * 4;
      *reinterpret_cast<f32x4_t*>(Sc + row * ldS + c4) = sp[sl][j];
      if constexpr (K::SPL) {
        uint2 ph, pm, pl;
        split3_pair(sp[sl][j].x, sp[sl][j].y, ph.x, pm.x, pl.x);
        split3_pair(sp[sl][j].z, sp[sl][j].w, ph.y, pm.y, pl.y);
        uint16_t* pb = Bpl + (K::NPB == 2 ? (c & 1) : 0) * 3 * K::plane + row * K::ldB + c4;
        *reinterpret_cast<uint2*>(pb) = ph;
        *reinterpret_cast<uint2*>(pb + K::plane) = pm;
        *reinterpret_cast<uint2*>(pb + 2 * K::plane) = pl;
      }
    }
#pragma unroll
    for (int j = 0; j < NC4; ++j) {
      const int e = 4 * (tid + NT * j), k = e / d;
      *reinterpret_cast<f32x4_t*>(Cc + k * d + cswz<d>(k, e % d)) = cp[slc][j];
    }
    load_s(c + PF, slot_tag);     // the slots just emptied
    load_c(c + PFC, cslot_tag);
    const float* mo = macc + (c & 1) * d;   // m_acc before segment c
    gst_write(c & 1);
    lds_barrier();
    put(pre + (size_t)c * F, mo, c & 1);
    const float rho = c == M - 1 ? rho_last : rho_full, rho2 = rho * rho;
    // G_acc^T <- rho^2 G_acc^T + G_c^T + rho (C_acc^T S_c[rows]^T): the
    // product takes the old C_acc, and rho is applied to its result
    if constexpr (K::SPL) {
      // MFMA step s, lane group g, element j: contraction index KS g + 8 s + j
      const uint16_t* pb = Bpl + (K::NPB == 2 ? (c & 1) : 0) * 3 * K::plane + n * K::ldB + KS * g;
      f32x4_t acc[RT][CT];
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[t][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS / 8; ++s) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          uint4 ah, am, al;
          split3_pair(cacc[ct][8 * s + 0], cacc[ct][8 * s + 1], ah.x, am.x, al.x);
          split3_pair(cacc[ct][8 * s + 2], cacc[ct][8 * s + 3], ah.y, am.y, al.y);
          split3_pair(cacc[ct][8 * s + 4], cacc[ct][8 * s + 5], ah.z, am.z, al.z);
          split3_pair(cacc[ct][8 * s + 6], cacc[ct][8 * s + 7], ah.w, am.w, al.w);
          const bf16x8_t a1 = __builtin_bit_cast(bf16x8_t, ah), a2 = __builtin_bit_cast(bf16x8_t, am),
                         a3 = __builtin_bit_cast(bf16x8_t, al);
#pragma unroll
          for (int t = 0; t < RT; ++t) {
            const uint16_t* bp = pb + 16 * t * K::ldB + 8 * s;
            const bf16x8_t b1 = *reinterpret_cast<const bf16x8_t*>(bp);
            const bf16x8_t b2 = *reinterpret_cast<const bf16x8_t*>(bp + K::plane);
            const bf16x8_t b3 = *reinterpret_cast<const bf16x8_t*>(bp + 2 * K::plane);
            f32x4_t x = acc[t][ct];
            x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, b1, x, 0, 0, 0);
            x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b2, x, 0, 0, 0);
            x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b3, x, 0, 0, 0);
            x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, b1, x, 0, 0, 0);
            x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b2, x, 0, 0, 0);
            acc[t][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, x, 0, 0, 0);
          }
        }
      }
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) gacc[ct][t] = rho2 * gacc[ct][t] + gc[sl][ct][t] + rho * acc[t][ct];
    } else
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      f32x4_t acc[CT];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const float* brow = Sc + (16 * t + n) * ldS + KS * g;
#pragma unroll
      for (int s4 = 0; s4 < KS; s4 += 4) {
        const f32x4_t b4 = *reinterpret_cast<const f32x4_t*>(brow + s4);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(cacc[ct][s4], b4.x, acc[ct], 0, 0, 0);
          acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(cacc[ct][s4 + 1], b4.y, acc[ct], 0, 0, 0);
          acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(cacc[ct][s4 + 2], b4.z, acc[ct], 0, 0, 0);
          acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(cacc[ct][s4 + 3], b4.w, acc[ct], 0, 0, 0);
        }
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) gacc[ct][t] = rho2 * gacc[ct][t] + gc[sl][ct][t] + rho * acc[ct];
    }
    // h_acc += h_c + S_c[rows] m_acc (old m_acc) of row tile t in wave t
    // alone (the wave that stores it); m_acc += m_c into the other parity
    // buffer (its readers, segment c - 1, are past the barrier)
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      if (w != t) continue;
      const float* arow = Sc + (16 * t + n) * ldS + KS * g;
      float e = 0.f;
#pragma unroll
      for (int s4 = 0; s4 < KS; s4 += 4) {
        const f32x4_t a4 = *reinterpret_cast<const f32x4_t*>(arow + s4);
        const f32x4_t m4 = *reinterpret_cast<const f32x4_t*>(mo + KS * g + s4);
        e += a4.x * m4.x + a4.y * m4.y + a4.z * m4.z + a4.w * m4.w;
      }
      e += __shfl_xor(e, 16);
      e += __shfl_xor(e, 32);
      hacc[t] = rho2 * hacc[t] + hc[sl][t] + rho * e;
    }
    if (w == 0) {
      float* mn = macc + ((c + 1) & 1) * d;
#pragma unroll
      for (int j = 0; j < NM; ++j)
        if (l + 64 * j < d) mn[l + 64 * j] = rho * mo[l + 64 * j] + mc[sl][j];
    }
    load_g(c + PF, slot_tag);
    // S_acc <- rho S_acc + S_c, C_acc <- rho C_acc + C_c
#pragma unroll
    for (int j = 0; j < NCO; ++j) {
      const int e = 4 * (tid + NT * j);
      sown[j] = rho * sown[j] + *reinterpret_cast<const f32x4_t*>(Sc + (e / d) * ldS + e % d);
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const int k = KS * g + s;
        cacc[ct][s] = rho * cacc[ct][s] + Cc[k * d + cswz<d>(k, cw + 16 * ct + n)];
      }
#pragma unroll
    for (int j = 0; j < NCO; ++j) {
      const int e = 4 * (tid + NT * j), k = r0 + e / d;
      cown[j] = rho * cown[j] + *reinterpret_cast<const f32x4_t*>(Cc + k * d + cswz<d>(k, e % d));
    }
  };
  if (M > 0) {
#define HLA_RB_LOAD(J) load_s(J, integral_constant<int, J>()), load_g(J, integral_constant<int, J>())
    HLA_RB_LOAD(0);
    if constexpr (PF > 1) HLA_RB_LOAD(1);
    if constexpr (PF > 2) HLA_RB_LOAD(2);
    if constexpr (PF > 3) HLA_RB_LOAD(3);
#undef HLA_RB_LOAD
    load_c(0, integral_constant<int, 0>());
    if constexpr (PFC > 1) load_c(1, integral_constant<int, 1>());
    if constexpr (PFC > 2) load_c(2, integral_constant<int, 2>());
    if constexpr (PFC > 3) load_c(3, integral_constant<int, 3>());
#define HLA_RB_STEP(J) step(c + J, integral_constant<int, J % PF>(), integral_constant<int, J % PFC>())
    int c = 0;
    for (; c + GRP <= M; c += GRP) {     // whole groups: no branch around a step
      HLA_RB_STEP(0);
      if constexpr (GRP > 1) HLA_RB_STEP(1);
      if constexpr (GRP > 2) HLA_RB_STEP(2);
      if constexpr (GRP > 3) HLA_RB_STEP(3);
    }
    if (c < M) HLA_RB_STEP(0);
    if constexpr (GRP > 1) if (c + 1 < M) HLA_RB_STEP(1);
    if constexpr (GRP > 2) if (c + 2 < M) HLA_RB_STEP(2);
#undef HLA_RB_STEP
  }
  if (total) {
    gst_write(M & 1);                       // the last put read the other buffer
    lds_barrier();                          // and m_acc of parity M is written by wave 0
    put(total + (size_t)bh * tot_stride, macc + (M & 1) * d, M & 1);
  }
}

hipError_t launch_scan(const float* states, const float* init, float* prefix, float* total,
                       int BH, int M, int d, int dv, hipStream_t s, float rho, float rho_last) {
  const size_t F = state_floats(d, dv);
  return launch_scan_strided(states, init, prefix, total, BH, M, d, dv, (size_t)M * F, (size_t)M * F, F, s, rho,
                             rho_last);
}

hipError_t launch_scan_strided(const float* states, const float* init, float* prefix, float* total, int BH, int M,
                               int d, int dv, size_t in_stride, size_t pre_stride, size_t tot_stride,
                               hipStream_t s, float rho, float rho_last) {
  const int groups = (BH + 7) / 8;
  if (d == dv) {
    const void* kern = nullptr;
    size_t lds = 0;
    int nt = 0, rbn = 0;
#define HLA_SCAN_RB(D_)                                      \
  if (d == D_) {                                             \
    kern = (const void*)k_scan_rb<D_>;                       \
    lds = RbCfg<D_>::lds_bytes;                              \
    nt = RbCfg<D_>::NT;                                      \
    rbn = RbCfg<D_>::RB;                                     \
  }
    HLA_SCAN_RB(16) HLA_SCAN_RB(32) HLA_SCAN_RB(64) HLA_SCAN_RB(128)
#undef HLA_SCAN_RB
    if (!kern) return hipErrorInvalidValue;
    hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    void* args[] = {&states, &init, &prefix, &total, &BH, &M, &in_stride, &pre_stride, &tot_stride, &rho, &rho_last};
    e = prof_launch(kern, dim3(groups * 8 * rbn), dim3(nt), args, lds, s);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  const int cb = scan_cols(d);
  const int nblk = (dv + cb - 1) / cb;
  const void* kern = nullptr;
  size_t lds = 0;
#define HLA_SCAN_CASE(D_, B_)                                 \
  if (d == D_ && nblk == B_) {                                \
    kern = (const void*)k_scan<D_, B_>;                       \
    lds = ScanCfg<D_>::lds_floats * sizeof(float);            \
  }
  HLA_SCAN_CASE(16, 1) HLA_SCAN_CASE(16, 2) HLA_SCAN_CASE(16, 4) HLA_SCAN_CASE(16, 8)
  HLA_SCAN_CASE(32, 2) HLA_SCAN_CASE(32, 4) HLA_SCAN_CASE(32, 8) HLA_SCAN_CASE(32, 16)
  HLA_SCAN_CASE(64, 4) HLA_SCAN_CASE(64, 8) HLA_SCAN_CASE(64, 16) HLA_SCAN_CASE(64, 32)
  HLA_SCAN_CASE(128, 1) HLA_SCAN_CASE(128, 2) HLA_SCAN_CASE(128, 4) HLA_SCAN_CASE(128, 8)
#undef HLA_SCAN_CASE
  if (!kern) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  void* args[] = {&states,    &init,       &prefix,     &total, &BH,     &M,       &dv, const_cast<int*>(&nblk),
                  &in_stride, &pre_stride, &tot_stride, &rho,   &rho_last};
  e = prof_launch(kern, dim3(groups * 8 * nblk), dim3(256), args, lds, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace hla
