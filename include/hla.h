/*
 * hla.h — C ABI of the MI355X (gfx950) Higher-order Linear Attention library.
 *
 * The library computes the strictly causal (masked) second-order HLA of
 * "Higher-order Linear Attention" (arXiv 2510.27258):
 *
 *     o_t = q_t^T (S_t C_t - G_t)                               (Thm. 1)
 *         = sum_{j<=t} sum_{i<=j} (q_t.k_i)(q_j.k_i) v_j        (Sec. 3.1)
 *
 * with S_t = sum k k^T, C_t = sum q v^T, m_t = sum q and the masking summaries
 * G_t = sum_i k_i k_i^T C_{i-1}, h_t = sum_i k_i k_i^T m_{i-1} (Sec. 3 and
 * 3.1), its ratio-normalised form num/(den + eps) with den_t = q_t^T(S_t m_t -
 * h_t) (Thm. 1), and the unmasked operator q_t^T S_t C_t (Eq. hla-unnorm,
 * Eq. hla-row).  Sequences are processed by the chunk-parallel associative
 * scan of Sec. 4 (Eq. semidirect, Thm. 2, Rem. scan-modes); the decode step
 * applies the online updates of Sec. 3.1.
 *
 * Conventions for every call
 *   - Pointers to tensors are DEVICE pointers.  The caller owns all memory,
 *     including workspaces sized by the *_workspace_bytes queries.  The library
 *     never allocates device memory, never synchronises, and enqueues work
 *     only on `stream` (a hipStream_t; NULL = the default stream).  Results
 *     are available once that stream reaches the enqueued work.
 *   - Tensors are row-major and contiguous:
 *       q, k [B, H, n, d]   v [B, H, n, dv]   out [B, H, n, dv]
 *     q/k/v are `dtype` (HLA_FP32 or HLA_BF16: raw bfloat16 bit patterns);
 *     outputs and states are always fp32.  Base pointers must be 16-byte
 *     aligned.  Inputs are read-only; inputs and outputs must not alias.
 *   - A head's second-order state is one fp32 record of
 *     F = d*d + 2*d*dv + 2*d floats (hla2_state_floats), in the order
 *       S [d][d] | C [d][dv] | m [d] | G [d][dv] | h [d]
 *     i.e. (S^K, C^QV, m^Q, G, h) of Sec. 3.1.  A state array [B, H, F]
 *     stores the records of all heads back to back.  The all-zero record is
 *     the identity segment (Thm. 2).
 *   - Supported sizes: d, dv in {16, 32, 64, 128}; chunk in {16, 32, 64,
 *     128}; any n >= 1 (a short last chunk is exact) with
 *     n * max(d, dv) * 4 < 2^31 (one head's fp32 rows stay within 32-bit
 *     byte offsets: n < 4 194 304 at d = dv = 128), else HLA_ERR_UNSUPPORTED;
 *     B*H <= 65535.
 *     masked, normalized in {0, 1}; eps finite and >= 0 (added to the
 *     denominator as is, den + eps).  Decay is 1 (hla2_forward_decay takes
 *     a decay) and the ridge 0.
 *   - Every call returns an hla_status.  On failure nothing is enqueued and
 *     hla_last_error() describes the reason (a thread-local string).
 *     Results are deterministic: the same inputs give bit-identical outputs.
 *   - Size queries returning size_t (*_workspace_bytes, hla2_state_bytes)
 *     return 0 exactly when the arguments would be rejected, and then set
 *     hla_last_error(); every accepted argument list gives a size > 0.
 *     hla2_workspace_query returns the status itself.
 *   - The environment variable HLA_FUSED_SEGMENTS=<p>, when set, overrides
 *     how many segments per head the segment-walk plans (fused forward and
 *     its decayed form, AHLA, backward, third order) cut each head into, for
 *     testing and tuning; any p >= 1 gives the same result up to fp32
 *     rounding order.  Workspace queries read it too: set it before the
 *     query.  A call checks its workspace against its own plan.
 *   - At d = dv = 128 (chunk 64 or 128, bf16, masked, no states) the fused
 *     forward writes every output row once: a summary walk gives each
 *     segment's bracket, and one walk per segment starts from its true carry.
 *     HLA_FUSED_LEGACY=1 selects instead the walk whose outputs a second
 *     kernel corrects by the carry (the form prefill with states uses), for
 *     testing; both give the same result up to fp32 rounding order.
 */
#ifndef HLA_H
#define HLA_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HLA_OK = 0,
  HLA_ERR_INVALID = 1,      /* null pointer, bad size, flag or alignment */
  HLA_ERR_UNSUPPORTED = 2,  /* valid but not implemented (e.g. d = 96)  */
  HLA_ERR_WORKSPACE = 3,    /* workspace missing or too small           */
  HLA_ERR_HIP = 4           /* a HIP launch or runtime call failed      */
} hla_status;

typedef enum { HLA_FP32 = 0, HLA_BF16 = 1 } hla_dtype;

/* Forward algorithms selectable through hla2_forward_ex. */
typedef enum {
  HLA_ALGO_AUTO = 0,     /* library choice (fused when supported)             */
  HLA_ALGO_CHUNKED = 1,  /* per-chunk summaries, (+)-scan, per-chunk readout  */
  HLA_ALGO_FUSED = 2     /* segment walk with the carry state kept on chip    */
} hla_algo;

/* Reason for the last failed call on this thread ("" if none). */
const char *hla_last_error(void);

/* Floats in one second-order state record: d*d + 2*d*dv + 2*d. */
size_t hla2_state_floats(int d, int dv);

/* ---------------------------------------------------------------------------
 * hla2_forward — masked (or unmasked) second-order HLA over whole sequences.
 * Thm. 1 (output), Sec. 4 (chunk-parallel scan).  out[b,h,t,:] = o_t of head
 * (b,h); with normalized = 1, num_t / (den_t + eps).  `chunk` is the scan's
 * chunk size; results do not depend on it beyond rounding (Thm. 2).
 * workspace: at least hla2_workspace_bytes(...) bytes of device memory (its
 * contents on entry are ignored).  Returns HLA_ERR_WORKSPACE if smaller.
 * ------------------------------------------------------------------------- */
size_t hla2_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype);
int hla2_forward(const void *q, const void *k, const void *v, float *out,
                 int B, int H, int n, int d, int dv, int chunk, int masked, int normalized,
                 float eps, int dtype, void *workspace, size_t workspace_bytes, void *stream);

/* As hla2_forward with an explicit algorithm (hla_algo) and an optional
 * denominator output.  den: NULL, or (normalized = 1 only) fp32 [B, H, n]
 * receiving den_t of Thm. 1 (q_t^T (S_t m_t - h_t) masked, q_t^T S_t m_t
 * unmasked), without eps; den != NULL with normalized = 0 is HLA_ERR_INVALID.
 * HLA_ALGO_FUSED returns HLA_ERR_UNSUPPORTED for shapes it does not cover. */
size_t hla2_workspace_bytes_ex(int B, int H, int n, int d, int dv, int chunk, int dtype, int algo);
int hla2_forward_ex(const void *q, const void *k, const void *v, float *out, float *den,
                    int B, int H, int n, int d, int dv, int chunk, int masked, int normalized,
                    float eps, int dtype, void *workspace, size_t workspace_bytes, int algo,
                    void *stream);

/* Workspace size of hla2_forward_ex as a status: on HLA_OK *bytes holds the
 * size; otherwise *bytes is 0 and hla_last_error() says why.  bytes must not
 * be NULL (HLA_ERR_INVALID). */
int hla2_workspace_query(int B, int H, int n, int d, int dv, int chunk, int dtype, int algo, size_t *bytes);

/* The segment plan of the fused path for these arguments, as the forward
 * without initial or final state uses it: *segments gets the number of
 * segments each head is cut into (walked in parallel, composed by
 * Eq. semidirect), *tile the token tile the walk advances by, and, unless the
 * pointers are NULL, *first_tiles the tiles of segment 0 and
 * *tiles_per_segment those of every later segment (the last holds the rest).
 * Returns HLA_ERR_UNSUPPORTED when the fused path does not cover the shape
 * (bf16 inputs, masked).  Reads HLA_FUSED_SEGMENTS like the forward. */
int hla2_fused_plan(int B, int H, int n, int d, int dv, int chunk, int *segments, int *tile, int *first_tiles,
                    int *tiles_per_segment);

/* 1 if hla2_forward_ex would accept `algo` for these arguments, else 0.
 * HLA_ALGO_FUSED covers bf16 inputs, masked = 1, n * max(d, dv) * 4 < 2^31
 * and (tile, d, dv) in {(64,64,64), (32,32,32), (64,32,32), (32,64,64),
 * (64,64,32), (64,32,64), (64,128,128), (32,128,128)}, where the tile is the
 * chunk for chunk 32 and 64, and 64 for chunk 128 (the scan is exact for any
 * chunking, Thm. 2, so the tile changes only the rounding order). */
int hla2_algo_supported(int algo, int n, int d, int dv, int chunk, int dtype, int masked);

/* ---------------------------------------------------------------------------
 * hla2_forward_noalloc — hla2_forward for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, checks and results as hla2_forward
 * (algorithm HLA_ALGO_AUTO), without the workspace arguments: the workspace
 * is a fixed array of HLA_NOALLOC_SCRATCH_BYTES bytes in the library's own
 * device memory, one per GPU, held until the process ends.  Sizes whose
 * workspace (hla2_workspace_query of the algorithm HLA_ALGO_AUTO takes for
 * the call's masked flag) exceeds it return HLA_ERR_WORKSPACE before
 * anything is enqueued.  The call allocates nothing.  Every call on one GPU
 * shares that GPU's array (no call needs it cleared: the workspace's
 * contents on entry are ignored), so calls that overlap on one GPU (other
 * streams, other threads) race and must be ordered by the caller.
 * ------------------------------------------------------------------------- */
#define HLA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int hla2_forward_noalloc(const void *q, const void *k, const void *v, float *out,
                         int B, int H, int n, int d, int dv, int chunk, int masked, int normalized,
                         float eps, int dtype, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_chunk_summaries — the summary of every chunk of `chunk` tokens with a
 * zero carry-in: the (+)-product of its token segments (Sec. 4.2, Rem.
 * scan-modes: chunk summary).  states: [B, H, M, F], M = ceil(n / chunk);
 * chunk c covers tokens [c*chunk, min(n, (c+1)*chunk)).
 * ------------------------------------------------------------------------- */
int hla2_chunk_summaries(const void *q, const void *k, const void *v, float *states,
                         int B, int H, int n, int d, int dv, int chunk, int dtype, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_scan — exclusive scan under the masked semidirect product, Eq.
 * (semidirect): prefix[b,h,c] = init (+) states[b,h,0] (+) ... (+)
 * states[b,h,c-1] (Rem. scan-modes).  states, prefix: [B, H, M, F];
 * init: [B, H, F] or NULL (identity); total: [B, H, F] receives the inclusive
 * product of all M segments, or NULL.  prefix and total must not alias
 * states or init.
 * ------------------------------------------------------------------------- */
int hla2_scan(const float *states, const float *init, float *prefix, float *total,
              int B, int H, int M, int d, int dv, void *stream);

/* ---------------------------------------------------------------------------
 * Decode state (Sec. 3.1 online updates; Thm. 2 identity).  A descriptor
 * fixes, for the life of the state, the operator every prefill and step on
 * it applies (masked, normalized, eps) and the dtype of the tokens they take,
 * so a prefill and the steps after it cannot disagree.  The state itself is
 * caller-owned device memory holding one record of FP floats per head: the
 * fields of the record above with S packed symmetric (Sec. 5: only its upper
 * triangle is stored), FP = d(d+1)/2 + 2*d*dv + 2*d:
 *   S [d(d+1)/2] | C [d][dv] | m [d] | G [d][dv] | h [d].
 * S is stored as d/2 folded row pairs of d+1 floats: pair p holds row p of S
 * from column p (d-p values), then row d-1-p from column d-1-p (p+1 values);
 * element (a, j), a <= j, is at p*(d+1) + c with p = a, c = j-a when a < d/2,
 * else p = d-1-a, c = j+1.  hla2_state_export writes the full records.
 * S, C, m, G, h point at head 0's fields and head i's field X is
 * X + i * head_floats.  `check` is written by hla2_state_init: a call
 * given a descriptor whose other fields changed since then returns
 * HLA_ERR_INVALID.  The descriptor is a host object; pass it by pointer.
 * ------------------------------------------------------------------------- */
typedef struct {
  int B, H, d, dv;            /* heads B*H; key and value widths            */
  int masked, normalized;     /* operator of every prefill and step          */
  int dtype;                  /* HLA_FP32 or HLA_BF16: the tokens' dtype     */
  float eps;                  /* denominator offset, used when normalized    */
  float *data;                /* [B, H, FP] fp32 device memory, caller-owned */
  size_t head_floats;         /* FP = d*(d+1)/2 + 2*d*dv + 2*d               */
  float *S, *C, *m, *G, *h;   /* head 0's fields inside data                 */
  unsigned long long check;   /* set by hla2_state_init                      */
} hla2_state;

/* Device bytes of a state of B*H heads: B*H*FP*4 (0 if invalid). */
size_t hla2_state_bytes(int B, int H, int d, int dv);

/* Fill *st for the device buffer buf (at least hla2_state_bytes(B, H, d, dv)
 * bytes, 16-byte aligned) and enqueue its zeroing on `stream`: the all-zero
 * record is the identity segment of Thm. 2, the state before any token.
 * Argument rules as hla2_forward (sizes, flags, eps, dtype). */
int hla2_state_init(hla2_state *st, void *buf, size_t buf_bytes, int B, int H, int d, int dv, int masked,
                    int normalized, float eps, int dtype, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_prefill — continue every head's state over n new tokens:
 *   state <- state (+) summary(tokens)          (Thm. 2)
 * and, if out != NULL, write the outputs of those tokens ([B, H, n, dv]) as
 * the serial recurrence started from the given state would (Sec. 3.1,
 * Thm. 1), with the state's operator.  q, k: [B, H, n, d], v: [B, H, n, dv]
 * in the state's dtype.  workspace: at least hla2_prefill_workspace_bytes(st,
 * n, chunk) bytes.
 * ------------------------------------------------------------------------- */
size_t hla2_prefill_workspace_bytes(const hla2_state *st, int n, int chunk);
int hla2_prefill(hla2_state *st, const void *q, const void *k, const void *v, int n, int chunk, float *out,
                 void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_step — one decode step per head: the online updates of Sec. 3.1 and
 * the readout of Thm. 1 (Sec. 5 order), with the state's operator.
 * q_t, k_t: [B, H, d]; v_t: [B, H, dv] in the state's dtype; out_t: [B, H, dv]
 * fp32.  The state is updated in place.
 * ------------------------------------------------------------------------- */
int hla2_step(hla2_state *st, const void *q_t, const void *k_t, const void *v_t, float *out_t, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_state_export — the state as full records (the paper's 5-tuple with S
 * as a d x d matrix): full is [B, H, F] fp32 device memory, F =
 * hla2_state_floats(d, dv), caller-owned, 16-byte aligned, not aliasing the
 * state.  Enqueued on `stream`; the state is not changed.
 * ------------------------------------------------------------------------- */
int hla2_state_export(const hla2_state *st, float *full, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_forward_decay — second-order HLA with exponential time decay gamma
 * (decay section; decay-aware monoid of Sec. 4).  Token moments age as
 *   S_t = gamma S_{t-1} + k_t k_t^T,  C_t = gamma C_{t-1} + q_t v_t^T,  m_t = gamma m_{t-1} + q_t,
 * so the pair (i, j) enters row t with weight gamma^{(t-i)+(t-j)}:
 *   masked    o_t = sum_{j<=t} sum_{i<=j} gamma^{(t-i)+(t-j)} (q_t.k_i)(q_j.k_i) v_j
 *   unmasked  o_t = sum_{j<=t} sum_{i<=t} gamma^{(t-i)+(t-j)} (q_t.k_i)(q_j.k_i) v_j
 * i.e. q_t^T (S_t C_t - G_t) with G_t = gamma^2 G_{t-1} + gamma k_t k_t^T C_{t-1}
 * (the paper prints the cross-summary and the segment concatenation in two
 * forms that disagree; this is the reading whose masked output drops exactly
 * the pairs j < i of the unmasked decayed output and whose concatenation,
 * with rho^2 on G and h, is associative).  normalized divides by the same
 * sum without v_j, plus eps.  gamma = 1 is hla2_forward's operator.
 * bf16 inputs, masked, d = dv in {64, 128}, chunk 64 or 128 run on the fused
 * segment walk with decay (bf16 MFMA, every decay factor applied in fp32 before
 * the hi/lo split); everything else on the chunked path in fp32 (decayed
 * chunk summaries, the decayed (+)-scan, decayed readout).  Arguments as
 * hla2_forward, plus
 * gamma, finite, 0 < gamma <= 1 (else HLA_ERR_INVALID); gamma^(2*tile), with
 * tile = min(chunk, 64) the token tile both paths walk, must stay a normal
 * fp32 number (gamma >= 0.51 at chunk 64 and 128; HLA_ERR_UNSUPPORTED
 * otherwise).  workspace: hla2_forward_decay_workspace_bytes(...) bytes (enough
 * for either path).
 * ------------------------------------------------------------------------- */
size_t hla2_forward_decay_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype);
int hla2_forward_decay(const void *q, const void *k, const void *v, float *out,
                       int B, int H, int n, int d, int dv, int chunk, int masked, int normalized,
                       float eps, float gamma, int dtype, void *workspace, size_t workspace_bytes,
                       void *stream);

/* ---------------------------------------------------------------------------
 * hla3_forward — third-order HLA over whole sequences (Sec. 7).
 * masked = 1: out[b,h,t,:] = q_t^T F_t with F_t the corrected third-order
 * state (Eq. hla3-corrected-state, Thm. 3): the sum, over triples (i, u, j)
 * <= t whose largest index is attained at least twice, of
 * (q_t.k_i)(k_i.q_u)(q_u.k_j) v_j.  Computed in fp32 by the chunk-parallel
 * scan of Sec. 7.3 (operator (x)_3, Thm. 4).
 * masked = 0: out[b,h,t,:] = q_t^T S^K_t S^Q_t P_t (Sec. 7.1), the same sum
 * over all triples (i, u, j) <= t; the summaries only add, so each segment is
 * walked from the running sum of the moments before it.
 * With normalized = 1 the row is divided by (den_t + eps), den_t the same sum
 * without v_j (q_t^T eta_t masked, q_t^T S^K_t S^Q_t m^K_t unmasked).
 * q, k: [B, H, n, d]; v: [B, H, n, dv], fp32 or bf16 (dtype); out: [B, H, n, dv]
 * fp32; all device pointers, 16-byte aligned, caller-owned.
 * Supported: d and dv in {16, 32}, chunk in {16, 32, 64, 128}; chunks above
 * 32 are walked in 32-token tiles (exact for any chunking, Thm. 4).  Other
 * sizes return HLA_ERR_UNSUPPORTED.
 * workspace: at least hla3_workspace_bytes(...) bytes of device memory (its
 * contents on entry are ignored); HLA_ERR_WORKSPACE if smaller.
 * ------------------------------------------------------------------------- */
size_t hla3_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype);
int hla3_forward(const void *q, const void *k, const void *v, float *out,
                 int B, int H, int n, int d, int dv, int chunk, int masked, int normalized,
                 float eps, int dtype, void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * hla2_backward — gradients of the masked, unnormalised second-order HLA
 * (the reverse scan of Sec. 4.2, written out): for a loss L with upstream
 * gradient g = dL/dout,
 *   dq_j = Phi_j g_j + S_j u_j,   dv_j = U_j^T r_j,   dk_i = (Z_i + Z_i^T) k_i,
 * with S_j = sum_{i<=j} k_i k_i^T, r_j = S_j q_j, Phi_j = sum_{j'<=j} r_j' v_j'^T,
 * U_j = sum_{t>=j} q_t g_t^T, u_j = U_j v_j, Z_i = sum_{j>=i} u_j q_j^T.
 * Computed on bf16 MFMA (fp32 operands split hi/lo, fp32 accumulation) as
 * seven causal or anti-causal first-order chunk scans over 64-token tiles.
 * q, k, v [B, H, n, d] bf16 (dtype = HLA_BF16); g [B, H, n, dv] fp32;
 * dq, dk [B, H, n, d] and dv [B, H, n, dv] fp32, written (not accumulated).
 * Device pointers, 16-byte aligned, caller-owned; outputs must not alias
 * inputs or each other.  Supported: d = dv in {64, 128}, chunk any supported
 * value (the tiling does not change the result beyond rounding), any n >= 1;
 * everything else returns HLA_ERR_UNSUPPORTED.  workspace: at least
 * hla2_backward_workspace_bytes(...) bytes (contents on entry ignored).
 * ------------------------------------------------------------------------- */
size_t hla2_backward_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype);
int hla2_backward(const void *q, const void *k, const void *v, const float *g, float *dq, float *dk,
                  float *dv, int B, int H, int n, int d, int dv_dim, int chunk, int dtype,
                  void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * ahla_forward — asymmetric second-order HLA (AHLA, Sec. 6): the left-cascaded
 * product ((A A) (.) L) V with A = L (.) Q K^T (diagonal kept),
 *   o_t = sum_{j<=t} sum_{i=j..t} (q_t.k_i)(q_i.k_j) v_j     (Eq. AHLA-explicit)
 *       = q_t^T E_t,  E_t = E_{t-1} + k_t (q_t^T P_t),  P_t = P_{t-1} + k_t v_t^T
 * (Thm. AHLA; E_t uses P_t including token t).  With normalized = 1 the row
 * is divided by (q_t^T n_t + eps), n_t = n_{t-1} + k_t (q_t^T m_t), m_t the
 * key sum: the same double sum without v_j.  Decay is 1.
 * Computed on bf16 MFMA with fp32 accumulation by a segment scan under
 * (+)_AHLA (Eq. AHLA-semidirect): q, k, v [B, H, n, d] bf16 (dtype =
 * HLA_BF16), out [B, H, n, d] fp32; device pointers, 16-byte aligned,
 * caller-owned.  Supported: d = dv in {64, 128}, chunk in {64, 128} (walked
 * in 64-token tiles; exact for any chunking), any n >= 1; everything else
 * (fp32 inputs included) returns HLA_ERR_UNSUPPORTED.  workspace: at least
 * ahla_workspace_bytes(...) bytes of device memory (contents on entry
 * ignored); HLA_ERR_WORKSPACE if smaller.
 * ------------------------------------------------------------------------- */
size_t ahla_workspace_bytes(int B, int H, int n, int d, int dv, int chunk, int dtype);
int ahla_forward(const void *q, const void *k, const void *v, float *out,
                 int B, int H, int n, int d, int dv, int chunk, int normalized, float eps,
                 int dtype, void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Benchmark timing.  hla_profile_begin(max_records) creates 2*max_records HIP
 * events (host objects, no device memory) and starts bracketing every kernel
 * the library launches with events recorded on that kernel's stream;
 * hla_profile_end() stops.  After synchronising the stream,
 * hla_profile_summary(buf, len) writes one line per kernel name,
 * "name launches total_ms", and forgets the records.  Records beyond
 * max_records are not timed.  Not thread-safe; for benchmarks only.
 * ------------------------------------------------------------------------- */
int hla_profile_begin(int max_records);
int hla_profile_end(void);
int hla_profile_summary(char *buf, size_t len);

#ifdef __cplusplus
}
#endif

#endif /* HLA_H */
