"""Third-order HLA oracle in fp64 NumPy (test infrastructure only).

Every function takes per-head sequences with arbitrary leading batch axes:
q, k have shape [..., n, d] and v has shape [..., n, dv], upcast to float64.
Decay is fixed at gamma = 1 (the chunk-parallel algorithm of Sec. 7.3 is
stated for gamma = 1).

Serial state (Sec. 7.1, Thm. 3), in the paper's notation:
    (SK, SQ, P, m, G1, G2, G3, h1, h2, h3)
    SK = sum_i k_i k_i^T, SQ = sum_i q_i q_i^T, P = sum_i k_i v_i^T, m = sum_i k_i
    G1 = sum_i k_i k_i^T SQ_{i-1} P_{i-1}      h1 = sum_i k_i k_i^T SQ_{i-1} m_{i-1}
    G2 = sum_i SK_{i-1} q_i q_i^T P_{i-1}      h2 = sum_i SK_{i-1} q_i q_i^T m_{i-1}
    G3 = sum_i SK_{i-1} SQ_{i-1} k_i v_i^T     h3 = sum_i SK_{i-1} SQ_{i-1} k_i

Segment scan state (Sec. 7.3):
    (SK, SQ, P, m, F, eta, R, r, U, MP, Mm)
with F = SK SQ P - G1 - G2 - G3 and eta = SK SQ m - h1 - h2 - h3 (Eq.
hla3-corrected-state), R = sum D^Q D^P, r = sum D^Q d^m, U = sum D^K D^Q, and
the linear maps M^KQP, M^KQm held densely as tensors:
    M^KQP[Z]_{a e} = sum_{b c} MP[a, b, c, e] Z[b, c],   MP = sum_t k (x) k (x) k (x) v
    M^KQm[Z]_a     = sum_{b c} Mm[a, b, c] Z[b, c],      Mm = sum_t k (x) k (x) k
(d^3 dv and d^3 entries: only for the small shapes the tests use).

Functions
  hla3_definition_loops  the triple sum over the index set of Thm. 3, written out.
  hla3_definition        the same sum, vectorised per row (small n).
  hla3_serial            Alg. 3 (gamma = 1), masked or unmasked.
  hla3_corrected_serial  the corrected-state recurrence (Eq. hla3-corrected-recurrence).
  token_segment3, combine3   Alg. 4 token segments and the operator (x)_3
                         (Eqs. hla3-base-concat, hla3-corrected-concat).
  hla3_chunked           Alg. 4: intra- and inter-chunk exclusive scans, readout.
"""
import itertools

import numpy as np

from oracle.hla2 import blelloch_exclusive


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _outer(a, b):
    return np.einsum("...i,...j->...ij", a, b)


def _mv(M, x):
    return np.einsum("...ij,...j->...i", M, x)


def _vm(x, M):
    return np.einsum("...i,...ij->...j", x, M)


# ---------------------------------------------------------------------------
# Plain definition
# ---------------------------------------------------------------------------
def in_index_set(i, u, j, t, masked=True):
    """Triples (i, u, j) <= t summed by row t.  Unmasked (Sec. 7.1): all of
    [1, t]^3.  Masked: the corrections G1, G2, G3 of Thm. 3 remove the triples
    whose largest index is held by exactly one of i (G1), u (G2) or j (G3), so
    the masked row sums the triples whose maximum is attained at least twice."""
    if max(i, u, j) > t:
        return False
    if not masked:
        return True
    top = max(i, u, j)
    return (i == top) + (u == top) + (j == top) >= 2


def hla3_definition_loops(q, k, v, masked=True):
    """num_t = sum over the index set of (q_t.k_i)(k_i.q_u)(q_u.k_j) v_j and
    den_t the same sum without v_j (Thm. 3 with v := 1), by explicit loops
    over one head.  O(n^4); for tiny n only."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[0]
    num = np.zeros((n, v.shape[1]))
    den = np.zeros(n)
    for t in range(n):
        for i, u, j in itertools.product(range(t + 1), repeat=3):
            if not in_index_set(i, u, j, t, masked):
                continue
            w = (q[t] @ k[i]) * (k[i] @ q[u]) * (q[u] @ k[j])
            num[t] += w * v[j]
            den[t] += w
    return num, den


def hla3_definition(q, k, v, masked=True):
    """The same triple sum, vectorised per row with an explicit index-set
    mask (batched over leading axes; O(n^4) work, small n)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[-2]
    A = np.einsum("...td,...id->...ti", q, k)      # A[t, i] = q_t . k_i
    idx = np.arange(n)
    I, U, J = np.meshgrid(idx, idx, idx, indexing="ij")
    top = np.maximum(np.maximum(I, U), J)
    ties = (I == top).astype(int) + (U == top) + (J == top)
    num = np.zeros(q.shape[:-1] + (v.shape[-1],))
    den = np.zeros(q.shape[:-1])
    for t in range(n):
        mask = (top <= t) & ((ties >= 2) if masked else True)
        # w[i, u, j] = A[t, i] A[u, i] A[u, j]
        w = np.einsum("...i,...ui,...uj->...iuj", A[..., t, :], A, A) * mask
        wj = w.sum(axis=(-3, -2))
        num[..., t, :] = np.einsum("...j,...jv->...v", wj, v)
        den[..., t] = wj.sum(axis=-1)
    return num, den


# ---------------------------------------------------------------------------
# Serial recurrences
# ---------------------------------------------------------------------------
def zero_serial_state(batch, d, dv):
    z = np.zeros
    return (z(batch + (d, d)), z(batch + (d, d)), z(batch + (d, dv)), z(batch + (d,)),
            z(batch + (d, dv)), z(batch + (d, dv)), z(batch + (d, dv)),
            z(batch + (d,)), z(batch + (d,)), z(batch + (d,)))


def hla3_serial(q, k, v, masked=True, normalized=False, eps=1e-6, state=None, return_num_den=False):
    """Alg. 3 with gamma = 1.  Per token, with the previous moments
    (SK', SQ', P', m'):
      inclusive moments   SK = SK' + k k^T, SQ = SQ' + q q^T, P = P' + k v^T, m = m' + k
      G1 += k ((SQ' k)^T P'),   h1 += k ((SQ' k) . m')
      G2 += (SK' q)(q^T P'),    h2 += (SK' q)(q . m')
      G3 += (SK' SQ' k) v^T,    h3 += SK' SQ' k
      num = (SQ SK q)^T P - q^T (G1 + G2 + G3)   [masked; unmasked keeps only the first term]
      den = q^T (SK SQ m - h1 - h2 - h3)         [unmasked: q^T SK SQ m]
    Returns (result, final_state) or ((num, den), final_state)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch, n, d, dv = q.shape[:-2], q.shape[-2], q.shape[-1], v.shape[-1]
    st = zero_serial_state(batch, d, dv) if state is None else tuple(_f64(x).copy() for x in state)
    SK, SQ, P, m, G1, G2, G3, h1, h2, h3 = st
    num = np.zeros(batch + (n, dv))
    den = np.zeros(batch + (n,))
    for t in range(n):
        qt, kt, vt = q[..., t, :], k[..., t, :], v[..., t, :]
        SKp, SQp, Pp, mp = SK, SQ, P, m
        SK = SKp + _outer(kt, kt)
        SQ = SQp + _outer(qt, qt)
        P = Pp + _outer(kt, vt)
        m = mp + kt
        u1 = _mv(SQp, kt)
        G1 = G1 + _outer(kt, _vm(u1, Pp))
        h1 = h1 + kt * np.sum(u1 * mp, axis=-1)[..., None]
        a2 = _mv(SKp, qt)
        G2 = G2 + _outer(a2, _vm(qt, Pp))
        h2 = h2 + a2 * np.sum(qt * mp, axis=-1)[..., None]
        a3 = _mv(SKp, _mv(SQp, kt))
        G3 = G3 + _outer(a3, vt)
        h3 = h3 + a3
        z = _mv(SQ, _mv(SK, qt))
        nt = _vm(z, P)
        dt = np.sum(z * m, axis=-1)
        if masked:
            nt = nt - _vm(qt, G1 + G2 + G3)
            dt = dt - np.sum(qt * (h1 + h2 + h3), axis=-1)
        num[..., t, :] = nt
        den[..., t] = dt
    final = (SK, SQ, P, m, G1, G2, G3, h1, h2, h3)
    if return_num_den:
        return (num, den), final
    res = num / (den + eps)[..., None] if normalized else num
    return res, final


def hla3_corrected_serial(q, k, v, return_increments=False):
    """The corrected-state recurrence (Eq. hla3-corrected-recurrence), masked:
      F_t   = F_{t-1} + SK' D^Q D^P + D^K SQ' D^P + D^K D^Q P' + D^K D^Q D^P
      eta_t = eta_{t-1} + (the same with D^P replaced by d^m = k)
    with D^K = k k^T, D^Q = q q^T, D^P = k v^T and primes the moments before
    token t; num_t = q_t^T F_t, den_t = q_t^T eta_t.  Returns (num, den) and
    the final (SK, SQ, P, m, F, eta); with return_increments also the per-token
    increments of eta (for the denominator scale)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch, n, d, dv = q.shape[:-2], q.shape[-2], q.shape[-1], v.shape[-1]
    SK = np.zeros(batch + (d, d))
    SQ = np.zeros(batch + (d, d))
    P = np.zeros(batch + (d, dv))
    m = np.zeros(batch + (d,))
    F = np.zeros(batch + (d, dv))
    eta = np.zeros(batch + (d,))
    num = np.zeros(batch + (n, dv))
    den = np.zeros(batch + (n,))
    incs = np.zeros(batch + (n, d))
    for t in range(n):
        qt, kt, vt = q[..., t, :], k[..., t, :], v[..., t, :]
        DK, DQ, DP = _outer(kt, kt), _outer(qt, qt), _outer(kt, vt)
        dF = SK @ DQ @ DP + DK @ SQ @ DP + DK @ DQ @ P + DK @ DQ @ DP
        de = _mv(SK @ DQ, kt) + _mv(DK @ SQ, kt) + _mv(DK @ DQ, m) + _mv(DK @ DQ, kt)
        F = F + dF
        eta = eta + de
        incs[..., t, :] = de
        SK, SQ, P, m = SK + DK, SQ + DQ, P + DP, m + kt
        num[..., t, :] = _vm(qt, F)
        den[..., t] = np.sum(qt * eta, axis=-1)
    out = ((num, den), (SK, SQ, P, m, F, eta))
    return out + (incs,) if return_increments else out


def hla3_den_scale(q, k):
    """Scale for judging the masked denominator: D_t = sum_{j<=t} |q_t . de_j|,
    with de_j the increment of eta at token j (corrected recurrence), so
    |den_t| <= D_t."""
    q, k = _f64(q), _f64(k)
    v = np.zeros(q.shape[:-1] + (1,))
    _, _, incs = hla3_corrected_serial(q, k, v, return_increments=True)
    c = np.abs(np.einsum("...td,...jd->...tj", q, incs))
    n = q.shape[-2]
    return (c * np.tril(np.ones((n, n)))).sum(axis=-1)


def hla3_den_scale_unmasked(q, k):
    """Scale for judging the unmasked denominator (Sec. 7.1):
    D_t = sum_{i,u,j<=t} |q_t.k_i| |k_i.q_u| |q_u.k_j|, the sum of the absolute
    values of the terms of den_t, so |den_t| <= D_t.  Per head over leading
    batch axes; O(n^3) per head."""
    q, k = _f64(q), _f64(k)
    A = np.abs(np.einsum("...ud,...jd->...uj", q, k))     # A[u, j] = |q_u . k_j|
    n = q.shape[-2]
    out = np.empty(q.shape[:-1])
    for t in range(n):
        x = A[..., : t + 1, : t + 1].sum(-1)                             # over j, per u
        y = np.einsum("...ui,...u->...i", A[..., : t + 1, : t + 1], x)   # over u, per i
        out[..., t] = (A[..., t, : t + 1] * y).sum(-1)                   # over i
    return out


# ---------------------------------------------------------------------------
# Segment scan state and the operator (x)_3
# ---------------------------------------------------------------------------
def zero_scan_state(batch, d, dv):
    z = np.zeros
    return (z(batch + (d, d)), z(batch + (d, d)), z(batch + (d, dv)), z(batch + (d,)),
            z(batch + (d, dv)), z(batch + (d,)), z(batch + (d, dv)), z(batch + (d,)), z(batch + (d, d)),
            z(batch + (d, d, d, dv)), z(batch + (d, d, d)))


def apply_MP(MP, Z):
    return np.einsum("...abce,...bc->...ae", MP, Z)


def apply_Mm(Mm, Z):
    return np.einsum("...abc,...bc->...a", Mm, Z)


def token_segment3(qt, kt, vt):
    """The single-token segment of Alg. 4 (its second step)."""
    DK, DQ, DP = _outer(kt, kt), _outer(qt, qt), _outer(kt, vt)
    return (DK, DQ, DP, kt.copy(),
            DK @ DQ @ DP, _mv(DK @ DQ, kt),
            DQ @ DP, _mv(DQ, kt), DK @ DQ,
            np.einsum("...a,...b,...c,...e->...abce", kt, kt, kt, vt),
            np.einsum("...a,...b,...c->...abc", kt, kt, kt))


def combine3(A, B):
    """X_A (x)_3 X_B, Eqs. hla3-base-concat and hla3-corrected-concat."""
    SKa, SQa, Pa, ma, Fa, ea, Ra, ra, Ua, MPa, Mma = A
    SKb, SQb, Pb, mb, Fb, eb, Rb, rb, Ub, MPb, Mmb = B
    F = Fa + Fb + SKa @ Rb + apply_MP(MPb, SQa) + Ub @ Pa
    eta = ea + eb + _mv(SKa, rb) + apply_Mm(Mmb, SQa) + _mv(Ub, ma)
    return (SKa + SKb, SQa + SQb, Pa + Pb, ma + mb, F, eta, Ra + Rb, ra + rb, Ua + Ub, MPa + MPb, Mma + Mmb)


def segment_summary3(q, k, v):
    """Scan state of a token segment: the (x)_3-product of its token segments, in order."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    acc = zero_scan_state(q.shape[:-2], q.shape[-1], v.shape[-1])
    for t in range(q.shape[-2]):
        acc = combine3(acc, token_segment3(q[..., t, :], k[..., t, :], v[..., t, :]))
    return acc


def hla3_chunked(q, k, v, chunk, normalized=False, eps=1e-6, return_num_den=False):
    """Alg. 4 (masked, gamma = 1) for one head (q [n, d], k [n, d], v [n, dv]):
    token segments; per chunk an exclusive Blelloch scan over its tokens (local
    prefixes, and the chunk summary as the last prefix (x)_3 the last token);
    an exclusive Blelloch scan over chunk summaries (carry-ins); and per token
    I_t = carry (x)_3 local prefix (x)_3 token, o_t = q_t^T F(I_t)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, d, dv = q.shape[0], q.shape[1], v.shape[1]
    E = zero_scan_state((), d, dv)
    toks = [token_segment3(q[t], k[t], v[t]) for t in range(n)]
    bounds = [(c, min(n, c + chunk)) for c in range(0, n, chunk)]
    local, summaries = [], []
    for a, b in bounds:
        pre = blelloch_exclusive(toks[a:b], combine3, E)
        local.append(pre)
        summaries.append(combine3(pre[-1], toks[b - 1]))
    carries = blelloch_exclusive(summaries, combine3, E)
    num = np.zeros((n, dv))
    den = np.zeros(n)
    for ci, (a, b) in enumerate(bounds):
        for t in range(a, b):
            inc = combine3(combine3(carries[ci], local[ci][t - a]), toks[t])
            num[t] = q[t] @ inc[4]
            den[t] = q[t] @ inc[5]
    if return_num_den:
        return num, den
    return num / (den + eps)[:, None] if normalized else num
