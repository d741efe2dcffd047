"""Second-order HLA oracle in fp64 NumPy (test infrastructure only).

Every function takes per-head sequences with arbitrary leading batch axes:
q, k have shape [..., n, d] and v has shape [..., n, dv].  Inputs are upcast to
float64.  Decay is fixed at gamma = 1 and the ridge at lambda = 0: the exact
masked bilinear form (Sec. 5, remark after Alg. 1).

State tuples follow the paper's notation (Sec. 3 and Eq. (semidirect)):
    (S, C, m, G, h)
    S = S^K  = sum_i k_i k_i^T          [..., d, d]
    C = C^QV = sum_i q_i v_i^T          [..., d, dv]
    m = m^Q  = sum_i q_i                [..., d]
    G        = sum_i k_i k_i^T C_{i-1}  [..., d, dv]
    h        = sum_i k_i k_i^T m_{i-1}  [..., d]

Functions
  hla2_definition  the plain definition (Sec. 3.1 matrix identity; Sec. 3 for
                   the unmasked operator), by dense n x n products.
  hla2_serial      the online updates of Sec. 3.1 and the readout of Thm. 1.
  combine          the masked semidirect product, Eq. (semidirect).
  blelloch_exclusive  work-efficient exclusive scan (Sec. 4, Rem. scan-modes).
  hla2_chunked     the two-level chunk-parallel scan of Sec. 4 / Alg. 1.
  segment_summary  the summary of a token segment (the inclusive total of
                   its token deltas under combine).
  readout          Thm. 1 output from an inclusive state.
"""
import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _tri_lower(n):
    """Binary causal mask L: lower-triangular including the diagonal (Sec. 3.1)."""
    return np.tril(np.ones((n, n), dtype=np.float64))


# ---------------------------------------------------------------------------
# Plain definition
# ---------------------------------------------------------------------------
def hla2_definition(q, k, v, masked=True, normalized=False, eps=1e-6,
                    return_num_den=False):
    """Second-order HLA straight from its definition, O(n^2 d + n^3) per head.

    Masked (Sec. 3.1 matrix identity): with W = L (.) (Q K^T),
        O = [(W W^T) (.) L] V,
    i.e. o_t = sum_{j<=t} sum_{i<=j} (q_t.k_i)(q_j.k_i) v_j, and the masked
    denominator is the same row applied to the all-ones vector (Thm. 1 proof).

    Unmasked (Eq. hla-unnorm with the prefix moments of Sec. 3):
        o_t = q_t^T S_t C_t = sum_{i<=t} sum_{j<=t} (q_t.k_i)(k_i.q_j) v_j,
    den_t = q_t^T S_t m_t (Eq. hla-row).  Row t only sees indices <= t, so it
    is the t-th row of Q_{:t} K_{:t}^T K_{:t} Q_{:t}^T V_{:t}; it is evaluated
    row by row here.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[-2]
    L = _tri_lower(n)
    if masked:
        W = L * (q @ np.swapaxes(k, -1, -2))                 # [..., n, n]
        T2 = (W @ np.swapaxes(W, -1, -2)) * L                # [..., n, n]
        num = T2 @ v
        den = T2.sum(axis=-1)
    else:
        num = np.empty(q.shape[:-1] + (v.shape[-1],))
        den = np.empty(q.shape[:-1])
        for t in range(n):
            qt = q[..., t, :]
            Kp, Qp, Vp = k[..., : t + 1, :], q[..., : t + 1, :], v[..., : t + 1, :]
            a = np.einsum('...d,...id->...i', qt, Kp)        # q_t . k_i, i <= t
            b = np.einsum('...i,...id->...d', a, Kp)         # q_t^T S_t
            c = np.einsum('...d,...jd->...j', b, Qp)         # q_t^T S_t q_j, j <= t
            num[..., t, :] = np.einsum('...j,...jv->...v', c, Vp)
            den[..., t] = c.sum(axis=-1)
    if return_num_den:
        return num, den
    if normalized:
        return num / (den + eps)[..., None]
    return num


def hla2_definition_loops(q, k, v, masked=True):
    """The double sums written out with Python loops (tiny single-head inputs).

    masked:   o_t = sum_{j<=t} sum_{i<=j} (q_t.k_i)(q_j.k_i) v_j  (Thm. 1 proof)
    unmasked: o_t = sum_{j<=t} sum_{i<=t} (q_t.k_i)(q_j.k_i) v_j
    q, k: [n, d]; v: [n, dv].  Returns (num [n, dv], den [n]).
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, dv = q.shape[0], v.shape[1]
    num = np.zeros((n, dv))
    den = np.zeros(n)
    for t in range(n):
        for j in range(t + 1):
            imax = j if masked else t
            w = 0.0
            for i in range(imax + 1):
                w += float(q[t] @ k[i]) * float(q[j] @ k[i])
            num[t] += w * v[j]
            den[t] += w
    return num, den


# ---------------------------------------------------------------------------
# State algebra
# ---------------------------------------------------------------------------
def zero_state(batch, d, dv):
    """The identity segment E: all summaries zero (Thm. 2 proof)."""
    batch = tuple(batch)
    return (np.zeros(batch + (d, d)), np.zeros(batch + (d, dv)), np.zeros(batch + (d,)),
            np.zeros(batch + (d, dv)), np.zeros(batch + (d,)))


def token_segment(qt, kt, vt):
    """Elementary segment of one token (Sec. 4.1/4.2): (k k^T, q v^T, q, 0, 0)."""
    qt, kt, vt = _f64(qt), _f64(kt), _f64(vt)
    dS = kt[..., :, None] * kt[..., None, :]
    dC = qt[..., :, None] * vt[..., None, :]
    return (dS, dC, qt.copy(), np.zeros_like(dC), np.zeros_like(qt))


def combine(A, B):
    """Masked semidirect product, Eq. (semidirect): segment A followed by B.

    (S_A+S_B, C_A+C_B, m_A+m_B, G_A+G_B+S_B C_A, h_A+h_B+S_B m_A)
    """
    SA, CA, mA, GA, hA = A
    SB, CB, mB, GB, hB = B
    return (SA + SB, CA + CB, mA + mB,
            GA + GB + SB @ CA,
            hA + hB + (SB @ mA[..., :, None])[..., 0])


def readout(state, qt, masked=True, normalized=False, eps=1e-6, return_num_den=False):
    """Thm. 1 from an inclusive state, in the order of Sec. 5 (Compute):
    u = q^T S, num = u C - q^T G, den = u m - q^T h (unmasked: drop G and h)."""
    S, C, m, G, h = state
    qt = _f64(qt)
    u = np.einsum('...a,...ab->...b', qt, S)
    num = np.einsum('...a,...ab->...b', u, C)
    den = np.einsum('...a,...a->...', u, m)
    if masked:
        num = num - np.einsum('...a,...ab->...b', qt, G)
        den = den - np.einsum('...a,...a->...', qt, h)
    if return_num_den:
        return num, den
    if normalized:
        return num / (den + eps)[..., None]
    return num


# ---------------------------------------------------------------------------
# Serial recurrence
# ---------------------------------------------------------------------------
def hla2_serial(q, k, v, masked=True, normalized=False, eps=1e-6, state=None,
                return_states=False, return_num_den=False):
    """Serial left-to-right recurrence: online updates of Sec. 3.1, Thm. 1 readout.

    At each t:  G += k_t (k_t^T C_{t-1}),  h += k_t (k_t^T m_{t-1}),
                S += k_t k_t^T,  C += q_t v_t^T,  m += q_t,
    then the readout of Thm. 1 in the Sec. 5 order.  `state` (S, C, m, G, h)
    continues a previous run (the serial recurrence from that prefix).

    Returns out [..., n, dv] (or (num, den)), the final state, and, with
    return_states, the list of inclusive states after every token.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    if state is None:
        S, C, m, G, h = zero_state(batch, d, dv)
    else:
        S, C, m, G, h = (np.array(_f64(x), copy=True) for x in state)
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    states = []
    for t in range(n):
        qt, kt, vt = q[..., t, :], k[..., t, :], v[..., t, :]
        w = np.einsum('...a,...ab->...b', kt, C)      # k_t^T C_{t-1}
        s = np.einsum('...a,...a->...', kt, m)        # k_t^T m_{t-1}
        G = G + kt[..., :, None] * w[..., None, :]
        h = h + kt * s[..., None]
        S = S + kt[..., :, None] * kt[..., None, :]
        C = C + qt[..., :, None] * vt[..., None, :]
        m = m + qt
        nt, dt = readout((S, C, m, G, h), qt, masked=masked, return_num_den=True)
        num[..., t, :] = nt
        den[..., t] = dt
        if return_states:
            states.append((S.copy(), C.copy(), m.copy(), G.copy(), h.copy()))
    final = (S, C, m, G, h)
    if return_num_den:
        res = (num, den)
    elif normalized:
        res = num / (den + eps)[..., None]
    else:
        res = num
    if return_states:
        return res, final, states
    return res, final


# ---------------------------------------------------------------------------
# Chunk-parallel associative scan
# ---------------------------------------------------------------------------
def blelloch_exclusive(xs, op, identity):
    """Work-efficient exclusive scan (up-sweep / down-sweep) of a list under an
    associative, not necessarily commutative, operator (Rem. scan-modes):
    returns P_t = E (+) x_1 (+) ... (+) x_{t-1}."""
    n = len(xs)
    size = 1
    while size < max(n, 1):
        size *= 2
    a = list(xs) + [identity] * (size - n)
    step = 1
    while step < size:                       # up-sweep: a[i] <- left (+) right
        for i in range(2 * step - 1, size, 2 * step):
            a[i] = op(a[i - step], a[i])
        step *= 2
    a[size - 1] = identity
    step = size // 2
    while step >= 1:                         # down-sweep
        for i in range(2 * step - 1, size, 2 * step):
            left = a[i - step]
            a[i - step] = a[i]               # left child: prefix before the node
            a[i] = op(a[i], left)            # right child: prefix (+) left total
        step //= 2
    return a[:n]


def segment_summary(q, k, v):
    """Summary of a token segment: the (+)-product of its token deltas, in order."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch = q.shape[:-2]
    acc = zero_state(batch, q.shape[-1], v.shape[-1])
    for t in range(q.shape[-2]):
        acc = combine(acc, token_segment(q[..., t, :], k[..., t, :], v[..., t, :]))
    return acc


def hla2_chunked(q, k, v, chunk, masked=True, normalized=False, eps=1e-6,
                 return_num_den=False, return_final=False):
    """Two-level chunk-parallel scan (Sec. 4, Rem. scan-modes, Alg. 1), fp64.

    1. Split the sequence into chunks of `chunk` tokens (the last may be short).
    2. Within each chunk, an exclusive Blelloch scan over the token segments
       gives the local prefixes P_t (Alg. 1).
    3. Each chunk's summary is P_w (+) T_w; an exclusive scan over the chunk
       summaries gives the carry-in of every chunk (inter-chunk parallelism).
    4. Token t of chunk c uses carry (+) P_t (+) T_t as its inclusive state and
       is read out with Thm. 1.
    Returns the outputs and, with return_final, the state after the last token.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    E = zero_state(batch, d, dv)
    starts = list(range(0, n, chunk))
    local_prefix, summaries, tokens = [], [], []
    for s0 in starts:
        seg = [token_segment(q[..., t, :], k[..., t, :], v[..., t, :])
               for t in range(s0, min(s0 + chunk, n))]
        P = blelloch_exclusive(seg, combine, E)
        local_prefix.append(P)
        tokens.append(seg)
        summaries.append(combine(P[-1], seg[-1]))
    carry = blelloch_exclusive(summaries, combine, E)
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    for c, s0 in enumerate(starts):
        for r, Tt in enumerate(tokens[c]):
            inc = combine(combine(carry[c], local_prefix[c][r]), Tt)
            nt, dt = readout(inc, q[..., s0 + r, :], masked=masked, return_num_den=True)
            num[..., s0 + r, :] = nt
            den[..., s0 + r] = dt
    if return_num_den:
        res = (num, den)
    elif normalized:
        res = num / (den + eps)[..., None]
    else:
        res = num
    if return_final:
        final = combine(carry[-1], summaries[-1]) if starts else E
        return res, final
    return res


def chunk_summaries(q, k, v, chunk):
    """Summary of every chunk of `chunk` tokens, stacked on a new chunk axis
    placed after the batch axes: each component has shape [..., M, ...]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[-2]
    sums = [segment_summary(q[..., s:s + chunk, :], k[..., s:s + chunk, :], v[..., s:s + chunk, :])
            for s in range(0, n, chunk)]
    nb = q.ndim - 2
    return tuple(np.stack([s[i] for s in sums], axis=nb) for i in range(5))


def exclusive_scan_states(states):
    """Exclusive (+)-scan along the chunk axis of stacked states (as returned by
    chunk_summaries); returns (prefixes stacked the same way, total)."""
    S = states[0]
    nb = S.ndim - 3
    M = S.shape[nb]
    items = [tuple(x[(slice(None),) * nb + (c,)] for x in states) for c in range(M)]
    E = tuple(np.zeros_like(x) for x in items[0])
    pre = blelloch_exclusive(items, combine, E)
    total = combine(pre[-1], items[-1])
    return tuple(np.stack([p[i] for p in pre], axis=nb) for i in range(5)), total


def hla2_den_scale(q, k, masked=True):
    """Sum of the absolute values of the terms of den_t, in fp64, [..., n].

    masked:   D_t = sum_{j<=t} |q_t^T S_j q_j|   (Thm. 1 proof, v_j -> 1)
    unmasked: D_t = sum_{j<=t} |q_t^T S_t q_j|   (Eq. hla-row)
    It bounds |den_t| and is the scale against which a computed den_t is
    judged where den_t itself is near zero."""
    q, k = _f64(q), _f64(k)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    S = np.zeros(batch + (d, d))
    R = np.empty(q.shape)
    for t in range(n):
        S = S + k[..., t, :, None] * k[..., t, None, :]
        R[..., t, :] = np.einsum('...ab,...b->...a', S, q[..., t, :])       # r_t = S_t q_t
    D = np.empty(batch + (n,))
    blk = 1024
    for s in range(0, n, blk):
        e = min(n, s + blk)
        if masked:
            A = np.abs(q[..., s:e, :] @ np.swapaxes(R[..., :e, :], -1, -2))  # |q_t . r_j|
        else:
            A = np.abs(R[..., s:e, :] @ np.swapaxes(q[..., :e, :], -1, -2))  # |r_t . q_j|
        A = A * (np.arange(e)[None, :] <= np.arange(s, e)[:, None])
        D[..., s:e] = A.sum(-1)
    return D
