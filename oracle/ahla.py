"""Asymmetric second-order HLA (AHLA, Sec. 6) in fp64 NumPy (test infrastructure only).

AHLA applies the left-cascaded product A A V with A = L (.) (Q K^T) (L the
causal mask including the diagonal):

    o_t = sum_{j<=t} sum_{i=j..t} (q_t.k_i)(q_i.k_j) v_j       (Eq. AHLA-explicit)

and, normalised, num_t / (den_t + eps) with den_t the same sum with v_j = 1.
Decay is 1.  Streaming (Thm. AHLA and Alg. AHLA-stream):

    P_t = P_{t-1} + k_t v_t^T,   m_t = m_{t-1} + k_t,
    E_t = E_{t-1} + k_t (q_t^T P_t),   n_t = n_{t-1} + k_t (q_t^T m_t),
    o_t = q_t^T E_t,   den_t = q_t^T n_t.

E_t uses P_t including token t (the paper's Fig. 2 writes the carry with the
prefix before t; the theorem and the algorithm include t, and so does this
oracle).  Segments compose with the key-query cross moment R = sum k_i q_i^T
(Eq. AHLA-semidirect):

    (R, P, m, E, n)_A (+) (...)_B = (R_A + R_B, P_A + P_B, m_A + m_B,
                                     E_A + E_B + R_B P_A, n_A + n_B + R_B m_A).

Functions: ahla_definition_loops, ahla_definition, ahla_serial,
token_segment_ahla, combine_ahla, segment_summary_ahla, ahla_chunked,
ahla_den_scale.
"""
import numpy as np

from oracle.hla2 import blelloch_exclusive


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def ahla_definition_loops(q, k, v):
    """The double sum of Eq. AHLA-explicit with Python loops; q, k [n, d], v [n, dv].
    Returns (num [n, dv], den [n])."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, dv = q.shape[0], v.shape[1]
    num = np.zeros((n, dv))
    den = np.zeros(n)
    for t in range(n):
        for j in range(t + 1):
            w = 0.0
            for i in range(j, t + 1):
                w += float(q[t] @ k[i]) * float(q[i] @ k[j])
            num[t] += w * v[j]
            den[t] += w
    return num, den


def ahla_definition(q, k, v, normalized=False, eps=1e-6, return_num_den=False):
    """Dense form ((A A) (.) L) V with A = L (.) Q K^T (A A is already lower
    triangular), per head over leading batch axes."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[-2]
    L = np.tril(np.ones((n, n)))
    A = L * (q @ np.swapaxes(k, -1, -2))
    AA = (A @ A) * L
    num = AA @ v
    den = AA.sum(-1)
    if return_num_den:
        return num, den
    if normalized:
        return num / (den + eps)[..., None]
    return num


def ahla_serial(q, k, v, normalized=False, eps=1e-6, return_states=False, return_num_den=False):
    """The streaming recurrence (module header), readout after every token."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    P = np.zeros(batch + (d, dv))
    m = np.zeros(batch + (d,))
    E = np.zeros(batch + (d, dv))
    nn = np.zeros(batch + (d,))
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    states = []
    for t in range(n):
        qt, kt, vt = q[..., t, :], k[..., t, :], v[..., t, :]
        P = P + kt[..., :, None] * vt[..., None, :]
        m = m + kt
        r = np.einsum('...a,...ab->...b', qt, P)           # q_t^T P_t
        s = np.einsum('...a,...a->...', qt, m)             # q_t^T m_t
        E = E + kt[..., :, None] * r[..., None, :]
        nn = nn + kt * s[..., None]
        num[..., t, :] = np.einsum('...a,...ab->...b', qt, E)
        den[..., t] = np.einsum('...a,...a->...', qt, nn)
        if return_states:
            states.append((P.copy(), m.copy(), E.copy(), nn.copy()))
    final = (P, m, E, nn)
    if return_num_den:
        res = (num, den)
    elif normalized:
        res = num / (den + eps)[..., None]
    else:
        res = num
    if return_states:
        return res, final, states
    return res, final


def zero_state_ahla(batch, d, dv):
    batch = tuple(batch)
    return (np.zeros(batch + (d, d)), np.zeros(batch + (d, dv)), np.zeros(batch + (d,)),
            np.zeros(batch + (d, dv)), np.zeros(batch + (d,)))


def token_segment_ahla(qt, kt, vt):
    """One token: (k q^T, k v^T, k, (q.k) k v^T, (q.k) k)."""
    qt, kt, vt = _f64(qt), _f64(kt), _f64(vt)
    qk = np.einsum('...a,...a->...', qt, kt)
    R = kt[..., :, None] * qt[..., None, :]
    P = kt[..., :, None] * vt[..., None, :]
    return (R, P, kt.copy(), qk[..., None, None] * P, qk[..., None] * kt)


def combine_ahla(A, B):
    """Eq. AHLA-semidirect: segment A followed by B."""
    RA, PA, mA, EA, nA = A
    RB, PB, mB, EB, nB = B
    return (RA + RB, PA + PB, mA + mB, EA + EB + RB @ PA, nA + nB + (RB @ mA[..., :, None])[..., 0])


def segment_summary_ahla(q, k, v):
    q, k, v = _f64(q), _f64(k), _f64(v)
    acc = zero_state_ahla(q.shape[:-2], q.shape[-1], v.shape[-1])
    for t in range(q.shape[-2]):
        acc = combine_ahla(acc, token_segment_ahla(q[..., t, :], k[..., t, :], v[..., t, :]))
    return acc


def ahla_chunked(q, k, v, chunk, normalized=False, eps=1e-6, return_num_den=False, return_final=False):
    """Two-level chunked scan under (+)_AHLA (Sec. 6, scan equivalence): token
    prefixes inside a chunk and chunk carries by exclusive Blelloch scans; row t
    reads o_t = q_t^T E, den_t = q_t^T n of carry (+) prefix (+) token."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    E0 = zero_state_ahla(batch, d, dv)
    starts = list(range(0, n, chunk))
    local_prefix, summaries, tokens = [], [], []
    for s0 in starts:
        seg = [token_segment_ahla(q[..., t, :], k[..., t, :], v[..., t, :]) for t in range(s0, min(s0 + chunk, n))]
        P = blelloch_exclusive(seg, combine_ahla, E0)
        local_prefix.append(P)
        tokens.append(seg)
        summaries.append(combine_ahla(P[-1], seg[-1]))
    carry = blelloch_exclusive(summaries, combine_ahla, E0)
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    for c, s0 in enumerate(starts):
        for r, Tt in enumerate(tokens[c]):
            inc = combine_ahla(combine_ahla(carry[c], local_prefix[c][r]), Tt)
            qt = q[..., s0 + r, :]
            num[..., s0 + r, :] = np.einsum('...a,...ab->...b', qt, inc[3])
            den[..., s0 + r] = np.einsum('...a,...a->...', qt, inc[4])
    if return_num_den:
        res = (num, den)
    elif normalized:
        res = num / (den + eps)[..., None]
    else:
        res = num
    if return_final:
        return res, (combine_ahla(carry[-1], summaries[-1]) if starts else E0)
    return res


def ahla_den_scale(q, k):
    """D_t = sum_{j<=t} |(A A)_{t,j}|: the scale a computed den_t is judged
    against where den_t itself is near zero, [..., n]."""
    q, k = _f64(q), _f64(k)
    n = q.shape[-2]
    L = np.tril(np.ones((n, n)))
    A = L * (q @ np.swapaxes(k, -1, -2))
    return np.abs((A @ A) * L).sum(-1)
