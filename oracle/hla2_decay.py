"""Second-order HLA with exponential time decay, fp64 NumPy (test infrastructure only).

Decay gamma in (0, 1] (Sec. "Adding decay and regularization"; decay-aware
monoid of Sec. 4).  The paper prints the decayed moments

    S_t = gamma S_{t-1} + k_t k_t^T,   C_t = gamma C_{t-1} + q_t v_t^T,   m_t = gamma m_{t-1} + q_t,

so the unmasked output q_t^T S_t C_t weights the pair (i, j) by
gamma^{(t-i)+(t-j)}: each token's moments age from its own time to t.  Its
printed cross-summary update (gamma G_{t-1} + k_t k_t^T C_{t-1}) and its
printed decayed concatenation (rho_B G_A) are not consistent with each other,
and the concatenation is not associative (see the tests).  This module reads
the masked decayed operator as the unmasked one with the pairs j < i removed
at the same weights:

    o_t = sum_{j<=t} sum_{i<=j} gamma^{(t-i)+(t-j)} (q_t.k_i)(q_j.k_i) v_j,

which is what q_t^T (S_t C_t - G_t) gives when

    G_t = gamma^2 G_{t-1} + gamma k_t (k_t^T C_{t-1}),   h_t = gamma^2 h_{t-1} + gamma k_t (k_t^T m_{t-1}).

Segments compose associatively with attenuation rho = gamma^length:

    (S, C, m, G, h, rho)_A (+)_g (...)_B =
        (rho_B S_A + S_B, rho_B C_A + C_B, rho_B m_A + m_B,
         rho_B^2 G_A + G_B + rho_B S_B C_A, rho_B^2 h_A + h_B + rho_B S_B m_A, rho_A rho_B).

At gamma = 1 all of this is the undecayed operator of the other oracle module.

Functions
  hla2_decay_definition_loops  the double sums with Python loops (tiny inputs).
  hla2_decay_definition        the same by dense products.
  hla2_decay_serial            the recurrence above with the Thm. 1 readout.
  combine_decay, token_segment_decay, segment_summary_decay,
  hla2_decay_chunked           the two-level chunked scan under (+)_g.
  hla2_decay_den_scale         sum of |terms| of den_t (scale for judging den).
"""
import numpy as np

from oracle.hla2 import blelloch_exclusive, readout


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def hla2_decay_definition_loops(q, k, v, gamma, masked=True):
    """o_t = sum_{j<=t} sum_{i<=j (masked) or i<=t (unmasked)} gamma^{(t-i)+(t-j)}
    (q_t.k_i)(q_j.k_i) v_j, and den_t the same with v_j -> 1.
    q, k: [n, d]; v: [n, dv].  Returns (num [n, dv], den [n])."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, dv = q.shape[0], v.shape[1]
    num = np.zeros((n, dv))
    den = np.zeros(n)
    for t in range(n):
        for j in range(t + 1):
            imax = j if masked else t
            w = 0.0
            for i in range(imax + 1):
                w += gamma ** ((t - i) + (t - j)) * float(q[t] @ k[i]) * float(q[j] @ k[i])
            num[t] += w * v[j]
            den[t] += w
    return num, den


def _decay_matrix(n, gamma):
    """D[t][i] = gamma^(t-i) for i <= t, else 0."""
    t = np.arange(n)
    e = t[:, None] - t[None, :]
    return np.where(e >= 0, float(gamma) ** np.maximum(e, 0), 0.0)


def hla2_decay_definition(q, k, v, gamma, masked=True, normalized=False, eps=1e-6, return_num_den=False):
    """The decayed operator by dense products, per head.

    masked: with A[t][i] = gamma^(t-i) (q_t.k_i) (i <= t) and B[j][i] = (q_j.k_i)
    (i <= j), the weight of v_j in row t (j <= t) is gamma^(t-j) (A B^T)[t][j]:
    the sum over i runs over i <= min(t, j) = j.
    unmasked: row by row, sum over all i, j <= t."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[-2]
    D = _decay_matrix(n, gamma)
    L = (D > 0).astype(np.float64)
    if masked:
        QK = q @ np.swapaxes(k, -1, -2)
        A = D * QK
        B = L * QK
        T2 = D * (A @ np.swapaxes(B, -1, -2))
        num = T2 @ v
        den = T2.sum(axis=-1)
    else:
        num = np.empty(q.shape[:-1] + (v.shape[-1],))
        den = np.empty(q.shape[:-1])
        for t in range(n):
            w = float(gamma) ** (t - np.arange(t + 1))                   # gamma^(t-i), i <= t
            a = np.einsum('...d,...id->...i', q[..., t, :], k[..., : t + 1, :]) * w
            b = np.einsum('...i,...id->...d', a, k[..., : t + 1, :])      # q_t^T S_t
            c = np.einsum('...d,...jd->...j', b, q[..., : t + 1, :]) * w  # gamma^(t-j) q_t^T S_t q_j
            num[..., t, :] = np.einsum('...j,...jv->...v', c, v[..., : t + 1, :])
            den[..., t] = c.sum(axis=-1)
    if return_num_den:
        return num, den
    if normalized:
        return num / (den + eps)[..., None]
    return num


def zero_state_decay(batch, d, dv):
    """Identity: the zero-length segment, all summaries zero and rho = 1."""
    batch = tuple(batch)
    return (np.zeros(batch + (d, d)), np.zeros(batch + (d, dv)), np.zeros(batch + (d,)),
            np.zeros(batch + (d, dv)), np.zeros(batch + (d,)), np.ones(batch))


def token_segment_decay(qt, kt, vt, gamma):
    """One token: (k k^T, q v^T, q, 0, 0, gamma)."""
    qt, kt, vt = _f64(qt), _f64(kt), _f64(vt)
    dS = kt[..., :, None] * kt[..., None, :]
    dC = qt[..., :, None] * vt[..., None, :]
    return (dS, dC, qt.copy(), np.zeros_like(dC), np.zeros_like(qt), np.full(qt.shape[:-1], float(gamma)))


def combine_decay(A, B):
    """Decayed concatenation, segment A followed by B (see the module header)."""
    SA, CA, mA, GA, hA, rA = A
    SB, CB, mB, GB, hB, rB = B
    r1 = rB[..., None]
    r2 = rB[..., None, None]
    return (r2 * SA + SB, r2 * CA + CB, r1 * mA + mB,
            r2 * r2 * GA + GB + r2 * (SB @ CA),
            r1 * r1 * hA + hB + r1 * (SB @ mA[..., :, None])[..., 0],
            rA * rB)


def hla2_decay_serial(q, k, v, gamma, masked=True, normalized=False, eps=1e-6, state=None,
                      return_states=False, return_num_den=False):
    """Serial recurrence with decay (module header), Thm. 1 readout after each token:
        G = g^2 G + g k_t (k_t^T C_{t-1}),  h = g^2 h + g k_t (k_t^T m_{t-1}),
        S = g S + k_t k_t^T,  C = g C + q_t v_t^T,  m = g m + q_t.
    `state` = (S, C, m, G, h) continues from that prefix."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    g = float(gamma)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    if state is None:
        S, C, m, G, h, _ = zero_state_decay(batch, d, dv)
    else:
        S, C, m, G, h = (np.array(_f64(x), copy=True) for x in state)
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    states = []
    for t in range(n):
        qt, kt, vt = q[..., t, :], k[..., t, :], v[..., t, :]
        w = np.einsum('...a,...ab->...b', kt, C)      # k_t^T C_{t-1}
        s = np.einsum('...a,...a->...', kt, m)        # k_t^T m_{t-1}
        G = g * g * G + g * kt[..., :, None] * w[..., None, :]
        h = g * g * h + g * kt * s[..., None]
        S = g * S + kt[..., :, None] * kt[..., None, :]
        C = g * C + qt[..., :, None] * vt[..., None, :]
        m = g * m + qt
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


def segment_summary_decay(q, k, v, gamma):
    """The (+)_g-product of a segment's token deltas, in order."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    acc = zero_state_decay(q.shape[:-2], q.shape[-1], v.shape[-1])
    for t in range(q.shape[-2]):
        acc = combine_decay(acc, token_segment_decay(q[..., t, :], k[..., t, :], v[..., t, :], gamma))
    return acc


def hla2_decay_chunked(q, k, v, gamma, chunk, masked=True, normalized=False, eps=1e-6,
                       return_num_den=False, return_final=False):
    """Two-level chunked scan under (+)_g (the same skeleton as the undecayed
    chunked scan): token prefixes inside a chunk and chunk carries by exclusive
    Blelloch scans, each token read out (Thm. 1) from carry (+)_g prefix (+)_g token."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    E = zero_state_decay(batch, d, dv)
    starts = list(range(0, n, chunk))
    local_prefix, summaries, tokens = [], [], []
    for s0 in starts:
        seg = [token_segment_decay(q[..., t, :], k[..., t, :], v[..., t, :], gamma)
               for t in range(s0, min(s0 + chunk, n))]
        P = blelloch_exclusive(seg, combine_decay, E)
        local_prefix.append(P)
        tokens.append(seg)
        summaries.append(combine_decay(P[-1], seg[-1]))
    carry = blelloch_exclusive(summaries, combine_decay, E)
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    for c, s0 in enumerate(starts):
        for r, Tt in enumerate(tokens[c]):
            inc = combine_decay(combine_decay(carry[c], local_prefix[c][r]), Tt)
            nt, dt = readout(inc[:5], q[..., s0 + r, :], masked=masked, return_num_den=True)
            num[..., s0 + r, :] = nt
            den[..., s0 + r] = dt
    if return_num_den:
        res = (num, den)
    elif normalized:
        res = num / (den + eps)[..., None]
    else:
        res = num
    if return_final:
        final = combine_decay(carry[-1], summaries[-1]) if starts else E
        return res, final
    return res


def hla2_decay_den_scale(q, k, gamma, masked=True):
    """D_t = sum_{j<=t} |w_tj| with w_tj the weight of v_j in row t (den_t =
    sum_j w_tj): the scale a computed den_t is judged against where den_t
    itself is near zero.  Per head, [..., n]."""
    q, k = _f64(q), _f64(k)
    n = q.shape[-2]
    D = _decay_matrix(n, gamma)
    L = (D > 0).astype(np.float64)
    QK = q @ np.swapaxes(k, -1, -2)
    if masked:
        T2 = D * ((D * QK) @ np.swapaxes(L * QK, -1, -2))
    else:
        T2 = np.empty(q.shape[:-1] + (n,))
        for t in range(n):
            w = float(gamma) ** (t - np.arange(t + 1))
            a = QK[..., t, : t + 1] * w
            b = np.einsum('...i,...id->...d', a, k[..., : t + 1, :])
            T2[..., t, : t + 1] = np.einsum('...d,...jd->...j', b, q[..., : t + 1, :]) * w
            T2[..., t, t + 1:] = 0.0
    return np.abs(T2).sum(-1)
