"""Pins for the second-order oracle (CPU only).

Each test ties the oracle to something other than itself: the hand-worked
example, closed forms of special inputs, the streaming invariants recomputed
from scratch, brute force on tiny inputs, associativity, and planted
mistakes that these pins must catch.
"""
import os

import numpy as np
import pytest

from oracle import hla2 as H
from oracle import native

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape_q, dv, seed=0):
    rng = np.random.default_rng(seed)
    *b, n, d = shape_q
    q = rng.standard_normal(shape_q)
    k = rng.standard_normal(shape_q)
    v = rng.standard_normal(tuple(b) + (n, dv))
    return q, k, v


def _load_hand_example():
    rows = []
    with open(os.path.join(GOLDEN, "hla2_hand_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                left, right = line.split("|")
                rows.append((list(map(float, left.split())), list(map(float, right.split()))))
    q = np.array([r[0][1:3] for r in rows])
    k = np.array([r[0][3:5] for r in rows])
    v = np.array([[r[0][5]] for r in rows])
    exp = np.array([r[1] for r in rows])
    return q, k, v, exp


# --------------------------------------------------------------------- hand example
@pytest.mark.parametrize("impl", ["definition", "loops", "serial", "chunked", "c"])
def test_hand_example(impl):
    q, k, v, exp = _load_hand_example()
    for masked, cols in ((True, (0, 1)), (False, (2, 3))):
        if impl == "definition":
            num, den = H.hla2_definition(q, k, v, masked=masked, return_num_den=True)
        elif impl == "loops":
            num, den = H.hla2_definition_loops(q, k, v, masked=masked)
        elif impl == "serial":
            (num, den), _ = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
        elif impl == "chunked":
            num, den = H.hla2_chunked(q, k, v, 2, masked=masked, return_num_den=True)
        else:
            num, den, _, _ = native.hla2_serial_c(q, k, v, masked=masked)
        np.testing.assert_allclose(num[:, 0], exp[:, cols[0]], atol=1e-12)
        np.testing.assert_allclose(den, exp[:, cols[1]], atol=1e-12)


def test_hand_example_normalized():
    q, k, v, exp = _load_hand_example()
    eps = 0.25
    out, _ = H.hla2_serial(q, k, v, masked=True, normalized=True, eps=eps)
    np.testing.assert_allclose(out[:, 0], exp[:, 0] / (exp[:, 1] + eps), atol=1e-12)


# --------------------------------------------------------------------- brute force
@pytest.mark.parametrize("masked", [True, False])
def test_serial_matches_bruteforce_loops(masked):
    q, k, v = _rand((11, 4), 3, seed=1)
    num_l, den_l = H.hla2_definition_loops(q, k, v, masked=masked)
    (num_s, den_s), _ = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
    num_d, den_d = H.hla2_definition(q, k, v, masked=masked, return_num_den=True)
    np.testing.assert_allclose(num_s, num_l, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(den_s, den_l, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(num_d, num_l, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(den_d, den_l, rtol=1e-11, atol=1e-11)


def test_serial_matches_definition_batched():
    q, k, v = _rand((2, 3, 40, 8), 5, seed=2)
    for masked in (True, False):
        for normalized in (False, True):
            ref = H.hla2_definition(q, k, v, masked=masked, normalized=normalized, eps=0.5)
            out, _ = H.hla2_serial(q, k, v, masked=masked, normalized=normalized, eps=0.5)
            np.testing.assert_allclose(out, ref, rtol=1e-9, atol=1e-9)


# --------------------------------------------------------------------- invariants
def test_streaming_invariants_every_t():
    """Prefix summaries after each token equal their sums over i <= t (Sec. 3)."""
    q, k, v = _rand((9, 3), 2, seed=3)
    _, _, states = H.hla2_serial(q, k, v, return_states=True)
    n = q.shape[0]
    Cp = [np.zeros((3, 2))]          # C_{i} for i = 0..n
    mp = [np.zeros(3)]
    for i in range(n):
        Cp.append(Cp[-1] + np.outer(q[i], v[i]))
        mp.append(mp[-1] + q[i])
    for t in range(n):
        S, C, m, G, h = states[t]
        np.testing.assert_allclose(S, sum(np.outer(k[i], k[i]) for i in range(t + 1)), atol=1e-12)
        np.testing.assert_allclose(C, sum(np.outer(q[i], v[i]) for i in range(t + 1)), atol=1e-12)
        np.testing.assert_allclose(m, q[: t + 1].sum(0), atol=1e-12)
        np.testing.assert_allclose(G, sum(np.outer(k[i], k[i]) @ Cp[i] for i in range(t + 1)), atol=1e-12)
        np.testing.assert_allclose(h, sum(np.outer(k[i], k[i]) @ mp[i] for i in range(t + 1)), atol=1e-12)


# --------------------------------------------------------------------- scan equivalence
@pytest.mark.parametrize("masked", [True, False])
def test_chunked_equals_serial_every_chunk(masked):
    """Thm. 2: the two-level scan reproduces the serial recurrence for any chunk."""
    q, k, v = _rand((2, 13, 4), 3, seed=4)
    (ref_n, ref_d), ref_state = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
    for C in range(1, 15):
        (num, den), fin = H.hla2_chunked(q, k, v, C, masked=masked, return_num_den=True,
                                         return_final=True)
        np.testing.assert_allclose(num, ref_n, rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(den, ref_d, rtol=1e-10, atol=1e-10)
        for a, b in zip(fin, ref_state):
            np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)


def test_combine_associative_random():
    rng = np.random.default_rng(5)
    d, dv = 4, 3

    def rnd():
        return (rng.standard_normal((d, d)), rng.standard_normal((d, dv)), rng.standard_normal(d),
                rng.standard_normal((d, dv)), rng.standard_normal(d))

    for _ in range(5):
        A, B, C = rnd(), rnd(), rnd()
        l = H.combine(H.combine(A, B), C)
        r = H.combine(A, H.combine(B, C))
        for x, y in zip(l, r):
            np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-12)
    E = H.zero_state((), d, dv)
    A = rnd()
    for x, y in zip(H.combine(E, A), A):
        np.testing.assert_array_equal(x, y)
    for x, y in zip(H.combine(A, E), A):
        np.testing.assert_array_equal(x, y)


def test_phi_form_composition():
    """Eq. (semidirect) in the variables Phi = S C - G, eta = S m - h:
    Phi_{A(+)B} = Phi_A + Phi_B + S_A C_B and eta_{A(+)B} = eta_A + eta_B + S_A m_B
    (the form in which the fused path composes segments), on token segments."""
    q, k, v = _rand((2, 13, 4), 3, seed=41)
    A = H.segment_summary(q[:, :6], k[:, :6], v[:, :6])
    B = H.segment_summary(q[:, 6:], k[:, 6:], v[:, 6:])
    AB = H.combine(A, B)
    phi = lambda X: X[0] @ X[1] - X[3]
    eta = lambda X: np.einsum("...ij,...j->...i", X[0], X[2]) - X[4]
    np.testing.assert_allclose(phi(AB), phi(A) + phi(B) + A[0] @ B[1], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(eta(AB), eta(A) + eta(B) + np.einsum("...ij,...j->...i", A[0], B[2]),
                               rtol=1e-11, atol=1e-11)
    # Phi of a prefix state is sum_{j<=t} S_j q_j v_j^T (the proof of Thm. 1)
    _, fin = H.hla2_serial(q, k, v)
    direct = np.zeros_like(fin[1])
    S = np.zeros_like(fin[0])
    for t in range(q.shape[1]):
        S = S + np.einsum("...i,...j->...ij", k[:, t], k[:, t])
        direct += np.einsum("...i,...j->...ij", np.einsum("...ij,...j->...i", S, q[:, t]), v[:, t])
    np.testing.assert_allclose(phi(fin), direct, rtol=1e-11, atol=1e-11)


def test_segment_summary_equals_serial_state():
    q, k, v = _rand((3, 10, 5), 4, seed=6)
    summ = H.segment_summary(q, k, v)
    _, fin = H.hla2_serial(q, k, v)
    for a, b in zip(summ, fin):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-11)


def test_chunk_summaries_scan_total():
    q, k, v = _rand((2, 17, 4), 3, seed=7)
    sums = H.chunk_summaries(q, k, v, 5)
    pre, tot = H.exclusive_scan_states(sums)
    _, fin = H.hla2_serial(q, k, v)
    for a, b in zip(tot, fin):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-11)
    # prefix of chunk c equals the serial state after 5c tokens
    for c in range(pre[0].shape[1]):
        _, st = H.hla2_serial(q[:, :5 * c], k[:, :5 * c], v[:, :5 * c])
        for a, b in zip(pre, st):
            np.testing.assert_allclose(a[:, c], b, rtol=1e-11, atol=1e-11)


def test_blelloch_noncommutative():
    """The scan keeps operand order: string concatenation as the operator."""
    xs = list("abcdefg")
    assert H.blelloch_exclusive(xs, lambda a, b: a + b, "") == ["", "a", "ab", "abc", "abcd", "abcde", "abcdef"]


# --------------------------------------------------------------------- closed forms
@pytest.mark.parametrize("n", [1, 5, 12])
def test_constant_tokens_closed_form(n):
    """q_t = k_t = e, v_t = v: masked o_t = t(t+1)/2 v, unmasked o_t = t^2 v."""
    d, dv = 3, 2
    e = np.zeros(d); e[1] = 1.0
    vv = np.array([0.5, -2.0])
    q = np.tile(e, (n, 1)); k = q.copy(); v = np.tile(vv, (n, 1))
    t = np.arange(1, n + 1, dtype=np.float64)
    for fn in (lambda **kw: H.hla2_serial(q, k, v, return_num_den=True, **kw)[0],
               lambda **kw: H.hla2_definition(q, k, v, return_num_den=True, **kw)):
        num, den = fn(masked=True)
        np.testing.assert_allclose(num, np.outer(t * (t + 1) / 2, vv), atol=1e-12)
        np.testing.assert_allclose(den, t * (t + 1) / 2, atol=1e-12)
        num, den = fn(masked=False)
        np.testing.assert_allclose(num, np.outer(t * t, vv), atol=1e-12)
        np.testing.assert_allclose(den, t * t, atol=1e-12)


def test_one_hot_tokens():
    """q_t = k_t = e_t: only i = j = t survives, so o_t = v_t."""
    d = 6
    q = np.eye(d); k = np.eye(d)
    v = np.random.default_rng(8).standard_normal((d, 3))
    for masked in (True, False):
        out, _ = H.hla2_serial(q, k, v, masked=masked)
        np.testing.assert_allclose(out, v, atol=1e-12)
        np.testing.assert_allclose(H.hla2_definition(q, k, v, masked=masked), v, atol=1e-12)


def test_linear_attention_reduction():
    """S = I and C = G = 0 after d key-only tokens; afterwards k = 0, so the
    output is linear attention with kernel q_t.q_j (Sec. 3, connection with
    linear attention)."""
    d, dv, extra = 4, 3, 7
    rng = np.random.default_rng(9)
    q = np.concatenate([np.zeros((d, d)), rng.standard_normal((extra, d))])
    k = np.concatenate([np.eye(d), np.zeros((extra, d))])
    v = np.concatenate([np.zeros((d, dv)), rng.standard_normal((extra, dv))])
    out, _ = H.hla2_serial(q, k, v)
    Q, V = q[d:], v[d:]
    expect = np.tril(Q @ Q.T) @ V
    np.testing.assert_allclose(out[d:], expect, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out[:d], 0.0, atol=1e-15)


# --------------------------------------------------------------------- identities
def test_unmasked_minus_masked_is_qG():
    q, k, v = _rand((15, 4), 3, seed=10)
    om, _, states = H.hla2_serial(q, k, v, masked=True, return_states=True)
    ou, _ = H.hla2_serial(q, k, v, masked=False)
    for t in range(15):
        np.testing.assert_allclose(ou[t] - om[t], q[t] @ states[t][3], rtol=1e-10, atol=1e-10)


def test_den_is_output_with_unit_values():
    q, k, v = _rand((2, 14, 5), 3, seed=11)
    for masked in (True, False):
        (_, den), _ = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
        ones, _ = H.hla2_serial(q, k, np.ones(v.shape[:-1] + (1,)), masked=masked)
        np.testing.assert_allclose(den, ones[..., 0], rtol=1e-11, atol=1e-11)


def test_homogeneity():
    q, k, v = _rand((12, 4), 3, seed=12)
    a, b, c = 1.7, -0.6, 2.3
    o, _ = H.hla2_serial(q, k, v)
    o2, _ = H.hla2_serial(a * q, b * k, c * v)
    np.testing.assert_allclose(o2, a * a * b * b * c * o, rtol=1e-10, atol=1e-10)


def test_zero_token_padding_is_exact():
    q, k, v = _rand((10, 4), 3, seed=13)
    z4, z3 = np.zeros((5, 4)), np.zeros((5, 3))
    o, st = H.hla2_serial(q, k, v)
    op, stp = H.hla2_serial(np.concatenate([z4, q, z4]), np.concatenate([z4, k, z4]),
                            np.concatenate([z3, v, z3]))
    np.testing.assert_allclose(op[5:15], o, atol=1e-12)
    np.testing.assert_array_equal(op[:5], 0.0)
    for a_, b_ in zip(st, stp):
        np.testing.assert_allclose(a_, b_, atol=1e-12)


def test_serial_resume_from_state():
    """Running n1 tokens, then continuing from the state, equals one run."""
    q, k, v = _rand((2, 20, 4), 3, seed=14)
    full, fin = H.hla2_serial(q, k, v)
    a, st = H.hla2_serial(q[:, :7], k[:, :7], v[:, :7])
    b, fin2 = H.hla2_serial(q[:, 7:], k[:, 7:], v[:, 7:], state=st)
    np.testing.assert_allclose(np.concatenate([a, b], axis=1), full, rtol=1e-11, atol=1e-11)
    for x, y in zip(fin, fin2):
        np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-11)


# --------------------------------------------------------------------- C oracle
def test_c_oracle_matches_numpy():
    q, k, v = _rand((3, 2, 33, 8), 6, seed=15)
    for masked in (True, False):
        (num, den), fin = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
        cn, cd, cfin, used = native.hla2_serial_c(q, k, v, masked=masked, threads=3)
        assert used >= 1
        np.testing.assert_allclose(cn, num, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(cd, den, rtol=1e-12, atol=1e-12)
        for a, b in zip(cfin, fin):
            np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_c_oracle_resume():
    q, k, v = _rand((4, 30, 5), 4, seed=16)
    full, _, _, _ = native.hla2_serial_c(q, k, v)
    a, _, st, _ = native.hla2_serial_c(q[:, :11], k[:, :11], v[:, :11])
    b, _, _, _ = native.hla2_serial_c(q[:, 11:], k[:, 11:], v[:, 11:], state=st)
    np.testing.assert_allclose(np.concatenate([a, b], axis=1), full, rtol=1e-11, atol=1e-11)


# --------------------------------------------------------------------- planted mistakes
def test_pins_catch_dropped_cross_term(monkeypatch):
    q, k, v = _rand((9, 3), 2, seed=17)
    ref, _ = H.hla2_serial(q, k, v)

    def bad(A, B):
        SA, CA, mA, GA, hA = A
        SB, CB, mB, GB, hB = B
        return (SA + SB, CA + CB, mA + mB, GA + GB, hA + hB)

    monkeypatch.setattr(H, "combine", bad)
    out = H.hla2_chunked(q, k, v, 3)
    assert np.abs(out - ref).max() > 1e-3


def test_pins_catch_swapped_cross_term(monkeypatch):
    q, k, v = _rand((9, 3), 2, seed=18)
    ref, _ = H.hla2_serial(q, k, v)
    orig = H.combine

    def bad(A, B):
        SA, CA, mA, GA, hA = A
        SB, CB, mB, GB, hB = B
        return (SA + SB, CA + CB, mA + mB, GA + GB + SA @ CB, hA + hB + SA @ mB)

    monkeypatch.setattr(H, "combine", bad)
    out = H.hla2_chunked(q, k, v, 3)
    monkeypatch.setattr(H, "combine", orig)
    assert np.abs(out - ref).max() > 1e-3


def test_pins_catch_wrong_update_order():
    """Updating G with the new C_t instead of C_{t-1} breaks the hand example."""
    q, k, v, exp = _load_hand_example()
    S = np.zeros((2, 2)); C = np.zeros((2, 1)); G = np.zeros((2, 1))
    out = []
    for t in range(3):
        S = S + np.outer(k[t], k[t]); C = C + np.outer(q[t], v[t])
        G = G + np.outer(k[t], k[t]) @ C          # planted mistake
        out.append(float((q[t] @ (S @ C - G))[0]))
    assert np.abs(np.array(out) - exp[:, 0]).max() > 0.5


def test_pins_catch_mask_without_diagonal():
    """A strictly-lower mask would give o_1 = 0 in the constant-token case."""
    n = 4
    q = np.ones((n, 1)); k = np.ones((n, 1)); v = np.ones((n, 1))
    L = np.tril(np.ones((n, n)), -1)
    W = L * (q @ k.T)
    bad = ((W @ W.T) * L) @ v
    t = np.arange(1, n + 1)
    assert np.abs(bad[:, 0] - t * (t + 1) / 2).max() >= 1


def test_den_scale_bounds_den():
    q, k, v = _rand((2, 30, 4), 3, seed=19)
    for masked in (True, False):
        (_, den), _ = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
        D = H.hla2_den_scale(q, k, masked=masked)
        assert np.all(np.abs(den) <= D * (1 + 1e-12))
        # with q = k the diagonal term q_t^T S_t q_t >= 0 and all terms of t=1 coincide
        np.testing.assert_allclose(D[..., 0], np.abs(den[..., 0]), rtol=1e-12)
