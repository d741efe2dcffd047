"""Pins for the decayed second-order oracle (CPU only).

The reading of the decay section (module header of oracle.hla2_decay) is
pinned by a hand-worked example, the gamma = 1 reduction to the undecayed
oracle, brute force, closed forms of special inputs, associativity of the
decayed concatenation (and the failure of the printed rho_B G_A form), the
chunked scan against the serial recurrence, and planted mistakes.
"""
import os

import numpy as np
import pytest

from oracle import hla2 as H
from oracle import hla2_decay as D
from oracle import native

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
GAMMAS = [0.5, 0.9, 0.99, 1.0]


def _rand(b, n, d, dv, seed=0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(b + (n, d)), rng.standard_normal(b + (n, d)), rng.standard_normal(b + (n, dv)))


def _load_hand_example():
    rows = []
    with open(os.path.join(GOLDEN, "hla2_decay_hand_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                left, right = line.split("|")
                rows.append((list(map(float, left.split())), list(map(float, right.split()))))
    q = np.array([[r[0][1]] for r in rows])
    k = np.array([[r[0][2]] for r in rows])
    v = np.array([[r[0][3]] for r in rows])
    return q, k, v, np.array([r[1] for r in rows])


@pytest.mark.parametrize("impl", ["loops", "definition", "serial", "chunked", "c"])
def test_hand_example(impl):
    q, k, v, exp = _load_hand_example()
    for masked, cols in ((True, (0, 1)), (False, (2, 3))):
        if impl == "loops":
            num, den = D.hla2_decay_definition_loops(q, k, v, 0.5, masked=masked)
        elif impl == "definition":
            num, den = D.hla2_decay_definition(q, k, v, 0.5, masked=masked, return_num_den=True)
        elif impl == "serial":
            (num, den), _ = D.hla2_decay_serial(q, k, v, 0.5, masked=masked, return_num_den=True)
        elif impl == "chunked":
            num, den = D.hla2_decay_chunked(q, k, v, 0.5, 2, masked=masked, return_num_den=True)
        else:
            num, den, _, _ = native.hla2_decay_serial_c(q, k, v, 0.5, masked=masked)
        np.testing.assert_allclose(num[:, 0], exp[:, cols[0]], atol=1e-12)
        np.testing.assert_allclose(den, exp[:, cols[1]], atol=1e-12)


@pytest.mark.parametrize("masked", [True, False])
@pytest.mark.parametrize("gamma", GAMMAS)
def test_serial_matches_bruteforce_loops(masked, gamma):
    q, k, v = _rand((), 9, 3, 2, seed=1)
    n1, d1 = D.hla2_decay_definition_loops(q, k, v, gamma, masked=masked)
    (n2, d2), _ = D.hla2_decay_serial(q, k, v, gamma, masked=masked, return_num_den=True)
    n3, d3 = D.hla2_decay_definition(q, k, v, gamma, masked=masked, return_num_den=True)
    np.testing.assert_allclose(n2, n1, atol=1e-11)
    np.testing.assert_allclose(d2, d1, atol=1e-11)
    np.testing.assert_allclose(n3, n1, atol=1e-11)
    np.testing.assert_allclose(d3, d1, atol=1e-11)


@pytest.mark.parametrize("masked", [True, False])
def test_gamma_one_is_undecayed(masked):
    q, k, v = _rand((2,), 17, 4, 3, seed=2)
    (n1, d1), f1 = D.hla2_decay_serial(q, k, v, 1.0, masked=masked, return_num_den=True)
    (n2, d2), f2 = H.hla2_serial(q, k, v, masked=masked, return_num_den=True)
    np.testing.assert_allclose(n1, n2, atol=1e-11)
    np.testing.assert_allclose(d1, d2, atol=1e-11)
    for a, b in zip(f1, f2):
        np.testing.assert_allclose(a, b, atol=1e-11)


def test_state_definitions_every_t():
    """Each inclusive state equals its decayed sum recomputed from scratch."""
    g = 0.8
    q, k, v = _rand((), 8, 3, 2, seed=3)
    _, _, states = D.hla2_decay_serial(q, k, v, g, return_states=True)
    for t, (S, C, m, G, h) in enumerate(states):
        w = g ** (t - np.arange(t + 1))
        np.testing.assert_allclose(S, np.einsum('i,ia,ib->ab', w, k[:t + 1], k[:t + 1]), atol=1e-12)
        np.testing.assert_allclose(C, np.einsum('i,ia,ib->ab', w, q[:t + 1], v[:t + 1]), atol=1e-12)
        np.testing.assert_allclose(m, np.einsum('i,ia->a', w, q[:t + 1]), atol=1e-12)
        Gr = np.zeros_like(G)
        hr = np.zeros_like(h)
        for i in range(t + 1):
            for j in range(i):                      # pairs j < i at weight g^{(t-i)+(t-j)}
                Gr += g ** ((t - i) + (t - j)) * np.outer(k[i], k[i]) @ np.outer(q[j], v[j])
                hr += g ** ((t - i) + (t - j)) * np.outer(k[i], k[i]) @ q[j]
        np.testing.assert_allclose(G, Gr, atol=1e-12)
        np.testing.assert_allclose(h, hr, atol=1e-12)
        # the corrected state Phi = S C - G obeys Phi_t = g^2 Phi_{t-1} + S_t q_t v_t^T
        if t > 0:
            Sp, Cp, _, Gp, _ = states[t - 1]
            np.testing.assert_allclose(S @ C - G, g * g * (Sp @ Cp - Gp) + np.outer(S @ q[t], v[t]), atol=1e-12)


@pytest.mark.parametrize("masked", [True, False])
@pytest.mark.parametrize("gamma", [0.5, 0.93])
def test_chunked_equals_serial_every_chunk(masked, gamma):
    q, k, v = _rand((2,), 11, 3, 2, seed=4)
    (n0, d0), f0 = D.hla2_decay_serial(q, k, v, gamma, masked=masked, return_num_den=True)
    for chunk in range(1, 12):
        (n1, d1), f1 = D.hla2_decay_chunked(q, k, v, gamma, chunk, masked=masked, return_num_den=True,
                                            return_final=True)
        np.testing.assert_allclose(n1, n0, atol=1e-11)
        np.testing.assert_allclose(d1, d0, atol=1e-11)
        for a, b in zip(f1[:5], f0):
            np.testing.assert_allclose(a, b, atol=1e-11)
        np.testing.assert_allclose(f1[5], gamma ** 11)


def _rand_seg(rng, d, dv, rho):
    return (rng.standard_normal((d, d)), rng.standard_normal((d, dv)), rng.standard_normal(d),
            rng.standard_normal((d, dv)), rng.standard_normal(d), np.array(rho))


def test_combine_associative_and_identity():
    rng = np.random.default_rng(5)
    A, B, Cs = (_rand_seg(rng, 3, 2, r) for r in (0.7, 0.4, 0.9))
    left = D.combine_decay(D.combine_decay(A, B), Cs)
    right = D.combine_decay(A, D.combine_decay(B, Cs))
    for x, y in zip(left, right):
        np.testing.assert_allclose(x, y, atol=1e-12)
    E = D.zero_state_decay((), 3, 2)
    for x, y in zip(D.combine_decay(E, A), A):
        np.testing.assert_allclose(x, y, atol=1e-15)
    for x, y in zip(D.combine_decay(A, E), A):
        np.testing.assert_allclose(x, y, atol=1e-15)


def test_printed_rho_form_is_not_associative():
    """The printed concatenation scales G_A by rho_B (not rho_B^2); expanding
    (A+B)+C against A+(B+C) gives different S_B C_A coefficients, which is why
    this oracle reads the squared form."""
    def printed(A, B):
        SA, CA, mA, GA, hA, rA = A
        SB, CB, mB, GB, hB, rB = B
        return (rB * SA + SB, rB * CA + CB, rB * mA + mB, rB * GA + GB + SB @ (rB * CA),
                rB * hA + hB + SB @ (rB * mA), rA * rB)
    rng = np.random.default_rng(6)
    A, B, Cs = (_rand_seg(rng, 3, 2, r) for r in (0.7, 0.4, 0.9))
    left = printed(printed(A, B), Cs)
    right = printed(A, printed(B, Cs))
    assert np.abs(left[3] - right[3]).max() > 1e-3


def test_constant_tokens_closed_form():
    """q_t = k_t = e_1, v_t = 1: masked o_t = sum_{j<=t} sum_{i<=j} g^{2t-i-j}
    = sum_{j<=t} g^{t-j} g^{t-j} (1 - g^{j+1}) / (1 - g)."""
    g, n = 0.7, 12
    q = np.zeros((n, 2)); q[:, 0] = 1.0
    v = np.ones((n, 1))
    (num, den), _ = D.hla2_decay_serial(q, q, v, g, return_num_den=True)
    for t in range(n):
        exp = sum(g ** (2 * (t - j)) * (1 - g ** (j + 1)) / (1 - g) for j in range(t + 1))
        assert abs(num[t, 0] - exp) < 1e-12 and abs(den[t] - exp) < 1e-12
    # unmasked: (sum_{i<=t} g^{t-i})^2
    (num, _), _ = D.hla2_decay_serial(q, q, v, g, masked=False, return_num_den=True)
    for t in range(n):
        assert abs(num[t, 0] - ((1 - g ** (t + 1)) / (1 - g)) ** 2) < 1e-12


def test_one_hot_tokens():
    """Orthonormal q_t = k_t = e_t: only i = j = t survives, weight g^0: o_t = v_t."""
    n = 6
    e = np.eye(n)
    v = np.random.default_rng(7).standard_normal((n, 3))
    for g in (0.3, 0.9):
        out, _ = D.hla2_decay_serial(e, e, v, g)
        np.testing.assert_allclose(out, v, atol=1e-13)


def test_c_oracle_matches_numpy():
    q, k, v = _rand((2, 3), 40, 5, 4, seed=8)
    for masked in (True, False):
        (n1, d1), f1 = D.hla2_decay_serial(q, k, v, 0.95, masked=masked, return_num_den=True)
        n2, d2, f2, _ = native.hla2_decay_serial_c(q, k, v, 0.95, masked=masked)
        np.testing.assert_allclose(n2, n1, atol=1e-10)
        np.testing.assert_allclose(d2, d1, atol=1e-10)
        for a, b in zip(f2, f1):
            np.testing.assert_allclose(a, b, atol=1e-10)


def test_resume_from_state():
    q, k, v = _rand((2,), 20, 3, 2, seed=9)
    full, _ = D.hla2_decay_serial(q, k, v, 0.8)
    a, st = D.hla2_decay_serial(q[:, :7], k[:, :7], v[:, :7], 0.8)
    b, _ = D.hla2_decay_serial(q[:, 7:], k[:, 7:], v[:, 7:], 0.8, state=st)
    np.testing.assert_allclose(np.concatenate([a, b], axis=1), full, atol=1e-11)
    n1, _, _, _ = native.hla2_decay_serial_c(q[:, 7:], k[:, 7:], v[:, 7:], 0.8, state=st)
    np.testing.assert_allclose(n1, full[:, 7:], atol=1e-11)


def test_den_scale_bounds_den():
    q, k, v = _rand((2,), 15, 3, 2, seed=10)
    for masked in (True, False):
        (num, den), _ = D.hla2_decay_serial(q, k, v, 0.85, masked=masked, return_num_den=True)
        Ds = D.hla2_decay_den_scale(q, k, 0.85, masked=masked)
        assert np.all(np.abs(den) <= Ds * (1 + 1e-12) + 1e-12)


def test_printed_cross_summary_is_another_operator(monkeypatch):
    """The decay section prints the cross-summary update G_t = g G_{t-1} +
    k (k^T C_{t-1}).  With the printed decayed moments that recurrence gives an
    operator other than the one this build reads (pair (i, j) weighted by
    g^((t-i)+(t-j)), whose masked output drops exactly the pairs j < i of the
    decayed unmasked output).  This test pins the reading: it records that
    the two differ, so the oracle's choice is visible, and that the oracle
    follows the reading's double sum (the brute-force definition)."""
    q, k, v = _rand((), 8, 3, 2, seed=11)
    g = 0.8
    ref, _ = D.hla2_decay_definition_loops(q, k, v, g)
    S = np.zeros((3, 3)); C = np.zeros((3, 2)); G = np.zeros((3, 2))
    out = np.zeros((8, 2))
    for t in range(8):
        G = g * G + np.outer(k[t], k[t] @ C)
        S = g * S + np.outer(k[t], k[t])
        C = g * C + np.outer(q[t], v[t])
        out[t] = q[t] @ (S @ C - G)
    assert np.abs(out - ref).max() > 1e-3


def test_pins_catch_single_rho_on_g(monkeypatch):
    """Planted mistake: rho_B instead of rho_B^2 on G_A must fail chunked == serial."""
    q, k, v = _rand((2,), 9, 3, 2, seed=12)
    ref, _ = D.hla2_decay_serial(q, k, v, 0.7)
    good = D.combine_decay

    def bad(A, B):
        out = list(good(A, B))
        rB = B[5][..., None, None]
        out[3] = out[3] - rB * rB * A[3] + rB * A[3]
        return tuple(out)
    monkeypatch.setattr(D, "combine_decay", bad)
    got = D.hla2_decay_chunked(q, k, v, 0.7, 3)
    assert np.abs(got - ref).max() > 1e-6
