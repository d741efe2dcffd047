"""Pins for the AHLA oracle (CPU only).

The streaming recurrence, the (+)_AHLA concatenation and the chunked scan are
pinned by a hand-worked example, brute force over the double sum, closed forms
of special inputs (constant tokens, orthonormal tokens), associativity, and
planted mistakes that each pin must catch.
"""
import os

import numpy as np
import pytest

from oracle import ahla as A
from oracle import native

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(b, n, d, dv, seed=0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(b + (n, d)), rng.standard_normal(b + (n, d)), rng.standard_normal(b + (n, dv)))


def _load_hand_example():
    rows = []
    with open(os.path.join(GOLDEN, "ahla_hand_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                left, right = line.split("|")
                rows.append((list(map(float, left.split())), list(map(float, right.split()))))
    q = np.array([[r[0][1]] for r in rows])
    k = np.array([[r[0][2]] for r in rows])
    v = np.array([[r[0][3]] for r in rows])
    return q, k, v, np.array([r[1] for r in rows])


def _run(impl, q, k, v, chunk=2):
    if impl == "loops":
        return A.ahla_definition_loops(q, k, v)
    if impl == "definition":
        return A.ahla_definition(q, k, v, return_num_den=True)
    if impl == "serial":
        return A.ahla_serial(q, k, v, return_num_den=True)[0]
    if impl == "chunked":
        return A.ahla_chunked(q, k, v, chunk, return_num_den=True)
    num, den, _ = native.ahla_serial_c(q, k, v)
    return num, den


IMPLS = ["loops", "definition", "serial", "chunked", "c"]


@pytest.mark.parametrize("impl", IMPLS)
def test_hand_example(impl):
    q, k, v, exp = _load_hand_example()
    num, den = _run(impl, q, k, v)
    np.testing.assert_allclose(num[:, 0], exp[:, 0], atol=1e-12)
    np.testing.assert_allclose(den, exp[:, 1], atol=1e-12)


@pytest.mark.parametrize("impl", IMPLS[1:])
def test_matches_bruteforce_loops(impl):
    q, k, v = _rand((), 11, 3, 2, seed=1)
    n0, d0 = A.ahla_definition_loops(q, k, v)
    num, den = _run(impl, q, k, v, chunk=4)
    np.testing.assert_allclose(num, n0, atol=1e-11)
    np.testing.assert_allclose(den, d0, atol=1e-11)


@pytest.mark.parametrize("chunk", [1, 2, 3, 4, 8, 13, 32])
def test_chunked_matches_serial(chunk):
    q, k, v = _rand((2,), 13, 4, 3, seed=2)
    (n1, d1), f1 = A.ahla_serial(q, k, v, return_num_den=True)
    (n2, d2), f2 = A.ahla_chunked(q, k, v, chunk, return_num_den=True, return_final=True)
    np.testing.assert_allclose(n2, n1, atol=1e-10)
    np.testing.assert_allclose(d2, d1, atol=1e-10)
    for a, b in zip(f2[1:], f1):                       # (P, m, E, n) of the whole sequence
        np.testing.assert_allclose(a, b, atol=1e-10)


def test_constant_tokens_closed_form():
    # q_t = k_t = e_1: A is the all-ones lower triangle, (A A)_{t,j} = t - j + 1,
    # so den_t = (t+1)(t+2)/2 and num_t = sum_j (t - j + 1) v_j.
    n, d = 10, 3
    q = np.zeros((n, d))
    q[:, 0] = 1.0
    v = np.random.default_rng(3).standard_normal((n, 2))
    t = np.arange(n)
    exp_den = (t + 1) * (t + 2) / 2
    exp_num = np.stack([((tt - np.arange(tt + 1) + 1)[:, None] * v[: tt + 1]).sum(0) for tt in range(n)])
    for impl in IMPLS:
        num, den = _run(impl, q, q.copy(), v, chunk=3)
        np.testing.assert_allclose(den, exp_den, atol=1e-12)
        np.testing.assert_allclose(num, exp_num, atol=1e-12)


def test_orthonormal_tokens_give_identity():
    # q_t = k_t = e_t with n <= d: A = I, so o_t = v_t and den_t = 1.
    n = d = 6
    q = np.eye(n)
    v = np.random.default_rng(4).standard_normal((n, 3))
    for impl in IMPLS:
        num, den = _run(impl, q, q.copy(), v, chunk=4)
        np.testing.assert_allclose(num, v, atol=1e-12)
        np.testing.assert_allclose(den, np.ones(n), atol=1e-12)


def test_shifted_orthonormal_tokens():
    # k_t = e_t, q_t = e_t + e_{t-1}: A has ones on the diagonal and the first
    # sub-diagonal, so A A has 1, 2, 1 on the diagonal and the first two
    # sub-diagonals: o_t = v_t + 2 v_{t-1} + v_{t-2}.
    n = d = 7
    k = np.eye(n)
    q = np.eye(n) + np.eye(n, k=-1)
    v = np.random.default_rng(5).standard_normal((n, 2))
    exp = v.copy()
    exp[1:] += 2 * v[:-1]
    exp[2:] += v[:-2]
    for impl in IMPLS:
        num, _ = _run(impl, q, k, v, chunk=3)
        np.testing.assert_allclose(num, exp, atol=1e-12)


def test_concatenation_is_associative():
    rng = np.random.default_rng(6)
    d, dv = 3, 2
    segs = [A.segment_summary_ahla(*(rng.standard_normal((m, x)) for x in (d, d, dv))) for m in (2, 3, 4)]
    left = A.combine_ahla(A.combine_ahla(segs[0], segs[1]), segs[2])
    right = A.combine_ahla(segs[0], A.combine_ahla(segs[1], segs[2]))
    for a, b in zip(left, right):
        np.testing.assert_allclose(a, b, atol=1e-11)
    ident = A.zero_state_ahla((), d, dv)
    for a, b in zip(A.combine_ahla(ident, segs[0]), segs[0]):
        np.testing.assert_allclose(a, b, atol=0)
    for a, b in zip(A.combine_ahla(segs[0], ident), segs[0]):
        np.testing.assert_allclose(a, b, atol=0)


def test_segment_summary_matches_serial_state():
    q, k, v = _rand((), 9, 3, 2, seed=7)
    _, (P, m, E, nn) = A.ahla_serial(q, k, v)
    R, P2, m2, E2, n2 = A.segment_summary_ahla(q, k, v)
    np.testing.assert_allclose(R, k.T @ q, atol=1e-12)
    for a, b in ((P2, P), (m2, m), (E2, E), (n2, nn)):
        np.testing.assert_allclose(a, b, atol=1e-11)


def test_normalized_is_num_over_den():
    q, k, v = _rand((2,), 8, 3, 2, seed=8)
    num, den = A.ahla_definition(q, k, v, return_num_den=True)
    for out in (A.ahla_definition(q, k, v, normalized=True, eps=1e-3),
                A.ahla_serial(q, k, v, normalized=True, eps=1e-3)[0],
                A.ahla_chunked(q, k, v, 3, normalized=True, eps=1e-3)):
        np.testing.assert_allclose(out, num / (den + 1e-3)[..., None], atol=1e-10)


def test_den_scale_bounds_den():
    q, k, v = _rand((), 12, 4, 2, seed=9)
    _, den = A.ahla_definition(q, k, v, return_num_den=True)
    sc = A.ahla_den_scale(q, k)
    assert np.all(np.abs(den) <= sc + 1e-12)
    qc = np.zeros((5, 2)); qc[:, 0] = 1.0
    np.testing.assert_allclose(A.ahla_den_scale(qc, qc), (np.arange(5) + 1) * (np.arange(5) + 2) / 2)


def test_c_twin_matches_numpy_on_heads():
    q, k, v = _rand((3, 2), 21, 5, 4, seed=10)
    (n1, d1), _ = A.ahla_serial(q, k, v, return_num_den=True)
    n2, d2, used = native.ahla_serial_c(q, k, v, threads=2)
    assert used >= 1
    np.testing.assert_allclose(n2, n1, atol=1e-10)
    np.testing.assert_allclose(d2, d1, atol=1e-10)


# ----------------------------------------------------------------- planted mistakes

def _serial_with_prefix_before_t(q, k, v):
    """E built from P_{t-1} (the carry without token t)."""
    d, dv = q.shape[1], v.shape[1]
    P = np.zeros((d, dv)); E = np.zeros((d, dv))
    out = np.empty((q.shape[0], dv))
    for t in range(q.shape[0]):
        E = E + np.outer(k[t], q[t] @ P)
        P = P + np.outer(k[t], v[t])
        out[t] = q[t] @ E
    return out


def _combine_without_cross(Aa, Bb):
    RA, PA, mA, EA, nA = Aa
    RB, PB, mB, EB, nB = Bb
    return (RA + RB, PA + PB, mA + mB, EA + EB, nA + nB)


def _combine_transposed_cross(Aa, Bb):
    RA, PA, mA, EA, nA = Aa
    RB, PB, mB, EB, nB = Bb
    return (RA + RB, PA + PB, mA + mB, EA + EB + RB.T @ PA, nA + nB + RB.T @ mA)


def test_planted_prefix_before_t_fails_hand_example():
    q, k, v, exp = _load_hand_example()
    assert not np.allclose(_serial_with_prefix_before_t(q, k, v)[:, 0], exp[:, 0])


@pytest.mark.parametrize("bad", [_combine_without_cross, _combine_transposed_cross])
def test_planted_concatenation_mistakes_fail(monkeypatch, bad):
    q, k, v = _rand((), 9, 3, 2, seed=11)
    n0, _ = A.ahla_definition_loops(q, k, v)
    monkeypatch.setattr(A, "combine_ahla", bad)
    num = A.ahla_chunked(q, k, v, 3)
    assert not np.allclose(num, n0, atol=1e-6)
