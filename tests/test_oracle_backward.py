"""Pins for the written-out gradients of the masked second-order HLA (CPU).

The reverse-scan VJP of oracle.hla2_backward is checked against torch
autograd through the dense definition, central finite differences, a
hand-worked example, the single-token closed form, Euler's identities for the
homogeneous loss, and planted mistakes that each pin must catch."""
import os

import numpy as np
import pytest

from oracle import hla2_backward as B

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape_b, n, d, dv, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape_b + (n, d)), rng.standard_normal(shape_b + (n, d)),
            rng.standard_normal(shape_b + (n, dv)), rng.standard_normal(shape_b + (n, dv)))


def _hand():
    rows = []
    with open(os.path.join(GOLDEN, "hla2_backward_hand_example.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                left, right = line.split("|")
                rows.append((list(map(float, left.split())), list(map(float, right.split()))))
    col = lambda i: np.array([[r[0][i]] for r in rows])
    return col(1), col(2), col(3), col(4), np.array([r[1] for r in rows])


@pytest.mark.parametrize("impl", ["serial", "autograd"])
def test_hand_example(impl):
    q, k, v, g, exp = _hand()
    f = B.hla2_vjp_serial if impl == "serial" else B.hla2_vjp_autograd
    dq, dk, dv = f(q, k, v, g)
    np.testing.assert_allclose(dq[:, 0], exp[:, 0], atol=1e-12)
    np.testing.assert_allclose(dk[:, 0], exp[:, 1], atol=1e-12)
    np.testing.assert_allclose(dv[:, 0], exp[:, 2], atol=1e-12)
    assert abs(B.hla2_loss(q, k, v, g) - 19.0) < 1e-12


@pytest.mark.parametrize("n,d,dv", [(1, 3, 2), (7, 3, 2), (13, 4, 5), (20, 2, 3)])
def test_serial_matches_autograd(n, d, dv):
    q, k, v, g = _rand((2,), n, d, dv, seed=n + d)
    for a, b in zip(B.hla2_vjp_serial(q, k, v, g), B.hla2_vjp_autograd(q, k, v, g)):
        np.testing.assert_allclose(a, b, atol=1e-10, rtol=1e-10)


def test_finite_differences():
    q, k, v, g = _rand((), 5, 2, 2, seed=3)
    grads = B.hla2_vjp_serial(q, k, v, g)
    h = 1e-5
    for which, grad in zip(range(3), grads):
        base = [q, k, v]
        for idx in np.ndindex(base[which].shape):
            plus = [x.copy() for x in base]
            minus = [x.copy() for x in base]
            plus[which][idx] += h
            minus[which][idx] -= h
            fd = (B.hla2_loss(*plus, g) - B.hla2_loss(*minus, g)) / (2 * h)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (which, idx, fd, grad[idx])


def test_single_token_closed_form():
    # n = 1: o = (q.k)^2 v, so dq = 2 (q.k)(g.v) k, dk = 2 (q.k)(g.v) q, dv = (q.k)^2 g
    q, k, v, g = _rand((), 1, 4, 3, seed=4)
    qk, gv = float(q[0] @ k[0]), float(g[0] @ v[0])
    dq, dk, dv = B.hla2_vjp_serial(q, k, v, g)
    np.testing.assert_allclose(dq[0], 2 * qk * gv * k[0], atol=1e-12)
    np.testing.assert_allclose(dk[0], 2 * qk * gv * q[0], atol=1e-12)
    np.testing.assert_allclose(dv[0], qk * qk * g[0], atol=1e-12)


def test_euler_identities():
    # L is homogeneous of degree 2 in q, 2 in k and 1 in v
    q, k, v, g = _rand((3,), 17, 4, 3, seed=5)
    dq, dk, dv = B.hla2_vjp_serial(q, k, v, g)
    L = B.hla2_loss(q, k, v, g)
    assert abs((q * dq).sum() - 2 * L) < 1e-9 * max(1, abs(L))
    assert abs((k * dk).sum() - 2 * L) < 1e-9 * max(1, abs(L))
    assert abs((v * dv).sum() - L) < 1e-9 * max(1, abs(L))


def test_linear_in_upstream_gradient():
    q, k, v, g = _rand((), 9, 3, 3, seed=6)
    g2 = np.random.default_rng(7).standard_normal(g.shape)
    a = B.hla2_vjp_serial(q, k, v, g)
    b = B.hla2_vjp_serial(q, k, v, g2)
    c = B.hla2_vjp_serial(q, k, v, 2.0 * g - 3.0 * g2)
    for x, y, z in zip(a, b, c):
        np.testing.assert_allclose(z, 2.0 * x - 3.0 * y, atol=1e-10)


# ----------------------------------------------------------------- planted mistakes

def _vjp_variant(q, k, v, g, strict_u=False, no_zt=False, no_su=False):
    """hla2_vjp_serial with one planted mistake (single head)."""
    n, d = q.shape
    u = np.zeros((n, d))
    U = np.zeros((d, v.shape[1]))
    for j in range(n - 1, -1, -1):
        if strict_u:
            u[j] = U @ v[j]
        U = U + np.outer(q[j], g[j])
        if not strict_u:
            u[j] = U @ v[j]
    S = np.zeros((d, d)); Phi = np.zeros((d, v.shape[1])); r = np.zeros((n, d)); dq = np.zeros((n, d))
    for j in range(n):
        S = S + np.outer(k[j], k[j]); r[j] = S @ q[j]; Phi = Phi + np.outer(r[j], v[j])
        dq[j] = Phi @ g[j] + (0 if no_su else S @ u[j])
    U = np.zeros((d, v.shape[1])); Z = np.zeros((d, d)); dk = np.zeros((n, d)); dv = np.zeros_like(v)
    for j in range(n - 1, -1, -1):
        U = U + np.outer(q[j], g[j]); dv[j] = U.T @ r[j]
        Z = Z + np.outer(u[j], q[j]); dk[j] = (Z if no_zt else Z + Z.T) @ k[j]
    return dq, dk, dv


def test_variant_without_mistake_is_the_serial_form():
    q, k, v, g = _rand((), 6, 3, 2, seed=8)
    for a, b in zip(_vjp_variant(q, k, v, g), B.hla2_vjp_serial(q, k, v, g)):
        np.testing.assert_allclose(a, b, atol=1e-12)


@pytest.mark.parametrize("mistake", ["strict_u", "no_zt", "no_su"])
def test_planted_mistakes_fail_the_pins(mistake):
    q, k, v, g, exp = _hand()
    got = _vjp_variant(q, k, v, g, **{mistake: True})
    ok_hand = all(np.allclose(x[:, 0], exp[:, i]) for i, x in enumerate(got))
    q2, k2, v2, g2 = _rand((), 7, 3, 2, seed=9)
    ref = B.hla2_vjp_autograd(q2, k2, v2, g2)
    got2 = _vjp_variant(q2, k2, v2, g2, **{mistake: True})
    ok_rand = all(np.allclose(a, b, atol=1e-8) for a, b in zip(got2, ref))
    assert not (ok_hand and ok_rand)
    assert not ok_rand
