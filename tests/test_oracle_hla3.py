"""Pins of the third-order oracle against things other than itself (Sec. 7):
brute force over the index set of Thm. 3, the streaming recurrence, the
corrected recurrence, Alg. 4 for every chunk size, associativity of (x)_3,
closed forms and algebraic identities, and planted mistakes."""
import numpy as np
import pytest

from oracle import hla3 as H
from oracle import native


def _rand(n, d, dv, seed=0, batch=()):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(batch + (n, d)), rng.standard_normal(batch + (n, d)),
            rng.standard_normal(batch + (n, dv)))


def _tri_count(t):
    """|index set| at row t (1-based): triples in [1, t]^3 whose maximum is
    attained at least twice = t^3 - 3 sum_{m<=t} (m-1)^2."""
    return t ** 3 - t * (t - 1) * (2 * t - 1) // 2


def test_index_set_small_rows():
    """Row 2 sums exactly (1,1,1), (1,2,2), (2,1,2), (2,2,1), (2,2,2) (0-based here)."""
    got = {(i, u, j) for i in range(2) for u in range(2) for j in range(2) if H.in_index_set(i, u, j, 1)}
    assert got == {(0, 0, 0), (0, 1, 1), (1, 0, 1), (1, 1, 0), (1, 1, 1)}
    for t in range(1, 7):
        cnt = sum(H.in_index_set(i, u, j, t - 1) for i in range(t) for u in range(t) for j in range(t))
        assert cnt == _tri_count(t)


@pytest.mark.parametrize("masked", [True, False])
def test_serial_matches_bruteforce(masked):
    q, k, v = _rand(7, 3, 2, seed=1)
    nb, db = H.hla3_definition_loops(q, k, v, masked)
    (ns, ds), _ = H.hla3_serial(q, k, v, masked, return_num_den=True)
    np.testing.assert_allclose(ns, nb, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(ds, db, rtol=1e-11, atol=1e-11)
    nd, dd = H.hla3_definition(q[None], k[None], v[None], masked)
    np.testing.assert_allclose(nd[0], nb, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dd[0], db, rtol=1e-11, atol=1e-11)


def test_not_the_masked_tensor_product():
    """The masked set is not (L(.)QK^T)(L(.)QK^T)^T(L(.)QK^T): they differ at n = 2."""
    q, k, v = _rand(2, 3, 2, seed=2)
    W = np.tril(q @ k.T)
    (num, _), _ = H.hla3_serial(q, k, v, return_num_den=True)
    assert np.abs((W @ W.T @ W @ v)[1] - num[1]).max() > 1e-3


def test_corrected_recurrence_matches_serial():
    q, k, v = _rand(12, 4, 3, seed=3, batch=(2,))
    (nc, dc), fin_c = H.hla3_corrected_serial(q, k, v)
    (ns, ds), fin_s = H.hla3_serial(q, k, v, return_num_den=True)
    np.testing.assert_allclose(nc, ns, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dc, ds, rtol=1e-10, atol=1e-10)
    SK, SQ, P, m, G1, G2, G3, h1, h2, h3 = fin_s
    np.testing.assert_allclose(fin_c[4], SK @ SQ @ P - G1 - G2 - G3, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(fin_c[5], np.einsum("...ij,...j->...i", SK @ SQ, m) - h1 - h2 - h3,
                               rtol=1e-10, atol=1e-10)


def test_chunked_equals_serial_every_chunk():
    q, k, v = _rand(11, 3, 2, seed=4)
    (ns, ds), _ = H.hla3_serial(q, k, v, return_num_den=True)
    for C in range(1, 12):
        nk, dk = H.hla3_chunked(q, k, v, C, return_num_den=True)
        np.testing.assert_allclose(nk, ns, rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(dk, ds, rtol=1e-10, atol=1e-10)


def test_combine3_associative_and_identity():
    rng = np.random.default_rng(5)
    d, dv = 3, 2
    shapes = [(d, d), (d, d), (d, dv), (d,), (d, dv), (d,), (d, dv), (d,), (d, d), (d, d, d, dv), (d, d, d)]

    def rnd():
        return tuple(rng.standard_normal(s) for s in shapes)

    for _ in range(4):
        A, B, C = rnd(), rnd(), rnd()
        left = H.combine3(H.combine3(A, B), C)
        right = H.combine3(A, H.combine3(B, C))
        for x, y in zip(left, right):
            np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-11)
    E = H.zero_scan_state((), d, dv)
    A = rnd()
    for x, y in zip(H.combine3(E, A), A):
        np.testing.assert_array_equal(x, y)
    for x, y in zip(H.combine3(A, E), A):
        np.testing.assert_array_equal(x, y)


def test_segment_summary_is_the_state_after_the_segment():
    q, k, v = _rand(9, 3, 2, seed=6)
    X = H.segment_summary3(q, k, v)
    (_, _), fin = H.hla3_corrected_serial(q, k, v)
    for a, b in zip(X[:6], fin):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)
    # the extra summaries are their definitions
    delta = np.einsum("td,td->t", q, k)
    np.testing.assert_allclose(X[6], q.T @ (delta[:, None] * v), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(X[8], k.T @ (delta[:, None] * q), rtol=1e-11, atol=1e-11)
    Z = np.random.default_rng(7).standard_normal((3, 3))
    s = np.einsum("td,de,te->t", k, Z, k)
    np.testing.assert_allclose(H.apply_MP(X[9], Z), k.T @ (s[:, None] * v), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("n", [1, 2, 5])
def test_constant_tokens_closed_form(n):
    """q = k = x (unit), v = y: every term is (x.x)^3 y = y, so num_t = |index set| y,
    den_t = |index set|; unmasked: t^3."""
    x = np.array([0.6, 0.8, 0.0])
    y = np.array([1.5, -2.0])
    q = np.tile(x, (n, 1))
    v = np.tile(y, (n, 1))
    (num, den), _ = H.hla3_serial(q, q, v, return_num_den=True)
    (nu, du), _ = H.hla3_serial(q, q, v, masked=False, return_num_den=True)
    for t in range(1, n + 1):
        np.testing.assert_allclose(num[t - 1], _tri_count(t) * y, rtol=1e-12)
        np.testing.assert_allclose(den[t - 1], _tri_count(t), rtol=1e-12)
        np.testing.assert_allclose(nu[t - 1], t ** 3 * y, rtol=1e-12)


def test_one_hot_tokens():
    """q_t = k_t = e_t: only (t, t, t) survives, so o_t = v_t (masked and unmasked)."""
    n = 4
    q = np.eye(n)
    v = np.random.default_rng(8).standard_normal((n, 3))
    for masked in (True, False):
        (num, den), _ = H.hla3_serial(q, q, v, masked=masked, return_num_den=True)
        np.testing.assert_allclose(num, v, atol=1e-14)
        np.testing.assert_allclose(den, np.ones(n), atol=1e-14)


def test_unmasked_minus_masked_is_the_corrections():
    q, k, v = _rand(8, 3, 2, seed=9)
    (nm, _), _ = H.hla3_serial(q, k, v, return_num_den=True)
    (nu, _), _ = H.hla3_serial(q, k, v, masked=False, return_num_den=True)
    for t in range(8):
        _, st = H.hla3_serial(q[:t + 1], k[:t + 1], v[:t + 1])
        G = st[4] + st[5] + st[6]
        np.testing.assert_allclose(nu[t] - nm[t], q[t] @ G, rtol=1e-10, atol=1e-10)


def test_den_is_output_with_unit_values():
    q, k, v = _rand(8, 3, 2, seed=10)
    (_, den), _ = H.hla3_serial(q, k, v, return_num_den=True)
    (num1, _), _ = H.hla3_serial(q, k, np.ones((8, 1)), return_num_den=True)
    np.testing.assert_allclose(num1[:, 0], den, rtol=1e-11, atol=1e-11)


def test_homogeneity():
    q, k, v = _rand(6, 3, 2, seed=11)
    a, b, c = 1.7, -0.6, 2.3
    (n0, _), _ = H.hla3_serial(q, k, v, return_num_den=True)
    (n1, _), _ = H.hla3_serial(a * q, b * k, c * v, return_num_den=True)
    np.testing.assert_allclose(n1, (a ** 3) * (b ** 3) * c * n0, rtol=1e-10, atol=1e-12)


def test_zero_padding_and_resume():
    q, k, v = _rand(10, 3, 2, seed=12)
    (n0, d0), f0 = H.hla3_serial(q, k, v, return_num_den=True)
    z = np.zeros((3, 3))
    (n1, d1), f1 = H.hla3_serial(np.vstack([q, z]), np.vstack([k, z]), np.vstack([v, np.zeros((3, 2))]),
                                 return_num_den=True)
    np.testing.assert_allclose(n1[:10], n0, rtol=1e-12)
    np.testing.assert_array_equal(n1[10:], 0.0)
    for a, b in zip(f0, f1):
        np.testing.assert_allclose(a, b, rtol=1e-12)
    (na, da), fa = H.hla3_serial(q[:4], k[:4], v[:4], return_num_den=True)
    (nb, db), fb = H.hla3_serial(q[4:], k[4:], v[4:], state=fa, return_num_den=True)
    np.testing.assert_allclose(np.vstack([na, nb]), n0, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(np.concatenate([da, db]), d0, rtol=1e-11, atol=1e-11)


def test_den_scale_bounds_den():
    q, k, v = _rand(20, 4, 2, seed=13)
    (_, den), _ = H.hla3_serial(q, k, v, return_num_den=True)
    D = H.hla3_den_scale(q, k)
    assert np.all(np.abs(den) <= D * (1 + 1e-12) + 1e-12)


def test_unmasked_den_scale_bounds_den():
    """|den_t| <= D_t, with equality when every term is nonnegative (q = k
    with nonnegative entries); brute force over the triples on a tiny case."""
    q, k, v = _rand(9, 3, 1, seed=21)
    (_, den), _ = H.hla3_serial(q, k, v, masked=False, return_num_den=True)
    D = H.hla3_den_scale_unmasked(q, k)
    assert np.all(np.abs(den) <= D * (1 + 1e-12))
    n = 5
    brute = np.array([sum(abs(q[t] @ k[i]) * abs(k[i] @ q[u]) * abs(q[u] @ k[j])
                          for i in range(t + 1) for u in range(t + 1) for j in range(t + 1)) for t in range(n)])
    np.testing.assert_allclose(D[:n], brute, rtol=1e-12)
    p = np.abs(q)
    (_, dp), _ = H.hla3_serial(p, p, v, masked=False, return_num_den=True)
    np.testing.assert_allclose(H.hla3_den_scale_unmasked(p, p), dp, rtol=1e-12)


def test_c_oracle_matches_numpy():
    if not native.available():
        pytest.skip("C oracle not built")
    q, k, v = _rand(40, 4, 3, seed=14, batch=(3,))
    for masked in (True, False):
        num, den, _ = native.hla3_serial_c(q, k, v, masked=masked, threads=2)
        (n2, d2), _ = H.hla3_serial(q, k, v, masked=masked, return_num_den=True)
        np.testing.assert_allclose(num, n2, rtol=1e-12, atol=1e-10)
        np.testing.assert_allclose(den, d2, rtol=1e-12, atol=1e-10)


# ------------------------------------------------------------- planted mistakes
def _serial_variant(q, k, v, mistake):
    """Alg. 3 with one planted mistake; must disagree with the brute force."""
    n, d = q.shape
    dv = v.shape[1]
    SK = np.zeros((d, d)); SQ = np.zeros((d, d)); P = np.zeros((d, dv)); m = np.zeros(d)
    G = np.zeros((d, dv))
    num = np.zeros((n, dv))
    for t in range(n):
        qt, kt, vt = q[t], k[t], v[t]
        SKp, SQp, Pp = SK, SQ, P
        SK = SKp + np.outer(kt, kt); SQ = SQp + np.outer(qt, qt); P = Pp + np.outer(kt, vt)
        if mistake == "g2_inclusive":          # G2 with the inclusive S^K
            G += np.outer(kt, (SQp @ kt) @ Pp) + np.outer(SK @ qt, qt @ Pp) + np.outer(SKp @ SQp @ kt, vt)
        elif mistake == "drop_g3":
            G += np.outer(kt, (SQp @ kt) @ Pp) + np.outer(SKp @ qt, qt @ Pp)
        elif mistake == "g1_uses_sk":          # u1 = S^K k instead of S^Q k
            G += np.outer(kt, (SKp @ kt) @ Pp) + np.outer(SKp @ qt, qt @ Pp) + np.outer(SKp @ SQp @ kt, vt)
        else:                                  # "none": Alg. 3 as written
            G += np.outer(kt, (SQp @ kt) @ Pp) + np.outer(SKp @ qt, qt @ Pp) + np.outer(SKp @ SQp @ kt, vt)
        num[t] = (SQ @ SK @ qt) @ P - qt @ G
    return num


@pytest.mark.parametrize("mistake", ["g2_inclusive", "drop_g3", "g1_uses_sk"])
def test_pins_catch_planted_mistakes(mistake):
    q, k, v = _rand(6, 3, 2, seed=15)
    nb, _ = H.hla3_definition_loops(q, k, v)
    np.testing.assert_allclose(_serial_variant(q, k, v, "none"), nb, rtol=1e-10, atol=1e-10)
    bad = _serial_variant(q, k, v, mistake)
    assert np.abs(bad - nb).max() > 1e-6
