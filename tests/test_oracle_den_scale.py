"""Pins of the oracle's denominator scales D_t (the sums of |terms| of den_t
that the normalised GPU tests judge den by) against a hand-worked example
whose terms change sign (tests/golden/den_scale_hand_example.txt), plus
planted mistakes the example must catch.  CPU only.

Passages: HLA-2 den, Thm. 1 and its proof (v_j -> 1), Eq. hla-row for the
unmasked form; AHLA, Sec. 6; decay, the decay section (reading of the masked
decayed operator); HLA-3, Sec. 7 (Thm. 3, Eq. hla3-corrected-recurrence).
"""
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import ahla as A
from oracle import hla2 as H
from oracle import hla2_decay as DK
from oracle import hla3 as H3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "den_scale_hand_example.txt")
Q = np.array([(1, 0), (-1, 1), (1, -2)], dtype=np.float64)
K = np.array([(1, 0), (0, 1), (1, 1)], dtype=np.float64)
COLS = ["hla2_m", "hla2_u", "ahla", "decay_m", "decay_u", "hla3_m", "hla3_u"]


def _golden():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        parts = [p.split() for p in line.split("|")]
        rows.append([[float(Fraction(x)) for x in p] for p in parts[1:]])
    out = {}
    for c, name in enumerate(COLS):
        out[name] = (np.array([r[c][0] for r in rows]), np.array([r[c][1] for r in rows]))
    return out


G = _golden()


def _v1():
    return np.ones((3, 1))


def test_golden_has_sign_changes():
    """The example is chosen so that the terms of den_t change sign: D_t > |den_t| somewhere."""
    for name in COLS:
        D, den = G[name]
        assert np.all(D >= np.abs(den))
        assert np.any(D > np.abs(den) + 0.5), name


def test_hla2_den_scale_matches_hand_example():
    np.testing.assert_allclose(H.hla2_den_scale(Q, K, masked=True), G["hla2_m"][0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(H.hla2_den_scale(Q, K, masked=False), G["hla2_u"][0], rtol=0, atol=1e-12)
    for masked, name in ((True, "hla2_m"), (False, "hla2_u")):
        (_, den), _ = H.hla2_serial(Q, K, _v1(), masked=masked, return_num_den=True)
        np.testing.assert_allclose(den, G[name][1], atol=1e-12)


def test_hla2_den_scale_planted_mistakes_fail():
    """S_t in place of S_j, and |sum| in place of sum |.|, must both miss the hand values."""
    D = G["hla2_m"][0]
    S = np.cumsum(K[:, :, None] * K[:, None, :], axis=0)            # S_t, inclusive
    wrong_st = np.array([sum(abs(Q[t] @ S[t] @ Q[j]) for j in range(t + 1)) for t in range(3)])
    wrong_abs = np.array([abs(sum(Q[t] @ S[j] @ Q[j] for j in range(t + 1))) for t in range(3)])
    assert np.abs(wrong_st - D).max() >= 1
    assert np.abs(wrong_abs - D).max() >= 1


def test_ahla_den_scale_matches_hand_example():
    np.testing.assert_allclose(A.ahla_den_scale(Q, K), G["ahla"][0], atol=1e-12)
    _, den = A.ahla_definition(Q, K, _v1(), return_num_den=True)
    np.testing.assert_allclose(den, G["ahla"][1], atol=1e-12)


def test_ahla_den_scale_planted_mistakes_fail():
    """A A^T (the symmetric second-order form) or a mask without the diagonal must miss the hand values."""
    L = np.tril(np.ones((3, 3)))
    Am = L * (Q @ K.T)
    wrong_sym = np.abs((Am @ Am.T) * L).sum(-1)
    Ls = np.tril(np.ones((3, 3)), -1)
    As = Ls * (Q @ K.T)
    wrong_diag = np.abs((As @ As) * L).sum(-1)
    assert np.abs(wrong_sym - G["ahla"][0]).max() >= 1
    assert np.abs(wrong_diag - G["ahla"][0]).max() >= 1


def test_decay_den_scale_matches_hand_example():
    for masked, name in ((True, "decay_m"), (False, "decay_u")):
        np.testing.assert_allclose(DK.hla2_decay_den_scale(Q, K, 0.5, masked=masked), G[name][0], atol=1e-12)
        (_, den), _ = DK.hla2_decay_serial(Q, K, _v1(), 0.5, masked=masked, return_num_den=True)
        np.testing.assert_allclose(den, G[name][1], atol=1e-12)


def test_decay_den_scale_planted_mistake_fails():
    """One decay factor gamma^(t-i) only (the j factor dropped) must miss the hand values."""
    g = 0.5
    a = Q @ K.T
    wrong = np.array([sum(abs(sum(g ** (t - i) * a[t, i] * a[j, i] for i in range(j + 1))) for j in range(t + 1))
                      for t in range(3)])
    assert np.abs(wrong - G["decay_m"][0]).max() >= 0.25


def test_hla3_den_scale_matches_hand_example():
    np.testing.assert_allclose(H3.hla3_den_scale(Q, K), G["hla3_m"][0], atol=1e-12)
    np.testing.assert_allclose(H3.hla3_den_scale_unmasked(Q, K), G["hla3_u"][0], atol=1e-12)
    for masked, name in ((True, "hla3_m"), (False, "hla3_u")):
        (_, den), _ = H3.hla3_serial(Q, K, _v1(), masked=masked, return_num_den=True)
        np.testing.assert_allclose(den, G[name][1], atol=1e-12)


@pytest.mark.parametrize("group", ["last", "first"])
def test_hla3_den_scale_planted_mistake_fails(group):
    """Grouping the masked triples by their last (or first) index instead of
    the largest index must miss the hand values."""
    import itertools
    a = Q @ K.T
    qk = K @ Q.T        # qk[i, u] = k_i . q_u
    wrong = []
    for t in range(3):
        terms = [0.0] * (t + 1)
        for i, u, j in itertools.product(range(t + 1), repeat=3):
            mx = max(i, u, j)
            if [i, u, j].count(mx) < 2:
                continue
            terms[j if group == "last" else i] += a[t, i] * qk[i, u] * a[u, j]
        wrong.append(sum(abs(x) for x in terms))
    assert np.abs(np.array(wrong) - G["hla3_m"][0]).max() >= 1
