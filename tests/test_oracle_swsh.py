"""Pins of the oracle's spin-weighted spherical harmonics (CPU only).

Each test checks ``oracle.swsh`` against something other than itself: the closed
forms printed in App. A.1, the conjugation and parity relations printed there,
orthonormality (App. A), scipy's ordinary spherical harmonics at s = 0, and the
textbook Wigner small-d form of SWSH.
"""

import math
import os

import numpy as np
import pytest
from scipy.special import sph_harm_y

import oracle
from oracle.gaunt import gauss_legendre_grid

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(20260701)
THETA = np.concatenate([[0.0, math.pi, math.pi / 2], rng.uniform(0, math.pi, 13)])
PHI = rng.uniform(0, 2 * math.pi, THETA.shape)


def test_closed_forms_s1_l1():
    """App. A.1 worked example: 1Y10 and 1Y1(+-1)."""
    kinds = {
        "sin": np.sin,
        "one_minus_cos": lambda t: 1 - np.cos(t),
        "one_plus_cos": lambda t: 1 + np.cos(t),
    }
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "swsh_s1_l1_closed_forms.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 3
    for s, l, m, sign, num, den, kind in rows:
        s, l, m, sign, num, den = map(int, (s, l, m, sign, num, den))
        want = sign * math.sqrt(num / (den * math.pi)) * kinds[kind](THETA) * np.exp(1j * m * PHI)
        got = oracle.swsh(s, l, m, THETA, PHI)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)


@pytest.mark.parametrize("l", range(0, 5))
def test_conjugation_and_parity(l):
    """App. A.1: sY*_lm = (-1)^(s+m) (-s)Y_l(-m);  sY(pi-theta, phi+pi) = (-1)^l (-s)Y_lm."""
    for s in range(-min(l, 2), min(l, 2) + 1):
        for m in range(-l, l + 1):
            y = oracle.swsh(s, l, m, THETA, PHI)
            conj = (-1) ** ((s + m) % 2) * oracle.swsh(-s, l, -m, THETA, PHI)
            np.testing.assert_allclose(np.conj(y), conj, atol=1e-14)
            par = oracle.swsh(s, l, m, math.pi - THETA, PHI + math.pi)
            np.testing.assert_allclose(par, (-1) ** l * oracle.swsh(-s, l, m, THETA, PHI),
                                       atol=1e-14)


@pytest.mark.parametrize("L,tol", [(4, 1e-13), (8, 1e-13), (16, 1e-10)])
def test_orthonormality(L, tol):
    """App. A: int sY_lm conj(sY_l'm') dOmega = delta_ll' delta_mm' at fixed s."""
    theta, wt, phi, wp = gauss_legendre_grid(2 * L)
    TH, PH = np.meshgrid(theta, phi, indexing="ij")
    W = np.outer(wt, np.full(len(phi), wp))
    for s in (-1, 0, 1, 2):
        funcs = [oracle.swsh(s, l, m, TH, PH) for l in range(abs(s), L + 1) for m in range(-l, l + 1)]
        F = np.stack([f.ravel() for f in funcs])
        gram = (F * W.ravel()) @ F.conj().T
        np.testing.assert_allclose(gram, np.eye(len(funcs)), atol=tol)


@pytest.mark.parametrize("l", range(0, 7))
def test_s0_is_scipy_spherical_harmonic(l):
    """App. A: 0Y_lm = Y_lm (Condon-Shortley phase, as scipy's sph_harm_y)."""
    for m in range(-l, l + 1):
        want = sph_harm_y(l, m, THETA, PHI)
        np.testing.assert_allclose(oracle.swsh(0, l, m, THETA, PHI), want, atol=1e-13)


def _wigner_small_d(l, mp, m, beta):
    """Textbook Wigner small-d (explicit sum), with d^1_{1,0}(b) = -sin(b)/sqrt2."""
    out = np.zeros_like(beta)
    pre = math.sqrt(math.factorial(l + mp) * math.factorial(l - mp)
                    * math.factorial(l + m) * math.factorial(l - m))
    for k in range(0, 2 * l + 1):
        a, b, c, d = l + m - k, k, l - k - mp, k - m + mp
        if min(a, b, c, d) < 0:
            continue
        coef = (-1.0) ** ((k - m + mp) % 2) * pre / (
            math.factorial(a) * math.factorial(b) * math.factorial(c) * math.factorial(d))
        out = out + coef * np.cos(beta / 2) ** (2 * l - 2 * k + m - mp) * np.sin(beta / 2) ** (2 * k - m + mp)
    return out


@pytest.mark.parametrize("l", range(0, 6))
def test_wigner_d_form(l):
    """sY_lm = (-1)^s sqrt((2l+1)/4pi) d^l_{m,-s}(theta) e^{i m phi} for all |s| <= l."""
    for s in range(-l, l + 1):
        for m in range(-l, l + 1):
            want = (-1) ** (s % 2) * math.sqrt((2 * l + 1) / (4 * math.pi)) \
                * _wigner_small_d(l, m, -s, THETA) * np.exp(1j * m * PHI)
            np.testing.assert_allclose(oracle.swsh(s, l, m, THETA, PHI), want, atol=1e-13)
