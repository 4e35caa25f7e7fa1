"""Pins of the oracle's spin-weighted Gaunt coefficients (CPU only).

The oracle gets G by quadrature.  These tests compare it with exact Wigner-3j
values from sympy (an independent library routine), with sympy's ordinary
Gaunt coefficient at s = 0, with the selection rules of Sec. 3.1/3.2, and with
the closed form in the proof of the path-completion proposition (App. A.3).
"""

import math
import os

import numpy as np
import pytest
from sympy.physics.wigner import gaunt as sympy_gaunt
from sympy.physics.wigner import wigner_3j

import oracle
from oracle.gaunt import gauss_legendre_grid

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _grid(L1, L2, L3, margin=2):
    return gauss_legendre_grid(L1 + L2 + L3, margin)


def _g(l1, m1, s1, l2, m2, s2, l3, s3, margin=2):
    grid = _grid(l1, l2, l3, margin)
    G = oracle.gaunt_block(l1, s1, l2, s2, l3, s3, *grid)
    return G[m1 + l1, m2 + l2]


def _3j_form(l1, m1, s1, l2, m2, s2, l3, m3, s3):
    """(-1)^(m3+s3) sqrt(prod(2l+1)/4pi) (l1 l2 l3; m1 m2 -m3) (l1 l2 l3; -s1 -s2 s3).

    This is eq. generalized_gaunt with the phase that the SWSH convention of
    App. A.1 implies (conjugate the third harmonic with the App. A.1
    conjugation relation, then use the standard triple-product formula).
    """
    pre = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1) / (4 * math.pi))
    return (-1) ** ((m3 + s3) % 2) * pre * float(wigner_3j(l1, l2, l3, m1, m2, -m3)) \
        * float(wigner_3j(l1, l2, l3, -s1, -s2, s3))


def _printed_form(l1, m1, s1, l2, m2, s2, l3, m3, s3):
    """eq. generalized_gaunt exactly as printed (second 3j with s1 s2 -s3)."""
    pre = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1) / (4 * math.pi))
    return pre * float(wigner_3j(l1, l2, l3, m1, m2, -m3)) * float(wigner_3j(l1, l2, l3, s1, s2, -s3))


def _random_entries(n, lmax, smax, seed):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        l1, l2 = rng.integers(0, lmax + 1, 2)
        l3 = rng.integers(abs(l1 - l2), min(l1 + l2, lmax) + 1)
        s1 = rng.integers(-min(l1, smax), min(l1, smax) + 1)
        s2 = rng.integers(-min(l2, smax), min(l2, smax) + 1)
        s3 = s1 + s2
        if abs(s3) > l3:
            continue
        m1 = rng.integers(-l1, l1 + 1)
        m2 = rng.integers(-l2, l2 + 1)
        if abs(m1 + m2) > l3:
            continue
        out.append(tuple(int(v) for v in (l1, m1, s1, l2, m2, s2, l3, m1 + m2, s3)))
    return out


def test_quadrature_matches_3j_form():
    """Quadrature G equals the exact 3j form (App. A.1 phase) to 1e-13."""
    n_sign_flip = 0
    for (l1, m1, s1, l2, m2, s2, l3, m3, s3) in _random_entries(150, 4, 2, 7):
        g = _g(l1, m1, s1, l2, m2, s2, l3, s3)
        assert abs(g.imag) < 1e-14
        want = _3j_form(l1, m1, s1, l2, m2, s2, l3, m3, s3)
        assert abs(g.real - want) < 1e-13, (l1, m1, s1, l2, m2, s2, l3, m3, s3, g, want)
        printed = _printed_form(l1, m1, s1, l2, m2, s2, l3, m3, s3)
        assert abs(abs(printed) - abs(want)) < 1e-13
        if abs(want) > 1e-8 and np.sign(printed) != np.sign(want):
            n_sign_flip += 1
    # the printed phase disagrees with the App. A.1 convention on some entries
    assert n_sign_flip > 0


@pytest.mark.parametrize("lmax", [3])
def test_s0_is_ordinary_gaunt(lmax):
    """Sec. 3.1 eq. gaunt_bridge: at s = 0, G = int Y1 Y2 conj(Y3) = (-1)^m3 gaunt(l1,l2,l3,m1,m2,-m3)."""
    for l1 in range(lmax + 1):
        for l2 in range(lmax + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                grid = _grid(l1, l2, l3)
                G = oracle.gaunt_block(l1, 0, l2, 0, l3, 0, *grid)
                for m1 in range(-l1, l1 + 1):
                    for m2 in range(-l2, l2 + 1):
                        m3 = m1 + m2
                        if abs(m3) > l3:
                            continue
                        want = (-1) ** (m3 % 2) * float(sympy_gaunt(l1, l2, l3, m1, m2, -m3))
                        assert abs(G[m1 + l1, m2 + l2] - want) < 1e-13


def test_selection_rules():
    """Sec. 3.1: s = 0 kills odd l1+l2+l3; Sec. 3.2: spin channels restore them."""
    grid = _grid(1, 1, 1)
    G0 = oracle.gaunt_block(1, 0, 1, 0, 1, 0, *grid)
    assert np.abs(G0).max() < 1e-15
    # (1,1,1) through spin channels: (s1,s2) = (1,0) -> 1 and (1,-1) -> 0
    target = math.sqrt(27 / (4 * math.pi)) / 6
    for s1, s2 in ((1, 0), (1, -1), (-1, 1), (0, -1)):
        G = oracle.gaunt_block(1, s1, 1, s2, 1, s1 + s2, *grid)
        assert abs(np.abs(G).max() - target) < 1e-14
    # odd l-sum at s = 0 for a larger triple
    grid = _grid(3, 2, 2)
    assert np.abs(oracle.gaunt_block(3, 0, 2, 0, 2, 0, *grid)).max() < 1e-14


def test_path_completion_closed_form():
    """App. A.3 proposition: |G| at the boundary spins is sqrt(prod/4pi) S^2 with the printed |S|."""
    rows = [tuple(map(int, ln.split())) for ln in open(os.path.join(GOLDEN, "path_completion.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 10
    f = math.factorial
    for l1, l2, l3 in rows:
        assert abs(l1 - l2) <= l3 <= l1 + l2
        S = math.sqrt(f(2 * l1) * f(2 * l3) / (f(l1 - l2 + l3) * f(l1 + l2 + l3 + 1)))
        pre = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1) / (4 * math.pi))
        g = _g(l1, l1, l1, l2, l3 - l1, l3 - l1, l3, l3)
        # magnitude: the printed |S| closed form; sign: the App. A.1 convention
        # gives (-1)^(l1+l2+l3) relative to the printed G = sqrt(.) S^2
        want = (-1) ** ((l1 + l2 + l3) % 2) * pre * S * S
        assert abs(g - want) < 1e-13, (l1, l2, l3, g, want)


def test_off_diagonal_m_vanish_under_full_quadrature():
    """Brute force over the full 2D rule: entries with m3 != m1 + m2 vanish."""
    L = 2
    grid = _grid(L, L, L)
    worst = 0.0
    for s1, s2 in ((1, 0), (0, 0), (-1, 1)):
        s3 = s1 + s2
        for l1 in range(abs(s1), L + 1):
            for l2 in range(abs(s2), L + 1):
                for l3 in range(abs(s3), L + 1):
                    for m1 in range(-l1, l1 + 1):
                        for m2 in range(-l2, l2 + 1):
                            for m3 in range(-l3, l3 + 1):
                                g = oracle.gaunt_full_quadrature(l1, m1, s1, l2, m2, s2, l3, m3, s3, *grid)
                                if m3 != m1 + m2:
                                    worst = max(worst, abs(g))
                                else:
                                    ref = oracle.gaunt_block(l1, s1, l2, s2, l3, s3, *grid)[m1 + l1, m2 + l2]
                                    assert abs(g - ref) < 1e-15
    assert worst < 1e-15


def test_minimal_rule_is_exact():
    """The rule with n_theta = (l1+l2+l3+2)//2, n_phi = l1+l2+l3+1 already gives the exact value."""
    for (l1, m1, s1, l2, m2, s2, l3, m3, s3) in _random_entries(40, 6, 1, 11):
        a = _g(l1, m1, s1, l2, m2, s2, l3, s3, margin=1)
        b = _g(l1, m1, s1, l2, m2, s2, l3, s3, margin=3)
        assert abs(a - b) < 1e-14
