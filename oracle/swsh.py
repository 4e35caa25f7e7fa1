"""Spin-weighted spherical harmonics sY_lm by the explicit Goldberg sum.

Test infrastructure only (see ``oracle/__init__.py``).

Paper App. A.1 ("Explicit Formula") gives

    sY_lm(theta, phi) = A_slm sin^{2l}(theta/2) e^{i m phi}
                        * sum_{r=0}^{l-s} (-1)^r C(l-s, r) C(l+s, r+s-m) cot^{2r+s-m}(theta/2)

and leaves the prefactor A_slm unnamed.  Reading taken here (it is the one that
reproduces the worked examples 1Y10 and 1Y1(+-1) printed right below the
formula, and the conjugation / parity relations printed after them):

    A_slm = (-1)^{m+l-s} sqrt( (l+m)! (l-m)! (2l+1) / (4 pi (l+s)! (l-s)!) ).

The sum is evaluated in half-angle form: sin^{2l} cot^k = sin^{2l-k} cos^k with
k = 2r+s-m, which has no pole at theta = 0 or pi.
"""

import math

import numpy as np


def goldberg_prefactor(s: int, l: int, m: int) -> float:
    """A_slm of the Goldberg sum (reading stated in the module docstring)."""
    num = math.factorial(l + m) * math.factorial(l - m)
    den = math.factorial(l + s) * math.factorial(l - s)
    mag = math.sqrt((2 * l + 1) / (4.0 * math.pi) * (num / den))
    return (-1.0) ** ((m + l - s) % 2) * mag


def theta_part(s: int, l: int, m: int, theta) -> np.ndarray:
    """sY_lm(theta, 0), which is real; zero when |s| > l or |m| > l."""
    theta = np.asarray(theta, dtype=np.float64)
    if abs(s) > l or abs(m) > l:
        return np.zeros_like(theta)
    c = np.cos(theta / 2.0)
    sn = np.sin(theta / 2.0)
    total = np.zeros_like(theta)
    for r in range(0, l - s + 1):
        j = r + s - m
        if j < 0 or j > l + s:
            continue
        k = 2 * r + s - m
        coef = (-1.0) ** r * math.comb(l - s, r) * math.comb(l + s, j)
        total = total + coef * sn ** (2 * l - k) * c ** k
    return goldberg_prefactor(s, l, m) * total


def swsh(s: int, l: int, m: int, theta, phi) -> np.ndarray:
    """sY_lm(theta, phi), complex."""
    theta = np.asarray(theta, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    return theta_part(s, l, m, theta) * np.exp(1j * m * phi)
