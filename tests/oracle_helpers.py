"""Small textbook helpers for the oracle pins (Wigner D matrices).  Test code only."""

import math

import numpy as np


def wigner_small_d(l, mp, m, beta):
    """Explicit-sum Wigner small-d, convention d^1_{1,0}(b) = -sin(b)/sqrt2."""
    beta = np.asarray(beta, dtype=np.float64)
    out = np.zeros_like(beta)
    pre = math.sqrt(math.factorial(l + mp) * math.factorial(l - mp)
                    * math.factorial(l + m) * math.factorial(l - m))
    for k in range(0, 2 * l + 1):
        a, b, c, d = l + m - k, k, l - k - mp, k - m + mp
        if min(a, b, c, d) < 0:
            continue
        coef = (-1.0) ** ((k - m + mp) % 2) * pre / (
            math.factorial(a) * math.factorial(b) * math.factorial(c) * math.factorial(d))
        out = out + coef * np.cos(beta / 2) ** (2 * l - 2 * k + m - mp) \
            * np.sin(beta / 2) ** (2 * k - m + mp)
    return out


def wigner_D(l, alpha, beta, gamma):
    """D^l_{m'm}(alpha, beta, gamma) = e^{-i m' alpha} d^l_{m'm}(beta) e^{-i m gamma}."""
    ms = np.arange(-l, l + 1)
    D = np.zeros((2 * l + 1, 2 * l + 1), dtype=np.complex128)
    for i, mp in enumerate(ms):
        for j, m in enumerate(ms):
            D[i, j] = np.exp(-1j * mp * alpha) * wigner_small_d(l, mp, m, beta) * np.exp(-1j * m * gamma)
    return D


def block_D(spins, L, alpha, beta, gamma):
    """Rotation of a complex [n_spins][(L+1)^2] coefficient vector: D^l on m, same for all spins."""
    n = len(spins) * (L + 1) ** 2
    out = np.zeros((n, n), dtype=np.complex128)
    for si, s in enumerate(spins):
        for l in range(abs(s), L + 1):
            o = si * (L + 1) ** 2 + l * l
            out[o:o + 2 * l + 1, o:o + 2 * l + 1] = wigner_D(l, alpha, beta, gamma)
    return out


def valid_mask(spins, L):
    """True on slots with l >= |s|."""
    m = np.zeros((len(spins), (L + 1) ** 2), dtype=bool)
    for si, s in enumerate(spins):
        for l in range(abs(s), L + 1):
            m[si, l * l:(l + 1) ** 2] = True
    return m.ravel()
