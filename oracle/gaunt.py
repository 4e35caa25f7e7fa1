"""Spin-weighted Gaunt coefficients by brute-force quadrature.

Test infrastructure only (see ``oracle/__init__.py``).

Definition (paper Sec. 3.2, eq. generalized_gaunt, integral form; s3 = s1 + s2):

    G^{(l3,m3,s3)}_{(l1,m1,s1)(l2,m2,s2)} = int_{S^2} s1Y_l1m1 s2Y_l2m2 conj(s3Y_l3m3) dOmega.

The integral is taken with a tensor-product rule: Gauss-Legendre in cos(theta)
and a uniform rule in phi.  With s3 = s1 + s2 and m3 = m1 + m2 the theta part of
the integrand is a polynomial in cos(theta) of degree <= l1 + l2 + l3 (the
half-angle powers of the Goldberg sum add up to even numbers), and the phi part
is e^{i(m1+m2-m3) phi} with |m1+m2-m3| <= l1+l2+l3.  Hence
n_theta >= (l1+l2+l3+1)/2 Gauss nodes and n_phi >= l1+l2+l3+1 uniform points
integrate exactly; ``gauss_legendre_grid`` uses twice that for margin.

The printed 3j form of the same coefficient is NOT used here; the tests compare
the quadrature against it (with the phase that the SWSH convention of App. A.1
implies) as an independent check.
"""

import math

import numpy as np

from .swsh import theta_part


def gauss_legendre_grid(degree_sum: int, margin: int = 2):
    """Nodes for an exact rule on polynomials of total degree ``degree_sum``.

    Returns (theta [n_theta], w_theta [n_theta], phi [n_phi], w_phi) where
    int f dOmega ~= sum_j sum_k w_theta[j] * w_phi * f(theta_j, phi_k).
    """
    n_theta = margin * ((degree_sum + 2) // 2)
    n_phi = margin * (degree_sum + 1)
    x, w = np.polynomial.legendre.leggauss(n_theta)
    theta = np.arccos(x)
    phi = 2.0 * math.pi * np.arange(n_phi) / n_phi
    return theta, w, phi, 2.0 * math.pi / n_phi


def _phi_rule(M, phi, w_phi):
    """Uniform-rule value of int_0^{2pi} e^{i M phi} dphi for integer array M."""
    M = np.asarray(M)
    return (np.exp(1j * np.multiply.outer(M, phi)) * w_phi).sum(axis=-1)


def gaunt_block(l1, s1, l2, s2, l3, s3, theta, w_theta, phi, w_phi):
    """G[m1 + l1, m2 + l2] for m3 = m1 + m2 (entries with |m3| > l3 are 0).

    Only the m3 = m1 + m2 entries are formed: the others carry
    int e^{i(m1+m2-m3)phi} dphi = 0 (``gaunt_full_quadrature`` checks that by
    brute force in the tests).
    """
    m1 = np.arange(-l1, l1 + 1)
    m2 = np.arange(-l2, l2 + 1)
    T1 = np.stack([theta_part(s1, l1, m, theta) for m in m1])          # [2l1+1, nt]
    T2 = np.stack([theta_part(s2, l2, m, theta) for m in m2])          # [2l2+1, nt]
    T3 = np.stack([theta_part(s3, l3, m, theta) for m in range(-l3, l3 + 1)]
                  + [np.zeros_like(theta)])                             # last row = 0
    m3 = np.add.outer(m1, m2)
    row = np.where(np.abs(m3) <= l3, m3 + l3, 2 * l3 + 1)             # out of range -> 0 row
    phase = _phi_rule(np.zeros(1, dtype=int), phi, w_phi)[0]          # m1+m2-m3 = 0
    G = np.einsum("aj,bj,abj->ab", T1 * w_theta, T2, T3[row]) * phase
    return G


def gaunt_full_quadrature(l1, m1, s1, l2, m2, s2, l3, m3, s3, theta, w_theta, phi, w_phi):
    """One coefficient by the full 2D rule, without using m3 = m1 + m2."""
    t = theta_part(s1, l1, m1, theta) * theta_part(s2, l2, m2, theta) \
        * theta_part(s3, l3, m3, theta)
    return np.sum(w_theta * t) * _phi_rule(m1 + m2 - m3, phi, w_phi)
