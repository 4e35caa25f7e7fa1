"""Pins of the parity-labelled real basis (Sec. 3.4 eq. parity_basis, App. D).

* the Parity Equivariance proposition: every basis function R_p^{s,l,m} satisfies
  R(-x) = p R(x), checked pointwise with the Goldberg-sum SWSH at random points
  and their antipodes (spatial inversion: theta -> pi - theta, phi -> phi + pi);
* P is orthogonal and the basis is the paper's literal basis mixed by it;
* the product respects parity: inputs of definite parities p1, p2 give outputs
  with parity p1 p2 only (a consequence of f1(-x) f2(-x) = p1 p2 f1(x) f2(x));
* the parity-basis product equals P^T F_paper(P x1, P x2).
"""

import numpy as np
import pytest

import oracle
from oracle.realbasis import BASIS_PAPER, BASIS_PARITY, parity_mix, q_matrix, real_index
from tests.oracle_helpers import valid_mask

S3 = (-1, 0, 1)


def parity_label(spins, L):
    """The parity p of every slot of the parity basis: (-1)^l at s = 0, +1 in the
    -|s| block, -1 in the +|s| block; 0 where the slot does not exist."""
    p = np.zeros(len(spins) * (L + 1) ** 2)
    for s in spins:
        for l in range(abs(s), L + 1):
            for m in range(-l, l + 1):
                p[real_index(spins, L, s, l, m)] = (-1.0) ** l if s == 0 else (1.0 if s < 0 else -1.0)
    return p


def field(Q, spins, L, k, theta, phi):
    """Basis function k of the basis with change of basis Q at points (theta, phi)."""
    v = np.zeros(np.shape(theta), dtype=np.complex128)
    for s in spins:
        for l in range(abs(s), L + 1):
            for m in range(-l, l + 1):
                q = Q[real_index(spins, L, s, l, m), k]
                if q != 0:
                    v = v + q * oracle.swsh(s, l, m, theta, phi)
    return v


@pytest.mark.parametrize("L", [1, 3])
def test_parity_basis_has_definite_parity(L):
    rng = np.random.default_rng(5)
    theta = rng.uniform(0.1, np.pi - 0.1, 7)
    phi = rng.uniform(0, 2 * np.pi, 7)
    Q = q_matrix(S3, L, BASIS_PARITY)
    p = parity_label(S3, L)
    for k in np.nonzero(p)[0]:
        a = field(Q, S3, L, k, theta, phi)
        b = field(Q, S3, L, k, np.pi - theta, phi + np.pi)
        assert np.abs(b - p[k] * a).max() <= 1e-12 * max(1.0, np.abs(a).max()), k
    # the literal basis has no definite parity in the |s| = 1 blocks
    Ql = q_matrix(S3, L, BASIS_PAPER)
    k = real_index(S3, L, 1, 1, 1)
    a, b = field(Ql, S3, L, k, theta, phi), field(Ql, S3, L, k, np.pi - theta, phi + np.pi)
    assert min(np.abs(b - a).max(), np.abs(b + a).max()) > 1e-3


def test_parity_mix_is_orthogonal():
    P = parity_mix(S3, 4)
    assert np.allclose(P.T @ P, np.eye(P.shape[0]))
    assert np.allclose(q_matrix(S3, 4, BASIS_PARITY), q_matrix(S3, 4, BASIS_PAPER) @ P)


@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (3, 1, 3), (1, 3, 3)])
def test_product_parity_rule(L1, L2, Lout):
    T = oracle.RealGauntTensor(L1, L2, Lout, S3, BASIS_PARITY)
    p1, p2, p3 = parity_label(S3, L1), parity_label(S3, L2), parity_label(S3, Lout)
    rng = np.random.default_rng(L1 + 3 * L2)
    for a in (1.0, -1.0):
        for b in (1.0, -1.0):
            x1 = rng.standard_normal((3, len(p1))) * (p1 == a)
            x2 = rng.standard_normal((3, len(p2))) * (p2 == b)
            y = T.apply(x1, x2).reshape(3, -1)
            assert np.abs(y[:, p3 == -a * b]).max() <= 1e-13 * max(1.0, np.abs(y).max())
            assert np.abs(y[:, p3 == a * b]).max() > 1e-3


@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (3, 2, 4)])
def test_parity_product_is_the_mixed_paper_product(L1, L2, Lout):
    rng = np.random.default_rng(9)
    x1 = rng.standard_normal((4, 3 * (L1 + 1) ** 2)) * valid_mask(S3, L1)
    x2 = rng.standard_normal((4, 3 * (L2 + 1) ** 2)) * valid_mask(S3, L2)
    P1, P2, P3 = parity_mix(S3, L1), parity_mix(S3, L2), parity_mix(S3, Lout)
    a = oracle.RealGauntTensor(L1, L2, Lout, S3, BASIS_PARITY).apply(x1, x2).reshape(4, -1)
    b = oracle.RealGauntTensor(L1, L2, Lout, S3, BASIS_PAPER).apply(x1 @ P1.T, x2 @ P2.T).reshape(4, -1) @ P3
    assert np.abs(a - b).max() <= 1e-13 * max(1.0, np.abs(b).max())
