"""Pins of the oracle's reverse-mode derivative (CPU only).

* the bilinear-form identity: for y = T(x1, x2), sum g y = sum gx1 x1 = sum gx2 x2;
* brute force on unit vectors: gx1[k1] = g . T(e_k1, x2) through the forward map;
* the conjugation map of the real basis (App. A.1 conjugation relation): a signed
  permutation, the identity for the m = 0 paired basis and for spin {0};
* the transpose identity the GPU backward is built on:
  gx1 = T_(Lout, L2, L1)(g, J2 x2) and gx2 = T_(Lout, L1, L2)(g, J1 x1).
"""

import numpy as np
import pytest

import oracle
from oracle.realbasis import conjugation_map, real_index
from tests.oracle_helpers import valid_mask

S3 = (-1, 0, 1)


def _inputs(L1, L2, Lout, spins, U, seed):
    rng = np.random.default_rng(seed)
    x1 = rng.standard_normal((U, len(spins) * (L1 + 1) ** 2)) * valid_mask(spins, L1)
    x2 = rng.standard_normal((U, len(spins) * (L2 + 1) ** 2)) * valid_mask(spins, L2)
    g = rng.standard_normal((U, len(spins) * (Lout + 1) ** 2)) * valid_mask(spins, Lout)
    return x1, x2, g


@pytest.mark.parametrize("L1,L2,Lout,spins,basis", [
    (2, 2, 2, S3, 0), (2, 2, 2, S3, 1), (3, 1, 2, S3, 0), (1, 3, 3, S3, 1), (4, 4, 4, S3, 0), (3, 3, 3, (0,), 0)])
def test_vjp_bilinear_identity(L1, L2, Lout, spins, basis):
    T = oracle.RealGauntTensor(L1, L2, Lout, spins, basis)
    x1, x2, g = _inputs(L1, L2, Lout, spins, 6, 11 + L1 + 5 * L2)
    y = T.apply(x1, x2).reshape(6, -1)
    gx1, gx2 = T.vjp(x1, x2, g)
    e = np.einsum("uk,uk->u", g, y)
    np.testing.assert_allclose(np.einsum("uk,uk->u", gx1, x1), e, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(np.einsum("uk,uk->u", gx2, x2), e, rtol=1e-12, atol=1e-13)


def test_vjp_brute_force_unit_vectors():
    L, spins = 1, S3
    T = oracle.RealGauntTensor(L, L, L, spins, 0)
    x1, x2, g = _inputs(L, L, L, spins, 1, 5)
    gx1, gx2 = T.vjp(x1, x2, g)
    n = x1.shape[1]
    for k in range(n):
        e = np.zeros((1, n))
        e[0, k] = 1.0
        assert abs(gx1[0, k] - g[0] @ T.apply(e, x2).reshape(-1)) < 1e-14
        assert abs(gx2[0, k] - g[0] @ T.apply(x1, e).reshape(-1)) < 1e-14


@pytest.mark.parametrize("L", [1, 3, 5])
def test_conjugation_map(L):
    for basis in (0, 1):
        J = conjugation_map(S3, L, basis)
        live = valid_mask(S3, L)
        Jl = J[np.ix_(live, live)]
        assert np.allclose(np.abs(Jl).sum(0), 1.0) and np.allclose(np.abs(Jl).sum(1), 1.0)  # signed permutation
        if basis == 1:
            assert np.allclose(Jl, np.eye(Jl.shape[0]))
        else:
            # the paper's literal m = 0 basis: the (+1, l, 0) and (-1, l, 0) slots swap with a sign change
            want = np.eye(J.shape[0]) * live
            for l in range(1, L + 1):
                a, b = real_index(S3, L, -1, l, 0), real_index(S3, L, 1, l, 0)
                want[a, a] = want[b, b] = 0.0
                want[a, b] = want[b, a] = -1.0
            assert np.allclose(J, want)
    assert np.allclose(conjugation_map((0,), L, 0), np.eye((L + 1) ** 2))


@pytest.mark.parametrize("L1,L2,Lout,basis", [(2, 2, 2, 0), (3, 3, 3, 1), (1, 3, 3, 0), (3, 1, 2, 0), (2, 3, 4, 1)])
def test_transpose_identity(L1, L2, Lout, basis):
    T = oracle.RealGauntTensor(L1, L2, Lout, S3, basis)
    x1, x2, g = _inputs(L1, L2, Lout, S3, 5, 7 * L1 + L2 + Lout)
    gx1, gx2 = T.vjp(x1, x2, g)
    J1, J2 = conjugation_map(S3, L1, basis), conjugation_map(S3, L2, basis)
    a = oracle.RealGauntTensor(Lout, L2, L1, S3, basis).apply(g, x2 @ J2.T).reshape(gx1.shape)
    b = oracle.RealGauntTensor(Lout, L1, L2, S3, basis).apply(g, x1 @ J1.T).reshape(gx2.shape)
    assert np.abs(a - gx1).max() <= 1e-13 * max(1.0, np.abs(gx1).max())
    assert np.abs(b - gx2).max() <= 1e-13 * max(1.0, np.abs(gx2).max())
