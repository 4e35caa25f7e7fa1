"""Pins of the oracle's full SpinGTP map (CPU only)."""

import math

import numpy as np
import pytest
from sympy.physics.wigner import wigner_3j

import oracle
from oracle.gaunt import gauss_legendre_grid
from oracle.realbasis import BASIS_M0_PAIRED, BASIS_PAPER
from tests.oracle_helpers import block_D, valid_mask

S3 = (-1, 0, 1)


def _rand(spins, L, n, seed):
    x = np.random.default_rng(seed).standard_normal((n, len(spins) * (L + 1) ** 2))
    return x * valid_mask(spins, L)


def test_nnz_counts():
    """Structural size of T at L = 2, 4, 6 (spins -1,0,1) -- 1043 / 15696 / 86410."""
    for L, want in ((2, 1043), (4, 15696), (6, 86410)):
        assert oracle.RealGauntTensor(L, L, L, S3).nnz == want


@pytest.mark.parametrize("basis", [BASIS_PAPER, BASIS_M0_PAIRED])
@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (3, 1, 2), (2, 3, 4)])
def test_constant_function(L1, L2, Lout, basis):
    """x2 = c * Y00 multiplies the x1 field by c/sqrt(4 pi): y = c/sqrt(4pi) x1 (l <= Lout)."""
    T = oracle.RealGauntTensor(L1, L2, Lout, S3, basis)
    x1 = _rand(S3, L1, 5, 1)
    x2 = np.zeros((5, T.n2))
    c = np.array([0.7, -1.3, 2.0, 0.1, 5.0])
    x2[:, oracle.real_index(S3, L2, 0, 0, 0)] = c
    y = T.apply(x1, x2).reshape(5, -1)
    want = np.zeros_like(y)
    for si, s in enumerate(S3):
        for l in range(abs(s), min(L1, Lout) + 1):
            o1 = si * (L1 + 1) ** 2 + l * l
            o3 = si * (Lout + 1) ** 2 + l * l
            want[:, o3:o3 + 2 * l + 1] = x1[:, o1:o1 + 2 * l + 1] * (c / math.sqrt(4 * math.pi))[:, None]
    np.testing.assert_allclose(y, want, atol=1e-13)


@pytest.mark.parametrize("basis", [BASIS_PAPER, BASIS_M0_PAIRED])
def test_commutative(basis):
    """The pointwise product commutes: y(x1, x2) = y(x2, x1) when L1 = L2."""
    T = oracle.RealGauntTensor(3, 3, 3, S3, basis)
    x1, x2 = _rand(S3, 3, 4, 2), _rand(S3, 3, 4, 3)
    np.testing.assert_allclose(T.apply(x1, x2), T.apply(x2, x1), atol=1e-13)


@pytest.mark.parametrize("seed", [0, 1])
def test_equivariance_complex_basis(seed):
    """App. A.2 rotation law: c(D a1, D a2) = D c(a1, a2), one D^l per l-block for all spins."""
    L = 3
    T = oracle.RealGauntTensor(L, L, L, S3)
    rng = np.random.default_rng(seed)
    v = valid_mask(S3, L)
    a1 = (rng.standard_normal((2, T.n1)) + 1j * rng.standard_normal((2, T.n1))) * v
    a2 = (rng.standard_normal((2, T.n2)) + 1j * rng.standard_normal((2, T.n2))) * v
    D = block_D(S3, L, *rng.uniform(0, 2 * math.pi, 3))
    lhs = T.apply_complex(a1 @ D.T, a2 @ D.T)
    rhs = T.apply_complex(a1, a2) @ D.T
    np.testing.assert_allclose(lhs, rhs, atol=1e-13)


@pytest.mark.parametrize("spins,basis", [((0,), BASIS_PAPER), (S3, BASIS_M0_PAIRED)])
def test_equivariance_real_basis(spins, basis):
    """Real-basis equivariance where the basis is rotation-closed: R = Q^dagger D Q."""
    L = 3
    T = oracle.RealGauntTensor(L, L, L, spins, basis)
    rng = np.random.default_rng(5)
    Q = oracle.q_matrix(spins, L, basis)
    D = block_D(spins, L, *rng.uniform(0, 2 * math.pi, 3))
    R = Q.conj().T @ D @ Q
    assert np.abs(R.imag).max() < 1e-14
    R = R.real
    x1, x2 = _rand(spins, L, 3, 6), _rand(spins, L, 3, 7)
    lhs = T.apply(x1 @ R.T, x2 @ R.T).reshape(3, -1)
    rhs = T.apply(x1, x2).reshape(3, -1) @ R.T
    np.testing.assert_allclose(lhs, rhs, atol=1e-13)


@pytest.mark.parametrize("basis", [BASIS_PAPER, BASIS_M0_PAIRED])
@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (1, 2, 3)])
def test_functional_product_brute_force(L1, L2, Lout, basis):
    """App. B proof: y is the projection of the pointwise product of the two fields.

    Fields are summed from SWSH on a fine grid, multiplied spin pair by spin pair,
    integrated against conj(sY), then mapped back with Re(Q^dagger .).
    """
    theta, wt, phi, wp = gauss_legendre_grid(L1 + L2 + Lout, margin=3)
    TH, PH = np.meshgrid(theta, phi, indexing="ij")
    W = np.outer(wt, np.full(len(phi), wp))
    x1, x2 = _rand(S3, L1, 3, 8), _rand(S3, L2, 3, 9)
    Q1, Q2 = oracle.q_matrix(S3, L1, basis), oracle.q_matrix(S3, L2, basis)
    Q3 = oracle.q_matrix(S3, Lout, basis)
    a1, a2 = x1 @ Q1.T, x2 @ Q2.T

    def field(a, L, s):
        si = S3.index(s)
        f = np.zeros((a.shape[0],) + TH.shape, dtype=np.complex128)
        for l in range(abs(s), L + 1):
            for m in range(-l, l + 1):
                f += a[:, si * (L + 1) ** 2 + l * l + l + m, None, None] * oracle.swsh(s, l, m, TH, PH)
        return f

    F1 = {s: field(a1, L1, s) for s in S3}
    F2 = {s: field(a2, L2, s) for s in S3}
    c = np.zeros((3, len(S3) * (Lout + 1) ** 2), dtype=np.complex128)
    for s3 in S3:
        h = sum(F1[s1] * F2[s3 - s1] for s1 in S3 if (s3 - s1) in S3)
        for l in range(abs(s3), Lout + 1):
            for m in range(-l, l + 1):
                k = S3.index(s3) * (Lout + 1) ** 2 + l * l + l + m
                c[:, k] = (h * np.conj(oracle.swsh(s3, l, m, TH, PH)) * W).sum(axis=(1, 2))
    y_brute = (c @ Q3.conj()).real
    y = oracle.RealGauntTensor(L1, L2, Lout, S3, basis).apply(x1, x2).reshape(3, -1)
    np.testing.assert_allclose(y, y_brute, atol=1e-13)


def test_tensor_matches_3j_construction():
    """T rebuilt from exact sympy 3j values (App. A.1 phase) equals the quadrature T at L = 2."""
    L = 2
    T = oracle.RealGauntTensor(L, L, L, S3).dense()
    Q = oracle.q_matrix(S3, L)
    n = Q.shape[0]
    G = np.zeros((n, n, n))
    for s1 in S3:
        for s2 in S3:
            s3 = s1 + s2
            if s3 not in S3:
                continue
            for l1 in range(abs(s1), L + 1):
                for l2 in range(abs(s2), L + 1):
                    for l3 in range(abs(s3), L + 1):
                        pre = math.sqrt((2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1) / (4 * math.pi))
                        w_s = float(wigner_3j(l1, l2, l3, -s1, -s2, s3))
                        if w_s == 0.0:
                            continue
                        for m1 in range(-l1, l1 + 1):
                            for m2 in range(-l2, l2 + 1):
                                m3 = m1 + m2
                                if abs(m3) > l3:
                                    continue
                                g = (-1) ** ((m3 + s3) % 2) * pre * w_s \
                                    * float(wigner_3j(l1, l2, l3, m1, m2, -m3))
                                G[oracle.real_index(S3, L, s1, l1, m1),
                                  oracle.real_index(S3, L, s2, l2, m2),
                                  oracle.real_index(S3, L, s3, l3, m3)] = g
    T3j = np.einsum("ak,bl,abe,ef->klf", Q, Q, G, Q.conj()).real
    np.testing.assert_allclose(T, T3j, atol=1e-13)


def test_spin_head_path():
    """OC20 spin head (1,1)o x (1,1)o -> (1,0)e (App. F.3): nonzero only through spin channels."""
    L = 1
    T = oracle.RealGauntTensor(L, L, L, S3)
    x1, x2 = _rand(S3, L, 4, 10), _rand(S3, L, 4, 11)
    x1[:, 4:8] = 0.0  # clear the s = 0 block
    x2[:, 4:8] = 0.0
    y = T.apply(x1, x2)
    out_s0_l1 = y[:, 1, 1:4]
    assert np.linalg.norm(out_s0_l1) > 0.05 * np.linalg.norm(x1) * np.linalg.norm(x2) / 4
    # scalar GTP: the (1,1,1) path through s = 0 alone vanishes
    T0 = oracle.RealGauntTensor(L, L, L, (0,))
    z1, z2 = np.zeros((4, 4)), np.zeros((4, 4))
    z1[:, 1:4] = x1[:, 4 + 1:4 + 4] + 1.0
    z2[:, 1:4] = x2[:, 4 + 1:4 + 4] - 0.5
    assert np.abs(T0.apply(z1, z2)[:, 0, 1:4]).max() < 1e-15


def test_scalar_selection_rule_in_real_tensor():
    """With spins (0,) every T entry with odd l1+l2+l3 is zero; with spins it is not."""
    L = 3

    def lvec(spins):
        return np.array([l for _ in spins for l in range(L + 1) for _ in range(2 * l + 1)])

    T0 = oracle.RealGauntTensor(L, L, L, (0,)).dense()
    l0 = lvec((0,))
    odd = (l0[:, None, None] + l0[None, :, None] + l0[None, None, :]) % 2 == 1
    assert np.abs(T0[odd]).max() == 0.0
    T1 = oracle.RealGauntTensor(L, L, L, S3).dense()
    l1 = lvec(S3)
    odd1 = (l1[:, None, None] + l1[None, :, None] + l1[None, None, :]) % 2 == 1
    assert np.abs(T1[odd1]).max() > 0.1


def test_degree_zero_closed_form():
    """L1 = L2 = Lout = 0, spins (0,): y = x1 x2 int Y00^3 = x1 x2 / sqrt(4 pi)."""
    x1 = np.array([[1.5], [-2.0], [0.25]])
    x2 = np.array([[2.0], [3.0], [-4.0]])
    y = oracle.spingtp(x1, x2, 0, 0, 0, spins=(0,))
    np.testing.assert_allclose(y.reshape(3), (x1 * x2).ravel() / math.sqrt(4 * math.pi), atol=1e-15)


def test_invalid_slots_ignored_and_zero():
    """Slots with l < |s| are ignored on input and zero on output."""
    L = 2
    T = oracle.RealGauntTensor(L, L, L, S3)
    x1, x2 = _rand(S3, L, 2, 12), _rand(S3, L, 2, 13)
    inv = ~valid_mask(S3, L)
    g1, g2 = x1.copy(), x2.copy()
    g1[:, inv] = 1e3
    g2[:, inv] = -7.0
    np.testing.assert_array_equal(T.apply(x1, x2), T.apply(g1, g2))
    assert np.abs(T.apply(g1, g2).reshape(2, -1)[:, inv]).max() == 0.0
