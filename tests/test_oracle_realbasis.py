"""Pins of the oracle's real<->complex change of basis Q (CPU only)."""

import math
import os

import numpy as np
import pytest

import oracle
from oracle.realbasis import BASIS_M0_PAIRED, BASIS_PAPER
from tests.oracle_helpers import block_D, valid_mask

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_q_l1_s0_matches_paper_example():
    """App. C example: Q for l = 1, |s| = 0."""
    Q = oracle.q_matrix((0,), 1)
    block = Q[1:4, 1:4]  # l = 1 block, rows/cols m,k = -1, 0, 1
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "q_l1_s0.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 9
    for r, c, re, im in rows:
        want = (float(re) + 1j * float(im)) / math.sqrt(2)
        assert abs(block[int(r) + 1, int(c) + 1] - want) < 1e-15


@pytest.mark.parametrize("basis", [BASIS_PAPER, BASIS_M0_PAIRED])
@pytest.mark.parametrize("spins", [(0,), (-1, 0, 1), (-2, -1, 0, 1, 2)])
def test_q_unitary(spins, basis):
    """App. C: Q is unitary on the existing slots (l >= |s|)."""
    L = 4
    Q = oracle.q_matrix(spins, L, basis)
    v = valid_mask(spins, L)
    Qv = Q[np.ix_(v, v)]
    np.testing.assert_allclose(Qv.conj().T @ Qv, np.eye(v.sum()), atol=1e-15)
    assert np.abs(Q[~v]).max(initial=0) == 0 and np.abs(Q[:, ~v]).max(initial=0) == 0


def test_q_real_basis_functions_are_real_at_s0():
    """At s = 0 the columns of Q build real functions (the usual real SH)."""
    from oracle.swsh import swsh
    L = 4
    rng = np.random.default_rng(3)
    th, ph = rng.uniform(0, math.pi, 50), rng.uniform(0, 2 * math.pi, 50)
    Q = oracle.q_matrix((0,), L)
    Y = np.stack([swsh(0, l, m, th, ph) for l in range(L + 1) for m in range(-l, l + 1)])
    R = Q.T @ Y  # column k of Q combines complex harmonics into the real function R_k
    assert np.abs(R.imag).max() < 1e-14


def _rotation_in_real_basis(spins, L, basis, angles):
    Q = oracle.q_matrix(spins, L, basis)
    v = valid_mask(spins, L)
    D = block_D(spins, L, *angles)
    return (Q.conj().T @ D @ Q)[np.ix_(v, v)]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_rotation_closure(seed):
    """Q^dagger D Q is real for s = 0 (both conventions) and for the m0-paired basis.

    For the paper-literal basis with |s| > 0 it is not (reading recorded with the
    oracle): the l = 1 block keeps imaginary parts of order 0.5.
    """
    angles = np.random.default_rng(seed).uniform(0, 2 * math.pi, 3)
    for basis in (BASIS_PAPER, BASIS_M0_PAIRED):
        R0 = _rotation_in_real_basis((0,), 4, basis, angles)
        assert np.abs(R0.imag).max() < 1e-14
    Rp = _rotation_in_real_basis((-1, 0, 1), 4, BASIS_M0_PAIRED, angles)
    assert np.abs(Rp.imag).max() < 1e-14
    Rl = _rotation_in_real_basis((-1, 0, 1), 1, BASIS_PAPER, angles)
    assert np.abs(Rl.imag).max() > 1e-2
