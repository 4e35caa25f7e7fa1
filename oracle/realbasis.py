"""Real SWSH basis and the unitary change of basis Q (a_complex = Q a_real).

Test infrastructure only (see ``oracle/__init__.py``).

Storage layout (shared by real and complex coefficient vectors of one input):
``[n_spins][(L+1)^2]``, spin axis in the order of the ``spins`` tuple (ascending,
e.g. (-1, 0, +1) -- App. C orders the doubled matrix by the -|s| sector first),
flat index l^2 + l + k inside a spin block, k = -l..l ascending.  Slots with
l < |s| do not exist as basis functions (Sec. 3.2 requires |s| <= l); Q has
neither rows nor columns there.

Entries (paper eq. real_swsh, Sec. 3.3; App. C gives the s = 0 entries and the
l = 1 example).  For a real column (sigma, l, k) the real basis function is
sigma R_lk; writing it as a combination of complex sY gives the column of Q:

  k > 0 : Q[(sigma, k), (sigma, k)]    = 1/sqrt2
          Q[(-sigma, -k), (sigma, k)]  = (-1)^(k+sigma)/sqrt2
  k < 0 : Q[(sigma, |k|), (sigma, k)]  = i/sqrt2
          Q[(-sigma, k), (sigma, k)]   = -i (-1)^(|k|+sigma)/sqrt2
  k = 0 : BASIS_PAPER      -- sigma R_l0 = sigma Y_l0 literally (eq. real_swsh):
                              Q[(sigma, 0), (sigma, 0)] = 1.
          BASIS_M0_PAIRED  -- reading for a rotation-closed real basis when
                              |s| > 0: column (+|s|, 0) -> rows (+|s|, 0), (-|s|, 0)
                              with (1/sqrt2, (-1)^|s|/sqrt2); column (-|s|, 0) ->
                              (i/sqrt2, -i(-1)^|s|/sqrt2).  For s = 0 both
                              conventions give Q = 1.

At sigma = 0 these formulas reproduce App. C's scalar matrix exactly.  The
real-basis output is y = Re(Q^dagger c) (App. C).
"""

import math

import numpy as np

BASIS_PAPER = 0
BASIS_M0_PAIRED = 1
BASIS_PARITY = 2

_R2 = 1.0 / math.sqrt(2.0)


def real_index(spins, L, s, l, k) -> int:
    """Flat index of slot (s, l, k) in a [n_spins][(L+1)^2] vector."""
    si = list(spins).index(s)
    return si * (L + 1) ** 2 + l * l + l + k


def parity_mix(spins, L) -> np.ndarray:
    """Real orthogonal P with x_real = P x_parity for the parity-labelled basis.

    Sec. 3.4 eq. parity_basis / App. D: for |s| > 0,
    R_p^{s,l,m} = (R_{-s,l,m} + p (-1)^l R_{s,l,m}) / sqrt2, p = +-1.  Storage
    reading: the coefficient of p = +1 sits in the -|s| block, that of p = -1 in
    the +|s| block (App. C orders the -|s| sector first); s = 0 is unchanged.  So a
    function sum_p c_p R_p has real-basis coefficients
    x[-s,l,m] = (c_+ + c_-)/sqrt2 and x[s,l,m] = (-1)^l (c_+ - c_-)/sqrt2.
    """
    spins = tuple(spins)
    n = len(spins) * (L + 1) ** 2
    P = np.eye(n)
    for s in spins:
        if s <= 0:
            continue
        for l in range(s, L + 1):
            t = (-1.0) ** (l % 2)
            for m in range(-l, l + 1):
                a, b = real_index(spins, L, -s, l, m), real_index(spins, L, s, l, m)
                P[a, a], P[a, b] = _R2, _R2
                P[b, a], P[b, b] = t * _R2, -t * _R2
    return P


def q_matrix(spins, L, basis=BASIS_PAPER) -> np.ndarray:
    """Dense complex Q of shape [n, n], n = len(spins) * (L+1)^2.

    ``spins`` must be symmetric (contain -s for every s) so that every |s| > 0
    sector is doubled as the paper requires.  BASIS_PARITY is the parity-labelled
    basis built on the paper's literal real basis: Q = Q_paper P (parity_mix).
    """
    spins = tuple(spins)
    if basis == BASIS_PARITY:
        return q_matrix(spins, L, BASIS_PAPER) @ parity_mix(spins, L)
    for s in spins:
        if -s not in spins:
            raise ValueError("spin set must be symmetric")
    n = len(spins) * (L + 1) ** 2
    Q = np.zeros((n, n), dtype=np.complex128)
    idx = lambda s, l, k: real_index(spins, L, s, l, k)  # noqa: E731
    for sigma in spins:
        for l in range(abs(sigma), L + 1):
            for k in range(-l, l + 1):
                col = idx(sigma, l, k)
                if k > 0:
                    Q[idx(sigma, l, k), col] += _R2
                    Q[idx(-sigma, l, -k), col] += (-1.0) ** ((k + sigma) % 2) * _R2
                elif k < 0:
                    a = -k
                    Q[idx(sigma, l, a), col] += 1j * _R2
                    Q[idx(-sigma, l, k), col] += -1j * (-1.0) ** ((a + sigma) % 2) * _R2
                else:
                    if sigma == 0 or basis == BASIS_PAPER:
                        Q[idx(sigma, l, 0), col] = 1.0
                    elif basis == BASIS_M0_PAIRED:
                        sa = abs(sigma)
                        sign = (-1.0) ** (sa % 2)
                        if sigma > 0:
                            Q[idx(sa, l, 0), col] = _R2
                            Q[idx(-sa, l, 0), col] = sign * _R2
                        else:
                            Q[idx(sa, l, 0), col] = 1j * _R2
                            Q[idx(-sa, l, 0), col] = -1j * sign * _R2
                    else:
                        raise ValueError("unknown basis convention")
    return Q


def conjugation_map(spins, L, basis=BASIS_PAPER) -> np.ndarray:
    """Real matrix J with conj(f) = sum_k (J x)[k] R_k for f = sum_k x[k] R_k.

    From the conjugation relation of App. A.1, conj(sY_lm) = (-1)^(s+m) (-s)Y_l(-m):
    conjugating the complex column Q[:, k] gives the column Q'[:, k] with
    Q'[(-s, l, -m), k] = (-1)^(s+m) conj(Q[(s, l, m), k]), and J = Q^-1 Q' on the
    existing slots (zero rows and columns at l < |s|).  Raises if J is not real.
    """
    spins = tuple(spins)
    Q = q_matrix(spins, L, basis)
    n = Q.shape[0]
    Qc = np.zeros_like(Q)
    for s in spins:
        for l in range(abs(s), L + 1):
            for m in range(-l, l + 1):
                Qc[real_index(spins, L, -s, l, -m), :] = (-1.0) ** ((s + m) % 2) * np.conj(
                    Q[real_index(spins, L, s, l, m), :])
    live = [i for i in range(n) if np.abs(Q[:, i]).sum() > 0]
    J = np.zeros((n, n), dtype=np.complex128)
    J[np.ix_(live, live)] = np.linalg.solve(Q[np.ix_(live, live)], Qc[np.ix_(live, live)])
    if np.abs(J.imag).max() > 1e-12:
        raise AssertionError("conjugation is not a real map in this basis")
    return J.real
