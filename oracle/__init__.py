"""CPU oracle for the spin-weighted Gaunt tensor product (SpinGTP), float64.

TEST INFRASTRUCTURE ONLY.  Nothing in the product (the HIP library, its C ABI and
its Python binding) may import, call, link or execute this package.  Only the
test-suite, the smoke check and the CPU-baseline leg of the benchmark use it.

The oracle computes the plain definition of the operation and nothing else:

* ``swsh``      -- spin-weighted spherical harmonics from the explicit Goldberg sum
                   (paper App. A.1, "Explicit Formula").
* ``realbasis`` -- the unitary real<->complex change of basis Q (paper Sec. 3.3,
                   eq. real_swsh; App. C "The Unitary Q Matrix").
* ``gaunt``     -- spin-weighted Gaunt coefficients obtained by brute-force
                   quadrature of triple SWSH products (paper Sec. 3.2,
                   eq. generalized_gaunt, the integral form).
* ``spingtp``   -- the real bilinear map y = Re(Q^dagger c), c = sum G a1 a2,
                   a = Q x, written as an explicit sparse tensor T (paper
                   Sec. 3.5, eq. spin_gtp with unit weights and the elementwise
                   channel mode of App. E.1); ``vjp`` / ``spingtp_vjp`` give its
                   reverse-mode derivative by the chain rule on that definition;
                   ``PathWeightedTensor`` scales it by one weight per path
                   (block triple) of eq. spin_gtp; ``channel_weighted*``,
                   ``depthwise*`` and ``fully_connected*`` are the multiplicity
                   modes uuu, uvu and uvw of App. E.1 and their derivatives.

Readings of points where the paper is silent or ambiguous are listed in the
docstrings of the functions that take them.  Every function here is pinned by
``tests/test_oracle_*.py`` against closed forms, identities and independent
library routines (scipy, sympy).
"""

from .swsh import swsh, theta_part, goldberg_prefactor
from .realbasis import q_matrix, real_index, conjugation_map, parity_mix, BASIS_PAPER, BASIS_M0_PAIRED, BASIS_PARITY
from .gaunt import gauss_legendre_grid, gaunt_block, gaunt_full_quadrature
from .spingtp import (RealGauntTensor, PathWeightedTensor, slot_blocks, spingtp, spingtp_vjp, channel_weighted_v1,
                      channel_weighted_v1_vjp, channel_weighted, channel_weighted_vjp, depthwise, depthwise_vjp,
                      fully_connected, fully_connected_vjp)

__all__ = [
    "swsh", "theta_part", "goldberg_prefactor",
    "q_matrix", "real_index", "parity_mix", "BASIS_PAPER", "BASIS_M0_PAIRED", "BASIS_PARITY",
    "gauss_legendre_grid", "gaunt_block", "gaunt_full_quadrature",
    "RealGauntTensor", "PathWeightedTensor", "slot_blocks", "spingtp", "spingtp_vjp",
    "channel_weighted_v1", "channel_weighted_v1_vjp", "channel_weighted", "channel_weighted_vjp",
    "depthwise", "depthwise_vjp", "fully_connected", "fully_connected_vjp",
]
