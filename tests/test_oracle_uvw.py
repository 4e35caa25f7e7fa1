"""Pins of the oracle's fully connected product (App. E.1 mode uvw) and its derivative.

None of them retypes the definition: the product is held to the depthwise mode (uvu,
itself pinned in test_oracle_weights.py) when W is diagonal in (u, w), to the
path-weighted product with one channel each, to linearity in W, to the block it may
write, and its three gradients to central differences of the product (exact up to
rounding, the product being linear in each argument).
"""

import numpy as np
import pytest

import oracle
from tests.oracle_helpers import valid_mask

S3 = (-1, 0, 1)
SHAPES = [((1, 1, 1), S3, 0), ((2, 2, 2), S3, 0), ((2, 2, 2), S3, 2), ((1, 3, 3), S3, 1), ((2, 1, 2), (0,), 0)]


def _draw(rng, shape, L, spins, N, C):
    return rng.standard_normal((N, C, len(spins) * (L + 1) ** 2)) * valid_mask(spins, L)


def _n_paths(L1, L2, LO, spins, basis):
    return len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)


@pytest.mark.parametrize("degrees,spins,basis", SHAPES)
def test_uvw_with_diagonal_weights_is_depthwise(degrees, spins, basis):
    L1, L2, LO = degrees
    rng = np.random.default_rng(sum(degrees) + 7 * basis)
    N, U, V = 3, 4, 2
    x1, x2 = _draw(rng, None, L1, spins, N, U), _draw(rng, None, L2, spins, N, V)
    P = _n_paths(L1, L2, LO, spins, basis)
    Wd = rng.standard_normal((V, U, P))
    W = np.zeros((P, U, V, U))
    for u in range(U):
        W[:, u, :, u] = Wd[:, u, :].T
    y = oracle.fully_connected(x1, x2, W, L1, L2, LO, spins, basis)
    yd = oracle.depthwise(x1, x2, Wd, L1, L2, LO, spins, basis)
    assert np.abs(y - yd).max() <= 1e-12 * max(1.0, np.abs(yd).max())


@pytest.mark.parametrize("degrees,spins,basis", SHAPES)
def test_uvw_single_channels_is_path_weighted(degrees, spins, basis):
    L1, L2, LO = degrees
    rng = np.random.default_rng(11 + sum(degrees))
    N = 5
    x1, x2 = _draw(rng, None, L1, spins, N, 1), _draw(rng, None, L2, spins, N, 1)
    P = _n_paths(L1, L2, LO, spins, basis)
    w = rng.standard_normal(P)
    y = oracle.fully_connected(x1, x2, w.reshape(P, 1, 1, 1), L1, L2, LO, spins, basis).reshape(N, -1)
    yp = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, w).apply(x1[:, 0], x2[:, 0]).reshape(N, -1)
    assert np.abs(y - yp).max() <= 1e-12 * max(1.0, np.abs(yp).max())


@pytest.mark.parametrize("degrees,spins,basis", SHAPES[:3])
def test_uvw_linear_in_weights_and_single_path_block(degrees, spins, basis):
    L1, L2, LO = degrees
    rng = np.random.default_rng(23)
    N, U, V, Wc = 2, 3, 2, 4
    x1, x2 = _draw(rng, None, L1, spins, N, U), _draw(rng, None, L2, spins, N, V)
    paths = oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths
    P = len(paths)
    W1, W2 = rng.standard_normal((P, U, V, Wc)), rng.standard_normal((P, U, V, Wc))
    f = lambda W: oracle.fully_connected(x1, x2, W, L1, L2, LO, spins, basis)  # noqa: E731
    assert np.allclose(f(2.0 * W1 - 3.0 * W2), 2.0 * f(W1) - 3.0 * f(W2), rtol=0, atol=1e-11)
    blocks = oracle.slot_blocks(spins, LO)
    for p in (0, P // 2, P - 1):
        Wp = np.zeros_like(W1)
        Wp[p] = W1[p]
        y = f(Wp).reshape(N, Wc, -1)
        outside = blocks != paths[p][2]
        assert np.abs(y[:, :, outside]).max() == 0.0
        assert np.abs(y[:, :, ~outside]).max() > 0.0


@pytest.mark.parametrize("degrees,spins,basis", SHAPES)
def test_uvw_gradients_match_central_differences(degrees, spins, basis):
    L1, L2, LO = degrees
    rng = np.random.default_rng(31 + sum(degrees))
    N, U, V, Wc = 2, 2, 3, 2
    x1, x2 = _draw(rng, None, L1, spins, N, U), _draw(rng, None, L2, spins, N, V)
    P = _n_paths(L1, L2, LO, spins, basis)
    W = rng.standard_normal((P, U, V, Wc))
    g = rng.standard_normal((N, Wc, len(spins) * (LO + 1) ** 2)) * valid_mask(spins, LO)
    gx1, gx2, gW = oracle.fully_connected_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)

    def loss(a, b, w):
        return float((oracle.fully_connected(a, b, w, L1, L2, LO, spins, basis).reshape(g.shape) * g).sum())

    h = 1e-3
    for arr, grad, which in ((x1, gx1, 0), (x2, gx2, 1), (W, gW, 2)):
        flat = arr.reshape(-1)
        for i in rng.choice(flat.size, size=min(12, flat.size), replace=False):
            d = np.zeros_like(flat)
            d[i] = h
            args_p = [x1, x2, W]
            args_m = [x1, x2, W]
            args_p[which] = (flat + d).reshape(arr.shape)
            args_m[which] = (flat - d).reshape(arr.shape)
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            assert abs(fd - grad.reshape(-1)[i]) <= 1e-8 * max(1.0, abs(fd)), (which, i, fd, grad.reshape(-1)[i])
