"""Pins of the oracle's path-weighted product (eq. spin_gtp, Sec. 3.4).

The weighted tensor scales each entry of the unweighted T by the weight of its
path (block triple rho1, rho2 -> rho3).  Pinned against the unweighted oracle
(itself pinned to the paper) through properties a wrong block label, a dropped
path or a transposed role would break:
* unit weights reproduce the unweighted product exactly;
* the weight of one path alone gives the unweighted product of the inputs masked
  to that path's input blocks, read on its output block;
* the single-path products add up to the unweighted product (the paths partition
  T), and the product is linear in the weights;
* the gradients satisfy the bilinear identity <g, y> = <gx1, x1> = <gx2, x2>;
* every path obeys the degree triangle and the spin rule s3 = s1 + s2 of some
  signed spins of its blocks.
"""

import numpy as np
import pytest

import oracle
from oracle.spingtp import slot_blocks
from tests.oracle_helpers import valid_mask

S3 = (-1, 0, 1)
S5 = (-2, -1, 0, 1, 2)
CASES = [(2, 2, 2, S3, 0), (2, 1, 3, S3, 1), (2, 2, 2, S3, 2), (1, 2, 2, S5, 0), (2, 2, 2, S5, 2), (3, 2, 1, (0,), 0)]


def draw(spins, L, n, seed):
    return np.random.default_rng(seed).standard_normal((n, len(spins) * (L + 1) ** 2)) * valid_mask(spins, L)


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CASES)
def test_unit_weights_are_the_unweighted_product(L1, L2, LO, spins, basis):
    W = oracle.PathWeightedTensor(L1, L2, LO, spins, basis)
    x1, x2 = draw(spins, L1, 5, 1), draw(spins, L2, 5, 2)
    assert np.array_equal(W.apply(x1, x2), W.base.apply(x1, x2))


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CASES)
def test_one_path_is_the_block_restricted_product(L1, L2, LO, spins, basis):
    W0 = oracle.PathWeightedTensor(L1, L2, LO, spins, basis)
    P = W0.paths
    b1, b2, b3 = slot_blocks(spins, L1), slot_blocks(spins, L2), slot_blocks(spins, LO)
    x1, x2 = draw(spins, L1, 4, 3), draw(spins, L2, 4, 4)
    rng = np.random.default_rng(len(P))
    total = np.zeros((4, len(spins) * (LO + 1) ** 2))
    for p in range(len(P)):
        w = np.zeros(len(P))
        w[p] = 1.0
        y = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, w).apply(x1, x2).reshape(4, -1)
        total += y
        if p in set(rng.choice(len(P), size=min(12, len(P)), replace=False).tolist()):
            ref = W0.base.apply(x1 * (b1 == P[p, 0]), x2 * (b2 == P[p, 1])).reshape(4, -1) * (b3 == P[p, 2])
            assert np.abs(y - ref).max() <= 1e-13 * max(1.0, np.abs(ref).max())
    assert np.abs(total - W0.base.apply(x1, x2).reshape(4, -1)).max() <= 1e-12


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CASES)
def test_linear_in_the_weights_and_gradients(L1, L2, LO, spins, basis):
    n = len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)
    rng = np.random.default_rng(n)
    wa, wb = rng.standard_normal(n), rng.standard_normal(n)
    A = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, wa)
    B = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, wb)
    C = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, 2.0 * wa - 3.0 * wb)
    x1, x2 = draw(spins, L1, 3, 5), draw(spins, L2, 3, 6)
    g = draw(spins, LO, 3, 7)
    assert np.abs(C.apply(x1, x2) - (2.0 * A.apply(x1, x2) - 3.0 * B.apply(x1, x2))).max() <= 1e-12
    gx1, gx2 = A.vjp(x1, x2, g)
    e = float((g * A.apply(x1, x2).reshape(3, -1)).sum())
    assert abs(float((gx1 * x1).sum()) - e) <= 1e-12 * max(1.0, abs(e))
    assert abs(float((gx2 * x2).sum()) - e) <= 1e-12 * max(1.0, abs(e))


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CASES)
def test_paths_obey_the_selection_rules(L1, L2, LO, spins, basis):
    P = oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths
    assert len(P) == len({tuple(p) for p in P.tolist()})
    for i1, i2, i3 in P.tolist():
        (s1, l1), (s2, l2), (s3, l3) = ((spins[i // (L + 1)], i % (L + 1)) for i, L in ((i1, L1), (i2, L2), (i3, LO)))
        assert abs(l1 - l2) <= l3 <= l1 + l2
        assert any(a * s1 + b * s2 == c * s3 for a in (1, -1) for b in (1, -1) for c in (1, -1))


# --- per-channel path weights with the edge input shared by the channels (V = 1) ---
# Pinned against the path-weighted product above (itself pinned to the unweighted
# oracle) and by central differences of that forward: the product is linear in each
# of x1, x2 and W, so a central difference is exact up to rounding, and a gradient
# entry on a wrong path, slot or channel fails it.

CW_CASES = [(1, 1, 1, S3, 0), (2, 2, 2, S3, 2), (1, 3, 3, S3, 0), (2, 1, 2, S5, 1)]


def cw_inputs(L1, L2, LO, spins, basis, N, C, seed):
    P = len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)
    rng = np.random.default_rng(seed)
    x1 = draw(spins, L1, N * C, seed + 1).reshape(N, C, -1)
    x2 = draw(spins, L2, N, seed + 2)
    g = draw(spins, LO, N * C, seed + 3).reshape(N, C, -1)
    return x1, x2, rng.standard_normal((C, P)), g


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CW_CASES)
def test_channel_weighted_v1_is_the_path_weighted_product_per_channel(L1, L2, LO, spins, basis):
    x1, x2, W, _ = cw_inputs(L1, L2, LO, spins, basis, 3, 4, 11)
    y = oracle.channel_weighted_v1(x1, x2, W, L1, L2, LO, spins, basis).reshape(3, 4, -1)
    for c in range(4):
        ref = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, W[c]).apply(x1[:, c], x2).reshape(3, -1)
        assert np.abs(y[:, c] - ref).max() <= 1e-13 * max(1.0, np.abs(ref).max())
    ones = np.ones_like(W)
    y1 = oracle.channel_weighted_v1(x1, x2, ones, L1, L2, LO, spins, basis).reshape(3, 4, -1)
    base = oracle.spingtp(x1.reshape(12, -1), np.repeat(x2, 4, axis=0), L1, L2, LO, spins, basis).reshape(3, 4, -1)
    assert np.abs(y1 - base).max() <= 1e-12


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CW_CASES)
def test_channel_weighted_v1_gradients_homogeneity(L1, L2, LO, spins, basis):
    x1, x2, W, g = cw_inputs(L1, L2, LO, spins, basis, 4, 3, 21)
    y = oracle.channel_weighted_v1(x1, x2, W, L1, L2, LO, spins, basis).reshape(4, 3, -1)
    gx1, gx2, gW = oracle.channel_weighted_v1_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)
    e = float((g * y).sum())
    for grad, val in ((gx1, x1), (gx2, x2), (gW, W)):
        assert grad.shape == val.shape
        assert abs(float((grad * val).sum()) - e) <= 1e-11 * max(1.0, abs(e))


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CW_CASES)
def test_channel_weighted_v1_gradients_central_differences(L1, L2, LO, spins, basis):
    N, C = 3, 2
    x1, x2, W, g = cw_inputs(L1, L2, LO, spins, basis, N, C, 31)
    gx1, gx2, gW = oracle.channel_weighted_v1_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)

    def f(a, b, w):
        return float((g * oracle.channel_weighted_v1(a, b, w, L1, L2, LO, spins, basis).reshape(N, C, -1)).sum())

    rng = np.random.default_rng(7)
    for _ in range(6):  # weights: every sampled (channel, path)
        c, p = int(rng.integers(C)), int(rng.integers(W.shape[1]))
        d = np.zeros_like(W)
        d[c, p] = 1.0
        fd = (f(x1, x2, W + d) - f(x1, x2, W - d)) / 2.0
        assert abs(fd - gW[c, p]) <= 1e-11 * max(1.0, abs(fd))
    valid1 = np.flatnonzero(valid_mask(spins, L1).ravel())
    valid2 = np.flatnonzero(valid_mask(spins, L2).ravel())
    for _ in range(4):  # per-unit input and shared edge input
        n, c, k = int(rng.integers(N)), int(rng.integers(C)), int(rng.choice(valid1))
        d = np.zeros_like(x1)
        d[n, c, k] = 1.0
        fd = (f(x1 + d, x2, W) - f(x1 - d, x2, W)) / 2.0
        assert abs(fd - gx1[n, c, k]) <= 1e-11 * max(1.0, abs(fd))
        n, k = int(rng.integers(N)), int(rng.choice(valid2))
        d = np.zeros_like(x2)
        d[n, k] = 1.0
        fd = (f(x1, x2 + d, W) - f(x1, x2 - d, W)) / 2.0
        assert abs(fd - gx2[n, k]) <= 1e-11 * max(1.0, abs(fd))


# --- per-channel path weights with a per-unit second input (mode uuu) ---

def cu_inputs(L1, L2, LO, spins, basis, N, C, seed):
    P = len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)
    rng = np.random.default_rng(seed)
    x1 = draw(spins, L1, N * C, seed + 1).reshape(N, C, -1)
    x2 = draw(spins, L2, N * C, seed + 2).reshape(N, C, -1)
    g = draw(spins, LO, N * C, seed + 3).reshape(N, C, -1)
    return x1, x2, rng.standard_normal((C, P)), g


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CW_CASES)
def test_channel_weighted_reduces_to_the_shared_form(L1, L2, LO, spins, basis):
    # with x2 equal over the channels of an edge, the per-unit form is the V = 1 form
    x1, _, W, g = cu_inputs(L1, L2, LO, spins, basis, 3, 4, 41)
    x2s = draw(spins, L2, 3, 45)
    x2 = np.repeat(x2s[:, None, :], 4, axis=1)
    y = oracle.channel_weighted(x1, x2, W, L1, L2, LO, spins, basis)
    assert np.abs(y - oracle.channel_weighted_v1(x1, x2s, W, L1, L2, LO, spins, basis)).max() <= 1e-13
    gx1, gx2, gW = oracle.channel_weighted_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)
    r1, r2, rW = oracle.channel_weighted_v1_vjp(x1, x2s, W, g, L1, L2, LO, spins, basis)
    assert np.abs(gx1 - r1).max() <= 1e-12 and np.abs(gW - rW).max() <= 1e-12
    assert np.abs(gx2.sum(axis=1) - r2).max() <= 1e-12  # the shared input's gradient sums the units'


@pytest.mark.parametrize("L1,L2,LO,spins,basis", CW_CASES)
def test_channel_weighted_gradients_central_differences(L1, L2, LO, spins, basis):
    N, C = 3, 2
    x1, x2, W, g = cu_inputs(L1, L2, LO, spins, basis, N, C, 51)
    gx1, gx2, gW = oracle.channel_weighted_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)

    def f(a, b, w):
        return float((g * oracle.channel_weighted(a, b, w, L1, L2, LO, spins, basis).reshape(N, C, -1)).sum())

    e = f(x1, x2, W)
    for grad, val in ((gx1, x1), (gx2, x2), (gW, W)):  # homogeneity in each argument
        assert abs(float((grad * val).sum()) - e) <= 1e-11 * max(1.0, abs(e))
    rng = np.random.default_rng(9)
    for _ in range(5):
        c, p = int(rng.integers(C)), int(rng.integers(W.shape[1]))
        d = np.zeros_like(W)
        d[c, p] = 1.0
        assert abs((f(x1, x2, W + d) - f(x1, x2, W - d)) / 2.0 - gW[c, p]) <= 1e-11 * max(1.0, abs(gW[c, p]))
    valid2 = np.flatnonzero(valid_mask(spins, L2).ravel())
    for _ in range(4):
        n, c, k = int(rng.integers(N)), int(rng.integers(C)), int(rng.choice(valid2))
        d = np.zeros_like(x2)
        d[n, c, k] = 1.0
        fd = (f(x1, x2 + d, W) - f(x1, x2 - d, W)) / 2.0
        assert abs(fd - gx2[n, c, k]) <= 1e-11 * max(1.0, abs(fd))


# --- depthwise mode with V second-input channels (uvu, W[v, u, p]) ---

@pytest.mark.parametrize("L1,L2,LO,spins,basis", CW_CASES[:3])
def test_depthwise_definition_and_gradients(L1, L2, LO, spins, basis):
    N, U, V = 2, 3, 2
    P = len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)
    rng = np.random.default_rng(61)
    x1 = draw(spins, L1, N * U, 62).reshape(N, U, -1)
    x2 = draw(spins, L2, N * V, 63).reshape(N, V, -1)
    g = draw(spins, LO, N * U, 64).reshape(N, U, -1)
    W = rng.standard_normal((V, U, P))
    y = oracle.depthwise(x1, x2, W, L1, L2, LO, spins, basis).reshape(N, U, -1)
    # the definition per unit: sum over v and paths with the path-weighted tensor of W[v, u]
    for n in range(N):
        for u in range(U):
            ref = sum(oracle.PathWeightedTensor(L1, L2, LO, spins, basis, W[v, u]).apply(x1[n, u][None], x2[n, v][None])
                      .reshape(-1) for v in range(V))
            assert np.abs(y[n, u] - ref).max() <= 1e-12
    gx1, gx2, gW = oracle.depthwise_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)

    def f(a, b, w):
        return float((g * oracle.depthwise(a, b, w, L1, L2, LO, spins, basis).reshape(N, U, -1)).sum())

    e = f(x1, x2, W)
    for grad, val in ((gx1, x1), (gx2, x2), (gW, W)):
        assert grad.shape == val.shape
        assert abs(float((grad * val).sum()) - e) <= 1e-11 * max(1.0, abs(e))
    for idx in ((1, 2, P - 1), (0, 0, 0)):
        d = np.zeros_like(W)
        d[idx] = 1.0
        assert abs((f(x1, x2, W + d) - f(x1, x2, W - d)) / 2.0 - gW[idx]) <= 1e-11 * max(1.0, abs(gW[idx]))
    valid2 = np.flatnonzero(valid_mask(spins, L2).ravel())
    d = np.zeros_like(x2)
    d[1, 1, valid2[-1]] = 1.0
    assert abs((f(x1, x2 + d, W) - f(x1, x2 - d, W)) / 2.0 - gx2[1, 1, valid2[-1]]) <= 1e-11
