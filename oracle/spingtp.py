"""The SpinGTP bilinear map as an explicit sparse real tensor.

Test infrastructure only (see ``oracle/__init__.py``).

For one unit (edge n, channel c) with real-basis inputs x1 (degree <= L1) and
x2 (degree <= L2), both carrying the spins of ``spins``:

1. a_i = Q x_i                                  (App. C, a_complex = Q a_real)
2. c[s3,l3,m3] = sum_{s1+s2=s3} sum G^{(l3,m3,s3)}_{(l1,m1,s1)(l2,m2,s2)} a1[s1,l1,m1] a2[s2,l2,m2]
   for s3 in ``spins`` and l3 <= Lout        (Sec. 3.2 eq. generalized_gaunt;
                                              App. B proof: coefficient of the
                                              pointwise product of the two
                                              spin-weighted functions)
3. y = Re(Q^dagger c)                           (App. C, a_real = Re(Q^dagger a_complex))

This is y[k3] = sum_{k1,k2} T[k1,k2,k3] x1[k1] x2[k2] with
T = Re(conj(Q3) G Q1 Q2), built once per (L1, L2, Lout, spins, basis).

Readings where the paper is silent:
* output spins: every pair (s1, s2) of ``spins`` contributes to s3 = s1 + s2,
  pairs with equal s3 are summed with no normalisation, and s3 outside
  ``spins`` (e.g. +-2 for spins (-1,0,1)) is dropped;
* output degrees: l3 <= Lout only;
* slots with l < |s| are ignored on input and zero on output;
* unit path weights (W = 1) and the elementwise channel mode (App. E.1 "uuu"):
  x1 and x2 of the same (edge, channel) are multiplied.
"""

import functools

import numpy as np
import scipy.sparse as sp

from .gaunt import gauss_legendre_grid, gaunt_block
from .realbasis import BASIS_PAPER, q_matrix, real_index

_PRUNE = 1e-13


def _row_lists(Q):
    """Nonzero (column, value) pairs of each row of Q, padded to the longest row
    (two for the real bases of eq. real_swsh, four for the parity-labelled one)."""
    n = Q.shape[0]
    width = max(1, max(len(np.nonzero(Q[r])[0]) for r in range(n)))
    cols = np.zeros((n, width), dtype=np.int64)
    vals = np.zeros((n, width), dtype=np.complex128)
    for r in range(n):
        nz = np.nonzero(Q[r])[0]
        cols[r, :len(nz)] = nz
        vals[r, :len(nz)] = Q[r, nz]
    return cols, vals


class RealGauntTensor:
    """Sparse real tensor T[k1, k2, k3] of the SpinGTP map (see module docstring)."""

    def __init__(self, L1, L2, Lout, spins, basis=BASIS_PAPER, skip_triangle=True):
        spins = tuple(int(s) for s in spins)
        self.L1, self.L2, self.Lout, self.spins, self.basis = L1, L2, Lout, spins, basis
        self.n1 = len(spins) * (L1 + 1) ** 2
        self.n2 = len(spins) * (L2 + 1) ** 2
        self.n3 = len(spins) * (Lout + 1) ** 2
        theta, w_t, phi, w_p = gauss_legendre_grid(L1 + L2 + Lout)

        # Step 2: complex Gaunt entries (a, b, e, g) over complex slot indices.
        A, B, E, Gv = [], [], [], []
        for s1 in spins:
            for s2 in spins:
                s3 = s1 + s2
                if s3 not in spins:
                    continue
                for l1 in range(abs(s1), L1 + 1):
                    for l2 in range(abs(s2), L2 + 1):
                        for l3 in range(abs(s3), Lout + 1):
                            if skip_triangle and not (abs(l1 - l2) <= l3 <= l1 + l2):
                                continue
                            G = gaunt_block(l1, s1, l2, s2, l3, s3, theta, w_t, phi, w_p)
                            ia, ib = np.nonzero(G)
                            if len(ia) == 0:
                                continue
                            m1 = ia - l1
                            m2 = ib - l2
                            m3 = m1 + m2
                            A.append(real_index(spins, L1, s1, l1, 0) + m1)
                            B.append(real_index(spins, L2, s2, l2, 0) + m2)
                            E.append(real_index(spins, Lout, s3, l3, 0) + m3)
                            Gv.append(G[ia, ib])
        A = np.concatenate(A) if A else np.zeros(0, np.int64)
        B = np.concatenate(B) if B else np.zeros(0, np.int64)
        E = np.concatenate(E) if E else np.zeros(0, np.int64)
        Gv = np.concatenate(Gv) if Gv else np.zeros(0, np.complex128)
        self.n_gaunt = len(Gv)
        self._complex = (A, B, E, Gv)

        # Steps 1 and 3 folded in: T = Re(conj(Q3[e,k3]) G[a,b,e] Q1[a,k1] Q2[b,k2]).
        c1, v1 = _row_lists(q_matrix(spins, L1, basis))
        c2, v2 = _row_lists(q_matrix(spins, L2, basis))
        c3, v3 = _row_lists(q_matrix(spins, Lout, basis))
        K1, K2, K3, V = [], [], [], []
        for i in range(c1.shape[1]):
            for j in range(c2.shape[1]):
                for l in range(c3.shape[1]):
                    val = (v1[A, i] * v2[B, j] * Gv * np.conj(v3[E, l])).real
                    keep = val != 0.0
                    K1.append(c1[A, i][keep])
                    K2.append(c2[B, j][keep])
                    K3.append(c3[E, l][keep])
                    V.append(val[keep])
        K1, K2, K3, V = map(np.concatenate, (K1, K2, K3, V))
        rows = K1 * self.n2 + K2
        M = sp.coo_matrix((V, (rows, K3)), shape=(self.n1 * self.n2, self.n3)).tocsr()
        M.sum_duplicates()
        M.data[np.abs(M.data) <= _PRUNE] = 0.0
        M.eliminate_zeros()
        self.matrix = M  # rows (k1, k2) flattened, columns k3

    def apply_complex(self, a1, a2) -> np.ndarray:
        """Step 2 alone on complex coefficients: c[u,e] = sum G[a,b,e] a1[u,a] a2[u,b]."""
        A, B, E, Gv = self._complex
        a1 = np.asarray(a1, dtype=np.complex128).reshape(-1, self.n1)
        a2 = np.asarray(a2, dtype=np.complex128).reshape(-1, self.n2)
        c = np.zeros((a1.shape[0], self.n3), dtype=np.complex128)
        for u in range(a1.shape[0]):
            np.add.at(c[u], E, Gv * a1[u, A] * a2[u, B])
        return c

    @property
    def nnz(self) -> int:
        return self.matrix.nnz

    def dense(self) -> np.ndarray:
        """T as a dense [n1, n2, n3] array (small L only)."""
        return self.matrix.toarray().reshape(self.n1, self.n2, self.n3)

    def apply(self, x1, x2, chunk=None) -> np.ndarray:
        """y[u, k3] = sum T[k1,k2,k3] x1[u,k1] x2[u,k2] in float64.

        x1: [..., n1] (or [..., n_spins, (L1+1)^2]); x2 likewise; returns
        [..., n_spins, (Lout+1)^2].
        """
        x1 = np.asarray(x1, dtype=np.float64)
        x2 = np.asarray(x2, dtype=np.float64)
        ns = len(self.spins)
        if x1.ndim >= 2 and x1.shape[-2:] == (ns, (self.L1 + 1) ** 2):
            lead = x1.shape[:-2]
        else:
            lead = x1.shape[:-1]
        X1 = x1.reshape(-1, self.n1)
        X2 = x2.reshape(-1, self.n2)
        if X1.shape[0] != X2.shape[0]:
            raise ValueError("x1 and x2 hold different numbers of units")
        U = X1.shape[0]
        if chunk is None:
            chunk = max(1, min(U, (1 << 24) // max(1, self.n1 * self.n2)))
        Y = np.empty((U, self.n3))
        for u0 in range(0, U, chunk):
            u1 = min(U, u0 + chunk)
            P = (X1[u0:u1, :, None] * X2[u0:u1, None, :]).reshape(u1 - u0, -1)
            Y[u0:u1] = np.asarray(P @ self.matrix)
        return Y.reshape(lead + (len(self.spins), (self.Lout + 1) ** 2))


    def vjp(self, x1, x2, g, chunk=None):
        """Reverse-mode derivative of the bilinear map (float64).

        For a scalar loss with dL/dy = g, the chain rule on
        y[u,k3] = sum T[k1,k2,k3] x1[u,k1] x2[u,k2] gives
          gx1[u,k1] = sum_{k2,k3} T[k1,k2,k3] x2[u,k2] g[u,k3],
          gx2[u,k2] = sum_{k1,k3} T[k1,k2,k3] x1[u,k1] g[u,k3].
        Returns (gx1, gx2) shaped like x1 and x2.
        """
        x1 = np.asarray(x1, dtype=np.float64)
        x2 = np.asarray(x2, dtype=np.float64)
        X1 = x1.reshape(-1, self.n1)
        X2 = x2.reshape(-1, self.n2)
        G = np.asarray(g, dtype=np.float64).reshape(-1, self.n3)
        if not (X1.shape[0] == X2.shape[0] == G.shape[0]):
            raise ValueError("x1, x2 and g hold different numbers of units")
        U = X1.shape[0]
        if chunk is None:
            chunk = max(1, min(U, (1 << 24) // max(1, self.n1 * self.n2)))
        MT = self.matrix.T.tocsr()  # [k3, (k1, k2)]
        gx1 = np.empty((U, self.n1))
        gx2 = np.empty((U, self.n2))
        for u0 in range(0, U, chunk):
            u1 = min(U, u0 + chunk)
            R = np.asarray(G[u0:u1] @ MT).reshape(u1 - u0, self.n1, self.n2)  # sum_k3 T g
            gx1[u0:u1] = np.einsum("uab,ub->ua", R, X2[u0:u1])
            gx2[u0:u1] = np.einsum("uab,ua->ub", R, X1[u0:u1])
        return gx1.reshape(x1.shape), gx2.reshape(x2.shape)


@functools.lru_cache(maxsize=16)
def _cached_tensor(L1, L2, Lout, spins, basis):
    return RealGauntTensor(L1, L2, Lout, spins, basis)


def spingtp(x1, x2, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER) -> np.ndarray:
    """Oracle value of the SpinGTP forward for a batch of units (float64)."""
    return _cached_tensor(L1, L2, Lout, tuple(spins), basis).apply(x1, x2)


def spingtp_vjp(x1, x2, g, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Oracle gradients (gx1, gx2) of sum(g * spingtp(x1, x2)) (float64)."""
    return _cached_tensor(L1, L2, Lout, tuple(spins), basis).vjp(x1, x2, g)


def slot_blocks(spins, L) -> np.ndarray:
    """Block label of every slot of a [n_spins][(L+1)^2] vector: the irrep block
    (spin index i, degree l) as i (L+1) + l, and -1 on the slots with l < |s|.

    In the parity-labelled basis these blocks are the irreps (l, |s|, p) of the
    paper (Sec. 3.4; the -|s| block holds p = +1, the +|s| block p = -1); in the
    other bases they are the (signed spin, degree) sectors of the layout."""
    spins = tuple(spins)
    out = np.full(len(spins) * (L + 1) ** 2, -1, dtype=np.int64)
    for i, s in enumerate(spins):
        for l in range(abs(s), L + 1):
            out[i * (L + 1) ** 2 + l * l:i * (L + 1) ** 2 + (l + 1) ** 2] = i * (L + 1) + l
    return out


class PathWeightedTensor:
    """The instruction-weighted product of eq. spin_gtp (Sec. 3.4) with one weight
    per path (block triple rho1, rho2 -> rho3) shared by all channels:
    T_W[k1,k2,k3] = W[path(k1,k2,k3)] T[k1,k2,k3], path(k) = (block(k1), block(k2),
    block(k3)) of ``slot_blocks``.

    Paths are the block triples on which T has a nonzero entry, in ascending
    lexicographic order; ``weights`` holds one value per path in that order.
    Reading: the paper's W_uvw also mixes channels; this is its per-path part
    with the channel wiring of the unweighted product (elementwise, one weight
    for every channel)."""

    def __init__(self, L1, L2, Lout, spins, basis=BASIS_PAPER, weights=None):
        self.base = _cached_tensor(L1, L2, Lout, tuple(spins), basis)
        b = self.base
        M = b.matrix.tocoo()
        k1, k2 = M.row // b.n2, M.row % b.n2
        trip = np.stack([slot_blocks(spins, L1)[k1], slot_blocks(spins, L2)[k2],
                         slot_blocks(spins, Lout)[M.col]], axis=1)
        self.paths, index = np.unique(trip, axis=0, return_inverse=True)
        index = np.asarray(index).ravel()
        w = np.ones(len(self.paths)) if weights is None else np.asarray(weights, dtype=np.float64)
        if w.shape != (len(self.paths),):
            raise ValueError(f"{len(self.paths)} path weights expected")
        self.matrix = sp.csr_matrix((M.data * w[index], (M.row, M.col)), shape=M.shape)
        self.L1, self.L2, self.Lout, self.spins = L1, L2, Lout, tuple(spins)
        self.n1, self.n2, self.n3 = b.n1, b.n2, b.n3

    dense = RealGauntTensor.dense
    apply = RealGauntTensor.apply
    vjp = RealGauntTensor.vjp


def _path_entries(L1, L2, Lout, spins, basis):
    """The nonzeros of the unweighted T with their path: (k1, k2, k3, value, path),
    paths numbered as in PathWeightedTensor (ascending block triples)."""
    w = PathWeightedTensor(L1, L2, Lout, spins, basis)
    b = w.base
    M = b.matrix.tocoo()
    k1, k2, k3 = M.row // b.n2, M.row % b.n2, M.col
    trip = np.stack([slot_blocks(spins, L1)[k1], slot_blocks(spins, L2)[k2], slot_blocks(spins, Lout)[k3]], axis=1)
    lookup = {tuple(p): i for i, p in enumerate(w.paths.tolist())}
    path = np.array([lookup[tuple(t)] for t in trip.tolist()], dtype=np.int64)
    return k1, k2, k3, M.data.astype(np.float64), path, len(w.paths)


def channel_weighted_v1(x1, x2, weights, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Depthwise product with one weight per (channel, path) and the edge input
    shared by the channels (App. E.1 mode uvu with V = 1, eq. spin_gtp with
    per-channel path weights): out[n, c] = T_{W[c]}(x1[n, c], x2[n]), where
    T_{W[c]} is the PathWeightedTensor of channel c's weights.

    x1 [N, C, ...] (n1 values per unit), x2 [N, ...] (n2 per edge), weights [C, P]."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    N, C = x1.shape[:2]
    X1 = x1.reshape(N, C, -1)
    X2 = np.asarray(x2, dtype=np.float64).reshape(N, -1)
    W = np.asarray(weights, dtype=np.float64).reshape(C, -1)
    out = np.stack([PathWeightedTensor(L1, L2, Lout, spins, basis, W[c]).apply(X1[:, c], X2).reshape(N, -1)
                    for c in range(C)], axis=1) if C else np.zeros((N, 0, len(spins) * (Lout + 1) ** 2))
    return out.reshape((N, C, len(spins), (Lout + 1) ** 2))


def channel_weighted_v1_vjp(x1, x2, weights, g, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Reverse-mode derivative of channel_weighted_v1 for dL/dout = g (float64).

    The product is linear in each of x1, x2 and W, so with T_c = T_{W[c]}:
      gx1[n,c,k1] = sum_{k2,k3} T_c[k1,k2,k3] x2[n,k2] g[n,c,k3],
      gx2[n,k2]   = sum_c sum_{k1,k3} T_c[k1,k2,k3] x1[n,c,k1] g[n,c,k3]  (x2 is shared),
      gW[c,p]     = sum_n sum_{(k1,k2,k3) in path p} T[k1,k2,k3] x1[n,c,k1] x2[n,k2] g[n,c,k3].
    Returns (gx1 shaped like x1, gx2 shaped like x2, gW [C, P])."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    N, C = x1.shape[:2]
    X1 = x1.reshape(N, C, -1)
    X2 = x2.reshape(N, -1)
    G = np.asarray(g, dtype=np.float64).reshape(N, C, -1)
    W = np.asarray(weights, dtype=np.float64).reshape(C, -1)
    k1, k2, k3, val, path, n_paths = _path_entries(L1, L2, Lout, spins, basis)
    gx1 = np.zeros_like(X1)
    gx2 = np.zeros_like(X2)
    gW = np.zeros((C, n_paths))
    for c in range(C):
        a, b = PathWeightedTensor(L1, L2, Lout, spins, basis, W[c]).vjp(X1[:, c], X2, G[:, c])
        gx1[:, c] = a
        gx2 += b
        # per entry: sum over the edges of x1 x2 g, times T; then summed per path
        per_entry = (X1[:, c, k1] * X2[:, k2] * G[:, c, k3]).sum(axis=0) * val
        gW[c] = np.bincount(path, weights=per_entry, minlength=n_paths)
    return gx1.reshape(x1.shape), gx2.reshape(x2.shape), gW


def channel_weighted(x1, x2, weights, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Elementwise product with one weight per (channel, path) (App. E.1 mode uuu with
    per-channel path weights, eq. spin_gtp): out[n, c] = T_{W[c]}(x1[n, c], x2[n, c]),
    T_{W[c]} the PathWeightedTensor of channel c's weights.

    x1 [N, C, ...] (n1 values per unit), x2 [N, C, ...] (n2 per unit), weights [C, P]."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    N, C = x1.shape[:2]
    X1 = x1.reshape(N, C, -1)
    X2 = np.asarray(x2, dtype=np.float64).reshape(N, C, -1)
    W = np.asarray(weights, dtype=np.float64).reshape(C, -1)
    out = np.zeros((N, C, len(spins) * (Lout + 1) ** 2))
    for c in range(C):
        out[:, c] = PathWeightedTensor(L1, L2, Lout, spins, basis, W[c]).apply(X1[:, c], X2[:, c]).reshape(N, -1)
    return out.reshape((N, C, len(spins), (Lout + 1) ** 2))


def channel_weighted_vjp(x1, x2, weights, g, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Reverse-mode derivative of channel_weighted for dL/dout = g (float64): per unit
    the VJP of T_{W[c]}, and
      gW[c,p] = sum_n sum_{(k1,k2,k3) in path p} T[k1,k2,k3] x1[n,c,k1] x2[n,c,k2] g[n,c,k3].
    Returns (gx1 shaped like x1, gx2 shaped like x2, gW [C, P])."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    N, C = x1.shape[:2]
    X1 = x1.reshape(N, C, -1)
    X2 = x2.reshape(N, C, -1)
    G = np.asarray(g, dtype=np.float64).reshape(N, C, -1)
    W = np.asarray(weights, dtype=np.float64).reshape(C, -1)
    k1, k2, k3, val, path, n_paths = _path_entries(L1, L2, Lout, spins, basis)
    gx1 = np.zeros_like(X1)
    gx2 = np.zeros_like(X2)
    gW = np.zeros((C, n_paths))
    for c in range(C):
        a, b = PathWeightedTensor(L1, L2, Lout, spins, basis, W[c]).vjp(X1[:, c], X2[:, c], G[:, c])
        gx1[:, c] = a
        gx2[:, c] = b
        per_entry = (X1[:, c, k1] * X2[:, c, k2] * G[:, c, k3]).sum(axis=0) * val
        gW[c] = np.bincount(path, weights=per_entry, minlength=n_paths)
    return gx1.reshape(x1.shape), gx2.reshape(x2.shape), gW


def depthwise(x1, x2, weights, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Depthwise product (App. E.1 mode uvu) with V second-input channels per edge and one
    weight per (path, u, v): out[n, u] = sum_v sum_p W[v, u, p] T_p(x1[n, u], x2[n, v]),
    T_p the tensor restricted to path p (eq. spin_gtp).

    x1 [N, U, ...], x2 [N, V, ...], weights [V, U, P] (v-major, so that V = 1 is the
    layout of channel_weighted_v1)."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    N, U = x1.shape[:2]
    X2 = np.asarray(x2, dtype=np.float64).reshape(N, -1, len(spins) * (L2 + 1) ** 2)
    W = np.asarray(weights, dtype=np.float64).reshape(X2.shape[1], U, -1)
    out = np.zeros((N, U, len(spins), (Lout + 1) ** 2))
    for v in range(X2.shape[1]):
        out += channel_weighted_v1(x1, X2[:, v], W[v], L1, L2, Lout, spins, basis)
    return out


def depthwise_vjp(x1, x2, weights, g, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Reverse-mode derivative of depthwise for dL/dout = g (float64): by linearity in
    each argument, gx1 = sum_v of the V = 1 gradient for (x2[:, v], W[v]), and gx2[:, v]
    and gW[v] are the V = 1 gradients of that term.  Returns (gx1, gx2, gW) shaped like
    x1, x2 and weights."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    N, U = x1.shape[:2]
    X2 = x2.reshape(N, -1, len(spins) * (L2 + 1) ** 2)
    V = X2.shape[1]
    W = np.asarray(weights, dtype=np.float64).reshape(V, U, -1)
    gx1 = np.zeros(x1.shape)
    gx2 = np.zeros(X2.shape)
    gW = np.zeros(W.shape)
    for v in range(V):
        a, b, c = channel_weighted_v1_vjp(x1, X2[:, v], W[v], g, L1, L2, Lout, spins, basis)
        gx1 += a
        gx2[:, v] = b.reshape(N, -1)
        gW[v] = c
    return gx1, gx2.reshape(x2.shape), gW.reshape(np.asarray(weights).shape)


def fully_connected(x1, x2, weights, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Fully connected product (App. E.1 mode uvw, eq. spin_gtp): for every path p =
    (rho1, rho2 -> rho3) first
        R_p[n, u, v, k3] = sum_{(k1, k2, k3) in p} T[k1, k2, k3] x1[n, u, k1] x2[n, v, k2],
    then the dense channel mixing
        out[n, w, k3] = sum_p sum_{u, v} W[p, u, v, w] R_p[n, u, v, k3]   (k3 in rho3).
    Paths and their order as in PathWeightedTensor.

    x1 [N, U, ...] (n1 values per channel), x2 [N, V, ...] (n2), weights [P, U, V, W];
    returns [N, W, n_spins, (Lout+1)^2]."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    N, U = x1.shape[:2]
    X1 = x1.reshape(N, U, -1)
    X2 = np.asarray(x2, dtype=np.float64).reshape(N, -1, len(spins) * (L2 + 1) ** 2)
    V = X2.shape[1]
    k1, k2, k3, val, path, n_paths = _path_entries(L1, L2, Lout, spins, basis)
    Wt = np.asarray(weights, dtype=np.float64).reshape(n_paths, U, V, -1)
    out = np.zeros((N, Wt.shape[3], len(spins) * (Lout + 1) ** 2))
    for p in range(n_paths):
        e = path == p
        R = np.zeros((N, U, V, out.shape[2]))
        for a, b, c, t in zip(k1[e], k2[e], k3[e], val[e]):
            R[:, :, :, c] += t * X1[:, :, a, None] * X2[:, None, :, b]
        out += np.einsum("nuvk,uvw->nwk", R, Wt[p])
    return out.reshape((N, Wt.shape[3], len(spins), (Lout + 1) ** 2))


def fully_connected_vjp(x1, x2, weights, g, L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Reverse-mode derivative of fully_connected for dL/dout = g (float64), by the chain
    rule through R_p and the mixing:
      gR_p[n,u,v,k3] = sum_w W[p,u,v,w] g[n,w,k3],      gW[p,u,v,w] = sum_{n,k3 in p} R_p[n,u,v,k3] g[n,w,k3],
      gx1[n,u,k1]    = sum_p sum_v sum_{(k1,k2,k3) in p} T x2[n,v,k2] gR_p[n,u,v,k3],
      gx2[n,v,k2]    = sum_p sum_u sum_{(k1,k2,k3) in p} T x1[n,u,k1] gR_p[n,u,v,k3].
    Returns (gx1, gx2, gW) shaped like x1, x2 and weights."""
    spins = tuple(spins)
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    N, U = x1.shape[:2]
    X1 = x1.reshape(N, U, -1)
    X2 = x2.reshape(N, -1, len(spins) * (L2 + 1) ** 2)
    V = X2.shape[1]
    k1, k2, k3, val, path, n_paths = _path_entries(L1, L2, Lout, spins, basis)
    Wt = np.asarray(weights, dtype=np.float64).reshape(n_paths, U, V, -1)
    G = np.asarray(g, dtype=np.float64).reshape(N, Wt.shape[3], -1)
    gx1, gx2, gW = np.zeros_like(X1), np.zeros_like(X2), np.zeros_like(Wt)
    for p in range(n_paths):
        e = path == p
        R = np.zeros((N, U, V, G.shape[2]))
        for a, b, c, t in zip(k1[e], k2[e], k3[e], val[e]):
            R[:, :, :, c] += t * X1[:, :, a, None] * X2[:, None, :, b]
        gW[p] = np.einsum("nuvk,nwk->uvw", R, G)
        gR = np.einsum("uvw,nwk->nuvk", Wt[p], G)
        for a, b, c, t in zip(k1[e], k2[e], k3[e], val[e]):
            gx1[:, :, a] += t * (X2[:, None, :, b] * gR[:, :, :, c]).sum(axis=2)
            gx2[:, :, b] += t * (X1[:, :, a, None] * gR[:, :, :, c]).sum(axis=1)
    return gx1.reshape(x1.shape), gx2.reshape(x2.shape), gW.reshape(np.asarray(weights).shape)
