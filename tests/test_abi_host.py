"""Host-side tests of the C-ABI library (CPU only, no GPU calls that compute).

* the library loads and exports every function ``include/spingtp.h`` declares;
* argument checking of the host-only table entry point;
* the float64 plan tables, pushed through a numpy re-enactment of the kernel's
  five steps, reproduce the oracle.  This checks the plan builder's mathematics
  (grid, SWSH values, real-basis mixing, folded constants) before any GPU run.
"""

import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_01408_amd import _lib
from paper_2607_01408_amd.spingtp import dense_tensor_host, mfma_operands_host, plan_tables_host, pre_table_host
from tests.kernel_emulation import _operand_matrices as _operand_matrices_abi, emulate_mfma_kernel, kernel_parity_mix
from tests.oracle_helpers import valid_mask

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
S5 = (-2, -1, 0, 1, 2)
HEADER = os.path.join(ROOT, "include", "spingtp.h")


@pytest.fixture(scope="session", autouse=True)
def built_library():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2607_01408_amd import build
        build.build()
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_][a-z_0-9]*\s*\*?\s*(spingtp_[a-z_0-9]+)\s*\(",
                                 text, flags=re.M)))


def test_exports_every_declared_symbol(built_library):
    names = declared_functions()
    assert set(names) >= set(_lib.EXPORTED)
    for n in names:
        assert hasattr(built_library, n), n


def _spins(s):
    return (ctypes.c_int * len(s))(*s), len(s)


@pytest.mark.parametrize("args,status", [
    ((2, 2, 5, (-1, 0, 1), 0), 1),      # Lout > L1 + L2
    ((17, 2, 2, (-1, 0, 1), 0), 1),     # L1 > 16
    ((-1, 2, 2, (-1, 0, 1), 0), 1),     # negative degree
    ((2, 2, 2, (0, 1), 0), 1),          # not symmetric
    ((2, 2, 2, (1, 0, -1), 0), 1),      # not ascending
    ((2, 2, 2, (-1, 1), 0), 1),         # no spin 0
    ((2, 2, 2, (-2, -1, 0, 1, 2), 0), 2),  # valid; no Fourier tables for s_max = 2
    ((2, 2, 2, (-2, 0, 2), 0), 2),      # valid, not built
    ((2, 2, 2, (-1, 0, 1), 7), 1),      # unknown basis flag
    ((2, 2, 2, (-1, 0, 1), 3), 1),      # unknown basis flag
    ((2, 2, 2, (-1, 0, 1), 2), 0),      # parity-labelled basis
    ((2, 2, 2, (-1, 0, 1), 0), 0),
    ((3, 1, 4, (0,), 1), 0),
])
def test_table_entry_point_argument_checks(built_library, args, status):
    L1, L2, Lout, spins, flags = args
    arr, n = _spins(spins)
    count = ctypes.c_size_t(0)
    got = built_library.spingtp_plan_tables_host(L1, L2, Lout, arr, n, flags, None, 0, ctypes.byref(count), None)
    assert got == status


def test_status_strings(built_library):
    for s in range(7):
        assert len(_lib.message(s)) >= 2
    assert "scratch" in _lib.message(6)


def emulate_kernel(x1, x2, L1, L2, LO, spin, basis, backward=False):
    """float64 re-enactment of the forward kernel from the host tables (layout.h);
    with backward=True on the tables of spingtp_backward."""
    tab, dims = plan_tables_host(L1, L2, LO, (-1, 0, 1) if spin else (0,), basis | (0x800 if backward else 0))
    NT, NP, PB, GLOB = dims["n_theta"], dims["n_phi"], dims["per_theta_block"], dims["global_block"]
    LA, TM = max(L1, L2), max(L1, L2, LO)
    triA, triO = (LA + 1) * (LA + 2) // 2, (LO + 1) * (LO + 2) // 2
    tri = lambda L, t, l: t * (L + 1) - t * (t - 1) // 2 + (l - t)  # noqa: E731
    a0c, a0s, aup, aum, aw = 0, triA, 2 * triA, 3 * triA, 4 * triA
    e0c = aw + LA + 1
    e0s, e1p, e1m, e1z = e0c + triO, e0c + 2 * triO, e0c + 3 * triO, e0c + 4 * triO
    N0 = (tab[0:8].reshape(4, 2), tab[8:16].reshape(4, 2))  # input 1, input 2
    M0 = tab[16:24].reshape(2, 4)
    parity = tab[24] != 0.0
    COS = tab[28:28 + NP * (TM + 1)].reshape(NP, TM + 1)
    SIN = tab[28 + NP * (TM + 1):28 + 2 * NP * (TM + 1)].reshape(NP, TM + 1)
    NS = 3 if spin else 1
    U = x1.shape[0]
    assert parity == (spin and basis == 2)
    if parity:
        x1, x2 = kernel_parity_mix(x1, L1, False), kernel_parity_mix(x2, L2, False)

    def block(x, L, si):
        return x[:, si * (L + 1) ** 2:(si + 1) * (L + 1) ** 2]

    def fourier(x, L, tb, n0):
        x0 = block(x, L, 1 if spin else 0)
        P = {k: np.zeros((U, L + 1)) for k in ("Ac", "As", "Bc", "Bs", "Cc", "Cs")}
        for t in range(L + 1):
            for l in range(t, L + 1):
                P["Ac"][:, t] += x0[:, l * l + l + t] * tb[a0c + tri(LA, t, l)]
                if t:
                    P["As"][:, t] += x0[:, l * l + l - t] * tb[a0s + tri(LA, t, l)]
        d = e = np.zeros(U)
        if spin:
            xm, xp = block(x, L, 0), block(x, L, 2)
            for t in range(1, L + 1):
                up = vp = um = vm = 0.0
                for l in range(t, L + 1):
                    wp, wm = tb[aup + tri(LA, t, l)], tb[aum + tri(LA, t, l)]
                    up = up + xp[:, l * l + l + t] * wp
                    vp = vp + xp[:, l * l + l - t] * wp
                    um = um + xm[:, l * l + l + t] * wm
                    vm = vm + xm[:, l * l + l - t] * wm
                P["Bc"][:, t], P["Bs"][:, t] = up + um, -(vp + vm)
                P["Cc"][:, t], P["Cs"][:, t] = vp - vm, up - um
            wpl = sum(xp[:, l * l + l] * tb[aw + l] for l in range(1, L + 1)) if L else np.zeros(U)
            wmi = sum(xm[:, l * l + l] * tb[aw + l] for l in range(1, L + 1)) if L else np.zeros(U)
            v = n0 @ np.stack([wpl, wmi])
            P["Bc"][:, 0], P["Cc"][:, 0], d, e = v
        return P, d, e

    y = np.zeros((U, NS * (LO + 1) ** 2))
    for j in range(NT):
        tb = tab[GLOB + j * PB:GLOB + (j + 1) * PB]
        F1, d1, e1 = fourier(x1, L1, tb, N0[0])
        F2, d2, e2 = fourier(x2, L2, tb, N0[1])

        def val(P, key, L, k):
            return P[key + "c"] @ COS[k, :L + 1] + P[key + "s"] @ SIN[k, :L + 1]

        R0c, R0s, P1c, P1s, P2c, P2s = (np.zeros((U, LO + 1)) for _ in range(6))
        for k in range(NP):
            A, a = val(F1, "A", L1, k), val(F2, "A", L2, k)
            B, b = val(F1, "B", L1, k), val(F2, "B", L2, k)
            C, c = val(F1, "C", L1, k), val(F2, "C", L2, k)
            r0 = A * a + (B * b + C * c if spin else 0)
            p1, p2 = A * b + a * B, A * c + a * C
            R0c += np.outer(r0, COS[k, :LO + 1])
            R0s += np.outer(r0, SIN[k, :LO + 1])
            P1c += np.outer(p1, COS[k, :LO + 1])
            P1s += np.outer(p1, SIN[k, :LO + 1])
            P2c += np.outer(p2, COS[k, :LO + 1])
            P2s += np.outer(p2, SIN[k, :LO + 1])
        if spin:
            R0c[:, 0] += -0.5 * NP * (d1 * d2 + e1 * e2)
        B0 = (LO + 1) ** 2
        y0 = y[:, B0:2 * B0] if spin else y
        for t in range(LO + 1):
            for l in range(t, LO + 1):
                y0[:, l * l + l + t] += tb[e0c + tri(LO, t, l)] * R0c[:, t]
                if t:
                    y0[:, l * l + l - t] += tb[e0s + tri(LO, t, l)] * R0s[:, t]
        if spin:
            ym, yp = y[:, :B0], y[:, 2 * B0:]
            for t in range(1, LO + 1):
                for l in range(t, LO + 1):
                    wp, wm = tb[e1p + tri(LO, t, l)], tb[e1m + tri(LO, t, l)]
                    yp[:, l * l + l + t] += wp * (P1c[:, t] + P2s[:, t])
                    ym[:, l * l + l + t] += wm * (P1c[:, t] - P2s[:, t])
                    yp[:, l * l + l - t] += wp * (P2c[:, t] - P1s[:, t])
                    ym[:, l * l + l - t] += wm * (-P2c[:, t] - P1s[:, t])
            sP1, sP2 = math.sqrt(2) * P1c[:, 0], math.sqrt(2) * P2c[:, 0]
            sP4 = -NP * (d2 * F1["Ac"][:, 0] + d1 * F2["Ac"][:, 0])
            sP3 = NP * (e2 * F1["Ac"][:, 0] + e1 * F2["Ac"][:, 0])
            Z = M0 @ np.stack([(sP1 + sP4) / 2, (sP3 + sP2) / 2, (sP1 - sP4) / 2, (sP3 - sP2) / 2])
            for l in range(1, LO + 1):
                yp[:, l * l + l] += tb[e1z + l] * Z[0]
                ym[:, l * l + l] += tb[e1z + l] * Z[1]
    return kernel_parity_mix(y, LO, True) if parity else y


@pytest.mark.parametrize("L1,L2,LO,spin,basis", [
    (2, 2, 2, True, 0), (2, 2, 2, True, 1), (1, 1, 1, True, 0), (3, 2, 4, True, 0), (2, 3, 1, True, 1),
    (4, 4, 4, True, 0), (6, 6, 6, True, 0), (2, 2, 2, False, 0), (3, 1, 2, False, 0), (0, 0, 0, False, 0),
    (1, 3, 3, True, 0), (8, 8, 8, True, 0), (12, 12, 12, True, 1), (2, 4, 1, True, 0), (4, 1, 2, True, 1),
    (1, 3, 0, False, 0), (6, 1, 3, True, 0), (2, 2, 2, True, 2), (3, 2, 4, True, 2), (5, 5, 5, True, 2),
    (8, 8, 8, True, 2), (2, 3, 1, False, 2),
])
def test_plan_tables_reproduce_oracle(built_library, L1, L2, LO, spin, basis):
    S = (-1, 0, 1) if spin else (0,)
    rng = np.random.default_rng(L1 * 100 + L2 * 10 + LO)
    x1 = rng.standard_normal((6, len(S) * (L1 + 1) ** 2)) * valid_mask(S, L1)
    x2 = rng.standard_normal((6, len(S) * (L2 + 1) ** 2)) * valid_mask(S, L2)
    y = emulate_kernel(x1, x2, L1, L2, LO, spin, basis)
    yo = oracle.RealGauntTensor(L1, L2, LO, S, basis).apply(x1, x2).reshape(6, -1)
    assert np.abs(y - yo).max() <= 1e-12 * max(1.0, np.abs(yo).max())


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (2, 2, 2, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 1), (3, 2, 4, (-1, 0, 1), 0), (4, 4, 4, (-1, 0, 1), 1),
    (3, 1, 2, (0,), 0), (1, 1, 1, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 2), (3, 2, 4, (-1, 0, 1), 2),
    (2, 1, 2, (0,), 2), (2, 2, 2, S5, 0), (2, 2, 2, S5, 1), (2, 2, 2, S5, 2), (3, 1, 3, S5, 1),
])
def test_dense_tensor_matches_oracle(built_library, L1, L2, LO, spins, basis):
    """The library's explicit tensor (its own quadrature, the benchmark's comparator) equals the oracle's."""
    T = dense_tensor_host(L1, L2, LO, spins, basis)
    To = oracle.RealGauntTensor(L1, L2, LO, spins, basis).dense()
    assert T.shape == To.shape
    assert np.abs(T - To).max() < 1e-13


@pytest.mark.parametrize("L,basis", [(4, 0), (5, 0), (6, 0), (6, 1), (7, 0), (7, 2), (8, 0), (8, 1), (8, 2), (5, 2),
                                     (6, 2)])
def test_mfma_operand_tables_reproduce_oracle(built_library, L, basis):
    """The matrix-core kernel's data flow, re-enacted on the CPU with the exact fp16
    operand words the plan uploads, matches the oracle to fp32-like accuracy; a
    wrong lane, K or row permutation in any table gives O(1) errors."""
    S = (-1, 0, 1)
    rng = np.random.default_rng(900 + L)
    x1 = rng.standard_normal((8, 3 * (L + 1) ** 2)) * valid_mask(S, L) * 3.0
    x2 = rng.standard_normal((8, 3 * (L + 1) ** 2)) * valid_mask(S, L) * 0.01
    y = emulate_mfma_kernel(x1, x2, L, basis)
    yo = oracle.RealGauntTensor(L, L, L, S, basis).apply(x1, x2).reshape(8, -1)
    rel = np.linalg.norm(y - yo) / np.linalg.norm(yo)
    assert rel <= 1e-6, rel


def test_mfma_operands_argument_checks(built_library):
    count = ctypes.c_size_t(0)
    assert built_library.spingtp_mfma_operands_host(0, None, 0, ctypes.byref(count)) == 1
    assert built_library.spingtp_mfma_operands_host(9, None, 0, ctypes.byref(count)) == 1
    assert built_library.spingtp_mfma_operands_host(6, None, 0, None) == 1
    assert built_library.spingtp_mfma_operands_host(6, None, 0, ctypes.byref(count)) == 0
    assert count.value == 512 * (1 + 2 * 2)  # L = 6: n_phi = 19 points, two K blocks
    assert built_library.spingtp_mfma_operands_host(8, None, 0, ctypes.byref(count)) == 0
    assert count.value == 512 * (3 + 2 * 2)  # L = 8: step (B) K blocks 1, 2a, 2b; two step-(D) K blocks


def test_mfma_operands_degree8_slots(built_library):
    """At L = 8 the first step-(B) block carries sin(8 phi) at kappa 8; the second K
    block comes once per input, with cos(8 phi) only at kappa 16 (input 1) or only at
    kappa 24 (input 2), row = phi point; checked against the trig values."""
    L, NP = 8, 25
    w = mfma_operands_host(L)
    h1, l1 = _operand_matrices_abi(w[:512])
    phi = 2 * np.pi * np.arange(32) / NP
    live = np.arange(32) < NP
    assert np.abs((h1 + l1)[:, 8] - np.where(live, np.sin(8 * phi), 0.0)).max() < 1e-6
    for i in range(2):
        h2, l2 = _operand_matrices_abi(w[512 * (5 + i):512 * (6 + i)])
        k = 8 * i  # K element within the block: kappa 16 + k
        assert np.abs((h2 + l2)[:, k] - np.where(live, np.cos(8 * phi), 0.0)).max() < 1e-6
        rest = np.delete(h2, k, axis=1), np.delete(l2, k, axis=1)
        assert not np.any(rest[0]) and not np.any(rest[1])
    for k in range(1, 8):
        assert np.abs((h1 + l1)[:, 8 + k] - np.where(live, np.sin(k * phi), 0.0)).max() < 1e-6
        assert np.abs((h1 + l1)[:, k] - np.where(live, np.cos(k * phi), 0.0)).max() < 1e-6


PRE_THREADS = 256


def emulate_pre_kernel(words, x1, x2):
    """The precontracted kernel's data flow on the CPU with the exact table words:
    per k3 block, each thread's running fp32 sum over its items, stored at `last`,
    builds that block of the transposed edge kernel; the product runs in float64
    with the invalid x1 slots read as 0.  x1 [C, NC1] of one edge, x2 [NC2]."""
    nc1, nc2, nco, blk1, ks, nt, ipt, kst, nb3, rb, stride = (int(v) for v in words[:11])
    pairs = words[16:16 + 2 * nb3 * stride * PRE_THREADS].reshape(nb3, stride, PRE_THREADS, 2)
    X2 = x2.astype(np.float32)
    Kt = np.zeros((nb3 * rb, kst), dtype=np.float32)
    for b in range(nb3):
        items = pairs[b, :, :, 0]
        vals = pairs[b, :, :, 1].copy().view(np.float32)
        blk = np.zeros(rb * kst, dtype=np.float32)
        acc = np.zeros(PRE_THREADS, dtype=np.float32)
        for i in range(stride):
            w = items[i]
            acc = (vals[i].astype(np.float64) * X2[(w >> 16) & 0xFF] + acc).astype(np.float32)  # one fp32 rounding
            last = (w >> 24) != 0
            blk[(w & 0xFFFF)[last]] = acc[last]
            acc[last] = 0.0
        Kt[b * rb:(b + 1) * rb] = blk.reshape(rb, kst)
    K = Kt[:nco, :nc1].T.astype(np.float64)
    ns = int(words[11])
    k = np.arange(nc1)
    sa = np.abs(k // blk1 - ns // 2)
    x1 = np.where(k % blk1 >= sa * sa, x1, 0.0)  # slots with l < |s| are read as 0
    return x1 @ K, K


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (1, 1, 1, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 0), (1, 3, 3, (-1, 0, 1), 0), (3, 1, 2, (-1, 0, 1), 0),
    (4, 4, 4, (-1, 0, 1), 0), (4, 2, 3, (-1, 0, 1), 1), (3, 3, 3, (-1, 0, 1), 1), (7, 7, 7, (0,), 0),
    (5, 2, 6, (0,), 0), (5, 5, 5, (-1, 0, 1), 0), (6, 6, 6, (-1, 0, 1), 1), (1, 6, 6, (-1, 0, 1), 0),
    (6, 2, 5, (-1, 0, 1), 0), (3, 3, 3, (-1, 0, 1), 2), (6, 6, 6, (-1, 0, 1), 2), (2, 4, 3, (-1, 0, 1), 2),
    (2, 2, 2, S5, 0), (3, 3, 3, S5, 1), (4, 4, 4, S5, 0), (4, 4, 4, S5, 2), (1, 2, 3, S5, 0), (2, 1, 2, S5, 2),
    (0, 2, 2, S5, 0)])
def test_pre_table_reproduces_oracle(built_library, L1, L2, LO, spins, basis):
    """The precontracted kernel's table, re-enacted on the CPU, gives the oracle's
    edge kernel K[k1, k3] = sum_k2 T x2 and the oracle's outputs for channels that
    share x2; every entry has one writer, inside the padded LDS block."""
    words = pre_table_host(L1, L2, LO, spins, basis)
    nc1, nc2, nco, blk1, ks, nt, ipt, kst, nb3, rb, stride = (int(v) for v in words[:11])
    ns = len(spins)
    assert (nc1, nc2, nco) == (ns * (L1 + 1) ** 2, ns * (L2 + 1) ** 2, ns * (LO + 1) ** 2)
    assert blk1 == (L1 + 1) ** 2 and int(words[11]) == ns
    assert (ks, nt, kst) == (-(-nc1 // 16), -(-nco // 16), 16 * -(-nc1 // 16) + 4)
    assert (nb3, rb) == ((1, 16 * nt) if ks <= 5 and nt <= 5 else (-(-16 * nt // 48), 48))
    blocked = ks > 5 or nt > 5
    assert stride == (ipt + 16 if blocked else ipt) and ipt % (16 if blocked else 8) == 0
    assert words.size == 16 + 2 * nb3 * stride * PRE_THREADS
    assert int(words[12]) == nc1 and not words[13:16].any()
    assert not words[16:].reshape(nb3, stride, PRE_THREADS, 2)[:, ipt:].any()  # zero padding
    items = words[16::2].reshape(nb3, -1)
    vals = words[17::2].copy().view(np.float32)
    blocks = np.repeat(np.arange(nb3), items.shape[1]).reshape(nb3, -1)
    last = (items >> 24) != 0
    stores = (items & 0xFFFF)[last] + (blocks * rb * kst)[last]  # position in the whole kernel
    assert len(np.unique(stores)) == len(stores)  # one writer per entry
    assert np.all((items & 0xFFFF)[last] < rb * kst)  # inside the block
    items = items.ravel()
    assert np.all(stores % kst < nc1) and np.all(stores // kst < nco)
    assert np.all(((items >> 16) & 0xFF) < nc2)
    assert np.all(items[vals == 0] == 0)  # padding items are all-zero
    T = oracle.RealGauntTensor(L1, L2, LO, spins, basis).dense()
    pattern = np.abs(T).max(axis=1) > 1e-12  # entries (k1, k3) with a nonzero list
    assert len(stores) == pattern.sum()
    assert np.array_equal(np.sort(stores), np.sort((np.nonzero(pattern.T)[0] * kst + np.nonzero(pattern.T)[1])))
    rng = np.random.default_rng(31 + L1 + 7 * L2 + 49 * LO)
    C = 5
    x1 = rng.standard_normal((C, nc1))
    x2 = rng.standard_normal(nc2) * valid_mask(spins, L2)
    y, K = emulate_pre_kernel(words, x1 * valid_mask(spins, L1), x2)
    Kref = np.einsum("akb,k->ab", T, x2)
    assert np.abs(K - Kref).max() <= 1e-6 * np.abs(Kref).max()
    yo = oracle.RealGauntTensor(L1, L2, LO, spins, basis).apply(x1 * valid_mask(spins, L1),
                                                                np.broadcast_to(x2, (C, nc2))).reshape(C, -1)
    rel = np.linalg.norm(y - yo) / np.linalg.norm(yo)
    assert rel <= 1e-6, rel
    # the kernel ignores what the invalid slots of x1 hold
    if ns > 1:
        poisoned = x1.copy()
        poisoned[:, ~valid_mask(spins, L1)] = 1e30
        assert np.array_equal(emulate_pre_kernel(words, poisoned * 1.0, x2)[0], y)


def test_pre_table_argument_checks(built_library):
    count = ctypes.c_size_t(0)
    S = (ctypes.c_int * 3)(-1, 0, 1)
    assert built_library.spingtp_pre_table_host(7, 7, 7, S, 3, 0, None, 0, ctypes.byref(count)) == 2  # NC 192
    assert built_library.spingtp_pre_table_host(6, 7, 6, S, 3, 0, None, 0, ctypes.byref(count)) == 2
    S0 = (ctypes.c_int * 1)(0)
    assert built_library.spingtp_pre_table_host(8, 8, 8, S0, 1, 0, None, 0, ctypes.byref(count)) == 2  # KS = 6
    assert built_library.spingtp_pre_table_host(6, 6, 6, S, 3, 0, None, 0, ctypes.byref(count)) == 0
    assert built_library.spingtp_pre_table_host(4, 4, 4, S, 3, 0, None, 0, None) == 1
    assert built_library.spingtp_pre_table_host(-1, 4, 4, S, 3, 0, None, 0, ctypes.byref(count)) == 1
    assert built_library.spingtp_pre_table_host(4, 4, 4, S, 3, 0, None, 0, ctypes.byref(count)) == 0
    assert count.value > 8


def test_plan_create_route_flags(built_library):
    """Flag checks of spingtp_plan_create that return before any device call."""
    S = (ctypes.c_int * 3)(-1, 0, 1)
    plan = ctypes.c_void_p()
    # SPINGTP_V1_FOURIER and SPINGTP_V1_PRECONTRACT together
    assert built_library.spingtp_plan_create(2, 2, 2, S, 3, 0, 0x200 | 0x400, ctypes.byref(plan)) == 1
    # precontraction forced where no precontracted kernel is built (rows of 192)
    assert built_library.spingtp_plan_create(7, 7, 7, S, 3, 0, 0x400, ctypes.byref(plan)) == 2
    assert built_library.spingtp_plan_create(2, 2, 2, S, 3, 0, 0x800, ctypes.byref(plan)) == 1  # tables-only bit
    assert built_library.spingtp_plan_create(2, 2, 2, S, 3, 0, 0x4000, ctypes.byref(plan)) == 1  # unknown bit


@pytest.mark.parametrize("L", [0, 1, 2, 4, 6, 16])
@pytest.mark.parametrize("spins,basis", [((-1, 0, 1), 0), ((-1, 0, 1), 1), ((0,), 0), ((-1, 0, 1), 2), (S5, 0),
                                         (S5, 1), (S5, 2)])
def test_conj_map_matches_oracle(built_library, L, spins, basis):
    """The library's conjugation map (used by spingtp_backward) equals the oracle's J."""
    from oracle.realbasis import conjugation_map
    from paper_2607_01408_amd.spingtp import conj_map_host

    words = conj_map_host(L, spins, basis)
    n = len(spins) * (L + 1) ** 2
    assert words.size == n
    J = np.zeros((n, n))
    for j, w in enumerate(words):
        if w & (1 << 17):
            continue
        J[j, w & 0xFFFF] = -1.0 if w & (1 << 16) else 1.0
    if L <= 6:
        assert np.array_equal(J, conjugation_map(spins, L, basis))
    live = valid_mask(spins, L)
    assert np.array_equal((words & (1 << 17)) == 0, live)


@pytest.mark.parametrize("L,spin,basis", [(1, True, 0), (2, True, 0), (3, True, 1), (4, True, 0), (6, True, 0),
                                          (3, False, 0), (8, True, 0), (2, True, 2), (5, True, 2), (8, True, 2)])
def test_backward_tables_reproduce_oracle(built_library, L, spin, basis):
    """spingtp_backward runs the forward kernel on (grad_out, x2) with its backward
    tables; re-enacted on the CPU from those tables this is the oracle's grad_x1
    (and, with x1 in place of x2, its grad_x2)."""
    spins = (-1, 0, 1) if spin else (0,)
    rng = np.random.default_rng(70 + L)
    n = len(spins) * (L + 1) ** 2
    x1, x2, g = (rng.standard_normal((4, n)) * valid_mask(spins, L) for _ in range(3))
    r1, r2 = oracle.RealGauntTensor(L, L, L, spins, basis).vjp(x1, x2, g)
    y1 = emulate_kernel(g, x2, L, L, L, spin, basis, backward=True)
    y2 = emulate_kernel(g, x1, L, L, L, spin, basis, backward=True)
    assert np.abs(y1 - r1).max() <= 1e-12 * max(1.0, np.abs(r1).max())
    assert np.abs(y2 - r2).max() <= 1e-12 * max(1.0, np.abs(r2).max())
    if spin and basis == 0 and L > 0:
        # the paper basis needs the conjugation: the forward tables alone give a different map
        assert np.abs(emulate_kernel(g, x2, L, L, L, spin, basis) - r1).max() > 1e-3


@pytest.mark.parametrize("L,spins,basis", [(1, (-1, 0, 1), 0), (3, (-1, 0, 1), 0), (4, (-1, 0, 1), 1),
                                           (5, (-1, 0, 1), 0), (6, (-1, 0, 1), 0), (4, (0,), 0),
                                           (3, (-1, 0, 1), 2), (6, (-1, 0, 1), 2)])
def test_backward_pre_table_reproduces_oracle(built_library, L, spins, basis):
    """spingtp_backward_v1's grad_x1 on the precontracted kernel: its table (x2
    indices and signs through J), re-enacted on (grad_out, x2), gives the oracle's
    grad_x1 for channels that share x2."""
    words = pre_table_host(L, L, L, spins, basis, backward=True)
    rng = np.random.default_rng(200 + L)
    n = len(spins) * (L + 1) ** 2
    C = 3
    x1 = rng.standard_normal((C, n)) * valid_mask(spins, L)
    x2 = rng.standard_normal(n) * valid_mask(spins, L)
    g = rng.standard_normal((C, n)) * valid_mask(spins, L)
    y, _ = emulate_pre_kernel(words, g, x2)
    r1, _ = oracle.RealGauntTensor(L, L, L, spins, basis).vjp(x1, np.broadcast_to(x2, (C, n)), g)
    assert np.abs(y - r1).max() <= 1e-6 * max(1.0, np.abs(r1).max())


def emulate_direct_kernel(words, A, B):
    """The direct kernel (family 6) on the CPU from its exact table words: per
    output slot, its 16-entry batches in order, products A[a] * B[b] rounded to
    fp32 and added with one fp32 fma each into two alternating sums (even entries
    of a batch to the first), which are added at the end of the slot."""
    na, nb, no, sta, stb, sto, nbatch, per = (int(v) for v in words[:8])
    assert per == 16
    W = 4  # waves per workgroup, each with a contiguous range of output slots
    oseg, bseg = words[8:8 + W + 1].astype(np.int64), words[8 + W + 1:8 + 2 * W + 2].astype(np.int64)
    hdr = 8 + 2 * (W + 1)
    counts = words[hdr:hdr + no].astype(np.int64)
    assert counts.sum() == nbatch
    assert oseg[0] == 0 and oseg[-1] == no and np.all(np.diff(oseg) >= 0)
    assert np.array_equal(bseg, np.concatenate([[0], np.cumsum(counts)])[oseg])  # batch start of each range
    body = words[hdr + no:]
    assert body.size == 24 * (nbatch + 2) and not body[24 * nbatch:].any()  # the trailing zero batches
    batches = body[:24 * nbatch].reshape(nbatch, 24)
    idx = np.stack([batches[:, :8] & 0xFFFF, batches[:, :8] >> 16], axis=2).reshape(nbatch, 16)
    ent = (idx & 0xFF) | ((idx >> 8) << 16)  # as a | b << 16
    val = batches[:, 8:].copy().view(np.float32)
    U = A.shape[0]
    Az = np.zeros((U, sta), dtype=np.float32)
    Bz = np.zeros((U, stb), dtype=np.float32)
    Az[:, :na], Bz[:, :nb] = A, B
    out = np.zeros((U, no), dtype=np.float32)
    q = 0
    for o in range(no):
        acc = [np.zeros(U, dtype=np.float32), np.zeros(U, dtype=np.float32)]
        for _ in range(counts[o]):
            for i in range(16):
                a, b = int(ent[q, i] & 0xFFFF), int(ent[q, i] >> 16)
                p = (Az[:, a] * Bz[:, b]).astype(np.float32)
                acc[i % 2] = (val[q, i].astype(np.float64) * p + acc[i % 2]).astype(np.float32)
            q += 1
        out[:, o] = acc[0] + acc[1]
    return out.astype(np.float64)


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (2, 2, 2, S5, 0), (2, 2, 2, S5, 1), (2, 2, 2, S5, 2), (3, 3, 3, S5, 0), (1, 2, 2, S5, 0), (2, 1, 3, S5, 2),
    (0, 2, 2, S5, 0), (4, 4, 4, S5, 0), (3, 2, 4, (-1, 0, 1), 0), (2, 4, 3, (-1, 0, 1), 1), (5, 5, 5, (0,), 0),
    (2, 3, 4, (0,), 0)])
def test_direct_table_reproduces_oracle(built_library, L1, L2, LO, spins, basis):
    """The direct kernel's three tables, re-enacted on the CPU from the exact words,
    give the oracle's forward and both gradients (fp32 arithmetic: 1e-6); entries
    are exactly the nonzeros of T, padding points at the zero columns, and what the
    l < |s| input slots hold is never read."""
    from paper_2607_01408_amd.spingtp import direct_table_host

    ns = len(spins)
    n1, n2, no = ns * (L1 + 1) ** 2, ns * (L2 + 1) ** 2, ns * (LO + 1) ** 2
    G = oracle.RealGauntTensor(L1, L2, LO, spins, basis)
    T = G.dense()
    rng = np.random.default_rng(5 + L1 + 3 * L2 + 9 * LO + 27 * basis)
    U = 7
    x1 = rng.standard_normal((U, n1)) * valid_mask(spins, L1)
    x2 = rng.standard_normal((U, n2)) * valid_mask(spins, L2)
    g = rng.standard_normal((U, no)) * valid_mask(spins, LO)
    r1, r2 = G.vjp(x1, x2, g)
    y = G.apply(x1, x2).reshape(U, -1)
    for role, (A, B, ref, widths) in enumerate([(x1, x2, y, (n1, n2, no)), (g, x2, r1, (no, n2, n1)),
                                                (g, x1, r2, (no, n1, n2))]):
        w = direct_table_host(L1, L2, LO, spins, basis, role)
        na, nb, nout, sta, stb, sto, nbatch = (int(v) for v in w[:7])
        assert (na, nb, nout) == widths and w[7] == 16
        for n, st in ((na, sta), (nb, stb), (nout, sto)):
            assert st % 2 == 1 and st > n
        hdr = 18
        body = w[hdr + nout:hdr + nout + 24 * nbatch].reshape(nbatch, 24)
        # the four waves' shares of the batches are balanced (whole output slots each)
        shares = np.diff(w[13:18].astype(np.int64))
        assert shares.max() <= nbatch / 4 + w[hdr:hdr + nout].max()
        ent = np.stack([body[:, :8] & 0xFFFF, body[:, :8] >> 16], axis=2).ravel()
        val = body[:, 8:].copy().view(np.float32).ravel()
        pad = val == 0
        assert np.all(ent[pad] == (na | (nb << 8)))
        # the entries are the nonzeros of T in this role (k1, k2, k3 permuted)
        perm = [(0, 1, 2), (2, 1, 0), (2, 0, 1)][role]
        Tr = np.transpose(T, perm)  # [a][b][o] with a, b, o the role's indices
        assert (~pad).sum() == (np.abs(Tr) > 0).sum()
        out = emulate_direct_kernel(w, A, B)
        assert np.linalg.norm(out - ref) <= 1e-6 * max(np.linalg.norm(ref), 1e-30), role
        if ns > 1:  # poisoned invalid slots are never read
            Ap = np.where(valid_mask(spins, (L1, LO, LO)[role]), A, 1e30)
            Bp = np.where(valid_mask(spins, (L2, L2, L1)[role]), B, 1e30)
            assert np.array_equal(emulate_direct_kernel(w, Ap, Bp), out)


def test_direct_table_argument_checks(built_library):
    count = ctypes.c_size_t(0)
    S = (ctypes.c_int * 5)(-2, -1, 0, 1, 2)
    assert built_library.spingtp_direct_table_host(2, 2, 2, S, 5, 0, 3, None, 0, ctypes.byref(count)) == 1
    assert built_library.spingtp_direct_table_host(2, 2, 2, S, 5, 0, -1, None, 0, ctypes.byref(count)) == 1
    assert built_library.spingtp_direct_table_host(2, 2, 2, S, 5, 0, 0, None, 0, None) == 1
    # rows beyond the 8-bit entry indices: 320 slots at degree 7 with spins {-2..2}
    assert built_library.spingtp_direct_table_host(7, 7, 7, S, 5, 0, 0, None, 0, ctypes.byref(count)) == 2
    assert built_library.spingtp_direct_table_host(2, 2, 2, S, 5, 0, 0, None, 0, ctypes.byref(count)) == 0
    assert count.value > 8
    # the Fourier tables do not exist for spins {-2..2}
    n = ctypes.c_size_t(0)
    assert built_library.spingtp_plan_tables_host(2, 2, 2, S, 5, 0, None, 0, ctypes.byref(n), None) == 2


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [(2, 2, 2, S5, 0), (2, 1, 3, (-1, 0, 1), 1), (2, 2, 2, (-1, 0, 1), 2),
                                                   (3, 2, 1, (0,), 0), (4, 4, 4, (-1, 0, 1), 0)])
def test_paths_match_oracle(built_library, L1, L2, LO, spins, basis):
    """The library's path list (block triples with a nonzero tensor entry, in order) is the oracle's."""
    from paper_2607_01408_amd.spingtp import paths_host

    assert np.array_equal(paths_host(L1, L2, LO, spins, basis), oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)


def test_weighted_plan_argument_checks(built_library):
    """Checks of spingtp_plan_create_weighted that return before any device call."""
    from paper_2607_01408_amd.spingtp import paths_host

    S = (ctypes.c_int * 3)(-1, 0, 1)
    plan = ctypes.c_void_p()
    n = len(paths_host(2, 2, 2))
    w = (ctypes.c_double * (n + 1))(*([1.0] * (n + 1)))
    f = built_library.spingtp_plan_create_weighted
    assert f(2, 2, 2, S, 3, 0, 0, None, n, ctypes.byref(plan)) == 1  # no weights
    assert f(2, 2, 2, S, 3, 0, 0, w, n + 1, ctypes.byref(plan)) == 1  # one per path
    assert f(2, 2, 2, S, 3, 0, 0, w, n - 1, ctypes.byref(plan)) == 1
    assert f(2, 2, 2, S, 3, 0, 0x200, w, n, ctypes.byref(plan)) == 2  # the Fourier route has no path weights
    w[3] = float("nan")
    assert f(2, 2, 2, S, 3, 0, 0, w, n, ctypes.byref(plan)) == 1  # weights must be finite
    assert not plan.value


def emulate_pre_weighted(words, x1, x2, W):
    """The per-channel path-weighted precontracted kernel on the CPU from its exact
    table words: the edge kernel K[q][k3] over path slots q built like the unweighted
    one (fp32 running sums per thread), then out[c] = sum_q K[q] W[c, path(q)] x1[c, k1(q)]
    in float64.  x1 [C, NC1], x2 [NC2], W [C, n_paths]."""
    Q, nc2, nco, blk1, ks, nt, ipt, kst, nb3, rb, stride, ns, nc1, npaths, qoff = (int(v) for v in words[:15])
    assert nb3 == 1 and rb == 16 * nt and stride == ipt and Q <= 16 * ks
    pairs = words[16:16 + 2 * stride * PRE_THREADS].reshape(stride, PRE_THREADS, 2)
    X2 = x2.astype(np.float32)
    blk = np.zeros(rb * kst, dtype=np.float32)
    acc = np.zeros(PRE_THREADS, dtype=np.float32)
    vals = pairs[:, :, 1].copy().view(np.float32)
    for i in range(stride):
        w = pairs[i, :, 0]
        acc = (vals[i].astype(np.float64) * X2[(w >> 16) & 0xFF] + acc).astype(np.float32)
        last = (w >> 24) != 0
        blk[(w & 0xFFFF)[last]] = acc[last]
        acc[last] = 0.0
    K = blk.reshape(rb, kst)[:nco, :Q].T.astype(np.float64)  # [q, k3]
    qm = words[qoff:qoff + Q]
    k1, path = (qm & 0xFFFF).astype(np.int64), (qm >> 16).astype(np.int64)
    assert path.max() < npaths and k1.max() < nc1
    A = W[:, path] * x1[:, k1]  # [C, Q]
    return A @ K


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [(1, 1, 1, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 0),
                                                   (1, 3, 3, (-1, 0, 1), 1), (2, 2, 2, (0,), 0),
                                                   (4, 4, 4, (0,), 0), (2, 1, 2, (-1, 0, 1), 2)])
def test_channel_weighted_pre_table_reproduces_oracle(built_library, L1, L2, LO, spins, basis):
    """spingtp_forward_v1_weighted's table, re-enacted on the CPU with per-channel weights, gives for
    every channel the oracle's path-weighted product with that channel's weights."""
    from paper_2607_01408_amd.spingtp import paths_host

    words = pre_table_host(L1, L2, LO, spins, basis, channel_weights=True)
    P = paths_host(L1, L2, LO, spins, basis)
    assert int(words[13]) == len(P)
    rng = np.random.default_rng(3 + L1 + 5 * L2 + 25 * LO)
    C = 4
    W = rng.standard_normal((C, len(P)))
    x1 = rng.standard_normal((C, len(spins) * (L1 + 1) ** 2)) * valid_mask(spins, L1)
    x2 = rng.standard_normal(len(spins) * (L2 + 1) ** 2) * valid_mask(spins, L2)
    y = emulate_pre_weighted(words, x1, x2, W)
    for c in range(C):
        yo = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, W[c]).apply(x1[c:c + 1], x2[None]).reshape(-1)
        assert np.linalg.norm(y[c] - yo) <= 1e-6 * np.linalg.norm(yo), c


def emulate_bwd_v1w(words, x1, x2, W, g):
    """The arithmetic of spingtp_backward_v1_weighted on its entry lists, for one edge: x1 and g
    [C, n] rows of the edge's channels, x2 its shared row, W [C, n_paths].  Each list segment
    is summed as the kernel sums it (value times the gathered product), the zero columns past
    each row included.  Returns (gx1 [C, NC1], gx2 [NC2], gW [C, NP]) in float64."""
    nc1, nc2, nco, npth = (int(v) for v in words[:4])
    seg = [words[int(words[5 + i]):] for i in range(3)]
    lst = [words[int(words[8 + i]):] for i in range(3)]

    def entries(i, key):
        e0, e1 = int(seg[i][key]), int(seg[i][key + 1])
        assert e0 % 8 == 0 and e1 % 8 == 0
        w = lst[i][2 * e0:2 * e1].reshape(-1, 2)
        f = w[:, 0].astype(np.int64)
        return f & 0x3ff, (f >> 10) & 0x3ff, f >> 20, w[:, 1].view(np.float32).astype(np.float64)

    C = x1.shape[0]
    pad = lambda a: np.concatenate([a, np.zeros(a.shape[:-1] + (1,))], axis=-1)  # the zero column
    X1, X2, G, Wp = pad(x1), pad(x2), pad(g), pad(W)
    gx1 = np.zeros((C, nc1))
    gx2 = np.zeros(nc2)
    gW = np.zeros((C, npth))
    for k1 in range(nc1):
        p, k2, k3, v = entries(0, k1)
        gx1[:, k1] = (v * X2[k2] * Wp[:, p] * G[:, k3]).sum(axis=1)
    for k2 in range(nc2):
        p, a, k3, v = entries(1, k2)
        gx2[k2] = (v * Wp[:, p] * X1[:, a] * G[:, k3]).sum()
    for q in range(npth):
        a, b, k3, v = entries(2, q)
        gW[:, q] = (v * X2[b] * X1[:, a] * G[:, k3]).sum(axis=1)
    return gx1, gx2, gW


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [(1, 1, 1, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 2),
                                                   (1, 3, 3, (-1, 0, 1), 0), (2, 1, 2, (-2, -1, 0, 1, 2), 1),
                                                   (3, 2, 1, (0,), 0)])
def test_weighted_backward_lists_reproduce_oracle(built_library, L1, L2, LO, spins, basis):
    """spingtp_backward_v1_weighted's three entry lists, re-enacted on the CPU, give the oracle's
    gradients of the per-channel path-weighted product; every nonzero of T is in each list once."""
    from paper_2607_01408_amd.spingtp import paths_host

    words = pre_table_host(L1, L2, LO, spins, basis, backward=True, channel_weights=True)
    P = paths_host(L1, L2, LO, spins, basis)
    n1, n2, n3 = (len(spins) * (L + 1) ** 2 for L in (L1, L2, LO))
    assert [int(v) for v in words[:4]] == [n1, n2, n3, len(P)]
    for i, n in enumerate((n1, n2, len(P))):  # real entries per list: the tensor's nonzeros
        s = words[int(words[5 + i]):int(words[5 + i]) + n + 1].astype(np.int64)
        ent = words[int(words[8 + i]):][:2 * int(s[-1])].reshape(-1, 2)
        assert int((ent[:, 1] != 0).sum()) == int(words[4])
        assert np.all(np.diff(s) % 8 == 0) and s[0] == 0
        kr = words[16 + 5 * i:21 + 5 * i].astype(np.int64)  # the four waves' key ranges
        assert kr[0] == 0 and kr[-1] == n and np.all(np.diff(kr) >= 0)
        tail = words[int(words[8 + i]) + 2 * int(s[-1]):][:2 * 96].reshape(-1, 2)  # prefetch padding
        assert tail.shape == (96, 2) and not tail[:, 1].any()
    rng = np.random.default_rng(7 + L1 + 5 * L2 + 25 * LO)
    N, C = 2, 3
    W = rng.standard_normal((C, len(P)))
    x1 = rng.standard_normal((N, C, n1)) * valid_mask(spins, L1).ravel()
    x2 = rng.standard_normal((N, n2)) * valid_mask(spins, L2).ravel()
    g = rng.standard_normal((N, C, n3)) * valid_mask(spins, LO).ravel()
    r1, r2, rW = oracle.channel_weighted_v1_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)
    gW = np.zeros_like(W)
    for n in range(N):
        e1, e2, eW = emulate_bwd_v1w(words, x1[n], x2[n], W, g[n])
        assert np.linalg.norm(e1 - r1[n]) <= 1e-6 * np.linalg.norm(r1[n])
        assert np.linalg.norm(e2 - r2[n]) <= 1e-6 * np.linalg.norm(r2[n])
        gW += eW
    assert np.linalg.norm(gW - rW) <= 1e-6 * np.linalg.norm(rW)
    # the k3-ordered list (spingtp_forward_weighted, x2 per unit) and its key ranges
    s3 = words[int(words[11]):int(words[11]) + n3 + 1].astype(np.int64)
    l3 = words[int(words[12]):]
    kr = words[31:36].astype(np.int64)
    assert kr[0] == 0 and kr[-1] == n3 and np.all(np.diff(kr) >= 0) and np.all(np.diff(s3) % 8 == 0)
    x2u = rng.standard_normal((N, C, n2)) * valid_mask(spins, L2).ravel()
    ref = oracle.channel_weighted(x1, x2u, W, L1, L2, LO, spins, basis).reshape(N, C, -1)
    pad = lambda a: np.concatenate([a, np.zeros(a.shape[:-1] + (1,))], axis=-1)
    X1, X2, Wp = pad(x1), pad(x2u), pad(W)
    y = np.zeros((N, C, n3))
    for k3 in range(n3):
        w = l3[2 * int(s3[k3]):2 * int(s3[k3 + 1])].reshape(-1, 2)
        f = w[:, 0].astype(np.int64)
        p, a, b = f & 0x3ff, (f >> 10) & 0x3ff, f >> 20
        v = w[:, 1].view(np.float32).astype(np.float64)
        y[:, :, k3] = (v * Wp[None, :, p] * X1[:, :, a] * X2[:, :, b]).sum(axis=-1)
    assert np.linalg.norm(y - ref) <= 1e-6 * np.linalg.norm(ref)


@pytest.mark.parametrize("L1,L2,LO,spins,dtype,basis", [
    (6, 6, 6, (-1, 0, 1), 0, 0),     # matrix-core plan: tables, backward tables, operand words
    (2, 2, 2, (-1, 0, 1), 0, 2),     # precontracted v1 kernel and its conjugated table
    (2, 2, 2, S5, 1, 1),             # direct kernel with its two gradient tables
    (1, 3, 3, (-1, 0, 1), 0, 0),
])
def test_plan_upload_failure_releases_everything(built_library, L1, L2, LO, spins, dtype, basis):
    """Plan creation's device upload, driven on the host with an allocator that fails at
    each allocation in turn: the status is SPINGTP_ERR_OUT_OF_MEMORY and every buffer
    allocated before the failure has been released."""
    arr = (ctypes.c_int * len(spins))(*spins)
    n_allocs, n_live = ctypes.c_int(-1), ctypes.c_int(-1)
    st = built_library.spingtp_plan_upload_selftest_host(L1, L2, LO, arr, len(spins), dtype, basis, -1,
                                                         ctypes.byref(n_allocs), ctypes.byref(n_live))
    assert st == 0 and n_live.value == n_allocs.value   # a successful upload holds every buffer
    total = n_allocs.value
    assert total >= 2
    for k in range(total):
        st = built_library.spingtp_plan_upload_selftest_host(L1, L2, LO, arr, len(spins), dtype, basis, k,
                                                             ctypes.byref(n_allocs), ctypes.byref(n_live))
        assert st == 3, (k, st)              # SPINGTP_ERR_OUT_OF_MEMORY
        assert n_allocs.value == k + 1       # nothing attempted after the failure
        assert n_live.value == 0             # nothing leaked
    # argument rules are those of spingtp_plan_create
    bad = built_library.spingtp_plan_upload_selftest_host(17, 2, 2, arr, len(spins), dtype, basis, -1,
                                                          ctypes.byref(n_allocs), ctypes.byref(n_live))
    assert bad == 1


def emulate_uvw_table(words, x1, x2, W, nco, role=0):
    """float64 re-enactment of the fully connected product from an entry table: per
    output block and path, R from the entries (ka | kb << 16, value) of each component,
    then the channel mixing with the path's weights W [path][A][B][out].  role 0: the
    forward (x1, x2 -> out); 1: grad_x1 (x2, grad_out -> x1 slots); 2: grad_x2 (x1,
    grad_out -> x2 slots).  A path record's words 3..5 are its blocks of x1, x2, out."""
    ax_a, ax_b, ax_o = ((0, 1, 2), (1, 2, 0), (0, 2, 1))[role]
    w = np.asarray(words, dtype=np.uint32)
    n_paths, n_blocks, nc1, nc2, nco_t, max_d3, rec0, ent0 = (int(v) for v in w[:8])
    assert nco_t == nco
    vals = w.view(np.float32)
    N, U, V = x1.shape[0], x1.shape[1], x2.shape[1]
    out = np.zeros((N, W.shape[3], nco))
    seen = set()
    for b in range(n_blocks):
        o3, d3, first, count = (int(v) for v in w[8 + 4 * b:12 + 4 * b])
        assert d3 <= max_d3
        for r in range(first, first + count):
            pid, d3r, csr = (int(v) for v in w[rec0 + 6 * r:rec0 + 6 * r + 3])
            blocks = [int(v) for v in w[rec0 + 6 * r + 3:rec0 + 6 * r + 6]]
            assert d3r == d3 and pid not in seen
            assert (blocks[ax_o] & 0xFFFF, blocks[ax_o] >> 16) == (o3, d3)      # the path's output block
            ba, bb = blocks[ax_a], blocks[ax_b]
            seen.add(pid)
            for m3 in range(d3):
                for k in range(int(w[csr + m3]), int(w[csr + m3 + 1])):
                    ix = int(w[ent0 + 2 * k])
                    t = float(vals[ent0 + 2 * k + 1])
                    # the entry lies in the path's blocks of its two inputs
                    assert 0 <= (ix & 0xFFFF) - (ba & 0xFFFF) < ba >> 16 and 0 <= (ix >> 16) - (bb & 0xFFFF) < bb >> 16
                    R = t * x1[:, :, ix & 0xFFFF, None] * x2[:, None, :, ix >> 16]      # [N, U, V]
                    out[:, :, o3 + m3] += np.einsum("nuv,uvw->nw", R, W[pid])
    assert seen == set(range(n_paths))
    return out


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (1, 1, 1, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 2), (1, 3, 3, (-1, 0, 1), 1),
    (2, 1, 2, (0,), 0), (2, 2, 2, S5, 2),
])
def test_uvw_table_reproduces_oracle(built_library, L1, L2, LO, spins, basis):
    """The fully connected product's entry table, re-enacted in float64: every path
    appears once under its output block, and the result matches the oracle's uvw mode."""
    from paper_2607_01408_amd.spingtp import uvw_table_host
    words = uvw_table_host(L1, L2, LO, spins, basis)
    rng = np.random.default_rng(L1 + 10 * L2 + 100 * LO + basis)
    N, U, V, Wc = 3, 3, 2, 4
    x1 = rng.standard_normal((N, U, len(spins) * (L1 + 1) ** 2)) * valid_mask(spins, L1)
    x2 = rng.standard_normal((N, V, len(spins) * (L2 + 1) ** 2)) * valid_mask(spins, L2)
    P = len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)
    W = rng.standard_normal((P, U, V, Wc))
    nco = len(spins) * (LO + 1) ** 2
    y = emulate_uvw_table(words, x1, x2, W, nco)
    yo = oracle.fully_connected(x1, x2, W, L1, L2, LO, spins, basis).reshape(N, Wc, -1)
    assert np.abs(y - yo).max() <= 1e-6 * max(1.0, np.abs(yo).max())


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (1, 1, 1, (-1, 0, 1), 0), (2, 2, 2, (-1, 0, 1), 2), (1, 3, 3, (-1, 0, 1), 1), (3, 1, 2, (-1, 0, 1), 0),
    (2, 1, 2, (0,), 0), (2, 2, 2, S5, 2),
])
def test_uvw_gradient_tables_reproduce_oracle(built_library, L1, L2, LO, spins, basis):
    """The entry tables of the fully connected product's gradients w.r.t. x1 (the tensor
    read as T[k2, k3 -> k1]) and x2 (T[k1, k3 -> k2]), re-enacted in float64 as products
    of (x2, grad_out) and (x1, grad_out) mixed by the permuted weights, against the
    oracle's reverse mode."""
    from paper_2607_01408_amd.spingtp import uvw_table_host
    t1, t2 = uvw_table_host(L1, L2, LO, spins, basis, backward=True)
    rng = np.random.default_rng(7 + L1 + 10 * L2 + 100 * LO + basis)
    N, U, V, Wc = 3, 3, 2, 4
    nc1, nc2, nco = (len(spins) * (L + 1) ** 2 for L in (L1, L2, LO))
    x1 = rng.standard_normal((N, U, nc1)) * valid_mask(spins, L1)
    x2 = rng.standard_normal((N, V, nc2)) * valid_mask(spins, L2)
    g = rng.standard_normal((N, Wc, nco)) * valid_mask(spins, LO)
    P = len(oracle.PathWeightedTensor(L1, L2, LO, spins, basis).paths)
    W = rng.standard_normal((P, U, V, Wc))
    g1 = emulate_uvw_table(t1, x2, g, W.transpose(0, 2, 3, 1), nc1, role=1)
    g2 = emulate_uvw_table(t2, x1, g, W.transpose(0, 1, 3, 2), nc2, role=2)
    r1, r2, _ = oracle.fully_connected_vjp(x1, x2, W, g, L1, L2, LO, spins, basis)
    for got, ref in ((g1, r1), (g2, r2)):
        assert np.abs(got - ref.reshape(got.shape)).max() <= 1e-6 * max(1.0, np.abs(ref).max())
