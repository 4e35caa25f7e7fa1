"""CPU re-enactments of kernel data flows from the library's own host tables (test code).

``emulate_mfma_kernel`` follows the matrix-core kernel step by step: the per-unit
power-of-two scaling, step (A) from the plan tables, steps (B) and (D) as
products with the exact fp16 operand words the plan uploads (the data split into
fp16 hi + lo, or hi alone in the bf16 mode), the per-half output slots and the
m3 = 0 closed forms.  Tests compare it with the oracle (the tables are right) and
with the GPU output (the kernel does what its tables say, word for word).
"""

import math

import numpy as np

from paper_2607_01408_amd.spingtp import mfma_operands_host, plan_tables_host
from tests.oracle_helpers import valid_mask


def kernel_parity_mix(x, L, inverse):
    """The kernels' in-LDS mixing of a [rows][3 (L+1)^2] tile for the parity basis:
    per slot of degree l >= 1, (a, b) of the -1 and +1 blocks become
    ((a + b)/sqrt2, (-1)^l (a - b)/sqrt2) on load and ((a + (-1)^l b)/sqrt2,
    (a - (-1)^l b)/sqrt2) before the store."""
    B = (L + 1) ** 2
    y = np.array(x, dtype=np.float64, copy=True)
    h = 1.0 / math.sqrt(2.0)
    for q in range(1, B):
        t = -1.0 if int(math.isqrt(q)) % 2 else 1.0
        a, b = x[:, q], x[:, 2 * B + q]
        if inverse:
            y[:, q], y[:, 2 * B + q] = (a + t * b) * h, (a - t * b) * h
        else:
            y[:, q], y[:, 2 * B + q] = (a + b) * h, t * (a - b) * h
    return y



def _operand_matrices(words):
    """64 lanes x 8 packed fp16 words -> the (hi, lo) 32 x 16 operand matrices:
    lane l holds row l % 32 and K elements 8 (l / 32) + e (the MFMA A/B layout)."""
    W = np.asarray(words, dtype=np.uint32).reshape(64, 8)
    halves = np.stack([W & 0xFFFF, W >> 16], axis=-1).astype(np.uint16).view(np.float16).astype(np.float64)
    hi, lo = np.zeros((32, 16)), np.zeros((32, 16))
    for lane in range(64):
        row, k0 = lane % 32, 8 * (lane // 32)
        hi[row, k0:k0 + 8] = halves[lane, 0:4].reshape(8)
        lo[row, k0:k0 + 8] = halves[lane, 4:8].reshape(8)
    return hi, lo


def _rtz16(x):
    """fp16 rounding toward zero (the kernel's v_cvt_pkrtz for the data's high parts)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -24)))
    q = np.ldexp(1.0, (np.maximum(e, -14) - 10).astype(int))   # fp16 spacing at |x| (subnormal below 2^-14)
    return np.sign(x) * np.floor(a / q) * q


def _split16(x):
    """Data split as the kernel does it: hi rounded toward zero, lo = fp16(x - hi) to nearest."""
    hi = _rtz16(x)
    return hi, (x - hi).astype(np.float16).astype(np.float64)


def _split_product(Mh, Ml, x, split=3):
    """(Mh + Ml) x with x split into fp16 hi + lo, summed as hi.hi + hi.lo + lo.hi
    (split = 3, the fp32 mode) or hi.hi alone (split = 1, the bf16 mode), in float64."""
    if split == 1:
        return x.astype(np.float16).astype(np.float64) @ Mh.T
    xh, xl = _split16(x)
    return xh @ Mh.T + xl @ Mh.T + xh @ Ml.T


def emulate_mfma_kernel(x1, x2, L, basis, split=3, theta_dtype=np.float64):
    """float64 re-enactment of the matrix-core kernel (L1 = L2 = Lout = L, spins
    {-1, 0, +1}) from the library's host tables: per-unit power-of-two scaling,
    step (A) from the plan tables, steps (B) and (D) as products with the fp16
    operand words exactly as uploaded (fp16 split of the data), the per-half
    output slots and the m3 = 0 closed forms.  ``split`` = 3 re-enacts the fp32
    mode, 1 the bf16 mode (high parts only); ``theta_dtype`` = np.float32 rounds the
    step-(A) results to fp32 as the kernel holds them, which moves some fp16
    roundings of the next step by one unit and so shows how far two faithful
    evaluations of the same arithmetic can drift apart."""
    tab, dims = plan_tables_host(L, L, L, (-1, 0, 1), basis)
    words = mfma_operands_host(L)
    NT, NP, PB, GLOB = dims["n_theta"], dims["n_phi"], dims["per_theta_block"], dims["global_block"]
    NB = (NP + 15) // 16
    KB = 2 if L >= 8 else 1
    assert words.size == 512 * (1 + 2 * NB + (2 if KB == 2 else 0))
    TB1 = _operand_matrices(words[:512])
    TBin = [TB1, TB1]
    if KB == 2:  # second K block after the step-(D) blocks: one table per input
        for i in range(2):
            T2 = _operand_matrices(words[512 * (1 + 2 * NB + i):512 * (2 + 2 * NB + i)])
            TBin[i] = (np.concatenate([TB1[0], T2[0]], axis=1), np.concatenate([TB1[1], T2[1]], axis=1))
    TD = [[_operand_matrices(words[512 * (1 + t * NB + b):512 * (2 + t * NB + b)]) for b in range(NB)]
          for t in range(2)]
    tri = lambda t, l: t * (L + 1) - t * (t - 1) // 2 + (l - t)  # noqa: E731
    triA = (L + 1) * (L + 2) // 2
    a0c, a0s, aup, aum, aw = 0, triA, 2 * triA, 3 * triA, 4 * triA
    e0c = aw + L + 1
    e1p, e1m, e1z = e0c + 2 * triA, e0c + 3 * triA, e0c + 4 * triA
    N0, M0 = tab[0:8].reshape(4, 2), tab[16:24].reshape(2, 4)  # forward tables: input 2 mixing = input 1
    BO = (L + 1) ** 2
    U = x1.shape[0]
    parity = tab[24] != 0.0
    assert parity == (basis == 2)
    if parity:
        x1, x2 = kernel_parity_mix(x1, L, False), kernel_parity_mix(x2, L, False)

    def scale(x):
        valid = valid_mask((-1, 0, 1), L).astype(bool)
        m = np.abs(np.where(valid, x, 0.0)).max(axis=1)
        _, e = np.frexp(m)
        return x * np.ldexp(1.0, -e)[:, None], e

    def theta_fourier(x, tb, inp):
        xm, x0, xp = x[:, :BO], x[:, BO:2 * BO], x[:, 2 * BO:]
        c, s = np.zeros((3, U, L + 1)), np.zeros((3, U, L + 1))
        for t in range(L + 1):
            for l in range(t, L + 1):
                c[0, :, t] += x0[:, l * l + l + t] * tb[a0c + tri(t, l)]
                if t:
                    s[0, :, t] += x0[:, l * l + l - t] * tb[a0s + tri(t, l)]
        for t in range(1, L + 1):
            up = vp = um = vm = 0.0
            for l in range(t, L + 1):
                wp, wm = tb[aup + tri(t, l)], tb[aum + tri(t, l)]
                up, vp = up + xp[:, l * l + l + t] * wp, vp + xp[:, l * l + l - t] * wp
                um, vm = um + xm[:, l * l + l + t] * wm, vm + xm[:, l * l + l - t] * wm
            c[1, :, t], s[1, :, t], c[2, :, t], s[2, :, t] = up + um, -(vp + vm), vp - vm, up - um
        wpl = sum(xp[:, l * l + l] * tb[aw + l] for l in range(1, L + 1))
        wmi = sum(xm[:, l * l + l] * tb[aw + l] for l in range(1, L + 1))
        c[1, :, 0], c[2, :, 0], d, e = N0 @ np.stack([wpl, wmi])
        # cos t at slot t, sin t at slot 8 + t; at L = 8 sin 8 at slot 8, cos 8 at 16
        kappa = np.zeros((3, U, 16 * KB))
        kappa[:, :, :min(L, 7) + 1] = c[:, :, :min(L, 7) + 1]
        kappa[:, :, 9:9 + min(L, 7)] = s[:, :, 1:min(L, 7) + 1]
        if L >= 8:  # cos 8 at kappa 16 (input 1, lanes 0..31) or 24 (input 2, lanes 32..63)
            kappa[:, :, 8] = s[:, :, 8]
            kappa[:, :, 16 + 8 * inp] = c[:, :, 8]
        return kappa.astype(theta_dtype).astype(np.float64), d, e, c[0, :, 0]

    holds = [8 * (v // 4) + v % 4 < NP for v in range(16)]
    x1s, ex1 = scale(x1)
    x2s, ex2 = scale(x2)
    y = np.zeros((U, 3 * BO))
    for j in range(NT):
        tb = tab[GLOB + j * PB:GLOB + (j + 1) * PB]
        K1, d1, e1, a1 = theta_fourier(x1s, tb, 0)
        K2, d2, e2, a2 = theta_fourier(x2s, tb, 1)
        f1 = [_split_product(*TBin[0], K1[p], split) for p in range(3)]  # (U, 32): row = phi point
        f2 = [_split_product(*TBin[1], K2[p], split) for p in range(3)]
        A, B, C = f1
        a, b, c = f2
        H = [A * a + B * b + C * c, A * b + a * B, A * c + a * C]
        spec = []
        for q in range(3):
            acc = np.zeros((U, 32))
            for blk in range(NB):
                Hb = np.zeros((U, 16))
                for kk in range(16):
                    v = 8 * blk + kk % 8
                    if v < 16 and holds[v]:
                        Hb[:, kk] = H[q][:, 8 * (v // 4) + 4 * (kk // 8) + v % 4]
                acc += _split_product(*TD[1 if q == 2 else 0][blk], Hb, split)
            spec.append(acc)

        def at(q, h, t):
            return spec[q][:, 8 * (t // 4) + 4 * h + t % 4]

        r0c0 = at(0, 0, 0) - 0.5 * NP * (d1 * d2 + e1 * e2)
        sP1, sP2 = math.sqrt(2) * at(1, 0, 0), math.sqrt(2) * at(2, 0, 0)
        sP4, sP3 = -NP * (d2 * a1 + d1 * a2), NP * (e2 * a1 + e1 * a2)
        Zp, Zm = M0 @ np.stack([(sP1 + sP4) / 2, (sP3 + sP2) / 2, (sP1 - sP4) / 2, (sP3 - sP2) / 2])
        for l in range(L + 1):
            y[:, BO + l * l + l] += tb[e0c + tri(0, l)] * r0c0
            if l:
                y[:, 2 * BO + l * l + l] += tb[e1z + l] * Zp
                y[:, l * l + l] += tb[e1z + l] * Zm
        for h, sg in ((0, 1.0), (1, -1.0)):
            for t in range(1, L + 1):
                sr = sg * at(0, h, t)
                sp = sg * at(1, h, t) + at(2, h, t)
                sm = sg * at(1, h, t) - at(2, h, t)
                m3 = t if h == 0 else -t
                for l in range(t, L + 1):
                    y[:, BO + l * l + l + m3] += tb[e0c + tri(t, l)] * sr
                    y[:, 2 * BO + l * l + l + m3] += tb[e1p + tri(t, l)] * sp
                    y[:, l * l + l + m3] += tb[e1m + tri(t, l)] * sm
    y = y * np.ldexp(1.0, ex1 + ex2)[:, None]
    return kernel_parity_mix(y, L, True) if parity else y
