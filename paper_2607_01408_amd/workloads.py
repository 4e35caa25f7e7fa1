"""Seeded synthetic inputs shaped like the atomistic edge batches of the paper.

Holds no arithmetic of the method: only seeded normal draws, the per-degree
scaling of a workload, and zeroing of the slots with l < |s| (which do not exist
as basis functions).  Both the HIP path and the CPU oracle are fed from here.

Shapes (units = edges x channels; every unit is independent, so only N and C
matter -- the paper's molecular datasets are not needed and none are read):

  small     L=2,  N=64,      C=8,   fp32, N(0,1)                       seeds 1001/1002
  molecule  L=4,  N=20,000,  C=64,  fp32, N(0,1)/sqrt(2l+1)            seeds 2001/2002
            (~30 atoms x ~20 neighbours x 32 graphs)
  organic   L=6,  N=100,000, C=128, fp32 and bf16, N(0,1)              seeds 3001/3002
            (20-100 atoms x ~25 neighbours x 64 graphs)
  catalyst  L=8,  N=400,000, C=128, bf16 in / fp32 accumulate, N(0,1)  seeds 4001/4002
            (~80 atoms x <=40 neighbours x 128 graphs)
  sweep     L in {2,4,8,12,16}, N=8,192, C=32, fp32, N(0,1)          seeds 5001+L/5101+L
  chiral    L=2, spins (-2..2), N=200,000, C=64, fp32, N(0,1)          seeds 6001/6002
            (the s_max = 2, L_max = 2 setting of the chirality experiments,
            App. F: small organic molecules, 64 channels)
Layout [N, C, n_spins, (L+1)^2] with spins (-1, 0, +1) unless a workload names
its own.
"""

import math

SPINS = (-1, 0, 1)

WORKLOADS = {
    "small": dict(L=2, N=64, C=8, dtypes=("fp32",), scale="unit", seeds=(1001, 1002)),
    "molecule": dict(L=4, N=20_000, C=64, dtypes=("fp32",), scale="inv_sqrt_2l1", seeds=(2001, 2002)),
    "organic": dict(L=6, N=100_000, C=128, dtypes=("fp32", "bf16"), scale="unit", seeds=(3001, 3002)),
    "catalyst": dict(L=8, N=400_000, C=128, dtypes=("bf16",), scale="unit", seeds=(4001, 4002)),
    "sweep": dict(L=(2, 4, 8, 12, 16), N=8_192, C=32, dtypes=("fp32",), scale="unit", seeds=(5001, 5101)),
    "chiral": dict(L=2, N=200_000, C=64, dtypes=("fp32",), scale="unit", seeds=(6001, 6002),
                   spins=(-2, -1, 0, 1, 2)),
}

_CHUNK_UNITS = 1 << 20  # units drawn per generator seed


def slot_scale(L, spins, scale):
    """[n_spins * (L+1)^2] multiplier: 0 on slots with l < |s|, else 1 or 1/sqrt(2l+1)."""
    out = []
    for s in spins:
        for l in range(L + 1):
            v = 0.0 if l < abs(s) else (1.0 if scale == "unit" else 1.0 / math.sqrt(2 * l + 1))
            out.extend([v] * (2 * l + 1))
    return out


def draw(L, N, C, seed, dtype="fp32", spins=SPINS, scale="unit", device="cuda"):
    """One input tensor [N, C, n_spins, (L+1)^2], drawn in fixed chunks of units.

    Chunk i uses the generator seed ``seed * 1_000_003 + i``; values are fp32 normal
    draws times the slot scale, then cast (round to nearest even) to ``dtype``.
    """
    import torch

    tdt = {"fp32": torch.float32, "bf16": torch.bfloat16}[dtype]
    ns, nc = len(spins), (L + 1) ** 2
    units = N * C
    out = torch.empty((N, C, ns, nc), dtype=tdt, device=device)
    flat = out.view(units, ns * nc)
    mult = torch.tensor(slot_scale(L, spins, scale), dtype=torch.float32, device=device)
    gen = torch.Generator(device=device)
    for i, u0 in enumerate(range(0, units, _CHUNK_UNITS)):
        u1 = min(units, u0 + _CHUNK_UNITS)
        gen.manual_seed(seed * 1_000_003 + i)
        v = torch.randn((u1 - u0, ns * nc), generator=gen, dtype=torch.float32, device=device)
        flat[u0:u1] = (v * mult).to(tdt)
    return out


def make_pair(name, dtype=None, L=None, device="cuda", N=None, C=None):
    """(x1, x2, meta) for a named workload; ``L`` picks one degree of the sweep."""
    w = WORKLOADS[name]
    if name == "sweep":
        if L is None:
            raise ValueError("the sweep needs L")
        s1, s2 = w["seeds"][0] + L, w["seeds"][1] + L
    else:
        L = w["L"]
        s1, s2 = w["seeds"]
    dtype = dtype or w["dtypes"][0]
    N = N or w["N"]
    C = C or w["C"]
    spins = w.get("spins", SPINS)
    x1 = draw(L, N, C, s1, dtype, spins, w["scale"], device)
    x2 = draw(L, N, C, s2, dtype, spins, w["scale"], device)
    meta = dict(workload=name, L=L, N=N, C=C, dtype=dtype, scale=w["scale"], seeds=(s1, s2), spins=spins)
    return x1, x2, meta
