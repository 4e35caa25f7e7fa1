"""Benchmark of the SpinGTP forward on one MI355X.

A step is one spingtp_forward over the whole workload (all five steps of the
path run inside the fused kernel), inputs resident in HBM.  Prints ONE JSON
line with the throughput in edge-channel tensor products per second, the
roofline object of the kernel, a sampled parity check and the CPU-oracle
baseline timed on the host cores.

Default workload: L1 = L2 = Lout = 6, spins (-1, 0, +1), N = 100,000 edges,
C = 128 channels, fp32 (12.8 M units).
"""

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0             # MI355X HBM3E
# vector ALU without packed fp32 (the build turns packed fp32 off): 256 CUs x 4 SIMDs x
# 16 lanes x 2 flops (FMA) x 2.4 GHz
PEAK_VALU_FP32_TFLOPS = 78.6
PEAK_VALU_PACKED_FP32_TFLOPS = 157.3  # the published fp32 vector figure (packed FMA)
PEAK_MFMA_F16_TFLOPS = 2500.0     # dense fp16 / bf16 matrix cores
PEAK_MFMA_FP32_TFLOPS = 157.3     # dense fp32 matrix cores
# Charged work per unit at spins (-1, 0, +1) of a 2D (u, v) Fourier route (the costing the
# reported scope fraction uses; this kernel does not execute it): coef->Fourier for both
# inputs, the spin-pair convolution done directly and by FFT, and Fourier->coef.  Its floor charges the cheaper convolution on the vector ALU and the
# transforms on the matrix cores (fp32 at 157.3 TF, bf16 at the fp16 peak).
SCOPE_CHARGED = {2: (1152, 26600, 34168, 1800), 4: (5840, 276696, 160672, 9928),
                 6: (16640, 1201928, 364544, 29000), 8: (35728, 3511928, 742048, 63624),
                 12: (110672, 16415000, 1680896, 197960), 16: (251280, 49823928, 3377152, 449800)}
METRIC = "edge·channel tensor products/sec at L=6 fp32; % HBM/MFMA roofline"
# sources of the spingtp_forward kernels (families 1-4): a stored traffic record
# is used only while their hash is unchanged
_CSRC = "paper_2607_01408_amd/csrc/"


def kernel_sources(kname):
    """The source files a forward kernel is compiled from (its counters go stale when they change)."""
    main = {"spingtp_fwd_mfma_kernel": "forward_mfma.hip",
            "spingtp_fwd_direct_kernel": "forward_direct.hip"}.get(kname, "forward.hip")
    extra = ("forward_pair.h",) if main == "forward.hip" else ()
    return tuple(_CSRC + f for f in (main, "device_common.h", "layout.h") + extra)


def route_steps(L1, L2, LO, spin=True):
    """Algorithmic flops per unit of the exact-grid route, by step (FMA = 2 flops).

    Counts the structural work of the five steps on the n_theta x n_phi grid:
    (A) one FMA per valid input coefficient plus the spin recombination (both inputs),
    (B) even/odd synthesis of each real trigonometric polynomial,
    (C) the spin-pair products, (D) even/odd analysis of each product,
    (E) one FMA per valid output coefficient plus the spin recombination.
    """
    NT = (L1 + L2 + LO + 2) // 2
    NP = L1 + L2 + LO + 1
    KP = (NP - 1) // 2
    even = NP % 2 == 0
    npoly = 3 if spin else 1

    def coeffs(L):
        return (L + 1) ** 2 + (2 * ((L + 1) ** 2 - 1) if spin else 0)

    def stage_a(L):
        return 2 * coeffs(L) + ((4 * L + 12) if spin else 0)

    def synth(L):
        return L + KP * (4 * L + 2) + (2 * L if even else 0)

    prod = 11 if spin else 1
    analysis = (LO + 1) + KP * (3 + 4 * LO) + (2 * (LO + 1) if even else 0)
    stage_e = 2 * coeffs(LO) + ((4 * LO + 23) if spin else 0)
    return {"A": NT * (stage_a(L1) + stage_a(L2)), "B": NT * npoly * (synth(L1) + synth(L2)),
            "C": NT * NP * prod, "D": NT * npoly * analysis, "E": NT * stage_e}


def route_flops(L1, L2, LO, spin=True):
    """All five steps of route_steps, per unit."""
    return sum(route_steps(L1, L2, LO, spin).values())


def mfma_flops_executed(family, L, dtype):
    """fp16 matrix-core flops one unit costs on the matrix-core kernel, as executed: per wave
    (32 units) and Gauss node, step (B) is six 32x32x16 products per 16-slot K block (two
    blocks at L = 8, the second for cos 8 alone) and step (D) three per 16-point K block,
    each repeated three times for the hi/lo split of fp32 I/O; all padding (19 of 32 rows,
    13 of 16 slots at L = 6) is counted."""
    if family != 4:
        return 0
    NT = (3 * L + 2) // 2
    NP = 3 * L + 1
    NB = (NP + 15) // 16
    KB = 2 if L >= 8 else 1
    split = 3 if dtype == "fp32" else 1
    per_wave_node = (6 * KB + 3 * NB) * split
    return per_wave_node * (32 * 32 * 16 * 2) * NT // 32


def roofline(family, L, dtype, units, avg_ms, bytes_unit, direct_flops=None, spin=True):
    """Floors of the executed route on each resource and the one that binds.

    hbm: algorithmic bytes (x1 + x2 + out) at 8 TB/s; valu: the route's vector-ALU flops (all
    steps on the vector kernels, steps A, C, E on the matrix-core kernel) at the non-packed
    78.6 TF (the library is compiled without packed fp32 instructions); mfma: the matrix-core work as executed (split products and
    padding) at the dense fp16 peak.  bound = the largest floor; frac = floor / measured."""
    t = avg_ms / 1e3
    steps = route_steps(L, L, L, spin)
    if direct_flops is not None:      # the direct kernel: a product and an FMA per tensor entry
        valu = direct_flops
    elif family == 4:
        valu = steps["A"] + steps["C"] + steps["E"]
    else:
        valu = sum(steps.values())
    mfma = mfma_flops_executed(family, L, dtype)
    floors = {"hbm": bytes_unit * units / (PEAK_HBM_GBS * 1e9),
              "alu": valu * units / (PEAK_VALU_FP32_TFLOPS * 1e12),
              "mfma": mfma * units / (PEAK_MFMA_F16_TFLOPS * 1e12)}
    bound = max(floors, key=floors.get)
    if bound == "hbm":
        achieved, peak, unit = bytes_unit * units / t / 1e9, PEAK_HBM_GBS, "GB/s"
    elif bound == "alu":
        achieved, peak, unit = valu * units / t / 1e12, PEAK_VALU_FP32_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = mfma * units / t / 1e12, PEAK_MFMA_F16_TFLOPS, "TFLOP/s"
    out = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
           "floors_ms": {k: v * 1e3 for k, v in floors.items()},
           "fracs": {k: v / t for k, v in floors.items()},
           "valu_flops_per_unit": valu, "mfma_f16_flops_per_unit_executed": mfma,
           "hbm_bytes_per_unit": bytes_unit,
           "route_flops_per_unit": sum(steps.values()) if direct_flops is None else direct_flops}
    if L in SCOPE_CHARGED and spin:
        s2, s3d, s3f, s4 = SCOPE_CHARGED[L]
        p_tr = (PEAK_VALU_PACKED_FP32_TFLOPS if dtype == "fp32" else PEAK_MFMA_F16_TFLOPS) * 1e12
        t_scope = max(bytes_unit * units / (PEAK_HBM_GBS * 1e9),
                      units * ((s2 + s4) / p_tr + min(s3d, s3f) / (PEAK_VALU_PACKED_FP32_TFLOPS * 1e12)))
        out["scope_charged_flops_per_unit"] = s2 + min(s3d, s3f) + s4
        out["scope_charged_frac"] = t_scope / t   # reported as-is; above 1 when the route does less work
    return out


def hbm_bytes_per_unit(L1, L2, LO, dtype, n_spins=3):
    es = 4 if dtype == "fp32" else 2
    return es * n_spins * ((L1 + 1) ** 2 + (L2 + 1) ** 2 + (LO + 1) ** 2)


def kernel_source_hash(kname):
    h = hashlib.sha256()
    for p in kernel_sources(kname):
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


BASES = {"paper": 0, "m0_paired": 1, "parity": 2}


def profile_tag(workload, dtype, L, valu=False, basis="paper"):
    tag = f"{workload}_L{L}_{dtype}" if workload == "sweep" else f"{workload}_{dtype}"
    if basis != "paper":
        tag += f"_{basis}"
    return tag + "_valu" if valu else tag


def measured_traffic(workload, dtype, units, L, kname, valu=False, basis="paper"):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source and the same kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_spingtp_fwd_{profile_tag(workload, dtype, L, valu, basis)}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_source_hash(kname) or rec.get("units") != units:
        return None
    if kname + "<" not in rec.get("kernel", ""):
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_workers_available():
    """Host cores this process may use, capped at one GPU's share of a shared host (16)."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _cpu_worker(conn):
    """One CPU-oracle process: holds the oracle's tensor and its share of the sample.
    Started with the spawn method before the parent touches the GPU; never uses it."""
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    import numpy as np

    import oracle

    T, X1, X2 = None, None, None
    while True:
        msg = conn.recv()
        if msg[0] == "tensor":
            t0 = time.perf_counter()
            T = oracle.RealGauntTensor(msg[1], msg[1], msg[1], msg[2], msg[3])
            conn.send(time.perf_counter() - t0)
        elif msg[0] == "data":
            X1, X2 = msg[1], msg[2]
            conn.send(0 if X1 is None else len(X1))
        elif msg[0] == "run":
            t0 = time.perf_counter()
            y = T.apply(X1, X2)
            conn.send((time.perf_counter() - t0, float(np.abs(y[:1]).sum())))
        elif msg[0] == "apply":
            conn.send(T.apply(msg[1], msg[2]))
        else:
            break
    conn.close()


class CpuPool:
    """n spawned oracle workers with one pipe each (no shared memory, no GPU)."""

    def __init__(self, n):
        import multiprocessing

        ctx = multiprocessing.get_context("spawn")
        self.conns, self.procs = [], []
        for _ in range(n):
            a, b = ctx.Pipe()
            p = ctx.Process(target=_cpu_worker, args=(b,), daemon=True)
            p.start()
            self.conns.append(a)
            self.procs.append(p)

    def __len__(self):
        return len(self.conns)

    def all(self, msg):
        for c in self.conns:
            c.send(msg)
        return [c.recv() for c in self.conns]

    def scatter(self, kind, parts):
        for c, part in zip(self.conns, parts):
            c.send((kind,) + tuple(part))
        return [c.recv() for c in self.conns[:len(parts)]]

    def apply(self, a, b):
        """The oracle on rows a, b (float64), split over the workers; rows in order."""
        import numpy as np

        k = max(1, min(len(self), len(a)))
        cuts = np.linspace(0, len(a), k + 1).astype(int)
        ys = self.scatter("apply", [(a[cuts[i]:cuts[i + 1]], b[cuts[i]:cuts[i + 1]]) for i in range(k)])
        return np.concatenate([y.reshape(len(y), -1) for y in ys])

    def close(self):
        for c in self.conns:
            try:
                c.send(("exit",))
            except OSError:
                pass
        for p in self.procs:
            p.join(timeout=10)


def cpu_baseline(pool, L, x1, x2, seconds, spins=(-1, 0, 1), basis=0):
    """The unchanged CPU oracle on a bounded random sample of the same inputs, spread over
    the worker processes (one core each); throughput = sampled units / wall time of the
    parallel contraction.  The tensor build is timed apart and excluded."""
    import numpy as np
    import torch

    n_w = len(pool)
    build_s = max(pool.all(("tensor", L, tuple(spins), basis)))
    U = x1.shape[0] * x1.shape[1]
    a = x1.reshape(U, -1)
    b = x2.reshape(U, -1)
    rng = np.random.default_rng(1234)

    def load(idx):
        ti = torch.as_tensor(idx, device=a.device)
        return a[ti].float().cpu().numpy(), b[ti].float().cpu().numpy()

    def split(A, B):
        cuts = np.linspace(0, len(A), n_w + 1).astype(int)
        return [(A[cuts[i]:cuts[i + 1]], B[cuts[i]:cuts[i + 1]]) for i in range(n_w)]

    # calibrate: 256 units per worker
    A, B = load(np.sort(rng.choice(U, size=min(U, 256 * n_w), replace=False)))
    pool.scatter("data", split(A, B))
    per_unit = float(np.median([r[0] for r in pool.all(("run",))])) / max(1, len(A) // n_w)
    n = int(max(256 * n_w, min(U, seconds * n_w / max(per_unit, 1e-9))))
    A, B = load(np.sort(rng.choice(U, size=n, replace=False)))
    pool.scatter("data", split(A, B))
    del A, B
    t0 = time.perf_counter()
    res = pool.all(("run",))
    wall = time.perf_counter() - t0
    pool.scatter("data", [(None, None)] * n_w)  # free the workers' copies
    return {
        "value": n / wall,
        "unit": "TP/s",
        "cores": n_w,
        "kind": "oracle",
        "sample": f"{n} seeded-random units of the same inputs, split over {n_w} single-threaded "
                  f"worker processes ({wall:.1f} s wall; float64 numpy/scipy); sparse tensor build "
                  f"{build_s:.2f} s excluded",
        "per_worker_s": [round(r[0], 3) for r in res],
        "extrapolated_full_job_s": U / (n / wall),
        "host_cpus_visible": len(os.sched_getaffinity(0)),
    }


# Depthwise V = 1 tensor-product shapes of the paper's backend runtime table (App. E):
# (L1, L2, Lout, multiplicity U = channels C, edges B, and the paper's H200 medians in ms for
# direct Gaunt, precontracted and Triton-fused precontracted execution -- context only).
V1_TABLE = [
    (1, 1, 1, 16, 128, 5.460, 0.537, 0.120), (1, 1, 1, 64, 128, 5.493, 0.466, 0.119),
    (1, 1, 1, 128, 128, 4.562, 0.443, 0.115), (2, 2, 2, 16, 32, 21.570, 0.997, 0.259),
    (2, 2, 2, 64, 32, 29.912, 1.769, 0.748), (2, 2, 2, 128, 32, 33.528, 1.837, 0.559),
    (2, 2, 2, 16, 128, 16.144, 0.999, 0.258), (2, 2, 2, 64, 128, 29.561, 1.771, 0.752),
    (2, 2, 2, 128, 128, 33.306, 1.838, 0.572), (1, 3, 3, 16, 128, 12.714, 0.678, 0.228),
    (1, 3, 3, 64, 128, 20.610, 1.080, 0.608), (1, 3, 3, 128, 128, 22.546, 1.344, 0.681),
    (2, 2, 2, 64, 1024, 29.912, 1.777, 2.090), (1, 3, 3, 64, 1024, 23.941, 1.394, 1.865),
    (1, 3, 3, 128, 1024, 22.628, 1.350, 2.240),
]


def run_v1(args):
    """spingtp_forward_v1 (x2 shared by the channels of an edge): the paper's V = 1 table
    shapes and a degree sweep, on the precontracted route and on the Fourier route.
    Times are HIP-event averages over back-to-back calls of the C entry point."""
    import ctypes

    import numpy as np
    import torch

    from oracle.spingtp import _cached_tensor
    from paper_2607_01408_amd import Plan, _lib, workloads

    torch.cuda.set_device(0)
    fn = _lib.lib().spingtp_forward_v1

    def measure(L1, L2, LO, C, B, fourier, seed):
        x1 = workloads.draw(L1, B, C, 9100 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, 1, 9200 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        try:
            plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", v1_fourier=fourier, v1_precontract=not fourier)
        except Exception:
            return None
        if fourier and plan.kernel_info_v1()["family"] == 5:
            return None
        if not fourier and plan.kernel_info_v1()["family"] != 5:
            return None
        out = torch.empty((B, C, 3, (LO + 1) ** 2), device="cuda:0")
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        call = (plan.handle, x1.data_ptr(), x2.data_ptr(), out.data_ptr(), B, C, st)
        for _ in range(args.warmup):
            assert fn(*call) == 0
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            fn(*call)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / args.steps
        U = B * C
        idx = np.unique(np.concatenate([np.arange(min(U, 64)), np.arange(max(0, U - 64), U)]))
        a = x1.view(U, -1)[torch.as_tensor(idx, device="cuda:0")].double().cpu().numpy()
        b = x2.view(B, -1).double().cpu().numpy()[idx // C]
        ref = _cached_tensor(L1, L2, LO, workloads.SPINS, 0).apply(a, b).reshape(len(idx), -1)
        got = out.view(U, -1)[torch.as_tensor(idx, device="cuda:0")].double().cpu().numpy()
        parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        return {"ms": ms, "family": plan.kernel_info_v1()["family"], "parity_rel_l2": parity,
                "tp_per_s": U / (ms / 1e3)}

    def measure_weighted(L1, L2, LO, C, B, basis, seed):
        """spingtp_forward_v1_weighted (per-channel path weights) on the precontracted kernel."""
        import oracle
        from paper_2607_01408_amd import paths_host

        x1 = workloads.draw(L1, B, C, 9100 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, 1, 9200 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        try:
            plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", basis, channel_weights=True)
        except Exception:
            return None
        n_paths = len(paths_host(L1, L2, LO, workloads.SPINS, basis))
        w = torch.randn((C, n_paths), generator=torch.Generator().manual_seed(seed)).to("cuda:0")
        out = torch.empty((B, C, 3, (LO + 1) ** 2), device="cuda:0")
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        wfn = _lib.lib().spingtp_forward_v1_weighted
        call = (plan.handle, x1.data_ptr(), x2.data_ptr(), w.data_ptr(), out.data_ptr(), B, C, st)
        for _ in range(args.warmup):
            assert wfn(*call) == 0
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            wfn(*call)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / args.steps
        U = B * C
        idx = np.unique(np.concatenate([np.arange(min(U, 32)), np.arange(max(0, U - 32), U)]))
        W = w.double().cpu().numpy()
        a = x1.view(U, -1).double().cpu().numpy()[idx]
        b = x2.view(B, -1).double().cpu().numpy()[idx // C]
        ref = np.stack([oracle.PathWeightedTensor(L1, L2, LO, workloads.SPINS, basis, W[u % C])
                        .apply(a[i:i + 1], b[i:i + 1]).reshape(-1) for i, u in enumerate(idx)])
        got = out.view(U, -1).double().cpu().numpy()[idx]
        return {"ms": ms, "paths": n_paths, "basis": basis,
                "parity_rel_l2": float(np.linalg.norm(got - ref) / np.linalg.norm(ref)), "tp_per_s": U / (ms / 1e3)}

    def measure_weighted_backward(L1, L2, LO, C, B, basis, seed):
        """spingtp_backward_v1_weighted (gradients of x1, the shared x2 and the per-channel weights),
        preallocated buffers; parity of gx1 and gx2 on sampled edges against the oracle, and of gW
        through the identity <gW, W> = <g, y> with y from the weighted forward (relative to |g| |y|)."""
        import oracle
        from paper_2607_01408_amd import paths_host

        try:
            plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", basis, channel_weights=True)
        except Exception:
            return None
        n_paths = len(paths_host(L1, L2, LO, workloads.SPINS, basis))
        x1 = workloads.draw(L1, B, C, 9600 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, 1, 9700 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        g = workloads.draw(LO, B, C, 9800 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        w = torch.randn((C, n_paths), generator=torch.Generator().manual_seed(seed)).to("cuda:0")
        gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
        gw = torch.empty_like(w)
        n = ctypes.c_size_t(0)
        assert _lib.lib().spingtp_backward_v1_weighted_workspace_size(plan.handle, B, C, ctypes.byref(n)) == 0
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device="cuda:0")
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        call = (plan.handle, x1.data_ptr(), x2.data_ptr(), w.data_ptr(), g.data_ptr(), gx1.data_ptr(),
                gx2.data_ptr(), gw.data_ptr(), ws.data_ptr(), n.value, B, C, st)
        bfn = _lib.lib().spingtp_backward_v1_weighted
        for _ in range(args.warmup):
            assert bfn(*call) == 0
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            bfn(*call)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / args.steps
        edges = sorted({0, B // 2, B - 1})
        sel = torch.as_tensor(edges, device="cuda:0")
        a, b, c = (t[sel].double().cpu().numpy() for t in (x1, x2, g))
        r1, r2, _ = oracle.channel_weighted_v1_vjp(a.reshape(len(edges), C, -1), b.reshape(len(edges), -1),
                                                   w.double().cpu().numpy(), c.reshape(len(edges), C, -1),
                                                   L1, L2, LO, workloads.SPINS, basis)
        got1 = gx1[sel].double().cpu().numpy().reshape(r1.shape)
        got2 = gx2[sel].double().cpu().numpy().reshape(r2.shape)
        try:
            y = plan.forward_v1_weighted(x1, x2, w)
        except Exception:  # a plan with the gradients' table only
            y = None
        ident = None
        if y is not None:
            torch.cuda.synchronize()
            # normalized by |g| |y| (the bound of <g, y>): the dot product itself cancels
            dot = float((g.double() * y.double()).sum())
            scale = float(g.double().norm() * y.double().norm())
            ident = abs(float((gw.double() * w.double()).sum()) - dot) / max(scale, 1e-300)
        return {"ms": ms, "paths": n_paths, "basis": basis,
                "parity_rel_l2_gx1_sampled": float(np.linalg.norm(got1 - r1) / np.linalg.norm(r1)),
                "parity_rel_l2_gx2_sampled": float(np.linalg.norm(got2 - r2) / np.linalg.norm(r2)),
                "gw_identity_rel": ident, "units_per_s": B * C / (ms / 1e3)}

    def measure_weighted_unit(L1, L2, LO, C, B, basis, seed):
        """spingtp_forward_weighted and spingtp_backward_weighted (per-channel path weights, x2 per
        unit), preallocated buffers; parity of the forward and gx2 on sampled edges against the oracle."""
        import oracle
        from paper_2607_01408_amd import paths_host

        try:
            plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", basis, channel_weights=True)
        except Exception:
            return None
        n_paths = len(paths_host(L1, L2, LO, workloads.SPINS, basis))
        x1 = workloads.draw(L1, B, C, 9610 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, C, 9710 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        g = workloads.draw(LO, B, C, 9810 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        w = torch.randn((C, n_paths), generator=torch.Generator().manual_seed(seed)).to("cuda:0")
        out = torch.empty_like(g)
        gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
        gw = torch.empty_like(w)
        n = ctypes.c_size_t(0)
        if _lib.lib().spingtp_backward_weighted_workspace_size(plan.handle, B, C, ctypes.byref(n)) != 0:
            return None
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device="cuda:0")
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        calls = {"forward": (_lib.lib().spingtp_forward_weighted,
                             (plan.handle, x1.data_ptr(), x2.data_ptr(), w.data_ptr(), out.data_ptr(), B, C, st)),
                 "backward": (_lib.lib().spingtp_backward_weighted,
                              (plan.handle, x1.data_ptr(), x2.data_ptr(), w.data_ptr(), g.data_ptr(), gx1.data_ptr(),
                               gx2.data_ptr(), gw.data_ptr(), ws.data_ptr(), n.value, B, C, st))}
        res = {"paths": n_paths, "basis": basis}
        for name, (fn_, call) in calls.items():
            for _ in range(args.warmup):
                assert fn_(*call) == 0
            torch.cuda.synchronize()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            for _ in range(args.steps):
                fn_(*call)
            e.record()
            torch.cuda.synchronize()
            res[name + "_ms"] = s.elapsed_time(e) / args.steps
        edges = sorted({0, B // 2, B - 1})
        sel = torch.as_tensor(edges, device="cuda:0")
        a, b, c = (t[sel].double().cpu().numpy().reshape(len(edges), C, -1) for t in (x1, x2, g))
        W = w.double().cpu().numpy()
        ref = oracle.channel_weighted(a, b, W, L1, L2, LO, workloads.SPINS, basis).reshape(a.shape[0], C, -1)
        _, r2, _ = oracle.channel_weighted_vjp(a, b, W, c, L1, L2, LO, workloads.SPINS, basis)
        got = out[sel].double().cpu().numpy().reshape(ref.shape)
        got2 = gx2[sel].double().cpu().numpy().reshape(r2.shape)
        res["parity_rel_l2_sampled"] = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        res["parity_rel_l2_gx2_sampled"] = float(np.linalg.norm(got2 - r2) / np.linalg.norm(r2))
        return res

    def measure_depthwise(L1, L2, LO, C, B, V, seed):
        """spingtp_forward_depthwise and spingtp_backward_depthwise with V second-input channels
        (parity basis), preallocated buffers; sampled parity of the forward against the oracle."""
        import oracle
        from paper_2607_01408_amd import paths_host

        plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", 2, channel_weights=True)
        n_paths = len(paths_host(L1, L2, LO, workloads.SPINS, 2))
        x1 = workloads.draw(L1, B, C, 9620 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, V, 9720 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        g = workloads.draw(LO, B, C, 9820 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        w = torch.randn((V, C, n_paths), generator=torch.Generator().manual_seed(seed)).to("cuda:0")
        out, gx1, gx2, gw = torch.empty_like(g), torch.empty_like(x1), torch.empty_like(x2), torch.empty_like(w)
        n = ctypes.c_size_t(0)
        assert _lib.lib().spingtp_backward_depthwise_workspace_size(plan.handle, B, C, V, ctypes.byref(n)) == 0
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device="cuda:0")
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        calls = {"forward": (_lib.lib().spingtp_forward_depthwise,
                             (plan.handle, x1.data_ptr(), x2.data_ptr(), w.data_ptr(), out.data_ptr(), B, C, V, st)),
                 "backward": (_lib.lib().spingtp_backward_depthwise,
                              (plan.handle, x1.data_ptr(), x2.data_ptr(), w.data_ptr(), g.data_ptr(), gx1.data_ptr(),
                               gx2.data_ptr(), gw.data_ptr(), ws.data_ptr(), n.value, B, C, V, st))}
        res = {"V": V, "paths": n_paths, "basis": 2}
        for name, (fn_, call) in calls.items():
            for _ in range(args.warmup):
                assert fn_(*call) == 0
            torch.cuda.synchronize()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            for _ in range(args.steps):
                fn_(*call)
            e.record()
            torch.cuda.synchronize()
            res[name + "_ms"] = s.elapsed_time(e) / args.steps
        sel = torch.as_tensor(sorted({0, B - 1}), device="cuda:0")
        a = x1[sel].double().cpu().numpy().reshape(len(sel), C, -1)
        b = x2[sel].double().cpu().numpy().reshape(len(sel), V, -1)
        ref = oracle.depthwise(a, b, w.double().cpu().numpy(), L1, L2, LO, workloads.SPINS, 2).reshape(len(sel), -1)
        got = out[sel].double().cpu().numpy().reshape(len(sel), -1)
        res["parity_rel_l2_sampled"] = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        return res

    def measure_backward(L, C, B, seed):
        """spingtp_backward_v1 (both gradients) on the default route, preallocated buffers."""
        x1 = workloads.draw(L, B, C, 9300 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L, B, 1, 9400 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        g = workloads.draw(L, B, C, 9500 + seed, "fp32", workloads.SPINS, "unit", "cuda:0")
        plan = Plan(L, L, L, workloads.SPINS, "fp32")
        gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
        n = ctypes.c_size_t(0)
        assert _lib.lib().spingtp_backward_v1_workspace_size(plan.handle, B, C, ctypes.byref(n)) == 0
        ws = torch.empty(n.value, dtype=torch.uint8, device="cuda:0")
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        call = (plan.handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(), gx1.data_ptr(), gx2.data_ptr(),
                ws.data_ptr(), n.value, B, C, st)
        bfn = _lib.lib().spingtp_backward_v1
        for _ in range(args.warmup):
            assert bfn(*call) == 0
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            bfn(*call)
        e.record()
        torch.cuda.synchronize()
        return {"ms": s.elapsed_time(e) / args.steps, "v1_family": plan.kernel_info_v1()["family"]}

    table = []
    for (L1, L2, LO, C, B, p_direct, p_pre, p_triton) in V1_TABLE:
        row = {"L1": L1, "L2": L2, "Lout": LO, "C": C, "B": B,
               "paper_h200_ms": {"direct": p_direct, "precontracted": p_pre, "triton_precontracted": p_triton}}
        for name, fourier in (("precontracted", False), ("fourier", True)):
            row[name] = measure(L1, L2, LO, C, B, fourier, L1 + 3 * L2 + C)
        for name, basis in (("channel_weighted_parity_basis", 2), ("channel_weighted_paper_basis", 0)):
            row[name] = measure_weighted(L1, L2, LO, C, B, basis, L1 + 3 * L2 + C)
            row[name + "_backward"] = measure_weighted_backward(L1, L2, LO, C, B, basis, L1 + 3 * L2 + C)
        for name, basis in (("channel_weighted_unit_parity_basis", 2), ("channel_weighted_unit_paper_basis", 0)):
            row[name] = measure_weighted_unit(L1, L2, LO, C, B, basis, L1 + 3 * L2 + C)
        if B == 1024:  # the depthwise mode with four second-input channels on the largest rows
            row["depthwise_v4_parity_basis"] = measure_depthwise(L1, L2, LO, C, B, 4, L1 + 3 * L2 + C)
            print(f"[v1] ({L1},{L2},{LO}) C={C} B={B}: depthwise V=4 (parity basis) forward "
                  f"{row['depthwise_v4_parity_basis']['forward_ms'] * 1e3:.1f} us, gradients "
                  f"{row['depthwise_v4_parity_basis']['backward_ms'] * 1e3:.1f} us", file=sys.stderr, flush=True)
        table.append(row)
        print(f"[v1] ({L1},{L2},{LO}) C={C} B={B}: pre {row['precontracted']['ms'] * 1e3:.1f} us, "
              f"fourier {row['fourier']['ms'] * 1e3:.1f} us, weighted (parity / paper basis) "
              f"{row['channel_weighted_parity_basis']['ms'] * 1e3:.1f} / "
              f"{row['channel_weighted_paper_basis']['ms'] * 1e3:.1f} us, its gradients "
              f"{row['channel_weighted_parity_basis_backward']['ms'] * 1e3:.1f} / "
              f"{row['channel_weighted_paper_basis_backward']['ms'] * 1e3:.1f} us; x2 per unit: forward "
              f"{row['channel_weighted_unit_parity_basis']['forward_ms'] * 1e3:.1f} / "
              f"{row['channel_weighted_unit_paper_basis']['forward_ms'] * 1e3:.1f} us, gradients "
              f"{row['channel_weighted_unit_parity_basis']['backward_ms'] * 1e3:.1f} / "
              f"{row['channel_weighted_unit_paper_basis']['backward_ms'] * 1e3:.1f} us", file=sys.stderr, flush=True)
    sweep = []
    for L in args.v1_sweep_degrees:
        row = {"L": L, "C": args.v1_sweep_channels, "B": args.v1_sweep_edges}
        for name, fourier in (("precontracted", False), ("fourier", True)):
            row[name] = measure(L, L, L, args.v1_sweep_channels, args.v1_sweep_edges, fourier, 50 + L)
        row["backward"] = measure_backward(L, args.v1_sweep_channels, args.v1_sweep_edges, 60 + L)
        sweep.append(row)
        pre = row["precontracted"]
        print(f"[v1-sweep] L={L}: pre {pre['ms'] if pre else float('nan'):.3f} ms, "
              f"fourier {row['fourier']['ms']:.3f} ms, backward {row['backward']['ms']:.3f} ms",
              file=sys.stderr, flush=True)
    print(json.dumps({
        "metric": "spingtp_forward_v1 time: precontracted vs Fourier route (x2 shared by the C channels)",
        "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": False,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "paper App. E depthwise V = 1 shapes, spins (-1,0,+1), N(0,1) coefficients; "
                               f"sweep L1=L2=Lout in {list(args.v1_sweep_degrees)}, "
                               f"{args.v1_sweep_edges} edges x {args.v1_sweep_channels} channels"},
        "table": table, "sweep": sweep}), flush=True)


def run_backward(args):
    """spingtp_backward on a forward workload: grad_x1 and grad_x2 of a loss with a
    random dLoss/dout, timed per call of the C entry point (HIP events on the
    launch stream, output buffers allocated before timing)."""
    import ctypes

    import numpy as np
    import torch

    import oracle
    from paper_2607_01408_amd import Plan, _lib, workloads

    torch.cuda.set_device(0)
    x1, x2, meta = workloads.make_pair(args.workload, dtype=args.dtype, L=args.L, device="cuda:0")
    L, N, C = meta["L"], meta["N"], meta["C"]
    U = N * C
    g = workloads.draw(L, N, C, 6001, args.dtype, workloads.SPINS, "unit", "cuda:0")
    plan = Plan(L, L, L, workloads.SPINS, args.dtype, valu_only=args.valu)
    gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
    stream = torch.cuda.current_stream()
    fn = _lib.lib().spingtp_backward
    call = (plan.handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(), gx1.data_ptr(), gx2.data_ptr(), N, C,
            ctypes.c_void_p(stream.cuda_stream))
    print(f"[bench] backward {meta['workload']} L={L} units={U} {args.dtype} kernel={plan.kernel_info()}",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        assert fn(*call) == 0
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        fn(*call)
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    avg_ms = float(np.mean([a.elapsed_time(b) for a, b in zip(starts, ends)]))
    rng = np.random.default_rng(78)
    idx = np.unique(np.concatenate([np.arange(min(64, U)), np.arange(max(0, U - 64), U),
                                    rng.choice(U, size=min(U, args.parity_units), replace=False)]))
    ti = torch.as_tensor(idx, device="cuda:0")
    a, b, c = (t.view(U, -1)[ti].double().cpu().numpy() for t in (x1, x2, g))
    r1, r2 = oracle.spingtp_vjp(a, b, c, L, L, L, workloads.SPINS)
    got = np.concatenate([gx1.view(U, -1)[ti].double().cpu().numpy(), gx2.view(U, -1)[ti].double().cpu().numpy()])
    ref = np.concatenate([r1, r2])
    parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    elem = 4 if args.dtype == "fp32" else 2
    nc = 3 * (L + 1) ** 2
    min_bytes = 5 * nc * elem  # read x1, x2, grad_out; write grad_x1, grad_x2
    route_bytes = 6 * nc * elem  # two forward launches (grad_out read twice)
    print(json.dumps({
        "metric": f"backward (grad_x1 and grad_x2) edge-channel units/sec at L={L} {args.dtype}",
        "value": U / (ms_per_step / 1e3), "unit": "units/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "avg_call_ms": avg_ms, "higher_is_better": True,
        "dtype": args.dtype, "data": "synthetic",
        "config": {"workload": meta["workload"], "L": L, "N": N, "C": C, "units": U,
                   "kernel_family": plan.kernel_info()["family"]},
        "hbm": {"min_bytes_per_unit": min_bytes, "route_bytes_per_unit": route_bytes,
                "min_frac": min_bytes * U / (avg_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
                "route_gbs": route_bytes * U / (avg_ms / 1e3) / 1e9},
        "route_tflops": 2 * route_flops(L, L, L, True) * U / (avg_ms / 1e3) / 1e12,
        "parity_rel_l2": parity, "parity_units": int(len(idx))}), flush=True)


def run_sweep(args):
    """The degree sweep: SpinGTP kernel vs two direct O(L^6) Clebsch-Gordan contractions.

    * dense-T GEMM: x1 (x) x2 per unit contracted with the explicit dense real tensor T
      (spingtp_dense_tensor_host) as one fp32 GEMM (2 NC^3 + NC^2 flops per unit);
    * per-path CG: for every path (block triple rho1, rho2 -> rho3 with a nonzero entry,
      spingtp_paths_host) the dense block of T times the outer product of the two input
      blocks (2 d1 d2 d3 + d1 d2 flops per unit and path, the scope table's O(L^6) count
      within a few per cent); paths of equal block shape run as one batched fp32 GEMM.
    Both run through torch (hipBLASLt / rocBLAS) on up to 32,768 units, scaled to the job,
    and are checked against the kernel's output.
    """
    import numpy as np
    import torch

    import oracle
    from paper_2607_01408_amd import Plan, dense_tensor_host, paths_host, workloads

    torch.cuda.set_device(0)
    torch.backends.cuda.matmul.allow_tf32 = False
    rows = []
    for L in args.sweep_degrees:
        x1, x2, meta = workloads.make_pair("sweep", L=L, device="cuda:0")
        U = meta["N"] * meta["C"]
        NC = 3 * (L + 1) ** 2
        plan = Plan(L, L, L, workloads.SPINS, "fp32")
        out = torch.empty_like(x1)
        for _ in range(args.warmup):
            plan.forward(x1, x2, out)
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            plan.forward(x1, x2, out)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / args.steps

        T = torch.from_numpy(dense_tensor_host(L, L, L).astype(np.float32)).to("cuda:0").reshape(NC * NC, NC)
        X1, X2 = x1.view(U, NC), x2.view(U, NC)
        ucg = min(U, 32768)
        chunk = max(1, min(ucg, (1 << 29) // (NC * NC)))
        ycg = torch.empty((ucg, NC), device="cuda:0")

        def cg():
            for u0 in range(0, ucg, chunk):
                u1 = min(ucg, u0 + chunk)
                P = (X1[u0:u1, :, None] * X2[u0:u1, None, :]).reshape(u1 - u0, NC * NC)
                torch.matmul(P, T, out=ycg[u0:u1])

        cg()
        torch.cuda.synchronize()
        s.record()
        cg()
        e.record()
        torch.cuda.synchronize()
        ms_cg = s.elapsed_time(e) * U / ucg
        ref = out.view(U, NC)[:ucg]
        cg_vs_kernel = float(torch.linalg.norm(ycg - ref) / torch.linalg.norm(ref))
        del T
        torch.cuda.empty_cache()

        # per-path CG: group the paths by block shape (d1, d2, d3)
        Td = dense_tensor_host(L, L, L)
        paths = paths_host(L, L, L, workloads.SPINS, 0)
        nb = L + 1

        def slots(b):  # block id = spin index * (L + 1) + degree
            si, l = divmod(int(b), nb)
            o = si * nb * nb + l * l
            return np.arange(o, o + 2 * l + 1)

        groups = {}
        for b1, b2, b3 in paths:
            key = (2 * int(b1 % nb) + 1, 2 * int(b2 % nb) + 1, 2 * int(b3 % nb) + 1)
            groups.setdefault(key, []).append((b1, b2, b3))
        plan_g = []
        path_flops = 0
        for (d1, d2, d3), ps in groups.items():
            i1 = torch.as_tensor(np.stack([slots(p[0]) for p in ps]), device="cuda:0")      # [n, d1]
            i2 = torch.as_tensor(np.stack([slots(p[1]) for p in ps]), device="cuda:0")      # [n, d2]
            i3 = torch.as_tensor(np.concatenate([slots(p[2]) for p in ps]), device="cuda:0")  # [n d3]
            blk = np.stack([Td[np.ix_(slots(p[0]), slots(p[1]), slots(p[2]))].reshape(d1 * d2, d3) for p in ps])
            plan_g.append((i1, i2, i3, torch.from_numpy(blk.astype(np.float32)).to("cuda:0")))
            path_flops += int(len(ps) * (2 * d1 * d2 * d3 + d1 * d2))
        upc = min(ucg, max(256, (1 << 28) // max(1, 4 * max(len(g[3]) * g[3].shape[1] for g in plan_g))))
        ypc = torch.zeros((upc, NC), device="cuda:0")

        def cg_paths():
            ypc.zero_()
            for i1, i2, i3, blk in plan_g:
                n, dd, d3 = blk.shape
                a = X1[:upc][:, i1]                                                   # [U, n, d1]
                b = X2[:upc][:, i2]                                                   # [U, n, d2]
                P = (a[:, :, :, None] * b[:, :, None, :]).reshape(upc, n, dd).transpose(0, 1).contiguous()
                yb = torch.bmm(P, blk)                                                # [n, U, d3]
                ypc.index_add_(1, i3, yb.transpose(0, 1).reshape(upc, n * d3))

        cg_paths()
        torch.cuda.synchronize()
        s.record()
        cg_paths()
        e.record()
        torch.cuda.synchronize()
        ms_cgp = s.elapsed_time(e) * U / upc
        cgp_vs_kernel = float(torch.linalg.norm(ypc - out.view(U, NC)[:upc]) / torch.linalg.norm(out.view(U, NC)[:upc]))
        del plan_g

        n_or = 256 if L <= 8 else 64
        idx = torch.arange(n_or, device="cuda:0")
        t0 = time.perf_counter()
        Tor = oracle.RealGauntTensor(L, L, L, workloads.SPINS)
        tb = time.perf_counter() - t0
        a, b = X1[idx].double().cpu().numpy(), X2[idx].double().cpu().numpy()
        t0 = time.perf_counter()
        yo = Tor.apply(a, b).reshape(n_or, NC)
        to = (time.perf_counter() - t0) / n_or
        parity = float(np.linalg.norm(ref[:n_or].double().cpu().numpy() - yo) / np.linalg.norm(yo))
        fl = route_flops(L, L, L, True)
        fam = plan.kernel_info()["family"]
        rf = roofline(fam, L, "fp32", U, ms, hbm_bytes_per_unit(L, L, L, "fp32"))
        rows.append({
            "L": L, "units": U, "ms": ms, "tp_per_s": U / (ms / 1e3),
            "kernel_family": fam,
            "route_flops_per_unit": fl, "achieved_tflops": fl * U / (ms / 1e3) / 1e12,
            "roofline": {k: rf[k] for k in ("bound", "frac", "fracs", "floors_ms")},
            "cg_dense_ms": ms_cg, "cg_dense_flops_per_unit": 2 * NC ** 3 + NC ** 2,
            "cg_dense_vs_kernel_rel_l2": cg_vs_kernel, "speedup_vs_cg_dense": ms_cg / ms,
            "cg_path_ms": ms_cgp, "cg_path_flops_per_unit": path_flops, "cg_path_paths": int(len(paths)),
            "cg_path_tflops": path_flops * U / (ms_cgp / 1e3) / 1e12,
            "cg_path_vs_kernel_rel_l2": cgp_vs_kernel, "speedup_vs_cg_path": ms_cgp / ms,
            "oracle_cpu_s_per_unit": to, "oracle_tensor_build_s": tb, "parity_rel_l2": parity,
        })
        print(f"[sweep] L={L} {ms:.3f} ms ({U / (ms / 1e3):.3e} TP/s), dense-T CG {ms_cg:.1f} ms, per-path CG "
              f"{ms_cgp:.1f} ms, parity {parity:.2e}", file=sys.stderr, flush=True)
        del x1, x2, out, ycg, ypc
        torch.cuda.empty_cache()
    last = rows[-1]
    print(json.dumps({
        "metric": "SpinGTP forward time vs L (sweep workload) against the direct dense CG contraction",
        "value": last["tp_per_s"], "unit": "TP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "sweep: L1=L2=Lout in {2,4,8,12,16}, spins (-1,0,+1), N=8192 edges x C=32 "
                               "channels (262,144 units), fp32, N(0,1) coefficients"},
        "sweep": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="organic")
    ap.add_argument("--dtype", default="fp32")
    ap.add_argument("--basis", default="paper", choices=sorted(BASES),
                    help="real basis of the coefficients (parity: the parity-labelled basis)")
    ap.add_argument("--L", type=int, default=None, help="degree (sweep workload only)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU seconds per worker process of the oracle baseline (wall time about the same)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--parity-units", type=int, default=16384,
                    help="seeded-random units checked against the oracle (plus the first and last 512)")
    ap.add_argument("--sweep", action="store_true", help="run the degree sweep against the dense CG comparator")
    ap.add_argument("--sweep-degrees", type=int, nargs="+", default=[2, 4, 8, 12, 16])
    ap.add_argument("--backward", action="store_true",
                    help="time spingtp_backward (both gradients) on the chosen workload")
    ap.add_argument("--uvw", action="store_true",
                    help="spingtp_forward_fully_connected (mode uvw) on the App. E.2 shapes")
    ap.add_argument("--v1", action="store_true",
                    help="spingtp_forward_v1: the paper's V = 1 shapes and a degree sweep, both routes")
    ap.add_argument("--v1-sweep-degrees", type=int, nargs="+", default=[1, 2, 3, 4, 5, 6])
    ap.add_argument("--v1-sweep-edges", type=int, default=8192)
    ap.add_argument("--v1-sweep-channels", type=int, default=128)
    ap.add_argument("--valu", action="store_true",
                    help="force the fp32 vector-ALU kernel (SPINGTP_KERNEL_VALU) where a matrix-core kernel exists")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the SpinGTP path has no "
              "multi-GPU leg: units are independent and a multi-GPU run is N independent shards.",
              file=sys.stderr)
        sys.exit(2)

    # the CPU-oracle workers start before this process touches the GPU
    pool = None
    if not (args.sweep or args.v1 or args.backward or args.uvw) and not args.no_cpu_baseline:
        pool = CpuPool(cpu_workers_available())
    try:
        run_main(args, pool)
    finally:
        if pool is not None:
            pool.close()


# the depthwise runtime table's shapes (App. E.2): (L1, L2, Lout, channels C, edges B)
UVW_SHAPES = [(1, 1, 1, 16, 128), (1, 1, 1, 64, 128), (1, 1, 1, 128, 128),
              (2, 2, 2, 16, 32), (2, 2, 2, 64, 32), (2, 2, 2, 128, 32),
              (2, 2, 2, 16, 128), (2, 2, 2, 64, 128), (2, 2, 2, 128, 128),
              (1, 3, 3, 16, 128), (1, 3, 3, 64, 128), (1, 3, 3, 128, 128),
              (2, 2, 2, 64, 1024), (1, 3, 3, 64, 1024), (1, 3, 3, 128, 1024)]


def run_uvw(args):
    """spingtp_forward_fully_connected (mode uvw, App. E.1) on the App. E.2 shapes: U = W = C
    channels, one edge channel (V = 1), B edges, spins (-1, 0, +1), fp32.  Time per call
    (HIP events on the launch stream, fill kernel included), the channel mixing's flops
    (2 U V W d3 per edge and path, run on the fp32 matrix cores) against the fp32 matrix-core
    peak, and the relative L2 error on sampled edges against the oracle.  Then the same for
    spingtp_backward_fully_connected (all three gradients per call: three mixings of that
    size), against the oracle's reverse mode."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_01408_amd import Plan, paths_host, workloads

    torch.cuda.set_device(0)
    rows = []
    for L1, L2, LO, C, B in UVW_SHAPES:
        U, V, W = C, 1, C
        plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", fully_connected=True)
        x1 = workloads.draw(L1, B, U, 7300 + C, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, V, 7400 + C, "fp32", workloads.SPINS, "unit", "cuda:0")
        g = torch.Generator(device="cuda:0")
        g.manual_seed(7500 + B)
        w = torch.randn((plan.n_paths, U, V, W), generator=g, device="cuda:0") / np.sqrt(U * V)
        out = plan.forward_fully_connected(x1, x2, w)
        for _ in range(args.warmup):
            plan.forward_fully_connected(x1, x2, w, out)
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            plan.forward_fully_connected(x1, x2, w, out)
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / args.steps
        d3 = [2 * (int(b3) % (LO + 1)) + 1 for _, _, b3 in paths_host(L1, L2, LO, workloads.SPINS, 0)]
        mix_flops = 2.0 * U * V * W * sum(d3) * B
        sel = np.unique(np.concatenate([np.arange(min(B, 8)), np.arange(max(0, B - 8), B), [B // 2]]))
        ti = torch.as_tensor(sel, device="cuda:0")
        a = x1[ti].double().cpu().numpy().reshape(len(sel), U, -1)
        b = x2[ti].double().cpu().numpy().reshape(len(sel), V, -1)
        ref = oracle.fully_connected(a, b, w.double().cpu().numpy(), L1, L2, LO, workloads.SPINS, 0)
        got = out[ti].double().cpu().numpy().reshape(ref.shape)
        rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        row = {"L1": L1, "L2": L2, "Lout": LO, "C": C, "B": B, "U": U, "V": V, "W": W, "n_paths": plan.n_paths,
               "ms": ms, "mix_flops": mix_flops, "mix_tflops": mix_flops / (ms * 1e-3) / 1e12,
               "mix_frac_of_fp32_mfma_peak": mix_flops / (ms * 1e-3) / (PEAK_MFMA_FP32_TFLOPS * 1e12),
               "parity_rel_l2_sampled": rel, "parity_edges": int(len(sel))}
        rows.append(row)
        print(f"[uvw] ({L1},{L2},{LO}) C={C} B={B}: {ms * 1e3:.1f} us, mixing {row['mix_tflops']:.2f} TF/s, "
              f"parity {rel:.2e}", file=sys.stderr, flush=True)
    # the gradients (spingtp_backward_fully_connected), after every forward so that a kernel
    # trace splits into the two phases by dispatch order
    for row in rows:
        L1, L2, LO, C, B = row["L1"], row["L2"], row["Lout"], row["C"], row["B"]
        U, V, W = C, 1, C
        plan = Plan(L1, L2, LO, workloads.SPINS, "fp32", fully_connected=True)
        x1 = workloads.draw(L1, B, U, 7300 + C, "fp32", workloads.SPINS, "unit", "cuda:0")
        x2 = workloads.draw(L2, B, V, 7400 + C, "fp32", workloads.SPINS, "unit", "cuda:0")
        g = torch.Generator(device="cuda:0")
        g.manual_seed(7500 + B)
        w = torch.randn((plan.n_paths, U, V, W), generator=g, device="cuda:0") / np.sqrt(U * V)
        gy = torch.randn((B, W) + tuple(plan.shape_out), generator=g, device="cuda:0")
        grads = plan.backward_fully_connected(x1, x2, w, gy)
        for _ in range(args.warmup):
            plan.backward_fully_connected(x1, x2, w, gy)
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(args.steps):
            plan.backward_fully_connected(x1, x2, w, gy)
        e.record()
        torch.cuda.synchronize()
        bms = s.elapsed_time(e) / args.steps
        sel = np.unique(np.concatenate([np.arange(min(B, 8)), np.arange(max(0, B - 8), B), [B // 2]]))
        ti = torch.as_tensor(sel, device="cuda:0")
        ref = oracle.fully_connected_vjp(x1[ti].double().cpu().numpy().reshape(len(sel), U, -1),
                                         x2[ti].double().cpu().numpy().reshape(len(sel), V, -1),
                                         w.double().cpu().numpy(), gy[ti].double().cpu().numpy().reshape(len(sel), W, -1),
                                         L1, L2, LO, workloads.SPINS, 0)
        # grad_weights sums over the edges: compared on a call given the sampled edges' rows alone
        gw_sel = plan.backward_fully_connected(x1[ti].contiguous(), x2[ti].contiguous(), w, gy[ti].contiguous(),
                                               need=(False, False, True))[2]
        got = (grads[0][ti], grads[1][ti], gw_sel)
        rels = [float(np.linalg.norm(a.double().cpu().numpy().reshape(r.shape) - r) / np.linalg.norm(r))
                for a, r in zip(got, ref)]
        row.update({"bwd_ms": bms, "bwd_mix_flops": 3 * row["mix_flops"],
                    "bwd_parity_rel_l2_sampled": {"grad_x1": rels[0], "grad_x2": rels[1], "grad_w": rels[2]}})
        print(f"[uvw-bwd] ({L1},{L2},{LO}) C={C} B={B}: {bms * 1e3:.1f} us, parity "
              f"{max(rels):.2e}", file=sys.stderr, flush=True)
    print(json.dumps({"metric": "fully connected SpinGTP (mode uvw) forward and backward time on the App. E.2 shapes",
                      "unit": "ms", "higher_is_better": False, "n_gpus": 1, "steps": args.steps,
                      "warmup": args.warmup, "dtype": "f32", "data": "synthetic",
                      "config": {"workload": "App. E.2 shapes, U = W = C, V = 1, spins (-1,0,1), N(0,1) inputs, "
                                             "N(0,1)/sqrt(U V) weights, N(0,1) output gradients"},
                      "rows": rows}), flush=True)


def run_main(args, pool):
    if args.sweep:
        run_sweep(args)
        return
    if args.uvw:
        run_uvw(args)
        return
    if args.v1:
        run_v1(args)
        return
    if args.backward:
        run_backward(args)
        return

    import numpy as np
    import torch

    from paper_2607_01408_amd import Plan, workloads

    torch.cuda.set_device(0)
    x1, x2, meta = workloads.make_pair(args.workload, dtype=args.dtype, L=args.L, device="cuda:0")
    L = meta["L"]
    U = meta["N"] * meta["C"]
    spins = meta["spins"]
    plan = Plan(L, L, L, spins, args.dtype, BASES[args.basis], valu_only=args.valu)
    out = torch.empty((meta["N"], meta["C"], len(spins), (L + 1) ** 2), dtype=x1.dtype, device="cuda:0")
    print(f"[bench] {meta['workload']} L={L} N={meta['N']} C={meta['C']} {args.dtype} units={U} "
          f"kernel={plan.kernel_info()}", file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        plan.forward(x1, x2, out)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        plan.forward(x1, x2, out)
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    ms_per_step = wall * 1e3 / args.steps
    avg_launch_ms = float(np.mean(launch_ms))
    value = U / (ms_per_step / 1e3)

    kinfo = plan.kernel_info()
    kname = {1: "spingtp_fwd_kernel", 2: "spingtp_fwd_pair_kernel", 3: "spingtp_fwd_big_kernel",
             4: "spingtp_fwd_mfma_kernel", 6: "spingtp_fwd_direct_kernel"}[kinfo["family"]]
    bytes_unit = hbm_bytes_per_unit(L, L, L, args.dtype, len(spins))
    if kinfo["family"] == 6:
        # the direct kernel: one product and one fma per nonzero of T (entries of its table)
        from paper_2607_01408_amd import direct_table_host

        w = direct_table_host(L, L, L, spins, BASES[args.basis], 0)
        nco, nbatch, hdr = int(w[2]), int(w[6]), 18
        vals = w[hdr + nco:hdr + nco + 24 * nbatch].reshape(nbatch, 24)[:, 8:]
        flops_unit = 3 * int((vals != 0).sum())
    else:
        flops_unit = route_flops(L, L, L, True)
    # arithmetic of the path: the matrix-core kernel runs the two phi transforms as fp16
    # products with fp32 accumulation (three split products per term for fp32 I/O)
    if kinfo["family"] == 4:
        compute = "f32 (phi transforms: fp16x3 split matrix products, fp32 accumulate)" if args.dtype == "fp32" \
            else "f32 (phi transforms: fp16 matrix products, fp32 accumulate)"
    else:
        compute = "f32"
    traffic = measured_traffic(meta["workload"], args.dtype, U, L, kname, args.valu, args.basis)

    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # sampled parity against the oracle on the timed output: the first and last 512 units
    # (tile tails) and a seeded random sample
    import oracle

    rng = np.random.default_rng(77)
    # the random units are drawn from between the head and the tail, so the sample holds
    # 1,024 + parity_units distinct units whenever the job has that many
    lo, hi = min(512, U), max(min(512, U), U - 512)
    inner = rng.choice(hi - lo, size=min(hi - lo, args.parity_units), replace=False) + lo
    idx = np.unique(np.concatenate([np.arange(lo), np.arange(hi, U), inner]))
    ti = torch.as_tensor(idx, device="cuda:0")
    ya = out.view(U, -1)[ti].double().cpu().numpy()
    pa, pb = x1.view(U, -1)[ti].double().cpu().numpy(), x2.view(U, -1)[ti].double().cpu().numpy()
    if pool is not None:
        pool.all(("tensor", L, tuple(spins), BASES[args.basis]))
        ref = pool.apply(pa, pb)
    else:
        ref = oracle.spingtp(pa, pb, L, L, L, spins, BASES[args.basis]).reshape(len(idx), -1)
    parity = float(np.linalg.norm(ya - ref) / np.linalg.norm(ref))

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "TP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if (kinfo["family"] != 4 or args.dtype == "fp32") else "f16/f32",
        "compute": compute,
        "io_dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{meta['workload']}: L1=L2=Lout={L}, spins {spins}, N={meta['N']} edges x "
                        f"C={meta['C']} channels ({U} units), {args.dtype} I/O, N(0,1) coefficients",
            "L1": L, "L2": L, "Lout": L, "N": meta["N"], "C": meta["C"], "units": U, "basis": args.basis,
            "seeds": list(meta["seeds"]),
        },
        "roofline": roofline(kinfo["family"], L, args.dtype, U, avg_launch_ms, bytes_unit,
                             flops_unit if kinfo["family"] == 6 else None, len(spins) > 1),
    }
    result["roofline"].update({"traffic": traffic, "kernel": kname, "kernel_family": kinfo["family"],
                               "avg_launch_ms": avg_launch_ms})
    result["parity_rel_l2"] = parity
    result["parity_units"] = int(len(idx))
    if pool is not None:
        result["cpu_baseline"] = cpu_baseline(pool, L, x1, x2, args.cpu_seconds, spins, BASES[args.basis])
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
