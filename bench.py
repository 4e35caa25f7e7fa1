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

PEAK_FP32_VECTOR_TFLOPS = 157.3  # MI355X published fp32 vector peak
PEAK_HBM_GBS = 8000.0
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


def route_flops(L1, L2, LO, spin=True):
    """Algorithmic flops per unit of the exact-grid route (FMA = 2 flops).

    Counts the structural work of the five steps on the n_theta x n_phi grid:
    (A) one FMA per valid input coefficient plus the spin recombination,
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
    per_node = (stage_a(L1) + stage_a(L2) + npoly * (synth(L1) + synth(L2)) + NP * prod
                + npoly * analysis + stage_e)
    return NT * per_node


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


def cpu_baseline(L, x1, x2, seconds, spins=(-1, 0, 1), basis=0):
    """The CPU oracle on a bounded sample of the same inputs, on the host cores."""
    import numpy as np

    import oracle

    t0 = time.perf_counter()
    T = oracle.RealGauntTensor(L, L, L, spins, basis)
    build_s = time.perf_counter() - t0
    U = x1.shape[0] * x1.shape[1]
    a = x1.reshape(U, -1)
    b = x2.reshape(U, -1)
    # calibrate on 256 units, then size the sample to ~`seconds`
    probe = 256
    t0 = time.perf_counter()
    T.apply(a[:probe].double().cpu().numpy(), b[:probe].double().cpu().numpy())
    per_unit = (time.perf_counter() - t0) / probe
    n = int(max(probe, min(U, seconds / max(per_unit, 1e-9))))
    rng = np.random.default_rng(1234)
    import torch
    idx = torch.as_tensor(np.sort(rng.choice(U, size=n, replace=False)), device=a.device)
    A = a[idx].double().cpu().numpy()
    B = b[idx].double().cpu().numpy()
    t0 = time.perf_counter()
    T.apply(A, B)
    dt = time.perf_counter() - t0
    return {
        "value": n / dt,
        "unit": "TP/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"{n} seeded-random units of the same inputs ({dt:.1f} s of contraction, float64, "
                  f"single-threaded numpy/scipy); sparse tensor build {build_s:.2f} s excluded",
        "extrapolated_full_job_s": U / (n / dt),
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
    """The degree sweep: SpinGTP kernel vs the direct O(L^6) dense contraction.

    The comparator forms x1 (x) x2 per unit and contracts it with the explicit
    dense real tensor T (spingtp_dense_tensor_host) as one fp32 GEMM on the GPU
    (hipBLASLt through torch): the Clebsch-Gordan-style direct product on the same
    inputs.  Its time is measured on up to 32,768 units and scaled to the job.
    """
    import numpy as np
    import torch

    import oracle
    from paper_2607_01408_amd import Plan, dense_tensor_host, workloads

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
        rows.append({
            "L": L, "units": U, "ms": ms, "tp_per_s": U / (ms / 1e3),
            "kernel_family": plan.kernel_info()["family"],
            "route_flops_per_unit": fl, "achieved_tflops": fl * U / (ms / 1e3) / 1e12,
            "cg_dense_ms": ms_cg, "cg_dense_flops_per_unit": 2 * NC ** 3 + NC ** 2,
            "cg_dense_vs_kernel_rel_l2": cg_vs_kernel, "speedup_vs_cg_dense": ms_cg / ms,
            "oracle_cpu_s_per_unit": to, "oracle_tensor_build_s": tb, "parity_rel_l2": parity,
        })
        print(f"[sweep] L={L} {ms:.3f} ms ({U / (ms / 1e3):.3e} TP/s), dense CG {ms_cg:.1f} ms, "
              f"parity {parity:.2e}", file=sys.stderr, flush=True)
        del T, x1, x2, out, ycg
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
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--parity-units", type=int, default=2048)
    ap.add_argument("--sweep", action="store_true", help="run the degree sweep against the dense CG comparator")
    ap.add_argument("--sweep-degrees", type=int, nargs="+", default=[2, 4, 8, 12, 16])
    ap.add_argument("--backward", action="store_true",
                    help="time spingtp_backward (both gradients) on the chosen workload")
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

    if args.sweep:
        run_sweep(args)
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
    achieved_tflops = flops_unit * U / (avg_launch_ms / 1e3) / 1e12
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

    # sampled parity against the oracle on the timed output
    import oracle

    rng = np.random.default_rng(77)
    n_par = min(U, args.parity_units)
    idx = np.unique(np.concatenate([np.arange(min(64, U)), np.arange(max(0, U - 64), U),
                                    rng.choice(U, size=n_par, replace=False)]))
    ti = torch.as_tensor(idx, device="cuda:0")
    ya = out.view(U, -1)[ti].double().cpu().numpy()
    ref = oracle.spingtp(x1.view(U, -1)[ti].double().cpu().numpy(), x2.view(U, -1)[ti].double().cpu().numpy(),
                         L, L, L, spins, BASES[args.basis]).reshape(len(idx), -1)
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
        "roofline": {
            "bound": "alu",
            "achieved": achieved_tflops,
            "peak": PEAK_FP32_VECTOR_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved_tflops / PEAK_FP32_VECTOR_TFLOPS,
        } if kinfo["family"] != 6 else {
            # the direct kernel moves more bytes per flop than the fp32 ridge point: HBM bound
            "bound": "hbm",
            "achieved": bytes_unit * U / (avg_launch_ms / 1e3) / 1e9,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": bytes_unit * U / (avg_launch_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
            "alu_tflops": achieved_tflops,
            "alu_frac": achieved_tflops / PEAK_FP32_VECTOR_TFLOPS,
        },
    }
    result["roofline"].update({
            "traffic": traffic,
            "kernel": kname,
            "kernel_family": kinfo["family"],
            "avg_launch_ms": avg_launch_ms,
            "flops_per_unit": flops_unit,
            "hbm_bytes_per_unit": bytes_unit,
            "hbm_achieved_gbs": bytes_unit * U / (avg_launch_ms / 1e3) / 1e9,
            "hbm_frac": bytes_unit * U / (avg_launch_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
    })
    result["parity_rel_l2"] = parity
    result["parity_units"] = int(len(idx))
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(L, x1, x2, args.cpu_seconds, spins, BASES[args.basis])
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
