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
KERNEL_SOURCES = ("paper_2607_01408_amd/csrc/forward.hip", "paper_2607_01408_amd/csrc/layout.h")


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


def kernel_source_hash():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def profile_tag(workload, dtype, L):
    return f"{workload}_L{L}_{dtype}" if workload == "sweep" else f"{workload}_{dtype}"


def measured_traffic(workload, dtype, units, L):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_spingtp_fwd_{profile_tag(workload, dtype, L)}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_source_hash() or rec.get("units") != units:
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(L, x1, x2, seconds):
    """The CPU oracle on a bounded sample of the same inputs, on the host cores."""
    import numpy as np

    import oracle

    t0 = time.perf_counter()
    T = oracle.RealGauntTensor(L, L, L, (-1, 0, 1))
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


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="organic")
    ap.add_argument("--dtype", default="fp32")
    ap.add_argument("--L", type=int, default=None, help="degree (sweep workload only)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--parity-units", type=int, default=2048)
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the SpinGTP path has no "
              "multi-GPU leg: units are independent and a multi-GPU run is N independent shards.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_01408_amd import Plan, workloads

    torch.cuda.set_device(0)
    x1, x2, meta = workloads.make_pair(args.workload, dtype=args.dtype, L=args.L, device="cuda:0")
    L = meta["L"]
    U = meta["N"] * meta["C"]
    plan = Plan(L, L, L, workloads.SPINS, args.dtype)
    out = torch.empty((meta["N"], meta["C"], 3, (L + 1) ** 2), dtype=x1.dtype, device="cuda:0")
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

    flops_unit = route_flops(L, L, L, True)
    achieved_tflops = flops_unit * U / (avg_launch_ms / 1e3) / 1e12
    bytes_unit = hbm_bytes_per_unit(L, L, L, args.dtype)
    traffic = measured_traffic(meta["workload"], args.dtype, U, L)
    kinfo = plan.kernel_info()
    kname = {1: "spingtp_fwd_kernel", 2: "spingtp_fwd_pair_kernel", 3: "spingtp_fwd_big_kernel"}[kinfo["family"]]

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
                         L, L, L, workloads.SPINS).reshape(len(idx), -1)
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
        "dtype": "f32",
        "io_dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{meta['workload']}: L1=L2=Lout={L}, spins (-1,0,+1), N={meta['N']} edges x "
                        f"C={meta['C']} channels ({U} units), {args.dtype} I/O, N(0,1) coefficients",
            "L1": L, "L2": L, "Lout": L, "N": meta["N"], "C": meta["C"], "units": U,
            "seeds": list(meta["seeds"]),
        },
        "roofline": {
            "bound": "alu",
            "achieved": achieved_tflops,
            "peak": PEAK_FP32_VECTOR_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved_tflops / PEAK_FP32_VECTOR_TFLOPS,
            "traffic": traffic,
            "kernel": kname,
            "avg_launch_ms": avg_launch_ms,
            "flops_per_unit": flops_unit,
            "hbm_bytes_per_unit": bytes_unit,
            "hbm_achieved_gbs": bytes_unit * U / (avg_launch_ms / 1e3) / 1e9,
            "hbm_frac": bytes_unit * U / (avg_launch_ms / 1e3) / 1e9 / PEAK_HBM_GBS,
        },
        "parity_rel_l2": parity,
        "parity_units": int(len(idx)),
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(L, x1, x2, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
