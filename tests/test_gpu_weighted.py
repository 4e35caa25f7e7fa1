"""GPU parity of the path-weighted product (Sec. 3.4 eq. spin_gtp, one weight per
path shared by the channels) against the oracle's PathWeightedTensor.

Weighted plans run the direct kernel (forward and both gradients) and, for an
edge input shared by the channels, the precontracted kernel; their tables hold the
weighted tensor.  Bars as elsewhere: relative L2 1e-5 (fp32), 2e-2 (bf16).
"""

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

from paper_2607_01408_amd import Plan, SpinGTPError, paths_host, workloads  # noqa: E402

S3 = (-1, 0, 1)
S5 = (-2, -1, 0, 1, 2)
TOL = {"fp32": 1e-5, "bf16": 2e-2}


def rel_l2(y, ref):
    return float(np.linalg.norm(y - ref) / max(np.linalg.norm(ref), 1e-300))


def host(t, rows):
    return t.reshape(rows, -1).double().cpu().numpy()


def weights_for(L1, L2, LO, spins, basis, seed):
    n = len(paths_host(L1, L2, LO, spins, basis))
    w = np.random.default_rng(seed).standard_normal(n)
    w[::7] = 0.0  # some paths switched off
    return w


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [(2, 2, 2, S3, 0), (3, 3, 3, S3, 2), (2, 1, 3, S3, 1),
                                                   (2, 2, 2, S5, 0), (2, 2, 2, S5, 2), (4, 4, 4, (0,), 0)])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_weighted_forward_and_backward(L1, L2, LO, spins, basis, dtype):
    N, C = 23, 3
    w = weights_for(L1, L2, LO, spins, basis, L1 + 3 * L2 + 9 * LO + basis)
    print(f"[weighted] L=({L1},{L2},{LO}) spins={spins} basis={basis} {dtype} paths={len(w)}", flush=True)
    x1 = workloads.draw(L1, N, C, 10, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, C, 11, dtype, spins, "unit", "cuda")
    g = workloads.draw(LO, N, C, 12, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, weights=w)
    assert plan.kernel_info()["family"] == 6
    y = plan.forward(x1, x2)
    gx1, gx2 = plan.backward(x1, x2, g)
    torch.cuda.synchronize()
    U = N * C
    W = oracle.PathWeightedTensor(L1, L2, LO, spins, basis, w)
    a, b, c = host(x1, U), host(x2, U), host(g, U)
    r1, r2 = W.vjp(a, b, c)
    errs = (rel_l2(host(y, U), W.apply(a, b).reshape(U, -1)), rel_l2(host(gx1, U), r1), rel_l2(host(gx2, U), r2))
    print(f"[weighted]   rel_l2 {errs}", flush=True)
    assert max(errs) <= TOL[dtype], errs


def test_unit_weights_equal_the_unweighted_product():
    x1 = workloads.draw(3, 40, 4, 20, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(3, 40, 4, 21, "fp32", S3, "unit", "cuda")
    w = np.ones(len(paths_host(3, 3, 3)))
    y1 = Plan(3, 3, 3, S3, "fp32", weights=w).forward(x1, x2)
    y0 = Plan(3, 3, 3, S3, "fp32").forward(x1, x2)  # the Fourier kernel
    torch.cuda.synchronize()
    assert rel_l2(host(y1, 160), host(y0, 160)) <= 2e-6


@pytest.mark.parametrize("L1,L2,LO,spins,C", [(2, 2, 2, S3, 64), (3, 3, 3, S5, 17), (1, 3, 3, S3, 128)])
def test_weighted_v1(L1, L2, LO, spins, C):
    # edge input shared by the channels: the precontracted kernel on the weighted tensor, and the
    # gradients on the direct kernel
    N = 9
    w = weights_for(L1, L2, LO, spins, 0, C)
    x1 = workloads.draw(L1, N, C, 30, "fp32", spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, 1, 31, "fp32", spins, "unit", "cuda")
    g = workloads.draw(LO, N, C, 32, "fp32", spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, "fp32", weights=w)
    assert plan.kernel_info_v1()["family"] == 5
    y = plan.forward_v1(x1, x2)
    gx1, gx2 = plan.backward_v1(x1, x2, g)
    torch.cuda.synchronize()
    U = N * C
    W = oracle.PathWeightedTensor(L1, L2, LO, spins, 0, w)
    a, b, c = host(x1, U), np.repeat(host(x2, N), C, axis=0), host(g, U)
    r1, r2 = W.vjp(a, b, c)
    errs = (rel_l2(host(y, U), W.apply(a, b).reshape(U, -1)), rel_l2(host(gx1, U), r1),
            rel_l2(host(gx2, N), r2.reshape(N, C, -1).sum(axis=1)))
    print(f"[weighted-v1] L=({L1},{L2},{LO}) C={C} rel_l2 {errs}", flush=True)
    assert max(errs) <= 1e-5, errs


def test_weighted_plan_rules():
    w = np.ones(len(paths_host(2, 2, 2)))
    with pytest.raises(SpinGTPError):
        Plan(2, 2, 2, S3, "fp32", weights=w[:-1])
    with pytest.raises(SpinGTPError):
        Plan(2, 2, 2, S3, "fp32", v1_fourier=True, weights=w)


# --- per-channel path weights, x2 shared by the channels (spingtp_forward_v1_weighted) ---

def run_channel_weighted(L1, L2, LO, spins, N, C, basis=0, dtype="fp32", seed=0):
    P = paths_host(L1, L2, LO, spins, basis)
    print(f"[v1-weighted] L=({L1},{L2},{LO}) spins={spins} basis={basis} N={N} C={C} {dtype} paths={len(P)}",
          flush=True)
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((C, len(P)))
    x1 = workloads.draw(L1, N, C, 40 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, 1, 41 + seed, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, channel_weights=True)
    y = plan.forward_v1_weighted(x1, x2, torch.as_tensor(W, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    Wf = torch.as_tensor(W, dtype=torch.float32).double().numpy()  # the fp32 weights the kernel read
    a, b = host(x1, N * C).reshape(N, C, -1), host(x2, N)
    g = host(y, N * C).reshape(N, C, -1)
    ref = np.stack([oracle.PathWeightedTensor(L1, L2, LO, spins, basis, Wf[c]).apply(a[:, c], b).reshape(N, -1)
                    for c in range(C)], axis=1)
    err = rel_l2(g, ref)
    print(f"[v1-weighted]   rel_l2={err:.3e}", flush=True)
    assert err <= (1e-5 if dtype == "fp32" else 2e-2), err
    return plan, (x1, x2, W, y)


@pytest.mark.parametrize("shape,C", [((1, 1, 1), 16), ((1, 1, 1), 128), ((2, 2, 2), 64), ((2, 2, 2), 17),
                                     ((1, 3, 3), 128), ((1, 3, 3), 1)])
@pytest.mark.parametrize("basis", [0, 2])
def test_channel_weighted_v1_table_shapes(shape, C, basis):
    # the depthwise V = 1 shapes of the paper's runtime table (App. E.2), with per-channel path weights
    run_channel_weighted(*shape, S3, 11, C, basis, seed=C + sum(shape))


@pytest.mark.parametrize("L1,L2,LO,spins", [(2, 2, 2, (0,)), (4, 4, 4, (0,)), (2, 1, 2, S3), (0, 2, 2, S3)])
def test_channel_weighted_v1_other_shapes(L1, L2, LO, spins):
    run_channel_weighted(L1, L2, LO, spins, 7, 40, 1, seed=L1 + L2)


def test_channel_weighted_v1_bf16():
    run_channel_weighted(2, 2, 2, S3, 9, 48, 2, "bf16", seed=5)


def test_channel_weighted_unit_weights_equal_forward_v1():
    N, C = 13, 33
    n = len(paths_host(2, 2, 2))
    x1 = workloads.draw(2, N, C, 50, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(2, N, 1, 51, "fp32", S3, "unit", "cuda")
    plan = Plan(2, 2, 2, S3, "fp32", channel_weights=True)
    y1 = plan.forward_v1_weighted(x1, x2, torch.ones((C, n), device="cuda"))
    y0 = plan.forward_v1(x1, x2)
    torch.cuda.synchronize()
    assert rel_l2(host(y1, N * C), host(y0, N * C)) <= 1e-6


def test_channel_weighted_rules():
    x1 = torch.zeros((2, 3, 3, 9), device="cuda")
    x2 = torch.zeros((2, 1, 3, 9), device="cuda")
    n = len(paths_host(2, 2, 2))
    with pytest.raises(ValueError):  # the plan has no weighted table (and no path count)
        Plan(2, 2, 2, S3, "fp32").forward_v1_weighted(x1, x2, torch.zeros((3, n), device="cuda"))
    from paper_2607_01408_amd import _lib
    w = torch.zeros((3, n), device="cuda")
    y = torch.empty((2, 3, 3, 9), device="cuda")
    assert _lib.lib().spingtp_forward_v1_weighted(Plan(2, 2, 2, S3, "fp32").handle, x1.data_ptr(), x2.data_ptr(),
                                                  w.data_ptr(), y.data_ptr(), 2, 3, None) == 2
    plan = Plan(2, 2, 2, S3, "fp32", channel_weights=True)
    with pytest.raises(ValueError):
        plan.forward_v1_weighted(x1, x2, torch.zeros((2, n), device="cuda"))  # one row per channel
    with pytest.raises(ValueError):
        plan.forward_v1_weighted(x1, x2, torch.zeros((3, n - 1), device="cuda"))  # one weight per path
    y = plan.forward_v1_weighted(x1, x2, torch.zeros((3, n), device="cuda"))
    torch.cuda.synchronize()
    assert not y.any()
    # path slots beyond the precontracted kernel's instantiations (degree 3 with spins {-1, 0, +1},
    # parity basis): the forward runs on the entry lists only; with SPINGTP_V1_PRECONTRACT too, as
    # that route does not exist; in the paper basis (335 paths) nothing fits
    with pytest.raises(SpinGTPError):
        Plan(3, 3, 3, S3, "fp32", 0, channel_weights=True)
    for pre in (False, True):
        plan3 = Plan(3, 3, 3, S3, "fp32", 2, channel_weights=True, v1_precontract=pre)
        x13 = torch.ones((2, 3, 3, 16), device="cuda")
        y3 = plan3.forward_v1_weighted(x13, torch.ones((2, 1, 3, 16), device="cuda"),
                                       torch.zeros((3, plan3.n_paths), device="cuda"))
        torch.cuda.synchronize()
        assert not y3.any()
    with pytest.raises(SpinGTPError):  # neither fits: 2002 paths at degree 6
        Plan(6, 6, 6, S3, "fp32", channel_weights=True)


# --- gradients of the per-channel path-weighted product (spingtp_backward_v1_weighted) ---

def run_channel_weighted_backward(L1, L2, LO, spins, N, C, basis=0, dtype="fp32", seed=0):
    P = paths_host(L1, L2, LO, spins, basis)
    print(f"[v1-weighted-bwd] L=({L1},{L2},{LO}) spins={spins} basis={basis} N={N} C={C} {dtype} "
          f"paths={len(P)}", flush=True)
    rng = np.random.default_rng(100 + seed)
    W = torch.as_tensor(rng.standard_normal((C, len(P))), dtype=torch.float32, device="cuda")
    x1 = workloads.draw(L1, N, C, 60 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, 1, 61 + seed, dtype, spins, "unit", "cuda")
    g = workloads.draw(LO, N, C, 62 + seed, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, channel_weights=True)
    gx1, gx2, gW = plan.backward_v1_weighted(x1, x2, W, g)
    torch.cuda.synchronize()
    a, b, c = host(x1, N * C).reshape(N, C, -1), host(x2, N), host(g, N * C).reshape(N, C, -1)
    r1, r2, rW = oracle.channel_weighted_v1_vjp(a, b, W.double().cpu().numpy(), c, L1, L2, LO, spins, basis)
    e1 = rel_l2(host(gx1, N * C), r1.reshape(N * C, -1)) if N * C else 0.0
    e2 = rel_l2(host(gx2, N), r2) if N else 0.0
    eW = rel_l2(gW.double().cpu().numpy(), rW) if N * C else float(gW.abs().max()) if C else 0.0
    print(f"[v1-weighted-bwd]   rel_l2 gx1={e1:.3e} gx2={e2:.3e} gW={eW:.3e}", flush=True)
    tol = TOL[dtype]
    assert e1 <= tol and e2 <= tol and eW <= tol, (e1, e2, eW)
    return plan, (x1, x2, W, g), (gx1, gx2, gW)


@pytest.mark.parametrize("shape,C", [((1, 1, 1), 16), ((2, 2, 2), 64), ((2, 2, 2), 17), ((1, 3, 3), 128),
                                     ((1, 3, 3), 1)])
@pytest.mark.parametrize("basis", [0, 2])
def test_channel_weighted_backward_table_shapes(shape, C, basis):
    # the depthwise V = 1 shapes of the paper's runtime table (App. E.2)
    run_channel_weighted_backward(*shape, S3, 11, C, basis, seed=C + sum(shape))


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [(2, 1, 2, S3, 1), (2, 2, 2, (0,), 0), (3, 3, 3, S3, 2),
                                                   (2, 1, 2, S5, 0)])
def test_channel_weighted_backward_other_shapes(L1, L2, LO, spins, basis):
    # shapes without a weighted forward kernel too (degree 3): the gradients have their own
    # kernel, and plan creation keeps its table
    run_channel_weighted_backward(L1, L2, LO, spins, 5, 70, basis, seed=L1 + 3 * L2)


def test_channel_weighted_backward_many_edge_ranges():
    # 1500 edges over 3 channel tiles (130 channels, the last tile ragged): several edges
    # per workgroup, so the weight gradient adds partial sums over edge ranges
    run_channel_weighted_backward(1, 1, 1, S3, 1500, 130, 0, seed=3)


def test_channel_weighted_backward_bf16():
    run_channel_weighted_backward(2, 2, 2, S3, 9, 48, 2, "bf16", seed=5)


def test_channel_weighted_backward_empty():
    # no edges: grad_weights is an empty sum (zeros); no channels: grad_x2 is zeros
    plan = Plan(2, 2, 2, S3, "fp32", channel_weights=True)
    n = plan.n_paths
    x1, x2 = torch.zeros((0, 8, 3, 9), device="cuda"), torch.zeros((0, 1, 3, 9), device="cuda")
    gx1, gx2, gW = plan.backward_v1_weighted(x1, x2, torch.ones((8, n), device="cuda"), x1)
    torch.cuda.synchronize()
    assert gx1.shape == (0, 8, 3, 9) and gx2.shape == (0, 1, 3, 9)
    assert gW.shape == (8, n) and not gW.any()
    x1 = torch.zeros((4, 0, 3, 9), device="cuda")
    x2 = workloads.draw(2, 4, 1, 3, "fp32", S3, "unit", "cuda")
    gx1, gx2, gW = plan.backward_v1_weighted(x1, x2, torch.zeros((0, n), device="cuda"), x1)
    torch.cuda.synchronize()
    assert gx2.shape == (4, 1, 3, 9) and not gx2.any() and gW.shape == (0, n)


def test_channel_weighted_backward_matches_forward_identity():
    # oracle-free: the product is linear in each argument, so <g, y> = <gx1, x1> = <gx2, x2> = <gW, W>
    # with y from the forward kernel and the gradients from the backward kernel on the same device data
    plan, (x1, x2, W, g), (gx1, gx2, gW) = run_channel_weighted_backward(2, 2, 2, S3, 40, 96, 2, seed=9)
    y = plan.forward_v1_weighted(x1, x2, W)
    torch.cuda.synchronize()
    e = float((g.double() * y.double()).sum())
    for grad, val in ((gx1, x1), (gx2, x2), (gW, W)):
        d = float((grad.double() * val.double()).sum())
        assert abs(d - e) <= 1e-5 * max(1.0, abs(e)), (d, e)


def test_channel_weighted_backward_repeatable():
    # the partial sums are added in a fixed order: two calls give identical bits
    _, (x1, x2, W, g), (gx1, gx2, gW) = run_channel_weighted_backward(1, 3, 3, S3, 600, 64, 0, seed=4)
    plan = Plan(1, 3, 3, S3, "fp32", 0, channel_weights=True)
    hx1, hx2, hW = plan.backward_v1_weighted(x1, x2, W, g)
    torch.cuda.synchronize()
    assert torch.equal(gx1, hx1) and torch.equal(gx2, hx2) and torch.equal(gW, hW)


def test_channel_weighted_backward_rules():
    from paper_2607_01408_amd import _lib
    x1 = torch.zeros((2, 3, 3, 9), device="cuda")
    x2 = torch.zeros((2, 1, 3, 9), device="cuda")
    n = len(paths_host(2, 2, 2))
    W = torch.zeros((3, n), device="cuda")
    with pytest.raises(ValueError):  # weights need a plan created with channel_weights=True
        Plan(2, 2, 2, S3, "fp32").backward_v1_weighted(x1, x2, W, x1)
    size = ctypes_size_t()
    assert _lib.lib().spingtp_backward_v1_weighted_workspace_size(Plan(2, 2, 2, S3, "fp32").handle, 2, 3,
                                                                  size) == 2
    plan = Plan(2, 2, 2, S3, "fp32", channel_weights=True)
    with pytest.raises(ValueError):
        plan.backward_v1_weighted(x1, x2, W[:, :-1].contiguous(), x1)  # one weight per path
    assert _lib.lib().spingtp_backward_v1_weighted_workspace_size(plan.handle, 2, 3, size) == 0
    gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
    gW = torch.empty_like(W)
    ws = torch.empty(max(1, size.value), dtype=torch.uint8, device="cuda")
    args = [x1.data_ptr(), x2.data_ptr(), W.data_ptr(), x1.data_ptr(), gx1.data_ptr(), gx2.data_ptr(),
            gW.data_ptr(), ws.data_ptr()]
    if size.value > 0:  # too small a workspace
        assert _lib.lib().spingtp_backward_v1_weighted(plan.handle, *args, size.value - 1, 2, 3, None) == 1
    bad = list(args)
    bad[6] = None  # grad_weights missing
    assert _lib.lib().spingtp_backward_v1_weighted(plan.handle, *bad, size.value, 2, 3, None) == 1
    assert _lib.lib().spingtp_backward_v1_weighted(plan.handle, *args, size.value, 2, 3, None) == 0
    torch.cuda.synchronize()
    assert not gx1.any() and not gx2.any() and not gW.any()


def ctypes_size_t():
    import ctypes
    return ctypes.c_size_t(0)


# --- per-channel path weights with a per-unit second input (spingtp_forward_weighted and
# spingtp_backward_weighted, mode uuu) ---

def run_channel_weighted_unit(L1, L2, LO, spins, N, C, basis=0, dtype="fp32", seed=0):
    P = paths_host(L1, L2, LO, spins, basis)
    print(f"[weighted-unit] L=({L1},{L2},{LO}) spins={spins} basis={basis} N={N} C={C} {dtype} paths={len(P)}",
          flush=True)
    rng = np.random.default_rng(200 + seed)
    W = torch.as_tensor(rng.standard_normal((C, len(P))), dtype=torch.float32, device="cuda")
    x1 = workloads.draw(L1, N, C, 70 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, C, 71 + seed, dtype, spins, "unit", "cuda")
    g = workloads.draw(LO, N, C, 72 + seed, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, channel_weights=True)
    y = plan.forward_weighted(x1, x2, W)
    gx1, gx2, gW = plan.backward_weighted(x1, x2, W, g)
    torch.cuda.synchronize()
    a, b, c = (host(t, N * C).reshape(N, C, -1) for t in (x1, x2, g))
    Wd = W.double().cpu().numpy()
    ref = oracle.channel_weighted(a, b, Wd, L1, L2, LO, spins, basis).reshape(N * C, -1)
    r1, r2, rW = oracle.channel_weighted_vjp(a, b, Wd, c, L1, L2, LO, spins, basis)
    ey = rel_l2(host(y, N * C), ref)
    e1 = rel_l2(host(gx1, N * C), r1.reshape(N * C, -1))
    e2 = rel_l2(host(gx2, N * C), r2.reshape(N * C, -1))
    eW = rel_l2(gW.double().cpu().numpy(), rW)
    print(f"[weighted-unit]   rel_l2 y={ey:.3e} gx1={e1:.3e} gx2={e2:.3e} gW={eW:.3e}", flush=True)
    tol = TOL[dtype]
    assert max(ey, e1, e2, eW) <= tol, (ey, e1, e2, eW)
    return plan, (x1, x2, W, g), (y, gx1, gx2, gW)


@pytest.mark.parametrize("shape,C,basis", [((1, 1, 1), 16, 0), ((2, 2, 2), 64, 2), ((2, 2, 2), 70, 0),
                                           ((1, 3, 3), 128, 0), ((1, 3, 3), 33, 2)])
def test_channel_weighted_unit_shapes(shape, C, basis):
    run_channel_weighted_unit(*shape, S3, 9, C, basis, seed=C + sum(shape))


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [(2, 1, 2, S5, 0), (3, 3, 3, S3, 2), (2, 2, 2, (0,), 0)])
def test_channel_weighted_unit_other_shapes(L1, L2, LO, spins, basis):
    run_channel_weighted_unit(L1, L2, LO, spins, 5, 40, basis, seed=L1 + 5 * L2)


def test_channel_weighted_unit_many_edge_ranges():
    # 1500 edges over 3 channel tiles (130 channels): several edges per workgroup
    run_channel_weighted_unit(1, 1, 1, S3, 1500, 130, 0, seed=8)


def test_channel_weighted_unit_bf16():
    run_channel_weighted_unit(2, 2, 2, S3, 9, 48, 2, "bf16", seed=6)


def test_channel_weighted_unit_matches_the_shared_form():
    # x2 equal over the channels of an edge: the per-unit kernels agree with the V = 1 ones
    N, C = 21, 70
    n = len(paths_host(2, 2, 2))
    plan = Plan(2, 2, 2, S3, "fp32", 0, channel_weights=True)
    W = torch.randn((C, n), generator=torch.Generator().manual_seed(3)).to("cuda")
    x1 = workloads.draw(2, N, C, 80, "fp32", S3, "unit", "cuda")
    x2s = workloads.draw(2, N, 1, 81, "fp32", S3, "unit", "cuda")
    g = workloads.draw(2, N, C, 82, "fp32", S3, "unit", "cuda")
    x2 = x2s.expand(N, C, 3, 9).contiguous()
    y = plan.forward_weighted(x1, x2, W)
    y1 = plan.forward_v1_weighted(x1, x2s, W)
    gx1, gx2, gW = plan.backward_weighted(x1, x2, W, g)
    hx1, hx2, hW = plan.backward_v1_weighted(x1, x2s, W, g)
    torch.cuda.synchronize()
    assert rel_l2(host(y, N * C), host(y1, N * C)) <= 1e-6
    assert rel_l2(host(gx1, N * C), host(hx1, N * C)) <= 1e-6
    assert rel_l2(host(gx2.sum(dim=1, keepdim=True), N), host(hx2, N)) <= 1e-5
    assert rel_l2(gW.double().cpu().numpy(), hW.double().cpu().numpy()) <= 1e-6


def test_channel_weighted_unit_empty_and_rules():
    plan = Plan(2, 2, 2, S3, "fp32", channel_weights=True)
    n = plan.n_paths
    x1, x2 = torch.zeros((0, 8, 3, 9), device="cuda"), torch.zeros((0, 8, 3, 9), device="cuda")
    W = torch.ones((8, n), device="cuda")
    y = plan.forward_weighted(x1, x2, W)
    gx1, gx2, gW = plan.backward_weighted(x1, x2, W, x1)
    torch.cuda.synchronize()
    assert y.shape == (0, 8, 3, 9) and gW.shape == (8, n) and not gW.any()
    x1 = torch.zeros((2, 3, 3, 9), device="cuda")
    with pytest.raises(ValueError):  # a plan without channel weights has no path count
        Plan(2, 2, 2, S3, "fp32").forward_weighted(x1, x1, torch.zeros((3, n), device="cuda"))
    with pytest.raises(ValueError):  # x2 per unit
        plan.forward_weighted(x1, x1[:, :1].contiguous(), torch.zeros((3, n), device="cuda"))
    from paper_2607_01408_amd import _lib
    w = torch.zeros((3, n), device="cuda")
    y = torch.empty_like(x1)
    assert _lib.lib().spingtp_forward_weighted(Plan(2, 2, 2, S3, "fp32").handle, x1.data_ptr(), x1.data_ptr(),
                                               w.data_ptr(), y.data_ptr(), 2, 3, None) == 2
    assert _lib.lib().spingtp_forward_weighted(plan.handle, x1.data_ptr(), x1.data_ptr(), None, y.data_ptr(), 2, 3,
                                               None) == 1


@pytest.mark.parametrize("shape,basis", [((2, 2, 2), 2), ((1, 3, 3), 0), ((1, 1, 1), 0)])
def test_channel_weighted_v1_routes_agree(shape, basis):
    # the default entry-list route and the precontracted route (SPINGTP_V1_PRECONTRACT) of
    # spingtp_forward_v1_weighted on the same data
    N, C = 17, 70
    n = len(paths_host(*shape, S3, basis))
    W = torch.randn((C, n), generator=torch.Generator().manual_seed(11)).to("cuda")
    x1 = workloads.draw(shape[0], N, C, 90, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(shape[1], N, 1, 91, "fp32", S3, "unit", "cuda")
    y0 = Plan(*shape, S3, "fp32", basis, channel_weights=True).forward_v1_weighted(x1, x2, W)
    y1 = Plan(*shape, S3, "fp32", basis, channel_weights=True, v1_precontract=True).forward_v1_weighted(x1, x2, W)
    torch.cuda.synchronize()
    assert rel_l2(host(y0, N * C), host(y1, N * C)) <= 1e-6


# --- depthwise mode with V second-input channels (spingtp_forward_depthwise, uvu) ---

def run_depthwise(L1, L2, LO, spins, N, C, V, basis=0, dtype="fp32", seed=0):
    P = paths_host(L1, L2, LO, spins, basis)
    print(f"[depthwise] L=({L1},{L2},{LO}) spins={spins} basis={basis} N={N} C={C} V={V} {dtype}", flush=True)
    rng = np.random.default_rng(300 + seed)
    W = torch.as_tensor(rng.standard_normal((V, C, len(P))), dtype=torch.float32, device="cuda")
    x1 = workloads.draw(L1, N, C, 73 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, V, 74 + seed, dtype, spins, "unit", "cuda")
    g = workloads.draw(LO, N, C, 75 + seed, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, channel_weights=True)
    y = plan.forward_depthwise(x1, x2, W)
    gx1, gx2, gW = plan.backward_depthwise(x1, x2, W, g)
    torch.cuda.synchronize()
    a, c = host(x1, N * C).reshape(N, C, -1), host(g, N * C).reshape(N, C, -1)
    b = host(x2, N * V).reshape(N, V, -1)
    Wd = W.double().cpu().numpy()
    ref = oracle.depthwise(a, b, Wd, L1, L2, LO, spins, basis).reshape(N * C, -1)
    r1, r2, rW = oracle.depthwise_vjp(a, b, Wd, c, L1, L2, LO, spins, basis)
    errs = (rel_l2(host(y, N * C), ref), rel_l2(host(gx1, N * C), r1.reshape(N * C, -1)),
            rel_l2(host(gx2, N * V), r2.reshape(N * V, -1)), rel_l2(gW.double().cpu().numpy(), rW))
    print(f"[depthwise]   rel_l2 y={errs[0]:.3e} gx1={errs[1]:.3e} gx2={errs[2]:.3e} gW={errs[3]:.3e}", flush=True)
    assert max(errs) <= TOL[dtype], errs
    return plan, (x1, x2, W, g), (y, gx1, gx2, gW)


# V = 2..4 run as one launch of the fused kernel, V = 5, 6 as four channels and then the rest
@pytest.mark.parametrize("shape,C,V,basis", [((1, 1, 1), 16, 3, 0), ((2, 2, 2), 70, 2, 2), ((1, 3, 3), 33, 4, 0),
                                             ((2, 1, 2), 64, 2, 1), ((2, 2, 2), 40, 6, 0), ((1, 2, 2), 24, 5, 2)])
def test_depthwise_shapes(shape, C, V, basis):
    run_depthwise(*shape, S3, 11, C, V, basis, seed=C + V)


def test_depthwise_bf16():
    run_depthwise(2, 2, 2, S3, 9, 48, 2, 2, "bf16", seed=4)


def test_depthwise_one_channel_is_the_v1_form():
    plan, (x1, x2, W, g), (y, gx1, gx2, gW) = run_depthwise(2, 2, 2, S3, 13, 40, 1, 0, seed=2)
    y1 = plan.forward_v1_weighted(x1, x2, W[0].contiguous())
    hx1, hx2, hW = plan.backward_v1_weighted(x1, x2, W[0].contiguous(), g)
    torch.cuda.synchronize()
    assert torch.equal(y, y1) and torch.equal(gx1, hx1) and torch.equal(gx2, hx2) and torch.equal(gW[0], hW)


def test_depthwise_rules():
    plan = Plan(2, 2, 2, S3, "fp32", channel_weights=True)
    n = plan.n_paths
    x1 = torch.zeros((2, 3, 3, 9), device="cuda")
    with pytest.raises(SpinGTPError):  # V = 0: no second-input channel
        plan.forward_depthwise(x1, torch.zeros((2, 0, 3, 9), device="cuda"), torch.zeros((0, 3, n), device="cuda"))
    with pytest.raises(ValueError):  # one weight slice per second-input channel
        plan.forward_depthwise(x1, torch.zeros((2, 2, 3, 9), device="cuda"), torch.zeros((1, 3, n), device="cuda"))
