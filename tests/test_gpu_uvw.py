"""GPU parity of the fully connected product (mode uvw, spingtp_forward_fully_connected)
against the oracle, through the C ABI.  fp32; bar: relative L2 <= 1e-5 (the products
and sums are fp32 on both the vector ALU and the matrix cores).
"""

import ctypes

import numpy as np
import pytest

import oracle
from tests.oracle_helpers import valid_mask

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

from paper_2607_01408_amd import Plan, SpinGTPError, workloads  # noqa: E402
from paper_2607_01408_amd import _lib  # noqa: E402

S3 = (-1, 0, 1)
S5 = (-2, -1, 0, 1, 2)
TOL = 1e-5


def run_uvw(L1, L2, LO, spins, N, U, V, W, basis=0, seed=0, edges=None):
    print(f"[uvw] L=({L1},{L2},{LO}) spins={spins} N={N} U={U} V={V} W={W} basis={basis}", flush=True)
    plan = Plan(L1, L2, LO, spins, "fp32", basis, fully_connected=True)
    x1 = workloads.draw(L1, N, U, 5300 + seed, "fp32", spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, V, 5400 + seed, "fp32", spins, "unit", "cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(5500 + seed)
    w = torch.randn((plan.n_paths, U, V, W), generator=g, device="cuda") / np.sqrt(max(1, U * V))
    y = plan.forward_fully_connected(x1, x2, w)
    torch.cuda.synchronize()
    sel = np.arange(N) if edges is None else np.unique(np.asarray(edges))
    ti = torch.as_tensor(sel, device="cuda")
    a, b = x1[ti].double().cpu().numpy(), x2[ti].double().cpu().numpy()
    ref = oracle.fully_connected(a.reshape(len(sel), U, -1), b.reshape(len(sel), V, -1), w.double().cpu().numpy(),
                                 L1, L2, LO, spins, basis).reshape(len(sel), W, -1)
    got = y[ti].double().cpu().numpy().reshape(ref.shape)
    err = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
    print(f"[uvw]   rel_l2={err:.3e}", flush=True)
    assert err <= TOL, err
    # slots with l < |s| are 0
    assert np.all(got.reshape(len(sel), W, -1)[:, :, ~valid_mask(spins, LO)] == 0.0)
    return plan, (x1, x2, w), y


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (1, 1, 1, S3, 0), (2, 2, 2, S3, 0), (2, 2, 2, S3, 2), (1, 3, 3, S3, 1), (2, 1, 2, (0,), 0), (2, 2, 2, S5, 2),
    (3, 3, 3, S3, 0),
])
def test_uvw_small_ragged(L1, L2, LO, spins, basis):
    # 37 edges: one full 32-edge tile and a ragged tail; 6 (u, v) pairs, 5 output channels
    run_uvw(L1, L2, LO, spins, 37, 3, 2, 5, basis, seed=L1 + 10 * LO + basis)


@pytest.mark.parametrize("N,U,V,W", [(65, 7, 5, 130), (33, 1, 1, 1), (40, 33, 1, 64), (9, 2, 3, 257)])
def test_uvw_channel_counts(N, U, V, W):
    # pairs not a multiple of 32, output channels across several 128-channel groups and ragged
    run_uvw(2, 2, 2, S3, N, U, V, W, 0, seed=N + U + V + W)


def test_uvw_wide_blocks():
    # output degree 4: blocks of 9 components, two 8-component chunks
    run_uvw(2, 2, 4, S3, 35, 3, 2, 6, 0, seed=44)


@pytest.mark.parametrize("shape", [(1, 1, 1), (2, 2, 2), (1, 3, 3)])
@pytest.mark.parametrize("C", [16, 64, 128])
@pytest.mark.parametrize("B", [32, 128, 1024])
def test_uvw_runtime_table_shapes(shape, C, B):
    # the depthwise runtime table's shapes (App. E.2) in the fully connected mode: U = W = C
    # channels, one edge channel (V = 1), B edges; sampled edges against the oracle
    edges = np.concatenate([np.arange(min(B, 6)), np.arange(max(0, B - 6), B), [B // 2]])
    run_uvw(*shape, S3, B, C, 1, C, 2, seed=B + C, edges=edges)


def test_uvw_zero_channels_and_empty():
    plan = Plan(2, 2, 2, S3, "fp32", 0, fully_connected=True)
    x1 = torch.zeros((4, 0, 3, 9), device="cuda")
    x2 = torch.zeros((4, 1, 3, 9), device="cuda")
    w = torch.zeros((plan.n_paths, 0, 1, 3), device="cuda")
    y = torch.full((4, 3, 3, 9), float("nan"), device="cuda")
    plan.forward_fully_connected(x1, x2, w, out=y)
    torch.cuda.synchronize()
    assert float(y.abs().max()) == 0.0               # U = 0: an empty sum
    x1e = torch.zeros((0, 2, 3, 9), device="cuda")
    x2e = torch.zeros((0, 1, 3, 9), device="cuda")
    we = torch.zeros((plan.n_paths, 2, 1, 3), device="cuda")
    plan.forward_fully_connected(x1e, x2e, we)       # N = 0: no-op


def test_uvw_argument_checks():
    L = _lib.lib()
    plan = Plan(2, 2, 2, S3, "fp32", 0, fully_connected=True)
    plain = Plan(2, 2, 2, S3, "fp32", 0)
    bf = Plan(2, 2, 2, S3, "bf16", 0, fully_connected=True)
    x = torch.zeros((4, 2, 3, 9), device="cuda")
    w = torch.zeros((plan.n_paths, 2, 2, 2), device="cuda")
    y = torch.zeros((4, 2, 3, 9), device="cuda")
    args = (x.data_ptr(), x.data_ptr(), w.data_ptr(), y.data_ptr(), 4, 2, 2, 2, None)
    assert L.spingtp_forward_fully_connected(plan.handle, *args) == 0
    assert L.spingtp_forward_fully_connected(plain.handle, *args) == 2   # no entry table: unsupported
    assert L.spingtp_forward_fully_connected(bf.handle, *args) == 2      # fp32 only
    assert L.spingtp_forward_fully_connected(None, *args) == 1
    bad = list(args)
    bad[3] = y.data_ptr() + 4                                            # misaligned output
    assert L.spingtp_forward_fully_connected(plan.handle, *bad) == 1
    bad = list(args)
    bad[5] = -1
    assert L.spingtp_forward_fully_connected(plan.handle, *bad) == 1
    torch.cuda.synchronize()


def test_uvw_bitwise_deterministic():
    plan, (x1, x2, w), y = run_uvw(2, 2, 2, S3, 100, 8, 2, 40, 0, seed=7, edges=[0, 50, 99])
    y2 = plan.forward_fully_connected(x1, x2, w)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


# --- gradients (spingtp_backward_fully_connected) against the oracle's reverse mode ---

def run_uvw_backward(L1, L2, LO, spins, N, U, V, W, basis=0, seed=0, edges=None):
    """All three gradients on the device against oracle.fully_connected_vjp.  grad_x1 and
    grad_x2 are compared on the sampled edges; grad_weights sums over every edge, so with
    `edges` it is compared on a second call given only the sampled edges' rows.  Returns
    the gradients of the call over all N edges."""
    print(f"[uvw-bwd] L=({L1},{L2},{LO}) spins={spins} N={N} U={U} V={V} W={W} basis={basis}", flush=True)
    plan = Plan(L1, L2, LO, spins, "fp32", basis, fully_connected=True)
    x1 = workloads.draw(L1, N, U, 5600 + seed, "fp32", spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, V, 5700 + seed, "fp32", spins, "unit", "cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5800 + seed)
    w = torch.randn((plan.n_paths, U, V, W), generator=gen, device="cuda") / np.sqrt(max(1, U * V))
    gy = torch.randn((N, W) + tuple(plan.shape_out), generator=gen, device="cuda")
    gy.view(N, W, -1)[:, :, torch.as_tensor(~valid_mask(spins, LO), device="cuda")] = 0.0
    g1, g2, gw = plan.backward_fully_connected(x1, x2, w, gy)
    torch.cuda.synchronize()
    sel = np.arange(N) if edges is None else np.unique(np.asarray(edges))
    ti = torch.as_tensor(sel, device="cuda")
    a = x1[ti].double().cpu().numpy().reshape(len(sel), U, -1)
    b = x2[ti].double().cpu().numpy().reshape(len(sel), V, -1)
    g = gy[ti].double().cpu().numpy().reshape(len(sel), W, -1)
    r1, r2, rw = oracle.fully_connected_vjp(a, b, w.double().cpu().numpy(), g, L1, L2, LO, spins, basis)
    gw_all = gw
    if edges is not None:
        # grad_weights of the sampled edges alone: the same entry point on their rows
        _, _, gw = plan.backward_fully_connected(x1[ti].contiguous(), x2[ti].contiguous(), w, gy[ti].contiguous(),
                                                 need=(False, False, True))
        torch.cuda.synchronize()
    errs = []
    for got, ref, name in ((g1[ti], r1, "grad_x1"), (g2[ti], r2, "grad_x2"), (gw, rw, "grad_w")):
        got = got.double().cpu().numpy().reshape(ref.shape)
        err = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
        errs.append(err)
        print(f"[uvw-bwd]   {name} rel_l2={err:.3e}", flush=True)
        assert err <= TOL, (name, err)
    # slots with l < |s| of the input gradients are 0
    assert np.all(g1[ti].cpu().numpy().reshape(len(sel), U, -1)[:, :, ~valid_mask(spins, L1)] == 0.0)
    assert np.all(g2[ti].cpu().numpy().reshape(len(sel), V, -1)[:, :, ~valid_mask(spins, L2)] == 0.0)
    return plan, (x1, x2, w, gy), (g1, g2, gw_all)


@pytest.mark.parametrize("L1,L2,LO,spins,basis", [
    (1, 1, 1, S3, 0), (2, 2, 2, S3, 0), (2, 2, 2, S3, 2), (1, 3, 3, S3, 1), (2, 1, 2, (0,), 0), (2, 2, 2, S5, 2),
    (3, 3, 3, S3, 0), (2, 2, 4, S3, 0), (3, 1, 2, S3, 0),
])
def test_uvw_backward_small_ragged(L1, L2, LO, spins, basis):
    # 37 edges (a full 32-edge tile and a ragged tail), 6 (u, v) pairs, 5 output channels;
    # mixed degrees give the three roles different block widths
    run_uvw_backward(L1, L2, LO, spins, 37, 3, 2, 5, basis, seed=L1 + 10 * LO + basis)


@pytest.mark.parametrize("N,U,V,W", [(65, 7, 5, 130), (33, 1, 1, 1), (40, 33, 1, 64), (9, 2, 3, 257),
                                     (70, 130, 1, 3)])
def test_uvw_backward_channel_counts(N, U, V, W):
    # pair counts (v w, u w, u v) across 32-pair blocks, channel counts across 128-channel groups
    run_uvw_backward(2, 2, 2, S3, N, U, V, W, 0, seed=N + U + V + W)


@pytest.mark.parametrize("shape,C,B", [((1, 3, 3), 64, 128), ((2, 2, 2), 128, 1024)])
def test_uvw_backward_runtime_table_shapes(shape, C, B):
    # App. E.2 shapes: U = W = C, V = 1; sampled edges
    edges = np.concatenate([np.arange(min(B, 5)), np.arange(max(0, B - 5), B), [B // 2]])
    run_uvw_backward(*shape, S3, B, C, 1, C, 0, seed=B + C, edges=edges)


def test_uvw_backward_subsets_and_empty():
    plan, (x1, x2, w, gy), (g1, g2, gw) = run_uvw_backward(2, 2, 2, S3, 20, 4, 2, 6, 0, seed=3)
    # each gradient alone equals the one from the joint call
    for need, ref in (((True, False, False), g1), ((False, True, False), g2), ((False, False, True), gw)):
        got = plan.backward_fully_connected(x1, x2, w, gy, need=need)
        torch.cuda.synchronize()
        i = need.index(True)
        assert torch.equal(got[i], ref) and all(got[k] is None for k in range(3) if k != i)
    # N = 0: grad_weights is 0
    x1e = torch.zeros((0, 4, 3, 9), device="cuda")
    x2e = torch.zeros((0, 2, 3, 9), device="cuda")
    gye = torch.zeros((0, 6, 3, 9), device="cuda")
    _, _, gwe = plan.backward_fully_connected(x1e, x2e, w, gye)
    torch.cuda.synchronize()
    assert gwe.shape == w.shape and float(gwe.abs().max()) == 0.0
    # V = 0: the products are empty sums, grad_x1 is 0
    x2z = torch.zeros((20, 0, 3, 9), device="cuda")
    wz = torch.zeros((plan.n_paths, 4, 0, 6), device="cuda")
    g1z, _, _ = plan.backward_fully_connected(x1, x2z, wz, gy)
    torch.cuda.synchronize()
    assert float(g1z.abs().max()) == 0.0


def test_uvw_backward_argument_checks():
    L = _lib.lib()
    plan = Plan(2, 2, 2, S3, "fp32", 0, fully_connected=True)
    plain = Plan(2, 2, 2, S3, "fp32", 0)
    x = torch.zeros((4, 2, 3, 9), device="cuda")
    w = torch.zeros((plan.n_paths, 2, 2, 2), device="cuda")
    gy = torch.zeros((4, 2, 3, 9), device="cuda")
    g1 = torch.zeros_like(x)
    g2 = torch.zeros_like(x)
    gw = torch.zeros_like(w)
    args = [x.data_ptr(), x.data_ptr(), w.data_ptr(), gy.data_ptr(), g1.data_ptr(), g2.data_ptr(), gw.data_ptr(),
            4, 2, 2, 2, None]
    assert L.spingtp_backward_fully_connected(plan.handle, *args) == 0
    assert L.spingtp_backward_fully_connected(plain.handle, *args) == 2  # no entry tables: unsupported
    assert L.spingtp_backward_fully_connected(None, *args) == 1
    for i, bad in ((4, g1.data_ptr() + 4), (3, gy.data_ptr() + 8), (3, None), (8, -1)):
        a = list(args)
        a[i] = bad
        assert L.spingtp_backward_fully_connected(plan.handle, *a) == 1, i
    a = list(args)
    a[4] = a[5] = a[6] = None                                            # nothing requested: no-op
    assert L.spingtp_backward_fully_connected(plan.handle, *a) == 0
    torch.cuda.synchronize()


def test_uvw_backward_bitwise_deterministic():
    plan, (x1, x2, w, gy), (g1, g2, gw) = run_uvw_backward(2, 2, 2, S3, 100, 8, 2, 40, 0, seed=7,
                                                           edges=[0, 50, 99])
    h1, h2, hw = plan.backward_fully_connected(x1, x2, w, gy)
    torch.cuda.synchronize()
    assert torch.equal(g1, h1) and torch.equal(g2, h2) and torch.equal(gw, hw)
