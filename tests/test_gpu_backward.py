"""GPU parity of spingtp_backward against the oracle's reverse-mode derivative.

The oracle's vjp is the chain rule written out on the definition (pinned in
test_oracle_vjp.py).  Bars as for the forward: relative L2 1e-5 in fp32, 2e-2 in
bf16, 1e-6 for the matrix-core kernel (family 4) in fp32.  The oracle sees the
dtype-rounded inputs read back from the device.
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
TOL = {"fp32": 1e-5, "bf16": 2e-2}


def rel_l2(y, ref):
    return float(np.linalg.norm(y - ref) / max(np.linalg.norm(ref), 1e-300))


def draw3(L, spins, N, C, dtype, seed):
    x1 = workloads.draw(L, N, C, 600 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L, N, C, 700 + seed, dtype, spins, "unit", "cuda")
    g = workloads.draw(L, N, C, 800 + seed, dtype, spins, "unit", "cuda")
    return x1, x2, g


def run_backward(L, spins, N, C, dtype="fp32", basis=0, seed=0):
    print(f"[backward] L={L} spins={spins} N={N} C={C} {dtype} basis={basis}", flush=True)
    x1, x2, g = draw3(L, spins, N, C, dtype, seed)
    plan = Plan(L, L, L, spins, dtype, basis)
    gx1, gx2 = plan.backward(x1, x2, g)
    torch.cuda.synchronize()
    U = N * C
    a, b, c = (t.view(U, -1).double().cpu().numpy() for t in (x1, x2, g))
    r1, r2 = oracle.RealGauntTensor(L, L, L, spins, basis).vjp(a, b, c)
    e1 = rel_l2(gx1.view(U, -1).double().cpu().numpy(), r1)
    e2 = rel_l2(gx2.view(U, -1).double().cpu().numpy(), r2)
    fam = plan.kernel_info()["family"]
    print(f"[backward]   rel_l2 {e1:.3e} {e2:.3e} family={fam}", flush=True)
    bar = 1e-6 if (fam == 4 and dtype == "fp32") else TOL[dtype]
    assert e1 <= bar and e2 <= bar, (e1, e2)
    return plan, (x1, x2, g), (gx1, gx2)


@pytest.mark.parametrize("L", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("basis", [0, 1, 2])
def test_backward_matches_oracle(L, basis):
    run_backward(L, S3, 37, 3, "fp32", basis, seed=L + 10 * basis)


@pytest.mark.parametrize("L,N,C", [(8, 9, 3), (9, 7, 5), (12, 5, 2), (14, 3, 13), (16, 4, 9)])
def test_backward_large_degree(L, N, C):
    # the matrix-core kernel (L = 8, two step-(B) K blocks) and the large-degree kernel
    # (L = 9: rows held in registers, two rounds; L = 12: a split last round; L = 14, 16:
    # staging loads per round, L = 16 with a one-node last round split over the waves)
    run_backward(L, S3, N, C, "fp32", 0, seed=L)


@pytest.mark.parametrize("L,dtype", [(7, "fp32"), (8, "fp32"), (4, "bf16"), (6, "bf16"), (12, "fp32"),
                                     (16, "fp32")])
def test_backward_parity_basis(L, dtype):
    run_backward(L, S3, 17, 3, dtype, 2, seed=90 + L)


@pytest.mark.parametrize("L", [0, 3, 6])
def test_backward_scalar_spin(L):
    run_backward(L, (0,), 29, 5, "fp32", 0, seed=3 + L)


@pytest.mark.parametrize("L", [4, 6, 12, 16])
def test_backward_bf16(L):
    run_backward(L, S3, 41, 4, "bf16", 0, seed=20 + L)


def test_backward_ragged_many_tiles():
    # several 64-unit tiles with a ragged tail on the matrix-core kernel
    run_backward(6, S3, 521, 3, "fp32", 0, seed=5)


def test_backward_bilinear_identity():
    # oracle-free: sum g . y = sum gx1 . x1 = sum gx2 . x2 for the same device data
    x1, x2, g = draw3(5, S3, 64, 8, "fp32", 9)
    plan = Plan(5, 5, 5, S3, "fp32")
    y = plan.forward(x1, x2)
    gx1, gx2 = plan.backward(x1, x2, g)
    e = float((g.double() * y.double()).sum())
    a = float((gx1.double() * x1.double()).sum())
    b = float((gx2.double() * x2.double()).sum())
    assert abs(a - e) <= 1e-5 * abs(e) and abs(b - e) <= 1e-5 * abs(e), (e, a, b)


def test_backward_one_side_and_argument_rules():
    L = 3
    x1, x2, g = draw3(L, S3, 16, 4, "fp32", 2)
    plan = Plan(L, L, L, S3, "fp32", 0)
    full1, full2 = plan.backward(x1, x2, g)
    only1, none2 = plan.backward(x1, x2, g, need_x2=False)
    none1, only2 = plan.backward(x1, x2, g, need_x1=False)
    torch.cuda.synchronize()
    assert none1 is None and none2 is None
    assert torch.equal(only1, full1) and torch.equal(only2, full2)
    lib = _lib.lib()
    gx = torch.empty_like(x1)
    assert lib.spingtp_backward(plan.handle, x1.data_ptr(), x2.data_ptr(), None, gx.data_ptr(), None, 16, 4,
                                None) == 1  # grad_out missing
    assert lib.spingtp_backward(plan.handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(), gx.data_ptr() + 4, None,
                                16, 4, None) == 1  # misaligned output
    assert lib.spingtp_backward(plan.handle, None, None, None, None, None, 0, 4, None) == 0  # no units
    assert lib.spingtp_backward(plan.handle, None, None, None, None, None, 16, 4, None) == 0  # nothing asked
    assert lib.spingtp_backward(plan.handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(), gx.data_ptr(), None,
                                16, 4, None) == 0
    torch.cuda.synchronize()
    assert torch.equal(gx, full1)
    # with the paired basis (J = identity) the backward is the forward on (grad_out, x2)
    paired = Plan(L, L, L, S3, "fp32", 1)
    p1, _ = paired.backward(x1, x2, g, need_x2=False)
    assert torch.equal(p1, paired.forward(g, x2))
    # mixed degrees: the gradients run on the direct kernel (their numerics: test_gpu_direct.py)
    mixed = Plan(1, 3, 3, S3, "fp32")
    assert lib.spingtp_backward(mixed.handle, None, None, None, None, None, 4, 4, None) == 0  # nothing asked
    m1 = torch.zeros((2, 1, 3, 4), device="cuda")
    m2, mg = torch.zeros((2, 1, 3, 16), device="cuda"), torch.zeros((2, 1, 3, 16), device="cuda")
    assert lib.spingtp_backward(mixed.handle, m1.data_ptr(), m2.data_ptr(), None, m1.data_ptr(), None, 2, 1,
                                None) == 1  # grad_out missing
    g1, g2 = mixed.backward(m1, m2, mg)
    torch.cuda.synchronize()
    assert not g1.any() and not g2.any()


def test_backward_invalid_slots():
    # l < |s| slots of the inputs hold NaN / 1e30: the gradients ignore them and write 0 there
    L = 4
    x1, x2, g = draw3(L, S3, 23, 3, "fp32", 4)
    inv = torch.as_tensor(~valid_mask(S3, L), device="cuda").view(3, -1)
    ref1, ref2 = Plan(L, L, L, S3, "fp32").backward(x1, x2, g)
    for t, v in ((x1, float("nan")), (x2, 1e30), (g, float("nan"))):
        t[:, :, inv] = v
    gx1, gx2 = Plan(L, L, L, S3, "fp32").backward(x1, x2, g)
    torch.cuda.synchronize()
    assert (gx1[:, :, inv] == 0).all() and (gx2[:, :, inv] == 0).all()
    assert torch.equal(gx1, ref1) and torch.equal(gx2, ref2)


def test_backward_full_size_organic_sampled():
    # the benchmark's L = 6 workload at full size (12.8 M units), sampled against the oracle
    x1, x2, meta = workloads.make_pair("organic", dtype="fp32", device="cuda")
    U = meta["N"] * meta["C"]
    g = workloads.draw(6, meta["N"], meta["C"], 3003, "fp32", S3, "unit", "cuda")
    plan = Plan(6, 6, 6, S3, "fp32")
    gx1, gx2 = plan.backward(x1, x2, g)
    torch.cuda.synchronize()
    rng = np.random.default_rng(17)
    idx = np.unique(np.concatenate([np.arange(512), np.arange(U - 512, U), rng.integers(0, U, 4096)]))
    ti = torch.as_tensor(idx, device="cuda")
    a, b, c = (t.view(U, -1)[ti].double().cpu().numpy() for t in (x1, x2, g))
    r1, r2 = oracle.RealGauntTensor(6, 6, 6, S3, 0).vjp(a, b, c)
    e1 = rel_l2(gx1.view(U, -1)[ti].double().cpu().numpy(), r1)
    e2 = rel_l2(gx2.view(U, -1)[ti].double().cpu().numpy(), r2)
    print(f"[backward] organic full size: rel_l2 {e1:.3e} {e2:.3e}", flush=True)
    assert e1 <= 1e-6 and e2 <= 1e-6


# ---------------------------------------------------------------------------
# spingtp_backward_v1: x2 shared by the channels of an edge
# ---------------------------------------------------------------------------

def run_backward_v1(L, spins, N, C, dtype="fp32", basis=0, seed=0, fourier=False, precontract=False):
    print(f"[backward-v1] L={L} spins={spins} N={N} C={C} {dtype} basis={basis} fourier={fourier} "
          f"precontract={precontract}", flush=True)
    x1 = workloads.draw(L, N, C, 610 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L, N, 1, 710 + seed, dtype, spins, "unit", "cuda")
    g = workloads.draw(L, N, C, 810 + seed, dtype, spins, "unit", "cuda")
    plan = Plan(L, L, L, spins, dtype, basis, v1_fourier=fourier, v1_precontract=precontract)
    gx1, gx2 = plan.backward_v1(x1, x2, g)
    torch.cuda.synchronize()
    U, n = N * C, len(spins) * (L + 1) ** 2
    a = x1.view(U, n).double().cpu().numpy()
    b = np.repeat(x2.view(N, n).double().cpu().numpy(), C, axis=0)
    c = g.view(U, n).double().cpu().numpy()
    r1, r2 = oracle.RealGauntTensor(L, L, L, spins, basis).vjp(a, b, c)
    r2 = r2.reshape(N, C, n).sum(axis=1)
    e1 = rel_l2(gx1.view(U, n).double().cpu().numpy(), r1)
    e2 = rel_l2(gx2.view(N, n).double().cpu().numpy(), r2)
    fam = plan.kernel_info_v1()["family"]
    print(f"[backward-v1]   rel_l2 {e1:.3e} {e2:.3e} v1 family={fam}", flush=True)
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype], (e1, e2)
    return fam, (e1, e2)


@pytest.mark.parametrize("L", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("basis", [0, 1, 2])
def test_backward_v1_matches_oracle(L, basis):
    # default route: precontracted up to L = 4, Fourier at L = 5, 6
    fam, _ = run_backward_v1(L, S3, 13, 17, "fp32", basis, seed=L + 10 * basis)
    assert (fam == 5) == (L <= 4)


@pytest.mark.parametrize("L,C,fourier,precontract", [(3, 40, True, False), (4, 1, True, False),
                                                     (6, 33, False, True), (2, 130, False, False)])
def test_backward_v1_routes_and_channel_counts(L, C, fourier, precontract):
    run_backward_v1(L, S3, 7, C, "fp32", 0, seed=3 * L + C, fourier=fourier, precontract=precontract)


@pytest.mark.parametrize("L", [3, 6])
def test_backward_v1_scalar_spin_and_bf16(L):
    run_backward_v1(L, (0,), 9, 20, "fp32", 0, seed=L)
    run_backward_v1(L, S3, 9, 20, "bf16", 0, seed=L + 1)


def test_backward_v1_rules():
    L = 2
    N, C = 5, 6
    plan = Plan(L, L, L, S3, "fp32")
    x1 = workloads.draw(L, N, C, 1, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, 1, 2, "fp32", S3, "unit", "cuda")
    g = workloads.draw(L, N, C, 3, "fp32", S3, "unit", "cuda")
    full1, full2 = plan.backward_v1(x1, x2, g)
    only1, none2 = plan.backward_v1(x1, x2, g, need_x2=False)
    torch.cuda.synchronize()
    assert none2 is None and torch.equal(only1, full1)
    lib = _lib.lib()
    gx2 = torch.empty_like(x2)
    need = ctypes.c_size_t(0)
    assert lib.spingtp_backward_v1_workspace_size(plan.handle, N, C, ctypes.byref(need)) == 0
    assert need.value == N * C * 27 * 4
    ws = torch.empty(need.value, dtype=torch.uint8, device="cuda")
    args = (plan.handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(), None, gx2.data_ptr())
    assert lib.spingtp_backward_v1(*args, None, 0, N, C, None) == 1  # workspace missing
    assert lib.spingtp_backward_v1(*args, ws.data_ptr(), need.value - 1, N, C, None) == 1  # too small
    assert lib.spingtp_backward_v1(*args, ws.data_ptr(), need.value, N, C, None) == 0
    torch.cuda.synchronize()
    assert torch.equal(gx2, full2)
    # no channels: grad_x2 is the empty sum
    gx2.fill_(7.0)
    assert lib.spingtp_backward_v1(*args, None, 0, N, 0, None) == 0
    torch.cuda.synchronize()
    assert (gx2 == 0).all()
    # a shape without a Fourier kernel: its gradients run on the direct kernel, workspace [N][C][NC2]
    mixed = Plan(3, 1, 2, S3, "fp32")
    assert lib.spingtp_backward_v1_workspace_size(mixed.handle, N, C, ctypes.byref(need)) == 0
    assert need.value == N * C * 3 * 4 * 4
