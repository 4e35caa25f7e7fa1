"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bar (per element set, relative L2 over the compared units): 1e-5 in fp32 and
2e-2 in bf16.  The matrix-core kernel (family 4) with fp32 I/O is held to 1e-6
as well: its split fp16 products are fp32-like (about 2e-7 here), and an error
between the two bars means corrupted operand words, not rounding.  The oracle always sees the exact dtype-rounded inputs the GPU saw
(read back from the device).  Large workloads compare the first and last 512
units (tile tails) and a seeded random sample, at the full size and in the
launch configuration the benchmark times.
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
MATRIX_CORE_FP32_TOL = 1e-6


def check_matrix_core(plan, dtype, err):
    if plan.kernel_info()["family"] == 4 and dtype == "fp32":
        assert err <= MATRIX_CORE_FP32_TOL, f"matrix-core fp32 path off its split-precision bar: {err:.3e}"


def rel_l2(y, ref):
    return float(np.linalg.norm(y - ref) / max(np.linalg.norm(ref), 1e-300))


def run_and_compare(L1, L2, LO, spins, N, C, dtype="fp32", basis=0, seed=0, scale="unit", units=None,
                    valu_only=False):
    from oracle.spingtp import _cached_tensor
    print(f"[parity] L=({L1},{L2},{LO}) spins={spins} N={N} C={C} {dtype} basis={basis} valu_only={valu_only}",
          flush=True)
    x1 = workloads.draw(L1, N, C, 7000 + seed, dtype, spins, scale, "cuda")
    x2 = workloads.draw(L2, N, C, 8000 + seed, dtype, spins, scale, "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, valu_only=valu_only)
    if valu_only:
        assert plan.kernel_info()["family"] != 4
    y = plan.forward(x1, x2)
    torch.cuda.synchronize()
    U = N * C
    idx = np.arange(U) if units is None else units
    ti = torch.as_tensor(idx, device="cuda")
    a = x1.view(U, -1)[ti].double().cpu().numpy()
    b = x2.view(U, -1)[ti].double().cpu().numpy()
    g = y.view(U, -1)[ti].double().cpu().numpy()
    ref = _cached_tensor(L1, L2, LO, tuple(spins), basis).apply(a, b).reshape(len(idx), -1)
    err = rel_l2(g, ref)
    print(f"[parity]   rel_l2={err:.3e} family={plan.kernel_info()['family']}", flush=True)
    assert err <= TOL[dtype], err
    check_matrix_core(plan, dtype, err)
    return err


def sample_units(U, n_random, seed):
    rng = np.random.default_rng(seed)
    head = np.arange(min(512, U))
    tail = np.arange(max(0, U - 512), U)
    rnd = rng.choice(U, size=min(n_random, U), replace=False)
    return np.unique(np.concatenate([head, tail, rnd]))


@pytest.mark.parametrize("L", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("basis", [0, 1, 2])
def test_ragged_spin_shapes(L, basis):
    # 37 * 3 = 111 units: one full 64-unit tile and a ragged tail of 47
    run_and_compare(L, L, L, S3, 37, 3, "fp32", basis, seed=L)


@pytest.mark.parametrize("L", [4, 5, 6, 7, 8])
@pytest.mark.parametrize("basis", [0, 1, 2])
def test_ragged_valu_kernels(L, basis):
    # the fp32 vector-ALU kernels of the degrees that default to the matrix-core kernel
    run_and_compare(L, L, L, S3, 37, 3, "fp32", basis, seed=40 + L, valu_only=True)


@pytest.mark.parametrize("L", [4, 5, 6, 7, 8])
@pytest.mark.parametrize("N,C", [(64, 1), (65, 1), (125, 8), (4113, 1)])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_matrix_core_sizes(L, N, C, dtype):
    # one exact tile, one unit past it, several tiles with a ragged tail, many tiles
    run_and_compare(L, L, L, S3, N, C, dtype, 0, seed=50 + L + N % 7)


def _ulp_bf16(y):
    e = np.floor(np.log2(np.maximum(np.abs(y), 1e-300)))
    return np.ldexp(1.0, (e - 7).astype(int))


@pytest.mark.parametrize("L", [4, 5, 6, 7, 8])
@pytest.mark.parametrize("N,C,basis", [(37, 3, 0), (4113, 1, 0), (125, 8, 2)])
def test_matrix_core_bf16_against_reenactment(L, N, C, basis):
    """The bf16 mode of the matrix-core kernel (fp16 high parts only) against the
    CPU re-enactment of its own arithmetic from the library's operand words.

    The oracle bar for bf16 (2e-2) leaves room for a corrupted operand word, so every
    output element is also held to the re-enactment: within half a bf16 unit in the
    last place (the output's own rounding) plus 2^-10 of the unit's largest output.
    Two faithful evaluations drift apart by at most about 3e-4 of that scale (fp32
    versus float64 step-(A) results move some fp16 roundings of step (B) by one
    unit); a stale or wrong fp16 word in step (B) or (D) moves a field or spectrum
    value by a sizable fraction of itself, which this bound catches."""
    from tests.kernel_emulation import emulate_mfma_kernel
    print(f"[reenact] L={L} N={N} C={C} bf16 basis={basis}", flush=True)
    x1 = workloads.draw(L, N, C, 9100 + L, "bf16", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, C, 9200 + L, "bf16", S3, "unit", "cuda")
    plan = Plan(L, L, L, S3, "bf16", basis)
    assert plan.kernel_info()["family"] == 4
    y = plan.forward(x1, x2)
    torch.cuda.synchronize()
    U = N * C
    a = x1.view(U, -1).double().cpu().numpy()
    b = x2.view(U, -1).double().cpu().numpy()
    g = y.view(U, -1).double().cpu().numpy()
    emu = emulate_mfma_kernel(a, b, L, basis, split=1)
    scale = np.abs(emu).max(axis=1, keepdims=True)
    excess = (np.abs(g - emu) - 0.5 * _ulp_bf16(emu)) / np.maximum(scale, 1e-300)
    worst = float(excess.max())
    print(f"[reenact]   worst excess over half an ulp = {worst:.3e} of the unit scale", flush=True)
    assert worst <= 2.0 ** -10, worst


@pytest.mark.parametrize("L,basis", [(9, 0), (9, 1), (10, 0), (11, 0), (12, 0), (13, 0), (13, 1), (14, 0), (15, 0),
                                     (16, 0), (16, 1)])
def test_ragged_large_degree(L, basis):
    # 37 * 3 = 111 units: three full 32-unit tiles and a ragged tail of 15; every
    # degree, since each stages its input rows in its own chunks of degrees
    run_and_compare(L, L, L, S3, 37, 3, "fp32", basis, seed=L)


@pytest.mark.parametrize("L,basis,spins", [(9, 0, S3), (12, 0, S3), (13, 1, S3), (16, 0, S3), (12, 2, S3),
                                           (16, 2, S3), (12, 0, (0,)), (16, 0, (0,))])
def test_bf16_large_degree(L, basis, spins):
    # bf16 I/O on the large-degree kernels (rows widened as they are staged, the tile
    # rounded to nearest even as it is stored): every staging form, both bases, spin {0}
    run_and_compare(L, L, L, spins, 37, 3, "bf16", basis, seed=300 + L + basis)


@pytest.mark.parametrize("L", [9, 16])
def test_large_degree_many_tiles(L):
    # 41 tiles of 32 units (more than one workgroup per XCD) and a ragged tail of 7;
    # the oracle on the first, a middle and the last tiles
    units = np.r_[0:40, 600:640, 1279:1319]
    run_and_compare(L, L, L, S3, 1319, 1, "fp32", 0, seed=200 + L, units=units)


@pytest.mark.parametrize("L", [0, 1, 2, 3, 4, 6, 8, 12, 16])
def test_ragged_scalar_shapes(L):
    run_and_compare(L, L, L, (0,), 29, 5, "fp32", 0, seed=10 + L)


@pytest.mark.parametrize("L1,L2,LO", [(1, 3, 3), (2, 1, 3)])
def test_mixed_degrees(L1, L2, LO):
    run_and_compare(L1, L2, LO, S3, 50, 7, "fp32", 0, seed=20 + L1)


@pytest.mark.parametrize("L", [2, 4, 6, 8])
def test_bf16_small(L):
    run_and_compare(L, L, L, S3, 45, 6, "bf16", 0, seed=30 + L)


# --- the parity-labelled basis (Sec. 3.4): kernels mix their tiles on load and store ---

@pytest.mark.parametrize("L1,L2,LO", [(1, 3, 3), (2, 1, 3)])
def test_parity_basis_mixed_degrees(L1, L2, LO):
    run_and_compare(L1, L2, LO, S3, 50, 7, "fp32", 2, seed=60 + L1)


@pytest.mark.parametrize("L", [4, 6, 8])
def test_parity_basis_bf16(L):
    run_and_compare(L, L, L, S3, 45, 6, "bf16", 2, seed=70 + L)


@pytest.mark.parametrize("L", [5, 6])
def test_parity_basis_matrix_core_many_tiles(L):
    run_and_compare(L, L, L, S3, 125, 8, "fp32", 2, seed=80 + L)


def test_parity_basis_changes_the_map():
    # the same coefficients read in the two bases give different products (the mixing is applied)
    x1 = workloads.draw(4, 9, 2, 5, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(4, 9, 2, 6, "fp32", S3, "unit", "cuda")
    y0 = Plan(4, 4, 4, S3, "fp32", 0).forward(x1, x2)
    y2 = Plan(4, 4, 4, S3, "fp32", 2).forward(x1, x2)
    assert float((y0 - y2).abs().max()) > 1e-2


@pytest.mark.parametrize("L", [9, 10, 11, 12, 13, 14, 15, 16])
def test_parity_basis_large_degree(L):
    # the large-degree kernels mix the input rows as step (A) reads them from the staged
    # chunks; every degree, since these instantiations are built with their own
    # scheduling strategy
    run_and_compare(L, L, L, S3, 37, 3, "fp32", 2, seed=100 + L)


def test_parity_basis_scalar_spin_large_degree():
    # no |s| = 1 sector: the paper-basis kernel serves the parity plan
    run_and_compare(9, 9, 9, (0,), 29, 5, "fp32", 2, seed=109)


def test_small_workload_all_units():
    x1, x2, m = workloads.make_pair("small", device="cuda")
    plan = Plan(m["L"], m["L"], m["L"], S3, "fp32")
    y = plan.forward(x1, x2)
    torch.cuda.synchronize()
    ref = oracle.spingtp(x1.double().cpu().numpy(), x2.double().cpu().numpy(), m["L"], m["L"], m["L"], S3)
    assert rel_l2(y.double().cpu().numpy(), ref) <= 1e-5


@pytest.mark.parametrize("name,dtype,L", [("molecule", "fp32", None), ("organic", "fp32", None),
                                          ("organic", "bf16", None), ("catalyst", "bf16", None),
                                          ("sweep", "fp32", 2), ("sweep", "fp32", 4), ("sweep", "fp32", 8),
                                          ("sweep", "fp32", 12), ("sweep", "fp32", 16)])
def test_full_size_sampled(name, dtype, L):
    print(f"[parity] full-size {name} {dtype} L={L}", flush=True)
    x1, x2, m = workloads.make_pair(name, dtype=dtype, L=L, device="cuda")
    L, U = m["L"], m["N"] * m["C"]
    plan = Plan(L, L, L, S3, dtype)
    y = plan.forward(x1, x2)
    torch.cuda.synchronize()
    idx = sample_units(U, 8192 if L <= 8 else 1024, 99)
    ti = torch.as_tensor(idx, device="cuda")
    a = x1.view(U, -1)[ti].double().cpu().numpy()
    b = x2.view(U, -1)[ti].double().cpu().numpy()
    g = y.view(U, -1)[ti].double().cpu().numpy()
    del x1, x2, y
    torch.cuda.empty_cache()
    ref = oracle.spingtp(a, b, L, L, L, S3).reshape(len(idx), -1)
    err = rel_l2(g, ref)
    print(f"[parity]   rel_l2={err:.3e} over {len(idx)} units family={plan.kernel_info()['family']}", flush=True)
    assert err <= TOL[dtype]
    check_matrix_core(plan, dtype, err)


# Tensors of more than 2^31 fp32 elements (element offsets past the int32 range) on the
# matrix-core kernel (L = 6) and the large-degree kernel (L = 12); the last 512 units sit
# past that offset.  About 27 and 26 GB of device memory.
@pytest.mark.parametrize("L,N,C", [(6, 115_000, 128), (12, 33_600, 128)])
def test_beyond_2g_elements(L, N, C):
    U = N * C
    assert U * 3 * (L + 1) ** 2 > 2 ** 31
    print(f"[parity] beyond 2^31 elements L={L} units={U}", flush=True)
    x1, x2, m = workloads.make_pair("sweep", dtype="fp32", L=L, device="cuda", N=N, C=C)
    plan = Plan(L, L, L, S3, "fp32")
    y = plan.forward(x1, x2)
    torch.cuda.synchronize()
    idx = sample_units(U, 2048, 7)
    ti = torch.as_tensor(idx, device="cuda")
    a = x1.view(U, -1)[ti].double().cpu().numpy()
    b = x2.view(U, -1)[ti].double().cpu().numpy()
    g = y.view(U, -1)[ti].double().cpu().numpy()
    del x1, x2, y
    torch.cuda.empty_cache()
    ref = oracle.spingtp(a, b, L, L, L, S3).reshape(len(idx), -1)
    err = rel_l2(g, ref)
    tail = rel_l2(g[-512:], ref[-512:])
    print(f"[parity]   rel_l2={err:.3e} (last 512 units {tail:.3e}) family={plan.kernel_info()['family']}",
          flush=True)
    assert err <= TOL["fp32"] and tail <= TOL["fp32"]


def test_empty_is_noop():
    plan = Plan(2, 2, 2, S3, "fp32")
    x = torch.zeros((0, 4, 3, 9), device="cuda")
    out = plan.forward(x, x)
    assert out.shape == (0, 4, 3, 9)
    L = _lib.lib()
    assert L.spingtp_forward(plan.handle, None, None, None, 0, 5, None) == 0
    assert L.spingtp_forward(plan.handle, None, None, None, 7, 0, None) == 0


def test_invalid_arguments():
    plan = Plan(2, 2, 2, S3, "fp32")
    L = _lib.lib()
    x = torch.zeros((4, 2, 3, 9), device="cuda")
    y = torch.zeros_like(x)
    p = x.data_ptr()
    assert L.spingtp_forward(plan.handle, None, p, y.data_ptr(), 4, 2, None) == 1
    assert L.spingtp_forward(plan.handle, p + 4, p, y.data_ptr(), 4, 2, None) == 1  # misaligned
    assert L.spingtp_forward(plan.handle, p, p, y.data_ptr(), -1, 2, None) == 1
    assert L.spingtp_forward(None, p, p, y.data_ptr(), 4, 2, None) == 1
    with pytest.raises(SpinGTPError):
        Plan(2, 2, 2, (-2, 0, 2), "fp32")  # valid spin set, not built
    with pytest.raises(SpinGTPError):
        Plan(3, 3, 7, S3, "fp32")


@pytest.mark.parametrize("L", [3, 6])
def test_nan_poisoned_output_and_invalid_slots(L):
    N, C = 33, 5
    x1 = workloads.draw(L, N, C, 11, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, C, 12, "fp32", S3, "unit", "cuda")
    plan = Plan(L, L, L, S3, "fp32")
    ref = plan.forward(x1, x2).clone()
    inv = torch.as_tensor(~valid_mask(S3, L), device="cuda").view(3, -1)
    g1, g2 = x1.clone(), x2.clone()
    g1[:, :, inv] = float("nan")
    g2[:, :, inv] = 1e30
    out = torch.full_like(ref, float("nan"))
    plan.forward(g1, g2, out=out)
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()
    torch.testing.assert_close(out, ref, rtol=1e-6, atol=1e-6)
    assert (out[:, :, inv] == 0).all()


def test_gpu_invariants():
    """Oracle-free checks on the GPU path: constant function and commutativity."""
    L, N, C = 4, 20, 6
    x1 = workloads.draw(L, N, C, 21, "fp32", S3, "unit", "cuda")
    x2 = torch.zeros_like(x1)
    x2[:, :, 1, 0] = 2.5  # s = 0, l = 0
    plan = Plan(L, L, L, S3, "fp32")
    y = plan.forward(x1, x2)
    torch.testing.assert_close(y, x1 * (2.5 / np.sqrt(4 * np.pi)), rtol=2e-6, atol=2e-6)
    x3 = workloads.draw(L, N, C, 22, "fp32", S3, "unit", "cuda")
    torch.testing.assert_close(plan.forward(x1, x3), plan.forward(x3, x1), rtol=1e-5, atol=1e-6)


def test_plan_reuse_across_streams():
    L, N, C = 6, 300, 8
    x1 = workloads.draw(L, N, C, 31, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, C, 32, "fp32", S3, "unit", "cuda")
    plan = Plan(L, L, L, S3, "fp32")
    ref = plan.forward(x1, x2)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        a = plan.forward(x1, x2)
    with torch.cuda.stream(s2):
        b = plan.forward(x1, x2)
    torch.cuda.synchronize()
    torch.testing.assert_close(a, ref, rtol=1e-6, atol=1e-6)
    torch.testing.assert_close(b, ref, rtol=1e-6, atol=1e-6)


def test_bitwise_deterministic():
    """The node sums run in a fixed order (no atomics): repeated launches agree bit for bit."""
    L, N, C = 6, 700, 16
    x1 = workloads.draw(L, N, C, 41, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, C, 42, "fp32", S3, "unit", "cuda")
    plan = Plan(L, L, L, S3, "fp32")
    a = plan.forward(x1, x2)
    b = plan.forward(x1, x2)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# --- edge multiplicity one: x2 shared by the channels of an edge (spingtp_forward_v1) ---

def run_v1(L1, L2, LO, spins, N, C, dtype="fp32", fourier=False, seed=0, precontract=False, basis=0):
    from oracle.spingtp import _cached_tensor
    print(f"[parity-v1] L=({L1},{L2},{LO}) N={N} C={C} {dtype} fourier={fourier} basis={basis}", flush=True)
    x1 = workloads.draw(L1, N, C, 9000 + seed, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, 1, 9500 + seed, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis, v1_fourier=fourier, v1_precontract=precontract)
    fam = plan.kernel_info_v1()["family"]
    y = plan.forward_v1(x1, x2)
    torch.cuda.synchronize()
    U = N * C
    a = x1.view(U, -1).double().cpu().numpy()
    b = np.repeat(x2.view(N, -1).double().cpu().numpy(), C, axis=0)
    ref = _cached_tensor(L1, L2, LO, tuple(spins), basis).apply(a, b).reshape(U, -1)
    err = rel_l2(y.view(U, -1).double().cpu().numpy(), ref)
    print(f"[parity-v1]   rel_l2={err:.3e} family={fam}", flush=True)
    assert err <= TOL[dtype], err
    check_matrix_core(Plan(L1, L2, LO, spins, dtype, basis), dtype, err) if (fourier and fam == 4) else None
    if fam == 5 and dtype == "fp32":
        # fp32 products on the matrix cores and fp32 sums: well inside the fp32 bar
        assert err <= MATRIX_CORE_FP32_TOL, err
    return fam, err


@pytest.mark.parametrize("shape", [(1, 1, 1), (2, 2, 2), (1, 3, 3)])
@pytest.mark.parametrize("C", [16, 64, 128])
@pytest.mark.parametrize("fourier", [False, True])
def test_v1_table_shapes(shape, C, fourier):
    # the depthwise V = 1 shapes of the paper's tensor-product runtime table (App. E)
    fam, _ = run_v1(*shape, S3, 37, C, "fp32", fourier, seed=sum(shape) + C)
    assert (fam == 5) == (not fourier)


@pytest.mark.parametrize("shape,C", [((2, 2, 2), 1), ((2, 2, 2), 3), ((2, 2, 2), 65), ((4, 4, 4), 65),
                                     ((3, 1, 2), 9), ((0, 0, 0), 5), ((4, 4, 4), 129), ((4, 2, 3), 17),
                                     ((2, 4, 1), 40), ((4, 1, 2), 24), ((1, 3, 0), 8), ((3, 3, 3), 200)])
def test_v1_channel_counts(shape, C):
    # one channel, a ragged 16-channel tile, several tiles per wave, mixed degrees (some with one degree
    # above the sum of the other two), L = 0
    fam, _ = run_v1(*shape, S3, 11, C, "fp32", False, seed=3 * C)
    assert fam == 5


@pytest.mark.parametrize("shape", [(2, 2, 2), (4, 4, 4), (6, 6, 6)])
@pytest.mark.parametrize("fourier", [False, True])
def test_v1_bf16(shape, fourier):
    run_v1(*shape, S3, 23, 48, "bf16", fourier, seed=7)


@pytest.mark.parametrize("L,C", [(7, 5), (8, 5), (9, 4), (12, 3), (16, 3)])
def test_v1_fourier_route_large_degree(L, C):
    # beyond the precontracted kernel's size the v1 entry runs the forward kernel with x2 per edge
    fam, _ = run_v1(L, L, L, S3, 19, C, "fp32", False, seed=L)
    assert fam != 5


@pytest.mark.parametrize("shape,C,fourier", [
    ((5, 5, 5), 7, False), ((5, 5, 5), 130, False), ((6, 6, 6), 7, False), ((6, 6, 6), 128, False),
    ((1, 6, 6), 33, False), ((6, 2, 5), 17, False), ((6, 6, 4), 40, False), ((5, 5, 5), 130, True),
    ((6, 6, 6), 128, True)])
def test_v1_degree_5_and_6(shape, C, fourier):
    # the large precontracted instantiations (one resident workgroup per CU), forced where the Fourier
    # route is the default; mixed degrees here have no Fourier kernel, so this is their only route
    fam, _ = run_v1(*shape, S3, 21, C, "fp32", fourier, seed=C + sum(shape), precontract=not fourier)
    assert (fam == 5) == (not fourier)


@pytest.mark.parametrize("shape,family", [((4, 4, 4), 5), ((1, 3, 3), 5), ((5, 5, 5), 4), ((6, 6, 6), 4),
                                          ((6, 2, 5), 5)])
def test_v1_default_route(shape, family):
    # precontracted for rows <= 75 and where no Fourier kernel exists, the Fourier route beyond
    assert Plan(*shape, S3, "fp32").kernel_info_v1()["family"] == family


@pytest.mark.parametrize("shape,C,fourier,precontract", [
    ((2, 2, 2), 16, False, False), ((4, 4, 4), 65, False, False), ((5, 5, 5), 130, False, False),
    ((6, 6, 6), 128, False, True), ((6, 2, 5), 17, False, False), ((6, 6, 6), 40, False, False),
    ((3, 3, 3), 33, True, False), ((8, 8, 8), 5, False, False)])
def test_v1_parity_basis(shape, C, fourier, precontract):
    # the precontracted tables hold the parity-basis tensor itself; the Fourier route mixes tiles
    run_v1(*shape, S3, 19, C, "fp32", fourier, seed=C, precontract=precontract, basis=2)


@pytest.mark.parametrize("shape,C", [((3, 3, 3), 17), ((7, 7, 7), 33), ((5, 2, 6), 16)])
def test_v1_scalar_spins(shape, C):
    fam, _ = run_v1(*shape, (0,), 29, C, "fp32", False, seed=1)
    assert fam == 5


def test_v1_fourier_equals_forward_with_repeated_x2():
    """The Fourier route of forward_v1 reads x2 per edge; with x2 repeated over the
    channels, forward runs the same kernel on the same values: bitwise equal."""
    L, N, C = 6, 13, 9
    x1 = workloads.draw(L, N, C, 61, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, 1, 62, "fp32", S3, "unit", "cuda")
    plan = Plan(L, L, L, S3, "fp32", v1_fourier=True)
    a = plan.forward_v1(x1, x2)
    b = plan.forward(x1, x2.expand(N, C, *x2.shape[2:]).contiguous())
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_v1_invalid_slots_and_poisoned_output():
    L, N, C = 3, 17, 70
    x1 = workloads.draw(L, N, C, 71, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L, N, 1, 72, "fp32", S3, "unit", "cuda")
    plan = Plan(L, L, L, S3, "fp32")
    assert plan.kernel_info_v1()["family"] == 5
    ref = plan.forward_v1(x1, x2).clone()
    inv = torch.as_tensor(~valid_mask(S3, L), device="cuda").view(3, -1)
    g1, g2 = x1.clone(), x2.clone()
    g1[:, :, inv] = float("nan")
    g2[:, :, inv] = 1e30
    out = torch.full_like(ref, float("nan"))
    plan.forward_v1(g1, g2, out=out)
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()
    assert torch.equal(out, ref)
    assert (out[:, :, inv] == 0).all()


def test_v1_argument_checks():
    plan = Plan(2, 2, 2, S3, "fp32")
    L = _lib.lib()
    x = torch.zeros((4, 2, 3, 9), device="cuda")
    x2 = torch.zeros((4, 1, 3, 9), device="cuda")
    y = torch.zeros_like(x)
    assert L.spingtp_forward_v1(plan.handle, x.data_ptr(), None, y.data_ptr(), 4, 2, None) == 1
    assert L.spingtp_forward_v1(plan.handle, x.data_ptr() + 4, x2.data_ptr(), y.data_ptr(), 4, 2, None) == 1
    assert L.spingtp_forward_v1(plan.handle, None, None, None, 0, 2, None) == 0
    with pytest.raises(ValueError):
        plan.forward_v1(x, x)  # x2 must be [N, 1, ...]
    mixed = Plan(3, 1, 2, S3, "fp32")  # no Fourier-route kernel: forward on the direct kernel
    assert mixed.kernel_info_v1()["family"] == 5 and mixed.kernel_info()["family"] == 6
    a = torch.zeros((2, 3, 3, 16), device="cuda")
    b = torch.zeros((2, 3, 3, 4), device="cuda")
    y = mixed.forward(a, b)
    torch.cuda.synchronize()
    assert y.shape == (2, 3, 3, 9) and not y.any()


# --- mixed degrees beyond the direct kernel's rows: the large-degree kernel of the
# largest degree, inputs padded with zeros as it stages them, the product truncated ---

# the padded instantiations of every degree 9..16 (each its own kernel), both bases, spin {0}, bf16
@pytest.mark.parametrize("L1,L2,LO,spins,basis,dtype", [
    (9, 3, 10, S3, 0, "fp32"), (12, 12, 6, S3, 0, "fp32"), (16, 2, 16, S3, 0, "fp32"), (4, 12, 16, S3, 2, "fp32"),
    (16, 15, 14, (0,), 0, "fp32"), (12, 5, 9, S3, 0, "bf16"), (3, 10, 12, S3, 1, "fp32"),
    (9, 9, 4, S3, 2, "bf16"), (11, 4, 9, S3, 0, "fp32"), (5, 13, 13, S3, 2, "fp32"), (14, 3, 12, S3, 1, "bf16"),
    (15, 6, 15, (0,), 0, "fp32"), (13, 2, 15, S3, 0, "fp32"),
])
def test_mixed_large_degrees(L1, L2, LO, spins, basis, dtype):
    run_and_compare(L1, L2, LO, spins, 37, 3, dtype, basis, seed=400 + L1 + L2 + LO)
    assert Plan(L1, L2, LO, spins, dtype, basis).kernel_info()["family"] == 3


@pytest.mark.parametrize("L1,L2,LO,dtype", [(13, 5, 11, "fp32"), (4, 16, 9, "bf16")])
def test_mixed_large_degrees_many_tiles(L1, L2, LO, dtype):
    # 20,000 units (625 tiles of 32), x1 and x2 rows of different lengths; sampled
    N, C = 2000, 10
    U = N * C
    print(f"[parity] mixed many tiles L=({L1},{L2},{LO}) {dtype} units={U}", flush=True)
    x1 = workloads.draw(L1, N, C, 610 + L1, dtype, S3, "unit", "cuda")
    x2 = workloads.draw(L2, N, C, 620 + L2, dtype, S3, "unit", "cuda")
    plan = Plan(L1, L2, LO, S3, dtype)
    assert plan.kernel_info()["family"] == 3
    y = plan.forward(x1, x2)
    torch.cuda.synchronize()
    idx = sample_units(U, 1024, 5)
    ti = torch.as_tensor(idx, device="cuda")
    a = x1.view(U, -1)[ti].double().cpu().numpy()
    b = x2.view(U, -1)[ti].double().cpu().numpy()
    g = y.view(U, -1)[ti].double().cpu().numpy()
    ref = oracle.spingtp(a, b, L1, L2, LO, S3).reshape(len(idx), -1)
    err = rel_l2(g, ref)
    print(f"[parity]   rel_l2={err:.3e} over {len(idx)} units", flush=True)
    assert err <= TOL[dtype]


@pytest.mark.parametrize("L1,L2,LO,spins,basis,dtype", [
    (9, 3, 10, S3, 0, "fp32"), (13, 5, 11, S3, 2, "bf16"), (6, 15, 15, (0,), 0, "fp32"), (14, 4, 10, S3, 1, "fp32"),
])
def test_mixed_large_degrees_v1(L1, L2, LO, spins, basis, dtype):
    # the shared-x2 entry on the padded route
    fam, _ = run_v1(L1, L2, LO, spins, 13, 5, dtype, seed=11 + L1, basis=basis)
    assert fam == 3


@pytest.mark.parametrize("L1,L2,LO,spins,basis,dtype", [
    (9, 3, 10, S3, 0, "fp32"), (4, 12, 16, S3, 2, "fp32"), (12, 12, 6, S3, 1, "fp32"),
    (16, 15, 14, (0,), 0, "fp32"), (12, 5, 9, S3, 0, "bf16"),
    (9, 4, 9, S3, 1, "fp32"), (11, 11, 5, S3, 0, "fp32"), (13, 8, 14, S3, 2, "bf16"), (15, 6, 15, (0,), 0, "fp32"),
])
def test_mixed_large_degrees_backward(L1, L2, LO, spins, basis, dtype):
    # the gradients: the degree-L ones of the padded functions (grad_out, x2 -> grad_x1
    # and grad_out, x1 -> grad_x2 on the padded kernel), truncated
    print(f"[mixed-bwd] L=({L1},{L2},{LO}) spins={spins} basis={basis} {dtype}", flush=True)
    N, C = 11, 3
    x1 = workloads.draw(L1, N, C, 500 + L1, dtype, spins, "unit", "cuda")
    x2 = workloads.draw(L2, N, C, 510 + L2, dtype, spins, "unit", "cuda")
    g = workloads.draw(LO, N, C, 520 + LO, dtype, spins, "unit", "cuda")
    plan = Plan(L1, L2, LO, spins, dtype, basis)
    gx1, gx2 = plan.backward(x1, x2, g)
    torch.cuda.synchronize()
    U = N * C
    a, b, c = (t.view(U, -1).double().cpu().numpy() for t in (x1, x2, g))
    r1, r2 = oracle.RealGauntTensor(L1, L2, LO, spins, basis).vjp(a, b, c)
    e1 = rel_l2(gx1.view(U, -1).double().cpu().numpy(), r1)
    e2 = rel_l2(gx2.view(U, -1).double().cpu().numpy(), r2)
    print(f"[mixed-bwd]   rel_l2 {e1:.3e} {e2:.3e}", flush=True)
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype], (e1, e2)


def test_mixed_large_degrees_backward_v1():
    # x2 shared by the channels of an edge: grad_x2 summed over them
    L1, L2, LO, N, C = 10, 4, 12, 7, 6
    x1 = workloads.draw(L1, N, C, 530, "fp32", S3, "unit", "cuda")
    x2 = workloads.draw(L2, N, 1, 531, "fp32", S3, "unit", "cuda")
    g = workloads.draw(LO, N, C, 532, "fp32", S3, "unit", "cuda")
    plan = Plan(L1, L2, LO, S3, "fp32")
    gx1, gx2 = plan.backward_v1(x1, x2, g)
    torch.cuda.synchronize()
    U = N * C
    a = x1.view(U, -1).double().cpu().numpy()
    b = np.repeat(x2.view(N, -1).double().cpu().numpy(), C, axis=0)
    c = g.view(U, -1).double().cpu().numpy()
    r1, r2 = oracle.RealGauntTensor(L1, L2, LO, S3, 0).vjp(a, b, c)
    r2 = r2.reshape(N, C, -1).sum(axis=1)
    e1 = rel_l2(gx1.view(U, -1).double().cpu().numpy(), r1)
    e2 = rel_l2(gx2.view(N, -1).double().cpu().numpy(), r2)
    print(f"[mixed-bwd-v1]   rel_l2 {e1:.3e} {e2:.3e}", flush=True)
    assert e1 <= TOL["fp32"] and e2 <= TOL["fp32"], (e1, e2)
