"""spingtp_backward_v1_noalloc against spingtp_backward_v1 (GPU, through the C ABI).

The no-allocation entry point runs the same kernels in the same order as
spingtp_backward_v1, with the grad_x2 staging rows in the library's fixed device
scratch instead of a caller workspace, so its gradients must equal those of
spingtp_backward_v1 bit for bit.  Two calls in a row, the second smaller, show
that nothing of the first call's scratch contents leaks into the second.
"""

import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

from paper_2607_01408_amd import Plan, workloads  # noqa: E402
from paper_2607_01408_amd import _lib  # noqa: E402

S3 = (-1, 0, 1)
SCRATCH_BYTES = 64 << 20
TOO_LARGE = 6


def _inputs(L, N, C, dtype, seed):
    x1 = workloads.draw(L, N, C, 4400 + seed, dtype, S3, "unit", "cuda")
    x2 = workloads.draw(L, N, 1, 4500 + seed, dtype, S3, "unit", "cuda")
    g = workloads.draw(L, N, C, 4600 + seed, dtype, S3, "unit", "cuda")
    return x1, x2, g


def _noalloc(plan, x1, x2, g):
    """Direct C-ABI call; outputs pre-filled with NaN so an unwritten slot cannot pass."""
    N, C = x1.shape[0], x1.shape[1]
    gx1 = torch.full_like(x1, float("nan"))
    gx2 = torch.full_like(x2, float("nan"))
    stream = torch.cuda.current_stream()
    st = _lib.lib().spingtp_backward_v1_noalloc(plan._handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(),
                                                gx1.data_ptr(), gx2.data_ptr(), N, C,
                                                ctypes.c_void_p(stream.cuda_stream))
    assert st == 0, _lib.message(st)
    return gx1, gx2


@pytest.mark.parametrize("L,dtype,big,small", [
    (6, "fp32", (200, 64), (33, 7)),      # Fourier route; 7.5 MB of scratch, then 0.1 MB
    (2, "fp32", (1000, 128), (17, 5)),    # precontracted route for grad_x1
    (4, "bf16", (300, 96), (9, 3)),
])
def test_noalloc_matches_workspace_entry_point(L, dtype, big, small):
    plan = Plan(L, L, L, S3, dtype)
    for i, (N, C) in enumerate((big, small)):
        print(f"[noalloc] L={L} {dtype} call {i}: N={N} C={C}", flush=True)
        x1, x2, g = _inputs(L, N, C, dtype, 10 * L + i)
        ref1, ref2 = plan.backward_v1(x1, x2, g)
        gx1, gx2 = _noalloc(plan, x1, x2.view(N, 1, *x2.shape[2:]), g)
        torch.cuda.synchronize()
        assert torch.equal(gx1, ref1), float((gx1.float() - ref1.float()).abs().max())
        assert torch.equal(gx2, ref2.view_as(gx2)), float((gx2.float() - ref2.float().view_as(gx2)).abs().max())


def test_noalloc_rejects_requests_beyond_the_scratch():
    L, dtype = 6, "fp32"
    plan = Plan(L, L, L, S3, dtype)
    x1, x2, g = _inputs(L, 4, 2, dtype, 99)
    row = 3 * (L + 1) ** 2 * 4
    C = 128
    N = SCRATCH_BYTES // (row * C) + 1   # one edge more than the scratch holds
    gx2 = torch.full_like(x2, float("nan"))
    st = _lib.lib().spingtp_backward_v1_noalloc(plan._handle, x1.data_ptr(), x2.data_ptr(), g.data_ptr(), None,
                                                gx2.data_ptr(), N, C, None)
    assert st == TOO_LARGE
    assert "scratch" in _lib.message(st)
    torch.cuda.synchronize()
    assert torch.isnan(gx2).all()        # nothing was launched
    N_fit = SCRATCH_BYTES // (row * C)   # exactly fits: accepted by the size rule
    need = ctypes.c_size_t(0)
    assert _lib.lib().spingtp_backward_v1_workspace_size(plan._handle, N_fit, C, ctypes.byref(need)) == 0
    assert need.value <= SCRATCH_BYTES
