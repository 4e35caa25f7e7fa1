"""Python binding of the SpinGTP C ABI (``include/spingtp.h``).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libspingtp.so``.  torch provides device memory and the stream.
"""

import ctypes

import numpy as np

from . import _lib

BASIS_PAPER = 0
BASIS_M0_PAIRED = 1
BASIS_PARITY = 2
KERNEL_VALU = 0x100  # force the fp32 vector-ALU kernels (spingtp.h)
CHANNEL_WEIGHTS = 0x1000  # also build the per-channel path-weighted table (spingtp.h)
FULLY_CONNECTED = 0x2000  # also build the entry table of the fully connected product (spingtp.h)
V1_FOURIER = 0x200  # spingtp_forward_v1 on the Fourier route (spingtp.h)
V1_PRECONTRACT = 0x400  # spingtp_forward_v1 on the precontracted kernel wherever it is built
TABLES_BACKWARD = 0x800  # host table functions: the gradients' tables (spingtp.h)
FP32 = 0
BF16 = 1


def _spin_array(spins):
    spins = [int(s) for s in spins]
    return (ctypes.c_int * len(spins))(*spins), len(spins)


def plan_tables_host(L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Float64 plan tables and dims (host only, no GPU needed)."""
    arr, n = _spin_array(spins)
    count = ctypes.c_size_t(0)
    dims = (ctypes.c_int * 8)()
    _lib.check(_lib.lib().spingtp_plan_tables_host(L1, L2, Lout, arr, n, basis, None, 0,
                                                   ctypes.byref(count), dims), "spingtp_plan_tables_host")
    out = np.zeros(count.value, dtype=np.float64)
    _lib.check(_lib.lib().spingtp_plan_tables_host(
        L1, L2, Lout, arr, n, basis, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), out.size,
        ctypes.byref(count), dims), "spingtp_plan_tables_host")
    keys = ("n_theta", "n_phi", "L1", "L2", "Lout", "n_spins", "per_theta_block", "global_block")
    return out, dict(zip(keys, list(dims)))


def dense_tensor_host(L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """Dense float64 T[k1, k2, k3] of the operation (host only, no GPU needed)."""
    arr, n = _spin_array(spins)
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_dense_tensor_host(L1, L2, Lout, arr, n, basis, None, 0, ctypes.byref(count)),
               "spingtp_dense_tensor_host")
    T = np.zeros(count.value, dtype=np.float64)
    _lib.check(_lib.lib().spingtp_dense_tensor_host(L1, L2, Lout, arr, n, basis,
                                                    T.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), T.size,
                                                    ctypes.byref(count)), "spingtp_dense_tensor_host")
    nc = lambda L: len(spins) * (L + 1) ** 2  # noqa: E731
    return T.reshape(nc(L1), nc(L2), nc(Lout))


def mfma_operands_host(L):
    """spingtp_mfma_operands_host: the packed fp16 operand words of the matrix-core kernel (uint32)."""
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_mfma_operands_host(L, None, 0, ctypes.byref(count)), "spingtp_mfma_operands_host")
    out = np.zeros(count.value, dtype=np.uint32)
    _lib.check(_lib.lib().spingtp_mfma_operands_host(L, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
                                                     out.size, ctypes.byref(count)), "spingtp_mfma_operands_host")
    return out


def uvw_table_host(L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER, backward=False):
    """spingtp_pre_table_host with SPINGTP_FULLY_CONNECTED: the entry table of the fully
    connected product, or with backward=True the tables of its gradients w.r.t. x1 and x2
    (a pair, split at the end of the first one)."""
    arr, n = _spin_array(spins)
    flags = basis | FULLY_CONNECTED | (TABLES_BACKWARD if backward else 0)
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_pre_table_host(L1, L2, Lout, arr, n, flags, None, 0, ctypes.byref(count)),
               "spingtp_pre_table_host")
    out = np.zeros(count.value, dtype=np.uint32)
    _lib.check(_lib.lib().spingtp_pre_table_host(L1, L2, Lout, arr, n, flags,
                                                 out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), out.size,
                                                 ctypes.byref(count)), "spingtp_pre_table_host")
    if not backward:
        return out
    # length of the first table: its entries end where its last entry offset points
    n_paths, rec0, ent0 = int(out[0]), int(out[6]), int(out[7])
    csr0 = rec0 + 6 * n_paths
    n_ent = int(out[csr0:ent0].max()) if ent0 > csr0 else 0
    end = ent0 + 2 * n_ent
    return out[:end], out[end:]


def pre_table_host(L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER, backward=False, channel_weights=False):
    """spingtp_pre_table_host: the tensor table of the precontracted kernel (uint32 words); with
    backward=True the table of spingtp_backward_v1, with channel_weights=True that of
    spingtp_forward_v1_weighted, with both the entry lists of spingtp_backward_v1_weighted."""
    arr, n = _spin_array(spins)
    basis = basis | (TABLES_BACKWARD if backward else 0) | (CHANNEL_WEIGHTS if channel_weights else 0)
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_pre_table_host(L1, L2, Lout, arr, n, basis, None, 0, ctypes.byref(count)),
               "spingtp_pre_table_host")
    out = np.zeros(count.value, dtype=np.uint32)
    _lib.check(_lib.lib().spingtp_pre_table_host(L1, L2, Lout, arr, n, basis,
                                                 out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), out.size,
                                                 ctypes.byref(count)), "spingtp_pre_table_host")
    return out


def paths_host(L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """spingtp_paths_host: the [n_paths, 3] block triples of the path-weighted product."""
    arr, n = _spin_array(spins)
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_paths_host(L1, L2, Lout, arr, n, basis, None, 0, ctypes.byref(count)),
               "spingtp_paths_host")
    out = np.zeros((count.value, 3), dtype=np.int32)
    _lib.check(_lib.lib().spingtp_paths_host(L1, L2, Lout, arr, n, basis,
                                             out.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), count.value,
                                             ctypes.byref(count)), "spingtp_paths_host")
    return out


def direct_table_host(L1, L2, Lout, spins=(-1, 0, 1), basis=BASIS_PAPER, role=0):
    """spingtp_direct_table_host: the entry table of the direct kernel for one role of T
    (0 forward, 1 gradient w.r.t. x1, 2 gradient w.r.t. x2; uint32 words)."""
    arr, n = _spin_array(spins)
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_direct_table_host(L1, L2, Lout, arr, n, basis, role, None, 0, ctypes.byref(count)),
               "spingtp_direct_table_host")
    out = np.zeros(count.value, dtype=np.uint32)
    _lib.check(_lib.lib().spingtp_direct_table_host(L1, L2, Lout, arr, n, basis, role,
                                                    out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), out.size,
                                                    ctypes.byref(count)), "spingtp_direct_table_host")
    return out


def conj_map_host(L, spins=(-1, 0, 1), basis=BASIS_PAPER):
    """spingtp_conj_map_host: the conjugation map words of degree L (uint32)."""
    arr, n = _spin_array(spins)
    count = ctypes.c_size_t(0)
    _lib.check(_lib.lib().spingtp_conj_map_host(L, arr, n, basis, None, 0, ctypes.byref(count)),
               "spingtp_conj_map_host")
    out = np.zeros(count.value, dtype=np.uint32)
    _lib.check(_lib.lib().spingtp_conj_map_host(L, arr, n, basis, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
                                                out.size, ctypes.byref(count)), "spingtp_conj_map_host")
    return out


class Plan:
    """spingtp_plan_create / spingtp_forward / spingtp_plan_destroy.

    ``valu_only`` sets SPINGTP_KERNEL_VALU: the fp32 vector-ALU kernels even where
    the matrix-core kernel is the default.  ``v1_fourier`` sets SPINGTP_V1_FOURIER:
    ``forward_v1`` on the Fourier route even where the precontracted kernel is the
    default; ``v1_precontract`` sets SPINGTP_V1_PRECONTRACT: the precontracted kernel
    wherever it is built.
    """

    def __init__(self, L1, L2, Lout, spins=(-1, 0, 1), dtype="fp32", basis=BASIS_PAPER, valu_only=False,
                 v1_fourier=False, v1_precontract=False, weights=None, channel_weights=False,
                 fully_connected=False):
        import torch  # device memory and streams only

        self.L1, self.L2, self.Lout = int(L1), int(L2), int(Lout)
        self.spins = tuple(int(s) for s in spins)
        self.dtype_name = {"fp32": "fp32", "float32": "fp32", "bf16": "bf16", "bfloat16": "bf16"}[str(dtype)]
        self.torch_dtype = torch.float32 if self.dtype_name == "fp32" else torch.bfloat16
        self.basis = int(basis)
        self.valu_only = bool(valu_only)
        self.v1_fourier = bool(v1_fourier)
        self.v1_precontract = bool(v1_precontract)
        self._handle = ctypes.c_void_p()
        arr, n = _spin_array(self.spins)
        code = FP32 if self.dtype_name == "fp32" else BF16
        flags = (self.basis | (KERNEL_VALU if self.valu_only else 0) | (V1_FOURIER if self.v1_fourier else 0)
                 | (V1_PRECONTRACT if self.v1_precontract else 0) | (CHANNEL_WEIGHTS if channel_weights else 0)
                 | (FULLY_CONNECTED if fully_connected else 0))
        if weights is None:
            _lib.check(_lib.lib().spingtp_plan_create(self.L1, self.L2, self.Lout, arr, n, code, flags,
                                                      ctypes.byref(self._handle)), "spingtp_plan_create")
        else:  # one weight per path of paths_host, shared by the channels
            w = np.ascontiguousarray(np.asarray(weights, dtype=np.float64).ravel())
            _lib.check(_lib.lib().spingtp_plan_create_weighted(
                self.L1, self.L2, self.Lout, arr, n, code, flags, w.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                w.size, ctypes.byref(self._handle)), "spingtp_plan_create_weighted")
        self.device = torch.cuda.current_device()
        # paths of the per-channel weights (their count bounds the kernel's reads of a weight row)
        self.n_paths = (len(paths_host(self.L1, self.L2, self.Lout, self.spins, self.basis))
                        if channel_weights or fully_connected else 0)

    @property
    def handle(self):
        return self._handle

    def shape_in(self, which):
        L = self.L1 if which == 1 else self.L2
        return (len(self.spins), (L + 1) ** 2)

    @property
    def shape_out(self):
        return (len(self.spins), (self.Lout + 1) ** 2)

    def kernel_info(self):
        info = (ctypes.c_int * 4)()
        _lib.check(_lib.lib().spingtp_plan_kernel_info(self._handle, info), "spingtp_plan_kernel_info")
        return {"waves": info[0], "units_per_workgroup": info[1], "lds_bytes": info[2], "family": info[3]}

    def kernel_info_v1(self):
        info = (ctypes.c_int * 4)()
        _lib.check(_lib.lib().spingtp_plan_kernel_info_v1(self._handle, info), "spingtp_plan_kernel_info_v1")
        return {"waves": info[0], "units_per_workgroup": info[1], "lds_bytes": info[2], "family": info[3]}

    def forward(self, x1, x2, out=None, stream=None):
        """out[N, C, n_spins, (Lout+1)^2] = SpinGTP(x1, x2) on the current (or given) stream."""
        return self._run(x1, x2, out, stream, False)

    def forward_v1(self, x1, x2, out=None, stream=None):
        """spingtp_forward_v1: x2 is [N, n_spins, (L2+1)^2] (or [N, 1, ...]), shared by the C channels."""
        if x2.dim() == 3:
            x2 = x2.unsqueeze(1)
        return self._run(x1, x2, out, stream, True)

    def forward_v1_weighted(self, x1, x2, weights, out=None, stream=None):
        """spingtp_forward_v1_weighted: x2 shared by the C channels of an edge, weights a contiguous fp32
        [C, n_paths] device tensor (paths in paths_host order); the plan needs channel_weights=True."""
        import torch

        if x2.dim() == 3:
            x2 = x2.unsqueeze(1)
        C = x1.shape[1]
        if (weights.dtype != torch.float32 or not weights.is_contiguous() or tuple(weights.shape) != (C, self.n_paths)
                or weights.device != x1.device):
            raise ValueError(f"weights must be a contiguous fp32 [C, {self.n_paths}] tensor on the inputs' device "
                             "(a plan created with channel_weights=True)")
        return self._run(x1, x2, out, stream, True, weights)

    def _run(self, x1, x2, out, stream, shared, weights=None):
        import torch

        if x1.dim() != 4 or x2.dim() != 4:
            raise ValueError("x1 and x2 must be [N, C, n_spins, (L+1)^2]")
        N, C = x1.shape[0], x1.shape[1]
        if tuple(x1.shape[2:]) != self.shape_in(1) or tuple(x2.shape[2:]) != self.shape_in(2):
            raise ValueError(f"trailing shapes {tuple(x1.shape[2:])}, {tuple(x2.shape[2:])} do not match "
                             f"{self.shape_in(1)}, {self.shape_in(2)}")
        if tuple(x2.shape[:2]) != ((N, 1) if shared else (N, C)):
            raise ValueError("x2 must be [N, 1, ...] (forward_v1) or [N, C, ...] (forward)")
        for t in (x1, x2):
            if t.dtype != self.torch_dtype or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"inputs must be contiguous {self.torch_dtype} device tensors")
        if out is None:
            out = torch.empty((N, C) + self.shape_out, dtype=self.torch_dtype, device=x1.device)
        elif (tuple(out.shape) != (N, C) + self.shape_out or out.dtype != self.torch_dtype
              or not out.is_contiguous()):
            raise ValueError("out has the wrong shape, dtype or layout")
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        if weights is not None:
            _lib.check(_lib.lib().spingtp_forward_v1_weighted(self._handle, x1.data_ptr(), x2.data_ptr(),
                                                              weights.data_ptr(), out.data_ptr(), N, C,
                                                              ctypes.c_void_p(stream.cuda_stream)),
                       "spingtp_forward_v1_weighted")
            return out
        fn = _lib.lib().spingtp_forward_v1 if shared else _lib.lib().spingtp_forward
        _lib.check(fn(self._handle, x1.data_ptr(), x2.data_ptr(), out.data_ptr(), N, C,
                      ctypes.c_void_p(stream.cuda_stream)), "spingtp_forward_v1" if shared else "spingtp_forward")
        return out

    def backward(self, x1, x2, grad_out, need_x1=True, need_x2=True, stream=None):
        """spingtp_backward: (grad_x1, grad_x2) of a loss with dLoss/dout = grad_out (None where not
        requested)."""
        import torch

        N, C = x1.shape[0], x1.shape[1]
        for t, shape in ((x1, self.shape_in(1)), (x2, self.shape_in(2)), (grad_out, self.shape_out)):
            if (t.dim() != 4 or tuple(t.shape) != (N, C) + tuple(shape) or t.dtype != self.torch_dtype
                    or not t.is_cuda or not t.is_contiguous()):
                raise ValueError("x1, x2, grad_out must be contiguous [N, C, n_spins, (L+1)^2] device tensors "
                                 "of the plan's dtype")
        gx1 = torch.empty_like(x1) if need_x1 else None
        gx2 = torch.empty_like(x2) if need_x2 else None
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        _lib.check(_lib.lib().spingtp_backward(self._handle, x1.data_ptr(), x2.data_ptr(), grad_out.data_ptr(),
                                               gx1.data_ptr() if gx1 is not None else None,
                                               gx2.data_ptr() if gx2 is not None else None, N, C,
                                               ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward")
        return gx1, gx2

    def backward_v1(self, x1, x2, grad_out, need_x1=True, need_x2=True, stream=None):
        """spingtp_backward_v1: (grad_x1 [N, C, ...], grad_x2 [N, 1, ...]) through forward_v1; the workspace
        for grad_x2 comes from torch's allocator."""
        import torch

        if x2.dim() == 3:
            x2 = x2.unsqueeze(1)
        N, C = x1.shape[0], x1.shape[1]
        for t, shape in ((x1, (N, C) + tuple(self.shape_in(1))), (x2, (N, 1) + tuple(self.shape_in(2))),
                         (grad_out, (N, C) + tuple(self.shape_out))):
            if (tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda
                    or not t.is_contiguous()):
                raise ValueError("x1 [N, C, ...], x2 [N, 1, ...], grad_out [N, C, ...] must be contiguous device "
                                 "tensors of the plan's dtype")
        gx1 = torch.empty_like(x1) if need_x1 else None
        gx2 = torch.empty_like(x2) if need_x2 else None
        n = ctypes.c_size_t(0)
        _lib.check(_lib.lib().spingtp_backward_v1_workspace_size(self._handle, N, C, ctypes.byref(n)),
                   "spingtp_backward_v1_workspace_size")
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device=x1.device) if need_x2 else None
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        _lib.check(_lib.lib().spingtp_backward_v1(self._handle, x1.data_ptr(), x2.data_ptr(), grad_out.data_ptr(),
                                                  gx1.data_ptr() if gx1 is not None else None,
                                                  gx2.data_ptr() if gx2 is not None else None,
                                                  ws.data_ptr() if ws is not None else None,
                                                  n.value if ws is not None else 0, N, C,
                                                  ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward_v1")
        return gx1, gx2

    def backward_v1_noalloc(self, x1, x2, grad_out, grad_x1=None, grad_x2=None, stream=None):
        """spingtp_backward_v1_noalloc: the gradients of backward_v1 written into the caller's
        grad_x1 [N, C, ...] and/or grad_x2 [N, 1, ...] tensors; the library stages grad_x2 in its
        fixed device scratch, so the call allocates nothing."""
        import torch

        if x2.dim() == 3:
            x2 = x2.unsqueeze(1)
        N, C = x1.shape[0], x1.shape[1]
        for t, shape in ((x1, (N, C) + tuple(self.shape_in(1))), (x2, (N, 1) + tuple(self.shape_in(2))),
                         (grad_out, (N, C) + tuple(self.shape_out)), (grad_x1, (N, C) + tuple(self.shape_in(1))),
                         (grad_x2, (N, 1) + tuple(self.shape_in(2)))):
            if t is not None and (tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda
                                  or not t.is_contiguous()):
                raise ValueError("x1, grad_out, grad_x1 [N, C, ...], x2, grad_x2 [N, 1, ...] must be contiguous "
                                 "device tensors of the plan's dtype")
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        _lib.check(_lib.lib().spingtp_backward_v1_noalloc(
            self._handle, x1.data_ptr(), x2.data_ptr(), grad_out.data_ptr(),
            grad_x1.data_ptr() if grad_x1 is not None else None, grad_x2.data_ptr() if grad_x2 is not None else None,
            N, C, ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward_v1_noalloc")
        return grad_x1, grad_x2

    def backward_v1_weighted(self, x1, x2, weights, grad_out, stream=None):
        """spingtp_backward_v1_weighted: (grad_x1 [N, C, ...], grad_x2 [N, 1, ...], grad_weights [C, n_paths]
        fp32) through forward_v1_weighted; the workspace comes from torch's allocator."""
        import torch

        if x2.dim() == 3:
            x2 = x2.unsqueeze(1)
        N, C = x1.shape[0], x1.shape[1]
        for t, shape in ((x1, (N, C) + tuple(self.shape_in(1))), (x2, (N, 1) + tuple(self.shape_in(2))),
                         (grad_out, (N, C) + tuple(self.shape_out))):
            if (tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda
                    or not t.is_contiguous()):
                raise ValueError("x1 [N, C, ...], x2 [N, 1, ...], grad_out [N, C, ...] must be contiguous device "
                                 "tensors of the plan's dtype")
        if (weights.dtype != torch.float32 or not weights.is_contiguous() or tuple(weights.shape) != (C, self.n_paths)
                or weights.device != x1.device):
            raise ValueError(f"weights must be a contiguous fp32 [C, {self.n_paths}] tensor on the inputs' device "
                             "(a plan created with channel_weights=True)")
        gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
        gw = torch.empty((C, self.n_paths), dtype=torch.float32, device=x1.device)
        n = ctypes.c_size_t(0)
        _lib.check(_lib.lib().spingtp_backward_v1_weighted_workspace_size(self._handle, N, C, ctypes.byref(n)),
                   "spingtp_backward_v1_weighted_workspace_size")
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device=x1.device)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t.numel() else None

        _lib.check(_lib.lib().spingtp_backward_v1_weighted(
            self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(grad_out), ptr(gx1), ptr(gx2), ptr(gw),
            ws.data_ptr(), n.value, N, C, ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward_v1_weighted")
        return gx1, gx2, gw

    def _check_weighted(self, x1, x2, weights, grad_out=None):
        import torch

        N, C = x1.shape[0], x1.shape[1]
        shapes = [(x1, (N, C) + tuple(self.shape_in(1))), (x2, (N, C) + tuple(self.shape_in(2)))]
        if grad_out is not None:
            shapes.append((grad_out, (N, C) + tuple(self.shape_out)))
        for t, shape in shapes:
            if (tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda
                    or not t.is_contiguous()):
                raise ValueError("x1, x2 [N, C, ...] (and grad_out) must be contiguous device tensors of the "
                                 "plan's dtype")
        if (weights.dtype != torch.float32 or not weights.is_contiguous() or tuple(weights.shape) != (C, self.n_paths)
                or weights.device != x1.device):
            raise ValueError(f"weights must be a contiguous fp32 [C, {self.n_paths}] tensor on the inputs' device "
                             "(a plan created with channel_weights=True)")
        return N, C

    def forward_weighted(self, x1, x2, weights, out=None, stream=None):
        """spingtp_forward_weighted: per-channel path weights [C, n_paths] with x2 [N, C, ...] per unit."""
        import torch

        N, C = self._check_weighted(x1, x2, weights)
        if out is None:
            out = torch.empty((N, C) + self.shape_out, dtype=self.torch_dtype, device=x1.device)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t.numel() else None

        _lib.check(_lib.lib().spingtp_forward_weighted(self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(out), N, C,
                                                       ctypes.c_void_p(stream.cuda_stream)), "spingtp_forward_weighted")
        return out

    def backward_weighted(self, x1, x2, weights, grad_out, stream=None):
        """spingtp_backward_weighted: (grad_x1, grad_x2 [N, C, ...], grad_weights [C, n_paths] fp32) through
        forward_weighted; the workspace comes from torch's allocator."""
        import torch

        N, C = self._check_weighted(x1, x2, weights, grad_out)
        gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
        gw = torch.empty((C, self.n_paths), dtype=torch.float32, device=x1.device)
        n = ctypes.c_size_t(0)
        _lib.check(_lib.lib().spingtp_backward_weighted_workspace_size(self._handle, N, C, ctypes.byref(n)),
                   "spingtp_backward_weighted_workspace_size")
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device=x1.device)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t.numel() else None

        _lib.check(_lib.lib().spingtp_backward_weighted(
            self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(grad_out), ptr(gx1), ptr(gx2), ptr(gw),
            ws.data_ptr(), n.value, N, C, ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward_weighted")
        return gx1, gx2, gw

    def _check_depthwise(self, x1, x2, weights, grad_out=None):
        import torch

        N, C, V = x1.shape[0], x1.shape[1], x2.shape[1]
        shapes = [(x1, (N, C) + tuple(self.shape_in(1))), (x2, (N, V) + tuple(self.shape_in(2)))]
        if grad_out is not None:
            shapes.append((grad_out, (N, C) + tuple(self.shape_out)))
        for t, shape in shapes:
            if (tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda
                    or not t.is_contiguous()):
                raise ValueError("x1 [N, C, ...], x2 [N, V, ...] (and grad_out [N, C, ...]) must be contiguous "
                                 "device tensors of the plan's dtype")
        if (weights.dtype != torch.float32 or not weights.is_contiguous()
                or tuple(weights.shape) != (V, C, self.n_paths) or weights.device != x1.device):
            raise ValueError(f"weights must be a contiguous fp32 [V, C, {self.n_paths}] tensor on the inputs' "
                             "device (a plan created with channel_weights=True)")
        return N, C, V

    def forward_fully_connected(self, x1, x2, weights, out=None, stream=None):
        """spingtp_forward_fully_connected (mode uvw): x1 [N, U, ...], x2 [N, V, ...], weights
        [n_paths, U, V, W] fp32 -> out [N, W, ...]; plan created with fully_connected=True."""
        import torch

        if x1.dim() != 4 or x2.dim() != 4 or weights.dim() != 4:
            raise ValueError("x1 [N, U, ...], x2 [N, V, ...], weights [n_paths, U, V, W]")
        N, U, V, W = x1.shape[0], x1.shape[1], x2.shape[1], weights.shape[3]
        for t, shape in ((x1, (N, U) + tuple(self.shape_in(1))), (x2, (N, V) + tuple(self.shape_in(2)))):
            if tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda or not t.is_contiguous():
                raise ValueError("x1, x2 must be contiguous device tensors of the plan's dtype and shape")
        if (tuple(weights.shape) != (self.n_paths, U, V, W) or weights.dtype != torch.float32 or not weights.is_cuda
                or not weights.is_contiguous()):
            raise ValueError(f"weights must be a contiguous fp32 device tensor [{self.n_paths}, U, V, W]")
        if out is None:
            out = torch.empty((N, W) + self.shape_out, dtype=self.torch_dtype, device=x1.device)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t.numel() else None

        _lib.check(_lib.lib().spingtp_forward_fully_connected(self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(out),
                                                              N, U, V, W, ctypes.c_void_p(stream.cuda_stream)),
                   "spingtp_forward_fully_connected")
        return out

    def backward_fully_connected(self, x1, x2, weights, grad_out, need=(True, True, True), stream=None):
        """spingtp_backward_fully_connected: the gradients (grad_x1, grad_x2, grad_weights) of
        forward_fully_connected for grad_out [N, W, ...]; `need` picks which are computed
        (the others are returned as None)."""
        import torch

        if x1.dim() != 4 or x2.dim() != 4 or weights.dim() != 4 or grad_out.dim() != 4:
            raise ValueError("x1 [N, U, ...], x2 [N, V, ...], weights [n_paths, U, V, W], grad_out [N, W, ...]")
        N, U, V, W = x1.shape[0], x1.shape[1], x2.shape[1], weights.shape[3]
        for t, shape in ((x1, (N, U) + tuple(self.shape_in(1))), (x2, (N, V) + tuple(self.shape_in(2))),
                         (grad_out, (N, W) + tuple(self.shape_out))):
            if tuple(t.shape) != shape or t.dtype != self.torch_dtype or not t.is_cuda or not t.is_contiguous():
                raise ValueError("x1, x2, grad_out must be contiguous device tensors of the plan's dtype and shape")
        if (tuple(weights.shape) != (self.n_paths, U, V, W) or weights.dtype != torch.float32 or not weights.is_cuda
                or not weights.is_contiguous()):
            raise ValueError(f"weights must be a contiguous fp32 device tensor [{self.n_paths}, U, V, W]")
        g1 = torch.empty_like(x1) if need[0] else None
        g2 = torch.empty_like(x2) if need[1] else None
        gw = torch.empty_like(weights) if need[2] else None
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t is not None and t.numel() else None

        _lib.check(_lib.lib().spingtp_backward_fully_connected(
            self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(grad_out), ptr(g1), ptr(g2), ptr(gw), N, U, V, W,
            ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward_fully_connected")
        return g1, g2, gw

    def forward_depthwise(self, x1, x2, weights, out=None, stream=None):
        """spingtp_forward_depthwise: x2 [N, V, ...] with V >= 1 channels per edge, weights [V, C, n_paths]."""
        import torch

        N, C, V = self._check_depthwise(x1, x2, weights)
        if out is None:
            out = torch.empty((N, C) + self.shape_out, dtype=self.torch_dtype, device=x1.device)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t.numel() else None

        _lib.check(_lib.lib().spingtp_forward_depthwise(self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(out), N, C,
                                                        V, ctypes.c_void_p(stream.cuda_stream)),
                   "spingtp_forward_depthwise")
        return out

    def backward_depthwise(self, x1, x2, weights, grad_out, stream=None):
        """spingtp_backward_depthwise: (grad_x1 [N, C, ...], grad_x2 [N, V, ...], grad_weights [V, C, n_paths])."""
        import torch

        N, C, V = self._check_depthwise(x1, x2, weights, grad_out)
        gx1, gx2 = torch.empty_like(x1), torch.empty_like(x2)
        gw = torch.empty_like(weights)
        n = ctypes.c_size_t(0)
        _lib.check(_lib.lib().spingtp_backward_depthwise_workspace_size(self._handle, N, C, V, ctypes.byref(n)),
                   "spingtp_backward_depthwise_workspace_size")
        ws = torch.empty(max(1, n.value), dtype=torch.uint8, device=x1.device)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)

        def ptr(t):
            return t.data_ptr() if t.numel() else None

        _lib.check(_lib.lib().spingtp_backward_depthwise(
            self._handle, ptr(x1), ptr(x2), ptr(weights), ptr(grad_out), ptr(gx1), ptr(gx2), ptr(gw),
            ws.data_ptr(), n.value, N, C, V, ctypes.c_void_p(stream.cuda_stream)), "spingtp_backward_depthwise")
        return gx1, gx2, gw

    __call__ = forward

    def close(self):
        if self._handle is not None and self._handle.value:
            _lib.check(_lib.lib().spingtp_plan_destroy(self._handle), "spingtp_plan_destroy")
            self._handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
