"""ctypes loader for the in-tree ``libspingtp.so``.  Fails loudly when it is missing."""

import ctypes
import os

# SPINGTP_LIBRARY names another build of the same library (the sanitizer-checked copy
# the host tests use); by default the in-tree build.
LIB_PATH = os.environ.get("SPINGTP_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                               "libspingtp.so")

SPINGTP_OK = 0
STATUS_NAMES = {0: "OK", 1: "ERR_INVALID_ARG", 2: "ERR_UNSUPPORTED", 3: "ERR_OUT_OF_MEMORY",
                4: "ERR_HIP", 5: "ERR_INTERNAL", 6: "ERR_TOO_LARGE"}
EXPORTED = ("spingtp_plan_create", "spingtp_forward", "spingtp_plan_destroy", "spingtp_status_string",
            "spingtp_plan_tables_host", "spingtp_plan_kernel_info", "spingtp_dense_tensor_host",
            "spingtp_mfma_operands_host", "spingtp_forward_v1", "spingtp_plan_kernel_info_v1",
            "spingtp_pre_table_host", "spingtp_backward", "spingtp_conj_map_host", "spingtp_backward_v1",
            "spingtp_backward_v1_workspace_size", "spingtp_direct_table_host", "spingtp_paths_host",
            "spingtp_plan_create_weighted", "spingtp_forward_v1_weighted", "spingtp_backward_v1_weighted",
            "spingtp_backward_v1_weighted_workspace_size", "spingtp_forward_weighted", "spingtp_backward_weighted",
            "spingtp_backward_weighted_workspace_size", "spingtp_forward_depthwise", "spingtp_backward_depthwise",
            "spingtp_backward_depthwise_workspace_size", "spingtp_backward_v1_noalloc",
            "spingtp_plan_upload_selftest_host", "spingtp_forward_fully_connected",
            "spingtp_backward_fully_connected")

_lib = None


class SpinGTPError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({message(status)})")


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                               "(or python paper_2607_01408_amd/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        c_int_p = ctypes.POINTER(ctypes.c_int)
        L.spingtp_plan_create.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                          ctypes.c_int, ctypes.c_uint, ctypes.POINTER(ctypes.c_void_p)]
        L.spingtp_plan_create.restype = ctypes.c_int
        L.spingtp_plan_create_weighted.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                                   ctypes.c_int, ctypes.c_uint, ctypes.POINTER(ctypes.c_double),
                                                   ctypes.c_size_t, ctypes.POINTER(ctypes.c_void_p)]
        L.spingtp_plan_create_weighted.restype = ctypes.c_int
        L.spingtp_paths_host.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                         ctypes.c_uint, c_int_p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_paths_host.restype = ctypes.c_int
        L.spingtp_forward_v1_weighted.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        L.spingtp_forward_v1_weighted.restype = ctypes.c_int
        L.spingtp_backward_v1_weighted.argtypes = [ctypes.c_void_p] + [ctypes.c_void_p] * 8 + [
            ctypes.c_size_t, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        L.spingtp_backward_v1_weighted.restype = ctypes.c_int
        L.spingtp_backward_v1_weighted_workspace_size.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                                                  ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_backward_v1_weighted_workspace_size.restype = ctypes.c_int
        L.spingtp_forward_weighted.argtypes = L.spingtp_forward_v1_weighted.argtypes
        L.spingtp_forward_weighted.restype = ctypes.c_int
        L.spingtp_backward_weighted.argtypes = L.spingtp_backward_v1_weighted.argtypes
        L.spingtp_backward_weighted.restype = ctypes.c_int
        L.spingtp_backward_weighted_workspace_size.argtypes = L.spingtp_backward_v1_weighted_workspace_size.argtypes
        L.spingtp_backward_weighted_workspace_size.restype = ctypes.c_int
        L.spingtp_forward_depthwise.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int64] * 3 + [ctypes.c_void_p]
        L.spingtp_forward_depthwise.restype = ctypes.c_int
        L.spingtp_backward_depthwise.argtypes = [ctypes.c_void_p] * 9 + [ctypes.c_size_t] + [ctypes.c_int64] * 3 + [
            ctypes.c_void_p]
        L.spingtp_backward_depthwise.restype = ctypes.c_int
        L.spingtp_backward_depthwise_workspace_size.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                                                ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_backward_depthwise_workspace_size.restype = ctypes.c_int
        L.spingtp_forward.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        L.spingtp_forward.restype = ctypes.c_int
        L.spingtp_plan_destroy.argtypes = [ctypes.c_void_p]
        L.spingtp_plan_destroy.restype = ctypes.c_int
        L.spingtp_status_string.argtypes = [ctypes.c_int]
        L.spingtp_status_string.restype = ctypes.c_char_p
        L.spingtp_plan_tables_host.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                               ctypes.c_uint, ctypes.POINTER(ctypes.c_double), ctypes.c_size_t,
                                               ctypes.POINTER(ctypes.c_size_t), c_int_p]
        L.spingtp_plan_tables_host.restype = ctypes.c_int
        L.spingtp_dense_tensor_host.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                                ctypes.c_uint, ctypes.POINTER(ctypes.c_double), ctypes.c_size_t,
                                                ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_dense_tensor_host.restype = ctypes.c_int
        L.spingtp_plan_kernel_info.argtypes = [ctypes.c_void_p, c_int_p]
        L.spingtp_plan_kernel_info.restype = ctypes.c_int
        L.spingtp_mfma_operands_host.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_uint32), ctypes.c_size_t,
                                                 ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_mfma_operands_host.restype = ctypes.c_int
        L.spingtp_pre_table_host.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                             ctypes.c_uint, ctypes.POINTER(ctypes.c_uint32), ctypes.c_size_t,
                                             ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_pre_table_host.restype = ctypes.c_int
        L.spingtp_direct_table_host.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                                ctypes.c_uint, ctypes.c_int, ctypes.POINTER(ctypes.c_uint32),
                                                ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_direct_table_host.restype = ctypes.c_int
        L.spingtp_backward.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                       ctypes.c_void_p]
        L.spingtp_backward.restype = ctypes.c_int
        L.spingtp_backward_v1.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                          ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        L.spingtp_backward_v1.restype = ctypes.c_int
        L.spingtp_backward_v1_noalloc.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int64, ctypes.c_int64,
                                                                         ctypes.c_void_p]
        L.spingtp_backward_v1_noalloc.restype = ctypes.c_int
        L.spingtp_plan_upload_selftest_host.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, c_int_p, ctypes.c_int,
                                                        ctypes.c_int, ctypes.c_uint, ctypes.c_int, c_int_p, c_int_p]
        L.spingtp_plan_upload_selftest_host.restype = ctypes.c_int
        L.spingtp_forward_fully_connected.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int64] * 4 + [ctypes.c_void_p]
        L.spingtp_forward_fully_connected.restype = ctypes.c_int
        L.spingtp_backward_fully_connected.argtypes = [ctypes.c_void_p] * 8 + [ctypes.c_int64] * 4 + [ctypes.c_void_p]
        L.spingtp_backward_fully_connected.restype = ctypes.c_int
        L.spingtp_backward_v1_workspace_size.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                                         ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_backward_v1_workspace_size.restype = ctypes.c_int
        L.spingtp_conj_map_host.argtypes = [ctypes.c_int, c_int_p, ctypes.c_int, ctypes.c_uint,
                                            ctypes.POINTER(ctypes.c_uint32), ctypes.c_size_t,
                                            ctypes.POINTER(ctypes.c_size_t)]
        L.spingtp_conj_map_host.restype = ctypes.c_int
        L.spingtp_forward_v1.argtypes = list(L.spingtp_forward.argtypes)
        L.spingtp_forward_v1.restype = ctypes.c_int
        L.spingtp_plan_kernel_info_v1.argtypes = [ctypes.c_void_p, c_int_p]
        L.spingtp_plan_kernel_info_v1.restype = ctypes.c_int
        _lib = L
    return _lib


def message(status: int) -> str:
    return lib().spingtp_status_string(int(status)).decode()


def check(status: int, where: str) -> None:
    if status != SPINGTP_OK:
        raise SpinGTPError(status, where)
