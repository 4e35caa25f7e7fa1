"""SpinGTP on AMD MI355X: the spin-weighted Gaunt tensor product as a C-ABI HIP library.

``Plan`` wraps ``spingtp_plan_create`` / ``spingtp_forward`` (``include/spingtp.h``).
``workloads`` holds the seeded synthetic input generators.
"""

from ._lib import SpinGTPError, LIB_PATH
from .spingtp import Plan, plan_tables_host, dense_tensor_host, mfma_operands_host, pre_table_host, conj_map_host, direct_table_host, paths_host, uvw_table_host, BASIS_PAPER, BASIS_M0_PAIRED, BASIS_PARITY

__all__ = ["Plan", "plan_tables_host", "dense_tensor_host", "mfma_operands_host", "pre_table_host", "conj_map_host", "direct_table_host", "paths_host", "uvw_table_host", "SpinGTPError", "LIB_PATH", "BASIS_PAPER", "BASIS_M0_PAIRED", "BASIS_PARITY"]
