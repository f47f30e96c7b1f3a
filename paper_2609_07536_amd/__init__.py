"""MI355X (gfx950) MoE GEMM2 + combine with a launch-time partition selector.

The compute path is the HIP library libmoe_gemm2.so (C ABI in
include/moe_gemm2.h); ``binding`` marshals torch tensors into it.
"""
from . import binding  # noqa: F401
from .binding import (MoeError, Workspace, combine, default_params,  # noqa: F401
                      make_workload, select_evaluate, select_partition)
