"""MI355X-native snapshot-free delta-extraction hot path (AReaL-DTE).

The compute path is libdte.so (HIP kernels for gfx950 behind the C ABI of
include/dte.h).  This package holds its ctypes binding (`binding`, same
names as the C entry points), the transfer-plan builder for the receiver
layouts (`layouts`), and `pipeline`, which owns device buffers (allocated
with torch) and chains the three hot calls.  There is no CPU fallback: if
libdte.so is missing, every entry point raises.
"""
from .binding import (DTE_ERR_ARG, DTE_ERR_CAPACITY, DTE_ERR_HIP, DTE_ERR_PLAN,  # noqa: F401
                      DTE_OK, DteError, dte_adamw_forward, dte_apply, dte_derive_scalars,
                      dte_extract_delta, dte_plan_create, dte_plan_destroy, dte_plan_info,
                      dte_remap, dte_status_string)
