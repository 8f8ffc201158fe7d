"""FMMformer attention forward on AMD MI355X (gfx950) through hand-written HIP kernels.

The operator lives in libfmm_attn.so (C ABI: include/fmm_attn.h); `forward`
and friends are a thin ctypes binding that only marshals arguments.
"""

from .binding import (FmmError, forward, forward_ws, kernel_timing, kernel_timing_read,  # noqa: F401
                      lib, release_workspace, status_string, version, workspace_bytes)
