"""FMMformer attention on AMD MI355X (gfx950) through hand-written HIP kernels.

The operator lives in libfmm_attn.so (C ABI: include/fmm_attn.h); `forward`,
`backward` and friends are a thin ctypes binding that only marshals
arguments, and `fmm_attention` wraps the two as a torch.autograd function.
"""

from .binding import (FmmError, backward, fmm_attention, forward, forward_ws,  # noqa: F401
                      kernel_timing, kernel_timing_read, lib, release_workspace, status_string,
                      version, workspace_bytes)
