"""FMMformer attention on AMD MI355X (gfx950) through hand-written HIP kernels.

The operator lives in libfmm_attn.so (C ABI: include/fmm_attn.h); `forward`,
`backward` and friends are a thin ctypes binding that only marshals
arguments, and `fmm_attention` (and `fmm_fast_weight_attention` for the fast-weight
form) wrap forward and backward as torch.autograd functions.
"""

from .binding import (FmmError, backward, backward_fastweight, fmm_attention,  # noqa: F401
                      fmm_fast_weight_attention, forward, forward_fastweight, forward_ws,
                      kernel_timing, kernel_timing_read, lib, release_workspace, status_string,
                      version, workspace_bytes)
