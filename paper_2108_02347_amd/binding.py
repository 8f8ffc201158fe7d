"""ctypes binding of libfmm_attn.so (the C ABI declared in include/fmm_attn.h).

Argument marshalling only: every step of the operator runs in the HIP library.
PyTorch supplies device memory and the current stream.  If the library has not
been built, every call raises; there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfmm_attn.so")

FMM_OK = 0
FMM_ERR_INVALID_ARG = -1
FMM_ERR_UNSUPPORTED = -2
FMM_ERR_HIP = -3
FMM_ERR_OOM = -4
FMM_ERR_SCRATCH = -5

FMM_DTYPE_F32 = 0
FMM_DTYPE_BF16 = 1

FMM_FAR_NORM_PER_MAP = 0
FMM_FAR_NORM_JOINT = 1

KERNELS = {"seg_state": 0, "state_combine": 1, "band_apply": 2, "causal_apply": 3,
           "bwd_rows": 4, "bwd_keys": 5, "bwd_dw": 6, "layer_copy": 7, "fast_weight": 8,
           "bwd_seg_grad": 9}

EXPORTS = (
    "fmm_attn_forward", "fmm_attn_forward_bf16", "fmm_attn_workspace_bytes",
    "fmm_attn_forward_ws", "fmm_attn_status_string", "fmm_attn_release_workspace",
    "fmm_attn_version", "fmm_attn_kernel_timing", "fmm_attn_kernel_timing_read",
    "fmm_attn_forward_noalloc", "fmm_attn_noalloc_max_bytes", "fmm_attn_forward_ex",
    "fmm_attn_backward", "fmm_attn_backward_ex", "fmm_attn_layer_forward",
    "fmm_attn_layer_backward",
    "fmm_attn_forward_fastweight", "fmm_attn_backward_fastweight",
    "fmm_attn_set_one_launch",
)

_lib = None


class FmmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


def lib() -> ctypes.CDLL:
    """Load the HIP library (once); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2108_02347_amd.build_lib` "
            "(there is no non-HIP fallback)")
    h = ctypes.CDLL(LIB_PATH)
    vp, ci, cf = ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p
    fwd_args = [vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, ci, cf, cf, vp]
    for name in ("fmm_attn_forward", "fmm_attn_forward_bf16"):
        fn = getattr(h, name)
        fn.argtypes = fwd_args
        fn.restype = ci
    h.fmm_attn_forward_ws.argtypes = fwd_args[:-1] + [ci, vp, ctypes.c_size_t, vp]
    h.fmm_attn_forward_ws.restype = ci
    h.fmm_attn_forward_fastweight.argtypes = [vp] * 5 + [ci] * 6 + [cf, cf, ci, vp]
    h.fmm_attn_forward_fastweight.restype = ci
    h.fmm_attn_backward_fastweight.argtypes = [vp] * 11 + [ci] * 6 + [cf, cf, ci, vp]
    h.fmm_attn_backward_fastweight.restype = ci
    h.fmm_attn_layer_forward.argtypes = [vp] * 4 + [ci] * 7 + [cf, cf, ci, vp]
    h.fmm_attn_layer_forward.restype = ci
    h.fmm_attn_layer_backward.argtypes = [vp] * 9 + [ci] * 7 + [cf, cf, ci, vp]
    h.fmm_attn_layer_backward.restype = ci
    h.fmm_attn_backward.argtypes = [vp] * 9 + [ci] * 7 + [cf, cf, ci, vp]
    h.fmm_attn_backward.restype = ci
    h.fmm_attn_backward_ex.argtypes = [vp] * 9 + [ci] * 7 + [cf, cf, ci, ci, vp]
    h.fmm_attn_backward_ex.restype = ci
    h.fmm_attn_forward_ex.argtypes = fwd_args[:-1] + [ci, ci, vp]
    h.fmm_attn_forward_ex.restype = ci
    h.fmm_attn_forward_noalloc.argtypes = fwd_args[:-1] + [ci, vp]
    h.fmm_attn_forward_noalloc.restype = ci
    h.fmm_attn_noalloc_max_bytes.argtypes = []
    h.fmm_attn_noalloc_max_bytes.restype = ctypes.c_size_t
    h.fmm_attn_workspace_bytes.argtypes = [ci] * 6
    h.fmm_attn_workspace_bytes.restype = ctypes.c_size_t
    h.fmm_attn_status_string.argtypes = [ci]
    h.fmm_attn_status_string.restype = ctypes.c_char_p
    h.fmm_attn_release_workspace.argtypes = []
    h.fmm_attn_release_workspace.restype = None
    h.fmm_attn_version.argtypes = []
    h.fmm_attn_version.restype = ci
    h.fmm_attn_kernel_timing.argtypes = [ci]
    h.fmm_attn_kernel_timing.restype = ci
    h.fmm_attn_set_one_launch.argtypes = [ci]
    h.fmm_attn_set_one_launch.restype = ci
    h.fmm_attn_kernel_timing_read.argtypes = [ci, ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_longlong)]
    h.fmm_attn_kernel_timing_read.restype = ci
    _lib = h
    return h


def status_string(status: int) -> str:
    return lib().fmm_attn_status_string(status).decode()


def version() -> int:
    return lib().fmm_attn_version()


def release_workspace() -> None:
    lib().fmm_attn_release_workspace()


def workspace_bytes(B: int, H: int, N: int, d: int, rank: int, causal: int) -> int:
    return int(lib().fmm_attn_workspace_bytes(B, H, N, d, rank, int(causal)))


def _check(status: int) -> None:
    if status != FMM_OK:
        raise FmmError(status, status_string(status))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


# The raw handle of the current stream: torch's own accessor when the
# installed torch provides it (tens of nanoseconds), else the public Stream
# object (microseconds).
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream_of(t: torch.Tensor):
    if _raw_stream is not None:
        return ctypes.c_void_p(_raw_stream(t.device.index))
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


_DTYPES = (torch.float32, torch.bfloat16)


def _prep(q, k, v, w_near, w_far):
    """Checks the operands (same dtype, shape and device, contiguous, on the
    GPU; w of H float32 values) and returns (B, H, N, d).  Kept lean: at
    short sequences this runs once per call next to a few-microsecond
    kernel sequence."""
    dt, dev, shp = q.dtype, q.device, q.shape
    if len(shp) != 4:
        raise ValueError("q, k, v must be [B, H, N, d]")
    if dev.type != "cuda" or dt not in _DTYPES:
        raise ValueError("q, k, v must be float32 or bfloat16 CUDA/HIP tensors")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != dt or t.shape != shp or t.device != dev:
            raise ValueError("q, k, v must share dtype, shape and device")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous CUDA/HIP tensor")
    B, H, N, d = shp
    for name, w in (("w_near", w_near), ("w_far", w_far)):
        if (w.dtype != torch.float32 or w.device != dev or w.numel() != H
                or not w.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous float32 device tensor of H values")
    return B, H, N, d


def _check_out(out, q):
    """A caller-supplied output must match q exactly: the library receives only
    its address and writes B*H*N*d elements of q's dtype there."""
    if (not isinstance(out, torch.Tensor) or out.dtype != q.dtype or out.shape != q.shape
            or out.device != q.device or not out.is_contiguous()):
        raise ValueError("out must be a contiguous tensor with q's dtype, shape and device")


def forward(q, k, v, w_near, w_far, band_k: int, rank: int, causal: bool, out=None,
            joint: bool = False):
    """FMMformer attention forward; returns out (allocated if not given).
    joint=True normalises the far-field maps jointly (fmm_attn_forward_ex)."""
    B, H, N, d = _prep(q, k, v, w_near, w_far)
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_out(out, q)
    if joint:
        dt = FMM_DTYPE_BF16 if q.dtype == torch.bfloat16 else FMM_DTYPE_F32
        _check(lib().fmm_attn_forward_ex(
            _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, int(band_k), int(rank),
            int(bool(causal)), _ptr(w_near), _ptr(w_far), dt, FMM_FAR_NORM_JOINT, _stream_of(q)))
        return out
    fn = lib().fmm_attn_forward_bf16 if q.dtype == torch.bfloat16 else lib().fmm_attn_forward
    _check(fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, int(band_k), int(rank),
              int(bool(causal)), _ptr(w_near), _ptr(w_far), _stream_of(q)))
    return out


def forward_ws(q, k, v, w_near, w_far, band_k: int, rank: int, causal: bool, workspace,
               out=None):
    """Same operator with a caller-owned workspace (a contiguous device tensor on
    q's device; its size in bytes is passed to the library, which checks it)."""
    B, H, N, d = _prep(q, k, v, w_near, w_far)
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_out(out, q)
    if (not isinstance(workspace, torch.Tensor) or workspace.device != q.device
            or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous tensor on q's device")
    dt = FMM_DTYPE_BF16 if q.dtype == torch.bfloat16 else FMM_DTYPE_F32
    _check(lib().fmm_attn_forward_ws(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, int(band_k), int(rank),
        int(bool(causal)), _ptr(w_near), _ptr(w_far), dt, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream_of(q)))
    return out


def forward_noalloc(q, k, v, w_near, w_far, band_k: int, rank: int, causal: bool, out=None):
    """Same operator through the entry point that allocates nothing in the
    library (its scratch is a fixed per-GPU array); `out` may be given so that
    the call allocates nothing at all."""
    B, H, N, d = _prep(q, k, v, w_near, w_far)
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_out(out, q)
    dt = FMM_DTYPE_BF16 if q.dtype == torch.bfloat16 else FMM_DTYPE_F32
    _check(lib().fmm_attn_forward_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, N, d, int(band_k), int(rank),
        int(bool(causal)), _ptr(w_near), _ptr(w_far), dt, _stream_of(q)))
    return out


def noalloc_max_bytes() -> int:
    return int(lib().fmm_attn_noalloc_max_bytes())


def backward(q, k, v, dout, w_near, w_far, band_k: int, rank: int, causal: bool,
             joint: bool = False):
    """Gradients of the forward for dout = dL/d(out): returns (dq, dk, dv,
    dw_near, dw_far).  joint=True: of the forward with jointly normalised
    far-field maps (fmm_attn_backward_ex)."""
    B, H, N, d = _prep(q, k, v, w_near, w_far)
    _check_out(dout, q)
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    dwn = torch.empty_like(w_near)
    dwf = torch.empty_like(w_far)
    dt = FMM_DTYPE_BF16 if q.dtype == torch.bfloat16 else FMM_DTYPE_F32
    args = (_ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dwn),
            _ptr(dwf), B, H, N, d, int(band_k), int(rank), int(bool(causal)), _ptr(w_near),
            _ptr(w_far), dt)
    if joint:
        _check(lib().fmm_attn_backward_ex(*args, FMM_FAR_NORM_JOINT, _stream_of(q)))
    else:
        _check(lib().fmm_attn_backward(*args, _stream_of(q)))
    return dq, dk, dv, dwn, dwf


class _FmmAttention(torch.autograd.Function):
    """The operator as a torch.autograd function: its forward and backward
    are the library's entry points."""

    @staticmethod
    def forward(ctx, q, k, v, w_near, w_far, band_k, rank, causal, joint):
        ctx.save_for_backward(q, k, v, w_near, w_far)
        ctx.args = (int(band_k), int(rank), bool(causal), bool(joint))
        return forward(q, k, v, w_near, w_far, band_k, rank, causal, joint=bool(joint))

    @staticmethod
    def backward(ctx, g):
        q, k, v, w_near, w_far = ctx.saved_tensors
        band_k, rank, causal, joint = ctx.args
        dq, dk, dv, dwn, dwf = backward(q, k, v, g.contiguous(), w_near, w_far, band_k, rank,
                                        causal, joint=joint)
        return dq, dk, dv, dwn, dwf, None, None, None, None


def fmm_attention(q, k, v, w_near, w_far, band_k: int, rank: int, causal: bool,
                  joint: bool = False):
    """The operator as a differentiable function of q, k, v and the two blend
    logits (torch.autograd), for training through it: out = forward(...), and
    out's gradient reaches q, k, v, w_near and w_far through backward(...)."""
    return _FmmAttention.apply(q, k, v, w_near, w_far, band_k, rank, causal, joint)


class _FmmFastWeight(torch.autograd.Function):
    """The fast-weight operator (Appendix D) as a torch.autograd function over
    forward_fastweight and backward_fastweight."""

    @staticmethod
    def forward(ctx, q, k, v, beta, w_near, w_far, band_k, n_linear):
        ctx.save_for_backward(q, k, v, beta, w_near, w_far)
        ctx.args = (int(band_k), int(n_linear))
        return forward_fastweight(q, k, v, beta, w_near, w_far, band_k, n_linear)

    @staticmethod
    def backward(ctx, g):
        q, k, v, beta, w_near, w_far = ctx.saved_tensors
        dq, dk, dv, dbeta, dwn, dwf = backward_fastweight(q, k, v, beta, g.contiguous(), w_near,
                                                          w_far, *ctx.args)
        return dq, dk, dv, dbeta, dwn, dwf, None, None


def fmm_fast_weight_attention(q, k, v, beta, w_near, w_far, band_k: int, n_linear: int):
    """The fast-weight operator as a differentiable function of q, k, v, beta
    and the two blend logits (torch.autograd)."""
    return _FmmFastWeight.apply(q, k, v, beta, w_near, w_far, band_k, n_linear)


def layer_forward(x, w_qkv, w_out, heads: int, w_near, w_far, band_k: int, rank: int,
                  causal: bool, out=None):
    """The attention layer: [q | k | v] = x W_qkv, the operator per head, the
    heads concatenated per token times W_out.  x [B, N, E]; returns [B, N, E]."""
    if x.dim() != 3 or x.device.type != "cuda" or x.dtype not in _DTYPES:
        raise ValueError("x must be a [B, N, E] float32 or bfloat16 CUDA/HIP tensor")
    B, N, E = x.shape
    for name, t, shp in (("w_qkv", w_qkv, (E, 3 * E)), ("w_out", w_out, (E, E))):
        if t.dtype != x.dtype or t.device != x.device or tuple(t.shape) != shp:
            raise ValueError(f"{name} must be a {shp} tensor of x's dtype on x's device")
    for t in (x, w_qkv, w_out):
        if not t.is_contiguous():
            raise ValueError("x, w_qkv and w_out must be contiguous")
    for name, w in (("w_near", w_near), ("w_far", w_far)):
        if (w.dtype != torch.float32 or w.device != x.device or w.numel() != heads
                or not w.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous float32 device tensor of H values")
    if out is None:
        out = torch.empty_like(x)
    else:
        _check_out(out, x)
    dt = FMM_DTYPE_BF16 if x.dtype == torch.bfloat16 else FMM_DTYPE_F32
    _check(lib().fmm_attn_layer_forward(
        _ptr(x), _ptr(w_qkv), _ptr(w_out), _ptr(out), B, N, E, int(heads), int(band_k),
        int(rank), int(bool(causal)), _ptr(w_near), _ptr(w_far), dt, _stream_of(x)))
    return out


def layer_backward(x, w_qkv, w_out, dy, heads: int, w_near, w_far, band_k: int, rank: int,
                   causal: bool):
    """Gradients of the layer (layer_forward) for dy = dL/dy: returns (dx,
    dw_qkv, dw_out, dw_near, dw_far)."""
    if x.dim() != 3 or x.device.type != "cuda" or x.dtype not in _DTYPES:
        raise ValueError("x must be a [B, N, E] float32 or bfloat16 CUDA/HIP tensor")
    B, N, E = x.shape
    for name, t, shp in (("w_qkv", w_qkv, (E, 3 * E)), ("w_out", w_out, (E, E)),
                         ("dy", dy, (B, N, E))):
        if (not isinstance(t, torch.Tensor) or t.dtype != x.dtype or t.device != x.device
                or tuple(t.shape) != shp or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous {shp} tensor of x's dtype on x's device")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    for name, w in (("w_near", w_near), ("w_far", w_far)):
        if (w.dtype != torch.float32 or w.device != x.device or w.numel() != heads
                or not w.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous float32 device tensor of H values")
    dx, dwq, dwo = torch.empty_like(x), torch.empty_like(w_qkv), torch.empty_like(w_out)
    dwn, dwf = torch.empty_like(w_near), torch.empty_like(w_far)
    dt = FMM_DTYPE_BF16 if x.dtype == torch.bfloat16 else FMM_DTYPE_F32
    _check(lib().fmm_attn_layer_backward(
        _ptr(x), _ptr(w_qkv), _ptr(w_out), _ptr(dy), _ptr(dx), _ptr(dwq), _ptr(dwo), _ptr(dwn),
        _ptr(dwf), B, N, E, int(heads), int(band_k), int(rank), int(bool(causal)),
        _ptr(w_near), _ptr(w_far), dt, _stream_of(x)))
    return dx, dwq, dwo, dwn, dwf


def forward_fastweight(q, k, v, beta, w_near, w_far, band_k: int, n_linear: int, out=None):
    """FMMformer with the fast-weight far field (causal); beta: [B, H, N]
    float32 write strengths."""
    B, H, N, d = _prep(q, k, v, w_near, w_far)
    if (beta.dtype != torch.float32 or beta.device != q.device
            or tuple(beta.shape) != (B, H, N) or not beta.is_contiguous()):
        raise ValueError("beta must be a contiguous float32 [B, H, N] tensor on q's device")
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_out(out, q)
    dt = FMM_DTYPE_BF16 if q.dtype == torch.bfloat16 else FMM_DTYPE_F32
    _check(lib().fmm_attn_forward_fastweight(
        _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(out), B, H, N, d, int(band_k),
        int(n_linear), _ptr(w_near), _ptr(w_far), dt, _stream_of(q)))
    return out


def backward_fastweight(q, k, v, beta, dout, w_near, w_far, band_k: int, n_linear: int):
    """Gradients of the fast-weight operator (forward_fastweight) for dout =
    dL/d(out): returns (dq, dk, dv, dbeta, dw_near, dw_far)."""
    B, H, N, d = _prep(q, k, v, w_near, w_far)
    _check_out(dout, q)
    if (not isinstance(beta, torch.Tensor) or beta.dtype != torch.float32
            or beta.device != q.device or tuple(beta.shape) != (B, H, N)
            or not beta.is_contiguous()):
        raise ValueError("beta must be a contiguous float32 [B, H, N] tensor on q's device")
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    dbeta = torch.empty_like(beta)
    dwn = torch.empty_like(w_near)
    dwf = torch.empty_like(w_far)
    dt = FMM_DTYPE_BF16 if q.dtype == torch.bfloat16 else FMM_DTYPE_F32
    _check(lib().fmm_attn_backward_fastweight(
        _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv),
        _ptr(dbeta), _ptr(dwn), _ptr(dwf), B, H, N, d, int(band_k), int(n_linear),
        _ptr(w_near), _ptr(w_far), dt, _stream_of(q)))
    return dq, dk, dv, dbeta, dwn, dwf


def raw_forward(q_ptr, k_ptr, v_ptr, out_ptr, B, H, N, d, band_k, rank, causal, wn_ptr,
                wf_ptr, stream_ptr, bf16: bool) -> int:
    """Direct call of the C entry point with raw pointers; returns the status."""
    fn = lib().fmm_attn_forward_bf16 if bf16 else lib().fmm_attn_forward
    v = ctypes.c_void_p
    return fn(v(q_ptr), v(k_ptr), v(v_ptr), v(out_ptr), B, H, N, d, band_k, rank, causal,
              v(wn_ptr), v(wf_ptr), v(stream_ptr))


def set_one_launch(mode: int) -> int:
    """Mode of the one-launch path for short non-causal slices (0 never, 1 where
    it applies, 2 where it applies without the workgroups' exchange); returns
    the previous mode."""
    prev = lib().fmm_attn_set_one_launch(int(mode))
    if prev < 0:
        raise ValueError("one-launch mode must be 0, 1 or 2")
    return prev


def kernel_timing(enable: bool) -> None:
    _check(lib().fmm_attn_kernel_timing(int(bool(enable))))


def kernel_timing_read(kernel: str):
    """(total_ms, launches) of one kernel since the previous read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_longlong(0)
    _check(lib().fmm_attn_kernel_timing_read(KERNELS[kernel], ctypes.byref(ms),
                                             ctypes.byref(n)))
    return ms.value, n.value
