"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/fmm_attn.h declares, and rejects bad arguments on the
host before touching the HIP runtime."""

import ctypes
import os
import re

import pytest

from paper_2108_02347_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fmm_attn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fmm_attn_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = binding.lib()
    names = declared_functions()
    assert len(names) >= 9
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(binding.EXPORTS)


def test_status_strings_and_version():
    assert binding.version() == 10200
    for st in (0, -1, -2, -3, -4, -5):
        assert binding.status_string(st).startswith(
            {0: "FMM_OK", -1: "FMM_ERR_INVALID_ARG", -2: "FMM_ERR_UNSUPPORTED",
             -3: "FMM_ERR_HIP", -4: "FMM_ERR_OOM", -5: "FMM_ERR_SCRATCH"}[st])
    assert "unknown" in binding.status_string(17)


def test_workspace_bytes():
    ws = binding.workspace_bytes
    assert ws(1, 8, 65536, 64, 2, 1) > 0
    assert ws(1, 8, 65536, 64, 2, 1) % 256 == 0
    # one state record per segment plus one final record, rank * d * (d+1) floats
    assert ws(1, 1, 64, 16, 1, 0) >= 2 * 16 * 17 * 4
    assert ws(1, 1, 64, 48, 1, 0) == 0      # unsupported width
    assert ws(1, 1, 64, 16, 4, 0) == 0      # unsupported rank
    assert ws(1, 1, 64, 256, 1, 0) == 0     # unsupported width
    # rank 3 and d = 128 records: rank * d * (d+1) floats each
    assert ws(1, 1, 64, 128, 3, 1) >= 2 * 3 * 128 * 129 * 4
    assert ws(0, 1, 64, 16, 1, 0) == 0


FAKE = 1 << 20  # aligned non-null addresses; never dereferenced on the error paths


def call(q=FAKE, k=2 * FAKE, v=3 * FAKE, out=4 * FAKE, B=1, H=2, N=64, d=32, kw=5, r=2, c=0,
         wn=5 * FAKE, wf=6 * FAKE, bf16=False):
    return binding.raw_forward(q, k, v, out, B, H, N, d, kw, r, c, wn, wf, 0, bf16)


@pytest.mark.parametrize("kwargs,status", [
    (dict(q=0), binding.FMM_ERR_INVALID_ARG),
    (dict(out=0), binding.FMM_ERR_INVALID_ARG),
    (dict(wn=0), binding.FMM_ERR_INVALID_ARG),
    (dict(B=0), binding.FMM_ERR_INVALID_ARG),
    (dict(N=-3), binding.FMM_ERR_INVALID_ARG),
    (dict(kw=-1), binding.FMM_ERR_INVALID_ARG),
    (dict(c=2), binding.FMM_ERR_INVALID_ARG),
    (dict(q=FAKE + 8), binding.FMM_ERR_INVALID_ARG),          # misaligned
    (dict(out=FAKE + 64), binding.FMM_ERR_INVALID_ARG),       # overlaps q
    (dict(d=48), binding.FMM_ERR_UNSUPPORTED),
    (dict(d=256), binding.FMM_ERR_UNSUPPORTED),
    (dict(r=4), binding.FMM_ERR_UNSUPPORTED),
    (dict(r=0), binding.FMM_ERR_UNSUPPORTED),
    (dict(d=48, bf16=True), binding.FMM_ERR_UNSUPPORTED),
])
def test_host_validation(kwargs, status):
    assert call(**kwargs) == status


def test_timing_read_rejects_bad_kernel_id():
    lib = binding.lib()
    ms, n = ctypes.c_double(), ctypes.c_longlong()
    # ids run from 0 to FMM_KERNEL_COUNT - 1 (10 kernels)
    assert lib.fmm_attn_kernel_timing_read(10, ctypes.byref(ms), ctypes.byref(n)) == -1
    assert lib.fmm_attn_kernel_timing_read(-1, ctypes.byref(ms), ctypes.byref(n)) == -1


def test_binding_rejects_host_tensors_and_wrong_rank():
    # the Python binding checks its operands before any library call
    import torch
    q = torch.zeros(1, 2, 8, 16)
    w = torch.zeros(2)
    with pytest.raises(ValueError):
        binding.forward(q, q, q, w, w, 2, 1, 0)
    with pytest.raises(ValueError):
        binding.forward(q[0], q[0], q[0], w, w, 2, 1, 0)


def test_host_validation_huge_shapes():
    # element counts beyond int64 are rejected before any arithmetic can wrap
    big = 2**31 - 1
    assert call(B=big, H=big, N=big, d=64) == binding.FMM_ERR_INVALID_ARG
    assert call(B=big, H=big, N=big, d=16, bf16=True) == binding.FMM_ERR_INVALID_ARG
    # B*H beyond int32 (the launchers count slices in int): unsupported, with
    # addresses far enough apart that the operands do not overlap
    T = 1 << 40
    assert (binding.raw_forward(T, 2 * T, 3 * T, 4 * T, 65536, 65536, 1, 16, 0, 1, 0,
                                5 * T, 6 * T, 0, False) == binding.FMM_ERR_UNSUPPORTED)


def test_binding_rejects_bad_out_and_workspace():
    # out and workspace are checked by the binding: the library gets only
    # their addresses (and the workspace's size)
    import torch
    q = torch.zeros(1, 2, 8, 16)
    w = torch.zeros(2)
    with pytest.raises(ValueError):
        binding._check_out(torch.zeros(1, 2, 8, 16, dtype=torch.bfloat16), q)
    with pytest.raises(ValueError):
        binding._check_out(torch.zeros(1, 2, 8, 15), q)
    with pytest.raises(ValueError):
        binding._check_out(torch.zeros(1, 2, 16, 8).transpose(2, 3), q)
    with pytest.raises(ValueError):
        binding._check_out(None, q)
    binding._check_out(torch.zeros(1, 2, 8, 16), q)


def test_noalloc_host_checks():
    # argument errors come first; a shape needing more than the fixed array is
    # refused on the host (no GPU is touched on either path)
    lib = binding.lib()
    assert binding.noalloc_max_bytes() == 32 << 20
    T = 1 << 40
    vp = ctypes.c_void_p
    args = lambda q, H, N: (vp(q), vp(2 * T), vp(3 * T), vp(4 * T), 1, H, N, 64, 64, 2, 1,
                            vp(5 * T), vp(6 * T), 1, vp(0))
    assert lib.fmm_attn_forward_noalloc(*args(0, 1024, 64)) == binding.FMM_ERR_INVALID_ARG
    assert binding.workspace_bytes(1, 1024, 64, 64, 2, 1) > binding.noalloc_max_bytes()
    assert lib.fmm_attn_forward_noalloc(*args(T, 1024, 64)) == binding.FMM_ERR_SCRATCH


def test_forward_ex_rejects_unknown_normalisation():
    lib = binding.lib()
    T = 1 << 40
    vp = ctypes.c_void_p
    args = lambda norm, dt=0: (vp(T), vp(2 * T), vp(3 * T), vp(4 * T), 1, 2, 64, 32, 5, 2, 0,
                               vp(5 * T), vp(6 * T), dt, norm, vp(0))
    assert lib.fmm_attn_forward_ex(*args(2)) == binding.FMM_ERR_INVALID_ARG
    assert lib.fmm_attn_forward_ex(*args(-1)) == binding.FMM_ERR_INVALID_ARG
    assert lib.fmm_attn_forward_ex(*args(0, 7)) == binding.FMM_ERR_UNSUPPORTED


def test_backward_ex_rejects_unknown_normalisation():
    lib = binding.lib()
    T = 1 << 40
    vp = ctypes.c_void_p
    args = lambda norm, dt=0: (vp(T), vp(2 * T), vp(3 * T), vp(4 * T), vp(5 * T), vp(6 * T),
                               vp(7 * T), vp(8 * T), vp(9 * T), 1, 2, 64, 32, 5, 2, 0,
                               vp(10 * T), vp(11 * T), dt, norm, vp(0))
    assert lib.fmm_attn_backward_ex(*args(2)) == binding.FMM_ERR_INVALID_ARG
    assert lib.fmm_attn_backward_ex(*args(-1)) == binding.FMM_ERR_INVALID_ARG
    assert lib.fmm_attn_backward_ex(*args(0, 7)) == binding.FMM_ERR_UNSUPPORTED


def test_one_launch_knob_and_workspace():
    # the mode is process-wide: 0 never, 1 where it applies (default), 2
    # without the exchange; anything else is refused and changes nothing
    prev = binding.set_one_launch(1)
    try:
        assert prev == 1
        with pytest.raises(ValueError):
            binding.set_one_launch(3)
        assert binding.set_one_launch(2) == 1
        assert binding.set_one_launch(0) == 2
    finally:
        binding.set_one_launch(prev)
    # the workspace covers the one-launch path: per slice G = ceil(N / 128)
    # partial records, one total and 2 G stamps of 8 bytes (each part
    # 256-byte aligned); the N = 4096, B*H = 16, d = 32 shape qualifies
    rec = 2 * 32 * 33 * 4
    al = lambda x: (x + 255) // 256 * 256
    need = al(16 * 32 * rec) + al(16 * rec) + al(16 * 32 * 2 * 8)
    assert binding.workspace_bytes(8, 2, 4096, 32, 2, 0) >= need
