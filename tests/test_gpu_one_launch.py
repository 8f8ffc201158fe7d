"""The one-launch path for short non-causal slices (k_band_fused): the slice's
workgroups exchange partial far-field states through memory instead of three
dependent launches.

Checked here, through the C ABI: the output against the float64 oracle on
shapes that take the path (several tiles and ragged tails, one-tile slices,
both head widths and band classes, both ranks), that it really is one launch
(the kernel timer counts one apply and no state kernels), that the exchange
gives the same bits as every workgroup forming its slice's state itself
(mode 2), that repeated calls give the same bits, and that the three-launch
path (mode 0) agrees within the tolerance."""

import numpy as np
import pytest
import torch

from fmm_testlib import TOL, floored_mean_rel_error, log, slice_errors, upload
from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu

# (B, H, N, d, band_k, rank): B*H a multiple of 8, N <= 64 tiles of 128 rows
SHAPES = [
    (8, 2, 4096, 32, 20, 2),   # the 4K retrieval shape: 32 tiles per slice
    (4, 2, 1000, 64, 64, 2),   # ragged tail, widest band, exact-fit interior tiles
    (8, 1, 100, 32, 5, 1),     # one tile per slice, shorter than the tile
    (2, 8, 2077, 64, 40, 1),   # ragged, band between the two classes
    (8, 1, 8192, 32, 32, 2),   # 64 tiles per slice, exact-fit band of one unit
    (16, 2, 257, 32, 3, 2),    # three tiles, the last with one row
]


def _mode(m):
    return binding.set_one_launch(m)


def _run(tq, tk, tv, twn, twf, kw, rank):
    out = binding.forward(tq, tk, tv, twn, twf, kw, rank, 0)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("shape", SHAPES, ids=[f"B{s[0]}H{s[1]}N{s[2]}d{s[3]}k{s[4]}r{s[5]}"
                                               for s in SHAPES])
def test_one_launch_matches_oracle(shape):
    B, H, N, d, kw, rank = shape
    seed = 500 + N % 97
    log(f"one-launch case B={B} H={H} N={N} d={d} k={kw} r={rank} bf16 seed={seed}")
    q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), seed)
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, "bf16")
    prev = _mode(1)
    try:
        for name in binding.KERNELS:
            binding.kernel_timing_read(name)
        binding.kernel_timing(True)
        got = _run(tq, tk, tv, twn, twf, kw, rank)
        binding.kernel_timing(False)
        counts = {n: binding.kernel_timing_read(n)[1] for n in binding.KERNELS}
        assert counts["band_apply"] == 1 and counts["seg_state"] == 0 \
            and counts["state_combine"] == 0, counts
        again = [_run(tq, tk, tv, twn, twf, kw, rank) for _ in range(3)]
        _mode(2)
        alone = _run(tq, tk, tv, twn, twf, kw, rank)
        _mode(0)
        three = _run(tq, tk, tv, twn, twf, kw, rank)
    finally:
        binding.kernel_timing(False)
        _mode(prev)
    for a in again:
        assert torch.equal(a.view(torch.int16), got.view(torch.int16))
    # the exchange and the workgroups' own sums give the same bits
    assert torch.equal(alone.view(torch.int16), got.view(torch.int16))
    want = ref.fmm_attention_stream(q, k, v, wn, wf, kw, rank, False)
    g = got.float().cpu().numpy().astype(np.float64)
    t = three.float().cpu().numpy().astype(np.float64)
    err = slice_errors(g, want).max()
    err3 = slice_errors(t, want).max()
    fm = floored_mean_rel_error(g, want)
    log(f"  one launch {err:.3e} (floored mean {fm:.3e}), three launches {err3:.3e}")
    assert err <= TOL["bf16"] and err3 <= TOL["bf16"]


def test_one_launch_not_taken_when_slices_straddle_xcds():
    # B*H = 6 is not a multiple of 8: the three-launch path runs
    B, H, N, d = 2, 3, 1024, 32
    q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 77)
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, "bf16")
    for name in binding.KERNELS:
        binding.kernel_timing_read(name)
    binding.kernel_timing(True)
    try:
        got = _run(tq, tk, tv, twn, twf, 9, 2)
    finally:
        binding.kernel_timing(False)
    assert binding.kernel_timing_read("seg_state")[1] == 1
    want = ref.fmm_attention_stream(q, k, v, wn, wf, 9, 2, False)
    err = slice_errors(got.float().cpu().numpy().astype(np.float64), want).max()
    assert err <= TOL["bf16"]


def test_one_launch_interleaved_shapes_share_workspace():
    # calls of different shapes on one stream reuse the library's workspace,
    # so each call's stamps sit where another call's records were; every
    # call must still match its own first result bit for bit
    cases = []
    for i, (B, H, N, d, kw, rank) in enumerate(SHAPES[:4]):
        q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 900 + i)
        t = upload(q, k, v, wn, wf, "bf16")
        cases.append((t, kw, rank))
    first = [_run(*t, kw, rank) for t, kw, rank in cases]
    for rep in range(3):
        for i, (t, kw, rank) in enumerate(reversed(cases)):
            j = len(cases) - 1 - i
            out = _run(*t, kw, rank)
            assert torch.equal(out.view(torch.int16), first[j].view(torch.int16)), (rep, j)
