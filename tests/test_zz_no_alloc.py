"""The no-allocation entry point (fmm_attn_forward_noalloc) against the
entry points with a library-owned workspace: same kernels, same segment plan,
so the outputs must be identical bit for bit.  Two calls in a row share the
per-GPU array; the second is smaller, so stale records of the first call sit
beyond the second's and must not be read."""

import numpy as np
import pytest
import torch

from fmm_testlib import TOL, log, upload
from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
def test_noalloc_matches_owned_workspace(dtype, causal):
    shapes = [(2, 4, 3000, 64, 40, 2), (1, 2, 700, 32, 9, 1)]  # second call smaller
    for i, (B, H, N, d, kw, rank) in enumerate(shapes):
        log(f"noalloc call {i}: B={B} H={H} N={N} d={d} k={kw} r={rank} causal={causal} "
            f"{dtype}")
        q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, 1.0 / np.sqrt(d), 300 + i + causal)
        tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, dtype)
        assert binding.workspace_bytes(B, H, N, d, rank, causal) <= binding.noalloc_max_bytes()
        out = torch.empty_like(tq)
        got = binding.forward_noalloc(tq, tk, tv, twn, twf, kw, rank, causal, out=out)
        want = binding.forward(tq, tk, tv, twn, twf, kw, rank, causal)
        torch.cuda.synchronize()
        assert got.data_ptr() == out.data_ptr()
        bits = torch.int16 if dtype == "bf16" else torch.int32
        assert torch.equal(got.view(bits), want.view(bits))
        if i == 1:
            exp = ref.fmm_attention_stream(q, k, v, wn, wf, kw, rank, bool(causal))
            g = got.double().cpu().numpy()
            err = (np.abs(g - exp).max(axis=(2, 3)) / np.abs(exp).max(axis=(2, 3))).max()
            assert err <= TOL[dtype]


def test_noalloc_rejects_oversize_shape():
    # 1024 heads of width 64 need more segment records than the array
    B, H, N, d = 1, 1024, 64, 64
    assert binding.workspace_bytes(B, H, N, d, 2, 1) > binding.noalloc_max_bytes()
    t = [torch.zeros(B, H, N, d, dtype=torch.bfloat16, device="cuda:0") for _ in range(3)]
    out = torch.full_like(t[0], 2.0)
    w = torch.zeros(H, device="cuda:0")
    with pytest.raises(binding.FmmError) as ei:
        binding.forward_noalloc(t[0], t[1], t[2], w, w, 64, 2, 1, out=out)
    assert ei.value.status == binding.FMM_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool((out == 2.0).all())
