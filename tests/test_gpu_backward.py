"""Parity of the backward pass (fmm_attn_backward) with the float64 oracle's
gradients (oracle.fmm_ref.fmm_attention_backward_stream), through the C ABI.

dq, dk, dv: the worst (batch, head) slice of max|g - o| / max|o| within the
forward's tolerance (1e-4 fp32, 2e-2 bf16).  dw_near, dw_far are sums over
B N d products with cancellation, so each is held to the tolerance times the
sum of the absolute values of its terms (sigma' sum |dout . part| per head)."""

import numpy as np
import pytest
import torch

from fmm_testlib import TOL, log, slice_errors, upload
from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs, to_dtype

pytestmark = pytest.mark.gpu


def check_backward(B, H, N, d, kw, rank, causal, dtype, seed, std=1.0, shift=0.0, joint=False):
    q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, std, seed)
    if shift:
        q, k = to_dtype(q + shift, dtype), to_dtype(k + shift, dtype)
    g = to_dtype(np.random.default_rng(seed + 1).standard_normal(q.shape), dtype)
    log(f"backward B={B} H={H} N={N} d={d} k={kw} r={rank} causal={causal} {dtype} "
        f"joint={joint} seed={seed}")
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, dtype)
    tg = torch.from_numpy(np.asarray(g, dtype=np.float32)).to("cuda:0").to(tq.dtype)
    norm = "joint" if joint else "map"
    got = binding.backward(tq, tk, tv, tg, twn, twf, kw, rank, causal, joint=joint)
    torch.cuda.synchronize()
    got = [x.float().cpu().numpy().astype(np.float64) for x in got]
    want = ref.fmm_attention_backward_stream(q, k, v, wn, wf, g, kw, rank, bool(causal),
                                             norm=norm)
    errs = []
    for name, a, b in zip(("dq", "dk", "dv"), got[:3], want[:3]):
        assert np.isfinite(a).all(), f"non-finite {name}"
        errs.append(slice_errors(a, b).max())
    # dw: scale by the absolute sums of the terms
    near = ref.near_stream(q, k, v, kw, bool(causal))
    far = ref.far_stream(q, k, v, rank, bool(causal), norm=norm)
    sa, sc = ref.sigmoid(wn), ref.sigmoid(wf)
    scale_n = sa * (1 - sa) * np.einsum("bhic,bhic->h", np.abs(g), np.abs(near))
    scale_f = sc * (1 - sc) * np.einsum("bhic,bhic->h", np.abs(g), np.abs(far))
    e_wn = (np.abs(got[3] - want[3]) / np.maximum(scale_n, 1e-30)).max()
    e_wf = (np.abs(got[4] - want[4]) / np.maximum(scale_f, 1e-30)).max()
    log(f"  dq {errs[0]:.2e} dk {errs[1]:.2e} dv {errs[2]:.2e} dw_near {e_wn:.2e} "
        f"dw_far {e_wf:.2e}")
    tol = TOL[dtype]
    assert max(errs) <= tol, errs
    assert e_wn <= tol and e_wf <= tol
    return max(errs + [e_wn, e_wf])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
@pytest.mark.parametrize("d", [16, 32, 64, 128])
def test_backward_widths(d, causal, dtype):
    worst = 0.0
    for B, H, N, kw, rank in ((1, 2, 300, 5, 2), (2, 1, 777, 20, 1), (1, 1, 1500, 64, 2),
                              (1, 2, 64, 0, 2), (1, 1, 33, 40, 2)):
        worst = max(worst, check_backward(B, H, N, d, kw, rank, causal, dtype,
                                          2000 + d + N + kw, std=1.0 / np.sqrt(d) * 2))
    log(f"backward d={d} causal={causal} {dtype}: worst {worst:.2e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
def test_backward_wide_band_and_rank3(causal, dtype):
    # a band wider than one staging round, and the third feature map with
    # shifted inputs (tanh's denominator away from zero)
    check_backward(1, 2, 1200, 32, 300, 2, causal, dtype, 2100 + causal)
    check_backward(2, 1, 900, 64, 30, 3, causal, dtype, 2200 + causal, shift=1.0)
    check_backward(1, 1, 700, 128, 40, 3, causal, dtype, 2250 + causal, shift=1.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
def test_backward_joint_normalisation(causal, dtype):
    # the far maps normalised as one matrix (Sec. 1.2): every width, one to
    # three maps, several segments and staging rounds
    worst = 0.0
    for B, H, N, d, kw, rank in ((1, 2, 700, 32, 20, 2), (2, 1, 900, 64, 40, 3),
                                 (1, 1, 500, 128, 16, 2), (1, 2, 300, 16, 5, 1),
                                 (1, 1, 1500, 64, 64, 2)):
        worst = max(worst, check_backward(B, H, N, d, kw, rank, causal, dtype,
                                          2500 + d + N + causal, std=1.0 / np.sqrt(d) * 2,
                                          joint=True))
    log(f"joint backward causal={causal} {dtype}: worst {worst:.2e}")


@pytest.mark.parametrize("causal", [0, 1])
def test_backward_benchmark_shape_slices(causal):
    # the N = 4096 retrieval shape (B = 8, H = 2, d = 32, k = 20, bf16)
    check_backward(2, 2, 4096, 32, 20, 2, causal, "bf16", 2300 + causal)


@pytest.mark.parametrize("causal", [0, 1])
def test_backward_fp32_d128_several_segments(causal):
    # fp32 at d = 128 (its own translation unit): several state segments and
    # staging rounds per slice, a ragged tail
    check_backward(1, 2, 2500, 128, 64, 2, causal, "f32", 2400 + causal, std=0.18)
