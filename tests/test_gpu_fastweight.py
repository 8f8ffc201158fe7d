"""Parity of the fast-weight far field (fmm_attn_forward_fastweight, causal)
with the float64 oracle (oracle.fmm_ref.fmm_fast_weight_forward): the
language-model shape of the workloads (context 256, 8 heads of width 16)
and other widths, lengths and bands, with one and two far-field kernels."""

import numpy as np
import pytest
import torch

from fmm_testlib import TOL, log, slice_errors, upload
from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu


def check_fw(B, H, N, d, kw, n_linear, dtype, seed, std=1.0):
    q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, std, seed)
    beta = np.random.default_rng(seed + 7).uniform(0.0, 1.0, (B, H, N))
    log(f"fast weight B={B} H={H} N={N} d={d} k={kw} n_linear={n_linear} {dtype}")
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, dtype)
    tb = torch.from_numpy(beta.astype(np.float32)).to("cuda:0")
    got = binding.forward_fastweight(tq, tk, tv, tb, twn, twf, kw, n_linear)
    torch.cuda.synchronize()
    got = got.float().cpu().numpy().astype(np.float64)
    want = ref.fmm_fast_weight_forward(q, k, v, beta.astype(np.float32).astype(np.float64),
                                       wn, wf, kw, n_linear)
    assert np.isfinite(got).all()
    err = slice_errors(got, want).max()
    log(f"  max slice error {err:.3e}")
    assert err <= TOL[dtype]
    return err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_linear", [0, 1])
def test_fast_weight_lm_shape(n_linear, dtype):
    check_fw(16, 8, 256, 16, 20, n_linear, dtype, 4000 + n_linear)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
def test_fast_weight_widths(d, dtype):
    check_fw(2, 2, 700, d, 33, 1, dtype, 4100 + d, std=1.0 / np.sqrt(d))
    check_fw(1, 3, 65, d, 0, 0, dtype, 4200 + d)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [16, 32])
def test_fast_weight_short_and_ragged(d, dtype):
    # lengths below and between the steps the inputs are loaded ahead
    for i, n in enumerate((1, 2, 3, 5, 131)):
        check_fw(3, 2, n, d, 4, i % 2, dtype, 4300 + 10 * d + i)


# ------------------------------------------------------------------ backward

def check_fw_backward(B, H, N, d, kw, n_linear, dtype, seed, std=1.0):
    q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, std, seed)
    beta = np.random.default_rng(seed + 7).uniform(0.0, 1.0, (B, H, N)).astype(np.float32)
    g = make_inputs(B, H, N, d, dtype, 1.0, seed + 11)[0]
    log(f"fast weight backward B={B} H={H} N={N} d={d} k={kw} n_linear={n_linear} {dtype}")
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, dtype)
    tg = upload(g, g, g, wn, wf, dtype)[0]
    tb = torch.from_numpy(beta).to("cuda:0")
    got = binding.backward_fastweight(tq, tk, tv, tb, tg, twn, twf, kw, n_linear)
    torch.cuda.synchronize()
    got = [x.float().cpu().numpy().astype(np.float64) for x in got]
    want = ref.fmm_fast_weight_backward(q, k, v, beta.astype(np.float64), wn, wf, g, kw,
                                        n_linear)
    errs = {}
    # each slice's error against its largest gradient of q, k and v together:
    # with one position the output does not depend on q (fw_0 = beta_0 v_0),
    # so dq is zero up to rounding and cannot be its own scale
    scale = np.maximum.reduce([np.abs(x).max(axis=(-2, -1)) for x in want[:3]])
    for name, a, b in zip(("dq", "dk", "dv"), got[:3], want[:3]):
        assert np.isfinite(a).all(), f"non-finite {name}"
        errs[name] = (np.abs(a - b).max(axis=(-2, -1)) / np.maximum(scale, 1e-30)).max()
    # dbeta per slice against the slice's largest magnitude
    db_num = np.abs(got[3] - want[3]).max(axis=-1)
    errs["dbeta"] = (db_num / np.maximum(np.abs(want[3]).max(axis=-1), 1e-30)).max()
    # dw: against the absolute sums of the terms that form them
    a, c = ref.sigmoid(wn), ref.sigmoid(wf)
    near = ref.near_stream(q, k, v, kw, True)
    far = ref.fast_weight_stream(q, k, v, beta.astype(np.float64))
    if n_linear:
        far = far + ref.far_stream(q, k, v, 1, True)
    sn = a * (1 - a) * np.einsum("bhic,bhic->h", np.abs(g), np.abs(near))
    sf = c * (1 - c) * np.einsum("bhic,bhic->h", np.abs(g), np.abs(far))
    errs["dw_near"] = (np.abs(got[4] - want[4]) / np.maximum(sn, 1e-30)).max()
    errs["dw_far"] = (np.abs(got[5] - want[5]) / np.maximum(sf, 1e-30)).max()
    log("  " + " ".join(f"{kk} {vv:.2e}" for kk, vv in errs.items()))
    for kk, vv in errs.items():
        assert vv <= TOL[dtype], (kk, vv)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_linear", [0, 1])
def test_fast_weight_backward_lm_shape(n_linear, dtype):
    # the language-model shape with fewer slices (the oracle's recurrence is a
    # Python loop)
    check_fw_backward(2, 4, 256, 16, 20, n_linear, dtype, 4300 + n_linear)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
def test_fast_weight_backward_widths(d, dtype):
    check_fw_backward(1, 2, 150, d, 17, 1, dtype, 4400 + d, std=1.0 / np.sqrt(d))
    check_fw_backward(2, 1, 40, d, 0, 0, dtype, 4500 + d)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fast_weight_backward_short_and_many_slices(dtype):
    # one and two positions (the recurrence's first steps alone), and many
    # slices at once
    check_fw_backward(1, 1, 1, 16, 0, 0, dtype, 4600)
    check_fw_backward(3, 2, 2, 64, 5, 1, dtype, 4610)
    check_fw_backward(8, 8, 33, 32, 8, 1, dtype, 4620)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fast_weight_backward_narrow_lengths(dtype):
    # d = 16 (four lanes per row of W): lengths below, at and between the
    # steps the inputs are loaded ahead
    for i, n in enumerate((2, 3, 4, 5, 9, 130)):
        check_fw_backward(2, 3, n, 16, 3, i % 2, dtype, 4700 + i)
