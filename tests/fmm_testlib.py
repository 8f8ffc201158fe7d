"""Shared helpers for the GPU tests: upload seeded inputs, run the HIP path,
compare with the float64 oracle."""

from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

TOL = {"f32": 1e-4, "bf16": 2e-2}
TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def upload(q, k, v, wn, wf, dtype: str, device="cuda:0"):
    dt = TORCH_DT[dtype]
    t = [torch.from_numpy(np.asarray(x, dtype=np.float32)).to(device).to(dt).contiguous()
         for x in (q, k, v)]
    w = [torch.from_numpy(np.asarray(x, dtype=np.float32)).to(device) for x in (wn, wf)]
    return t[0], t[1], t[2], w[0], w[1]


def run_gpu(q, k, v, wn, wf, band_k, rank, causal, dtype):
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, dtype)
    out = binding.forward(tq, tk, tv, twn, twf, band_k, rank, causal)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


def slice_errors(got: np.ndarray, want: np.ndarray) -> np.ndarray:
    """max|g - o| / max|o| for every (b, h) slice."""
    num = np.abs(got - want).max(axis=(-2, -1))
    den = np.abs(want).max(axis=(-2, -1))
    return num / np.maximum(den, 1e-30)


def floored_mean_rel_error(got: np.ndarray, want: np.ndarray) -> float:
    """Mean over all elements of |g - o| / max(|o|, 1e-3 max|o|), the floor
    taken per (b, h) slice: an elementwise measure that the max-normalised
    slice error can hide on small outputs."""
    floor = 1e-3 * np.abs(want).max(axis=(-2, -1), keepdims=True)
    return float((np.abs(got - want) / np.maximum(np.abs(want), np.maximum(floor, 1e-30))).mean())


def check_full(B, H, N, d, band_k, rank, causal, dtype, seed, std=1.0, wn=None, wf=None):
    q, k, v, wn0, wf0 = make_inputs(B, H, N, d, dtype, std, seed)
    wn = wn0 if wn is None else wn
    wf = wf0 if wf is None else wf
    log(f"case B={B} H={H} N={N} d={d} k={band_k} r={rank} causal={int(causal)} "
        f"dtype={dtype} seed={seed}")
    got = run_gpu(q, k, v, wn, wf, band_k, rank, causal, dtype)
    want = ref.fmm_attention_stream(q, k, v, wn, wf, band_k, rank, bool(causal))
    assert np.isfinite(got).all(), "non-finite GPU output"
    err = slice_errors(got, want).max()
    log(f"  max slice error {err:.3e}, floored mean relative error "
        f"{floored_mean_rel_error(got, want):.3e}")
    assert err <= TOL[dtype], f"max slice error {err:.3e} > {TOL[dtype]}"
    return err
