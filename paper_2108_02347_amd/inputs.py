"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module draws random numbers and rounds them to the storage dtype; it holds
none of the operator's arithmetic.  Both the GPU path and the float64 oracle are
fed the arrays it returns, so the oracle always sees exactly the values the GPU
reads (bf16 values are exactly representable in float64).

Recipe (one numpy PCG64 generator per call, seeded):
  q, k, v = std * standard_normal((B, H, N, d))    drawn in this order
  w_near, w_far = standard_normal(H)               raw per-head blend logits
then q, k, v are rounded to the storage dtype: float64 -> float32 by
round-to-nearest-even, and for bf16 float32 -> bf16 by round-to-nearest-even.

The named workloads stand in for the paper's experiments (Sec. 4): the
long-range classification shapes (1K and 4K tokens, 2 heads of width 32), the
language-model shape (context 256, 8 heads of width 16, causal) and the
2^16-token length of the complexity study.  No dataset is read: values are
i.i.d. normal, which is what the attention operator sees after random
projections.
"""

from __future__ import annotations

import dataclasses

import numpy as np

__all__ = ["Workload", "WORKLOADS", "round_to_bf16", "make_inputs", "to_dtype"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    d: int
    band_k: int
    rank: int
    causal: tuple          # causal flags the workload is run with
    dtypes: tuple          # storage dtypes the workload is run with
    std: float             # standard deviation of q, k, v
    seed: int
    about: str


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 512, 32, 5, 1, (0,), ("f32",), 1.0, 1,
                     "tiny non-causal parity case, rank 1"),
    "lra1k": Workload("lra1k", 32, 2, 1024, 32, 20, 2, (0,), ("f32", "bf16"), 1.0, 2,
                      "long-range classification, 1K tokens, 2 heads x 32"),
    "lra4k": Workload("lra4k", 8, 2, 4096, 32, 20, 2, (0,), ("bf16",), 1.0, 3,
                      "long-range retrieval length, 4K tokens, 2 heads x 32"),
    "lm256": Workload("lm256", 16, 8, 256, 16, 20, 2, (1,), ("f32",), 1.0, 4,
                      "causal language model, context 256, 8 heads x 16"),
    "stress64k": Workload("stress64k", 1, 8, 65536, 64, 64, 2, (0, 1), ("bf16",),
                          1.0 / 8.0, 5,
                          "2^16 tokens, 8 heads x 64, std 1/sqrt(64)"),
}


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even), returned as float32.

    The input is first rounded to float32 (numpy's cast is round-to-nearest-
    even); the low 16 bits of the float32 pattern are then rounded away."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x32)):
        raise ValueError("round_to_bf16 expects finite values")
    bits = x32.view(np.uint32).astype(np.uint64)
    bias = 0x7FFF + ((bits >> 16) & 1)
    bits = ((bits + bias) & 0xFFFF0000).astype(np.uint32)
    return bits.view(np.float32)


def to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 data to the storage dtype; returns float64 holding the
    exactly rounded values."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_to_bf16(x).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def make_inputs(B: int, H: int, N: int, d: int, dtype: str = "f32",
                std: float = 1.0, seed: int = 0):
    """Return (q, k, v, w_near, w_far) as float64 arrays.

    q, k, v have shape [B, H, N, d] and hold values exactly representable in
    `dtype`; w_near and w_far have shape [H]."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, N, d)) * std
    k = rng.standard_normal((B, H, N, d)) * std
    v = rng.standard_normal((B, H, N, d)) * std
    w_near = rng.standard_normal(H)
    w_far = rng.standard_normal(H)
    return (to_dtype(q, dtype), to_dtype(k, dtype), to_dtype(v, dtype),
            w_near, w_far)


def workload_inputs(name: str, dtype: str | None = None):
    """make_inputs for a named workload (its own seed and scale)."""
    w = WORKLOADS[name]
    return make_inputs(w.B, w.H, w.N, w.d, dtype or w.dtypes[0], w.std, w.seed)
