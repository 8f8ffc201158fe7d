"""Float64 CPU oracle for the FMMformer attention forward operator.

TEST INFRASTRUCTURE ONLY.  This module exists to check the HIP kernels; it is
not part of the product path.  Only the test suite, the package smoke check and
the CPU-baseline leg of the benchmark may import it.  It shares no code with the
GPU library and imports nothing from it.

What it computes (FMMformer, arXiv 2108.02347):

  near field, Sec. 3.1, Eq. (3):
      D = softmax(band_k(Q K^T / sqrt(d)))
      Entries outside the band are excluded from the softmax (they are -inf
      before normalisation), and each row of D sums to one.  The band of row i
      is J(i) = [i-k, i+k] clipped to [0, N-1]; causal: [i-k, i].
  far field, Sec. 3.2.1, Eq. (7)-(9):
      far_i = sum_l  phi_l(q_i)^T S_l(i) / phi_l(q_i)^T z_l(i)
      S_l(i) = sum_{j in F(i)} phi_l(k_j) v_j^T,   z_l(i) = sum_{j in F(i)} phi_l(k_j)
      F(i) = [0, N-1]; causal: [0, i] (the sum truncated at i, Sec. 3.2.1).
  feature maps, Sec. 3.2.1 "Feature map selection":
      phi_1(x) = elu(x) + 1,  phi_2(x) = elu(-x) + 1  (elementwise, elu with alpha 1)
  blend, Sec. 3.3, Eq. (11):
      out = sigmoid(w_near[h]) * near + sigmoid(w_far[h]) * far

Readings where the paper leaves room (each is listed with its reason in the
design notes): "bandwidth k" is a half-width; band rows are truncated at the
sequence ends; the causal band and the causal far sum both include j = i; each
feature map is normalised on its own as Eq. (9) writes it; the far sum runs over
all of F(i) (the band is not excluded); there is no epsilon in the far
denominator; the 1/sqrt(d) scale applies to the near field only; the blend
weights are raw per-head logits passed through a sigmoid.

Three forms, all float64:
  * dense:     builds the N x N matrices of the definitions (tiny N only);
  * stream:    the same values through associativity (Eq. (5)) and an explicit
               running prefix sum for the causal far field; any N;
  * rows:      the stream form evaluated at a chosen set of rows of one
               (batch, head) slice, for spot checks at full problem sizes.

Parity pins: every function here is checked by the CPU test suite against
closed forms, library routines (torch's scaled_dot_product_attention in
float64), brute-force scalar loops and invariants; see tests/test_oracle_pins.py.
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "phi",
    "sigmoid",
    "band_mask",
    "near_dense",
    "far_dense",
    "fmm_attention_dense",
    "near_stream",
    "far_stream",
    "fmm_attention_stream",
    "fmm_attention_rows",
]


# ---------------------------------------------------------------- primitives

def _elu(x: np.ndarray) -> np.ndarray:
    """elu with alpha = 1: x for x > 0, exp(x) - 1 otherwise."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x, np.expm1(np.minimum(x, 0.0)))


def phi(x: np.ndarray, l: int) -> np.ndarray:
    """Feature map phi_l (Sec. 3.2.1): l = 1 -> elu(x)+1, l = 2 -> elu(-x)+1."""
    if l == 1:
        return _elu(x) + 1.0
    if l == 2:
        return _elu(-np.asarray(x, dtype=np.float64)) + 1.0
    raise ValueError(f"feature map {l} is not defined for this operator (rank 1 or 2)")


def sigmoid(w: np.ndarray) -> np.ndarray:
    """Logistic function used to keep the blend weights positive (Eq. (11))."""
    w = np.asarray(w, dtype=np.float64)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-w))


def band_mask(n: int, band_k: int, causal: bool) -> np.ndarray:
    """Boolean N x N mask of the near-field band (Eq. (3)); True = kept."""
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    if causal:
        return (j <= i) & (j >= i - band_k)
    return np.abs(i - j) <= band_k


def _check(q, k, v):
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if q.ndim != 4 or q.shape != k.shape or q.shape != v.shape:
        raise ValueError("q, k, v must share one shape [B, H, N, d]")
    return q, k, v


# ---------------------------------------------------------------- dense form

def near_dense(q, k, v, band_k: int, causal: bool) -> np.ndarray:
    """Near field, Eq. (3), with the full N x N score matrix masked to the band."""
    q, k, v = _check(q, k, v)
    _, _, n, d = q.shape
    keep = band_mask(n, band_k, causal)
    s = np.einsum("bhic,bhjc->bhij", q, k) / math.sqrt(d)
    s = np.where(keep, s, -np.inf)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.einsum("bhij,bhjc->bhic", p, v)


def far_dense(q, k, v, rank: int, causal: bool) -> np.ndarray:
    """Far field, Eq. (8)-(9): for each map the explicit N x N matrix
    phi_l(Q) phi_l(K)^T (lower triangle only when causal), each row divided by
    its own sum, applied to V; the r results are added."""
    q, k, v = _check(q, k, v)
    n = q.shape[2]
    out = np.zeros_like(v)
    lower = np.tril(np.ones((n, n), dtype=bool))
    for l in range(1, rank + 1):
        a = np.einsum("bhic,bhjc->bhij", phi(q, l), phi(k, l))
        if causal:
            a = np.where(lower, a, 0.0)
        w = a / a.sum(axis=-1, keepdims=True)
        out += np.einsum("bhij,bhjc->bhic", w, v)
    return out


def _blend(near, far, w_near, w_far):
    a = sigmoid(w_near)[None, :, None, None]
    b = sigmoid(w_far)[None, :, None, None]
    # sigmoid(-inf) = 0 must remove its part exactly, also when that part is
    # not finite, so multiply only where the weight is non-zero.
    return np.where(a > 0, a * near, 0.0) + np.where(b > 0, b * far, 0.0)


def fmm_attention_dense(q, k, v, w_near, w_far, band_k: int, rank: int,
                        causal: bool) -> np.ndarray:
    """out = sigmoid(w_near) D V + sigmoid(w_far) L V (Eq. (9), Eq. (11))."""
    return _blend(near_dense(q, k, v, band_k, causal),
                  far_dense(q, k, v, rank, causal), w_near, w_far)


# ---------------------------------------------------------------- stream form

def near_stream(q, k, v, band_k: int, causal: bool, row_chunk: int = 16384) -> np.ndarray:
    """Near field, Eq. (3), computing only the band entries: for every offset
    o = j - i in the band, score[i, o] = q_i . k_{i+o} / sqrt(d); offsets that
    fall outside [0, N-1] are excluded; softmax over the offsets; weighted sum
    of the rows v_{i+o}."""
    q, k, v = _check(q, k, v)
    b_, h_, n, d = q.shape
    kk = min(band_k, n - 1)
    offs = np.arange(-kk, 1 if causal else kk + 1)
    scale = 1.0 / math.sqrt(d)
    out = np.empty_like(v)
    for i0 in range(0, n, row_chunk):
        i1 = min(n, i0 + row_chunk)
        rows = np.arange(i0, i1)
        score = np.full((b_, h_, i1 - i0, len(offs)), -np.inf)
        for t, o in enumerate(offs):
            j = rows + o
            ok = (j >= 0) & (j < n)
            if not ok.any():
                continue
            score[:, :, ok, t] = np.einsum("bhic,bhic->bhi", q[:, :, rows[ok]],
                                           k[:, :, j[ok]]) * scale
        score = score - score.max(axis=-1, keepdims=True)
        p = np.exp(score)
        p = p / p.sum(axis=-1, keepdims=True)
        acc = np.zeros((b_, h_, i1 - i0, d))
        for t, o in enumerate(offs):
            j = rows + o
            ok = (j >= 0) & (j < n)
            if not ok.any():
                continue
            acc[:, :, ok] += p[:, :, ok, t, None] * v[:, :, j[ok]]
        out[:, :, i0:i1] = acc
    return out


def far_stream(q, k, v, rank: int, causal: bool, row_chunk: int = 512) -> np.ndarray:
    """Far field through associativity (Eq. (5), Eq. (7)).

    Non-causal: S_l = phi_l(K)^T V and z_l = phi_l(K)^T 1 once per slice, then
    far_i = sum_l phi_l(q_i)^T S_l / phi_l(q_i)^T z_l.
    Causal: the sums are truncated at i (Sec. 3.2.1); the running sums
    S_l(i), z_l(i) are formed as explicit cumulative sums of the outer products
    phi_l(k_j) v_j^T, carried from one row block to the next."""
    q, k, v = _check(q, k, v)
    b_, h_, n, d = q.shape
    out = np.zeros_like(v)
    for l in range(1, rank + 1):
        pq = phi(q, l)
        pk = phi(k, l)
        if not causal:
            s = np.einsum("bhjc,bhje->bhce", pk, v)
            z = pk.sum(axis=2)
            num = np.einsum("bhic,bhce->bhie", pq, s)
            den = np.einsum("bhic,bhc->bhi", pq, z)
            out += num / den[..., None]
            continue
        s_run = np.zeros((b_, h_, d, d))
        z_run = np.zeros((b_, h_, d))
        for i0 in range(0, n, row_chunk):
            i1 = min(n, i0 + row_chunk)
            outer = pk[:, :, i0:i1, :, None] * v[:, :, i0:i1, None, :]
            s_cum = s_run[:, :, None] + np.cumsum(outer, axis=2)
            z_cum = z_run[:, :, None] + np.cumsum(pk[:, :, i0:i1], axis=2)
            num = np.einsum("bhic,bhice->bhie", pq[:, :, i0:i1], s_cum)
            den = np.einsum("bhic,bhic->bhi", pq[:, :, i0:i1], z_cum)
            out[:, :, i0:i1] += num / den[..., None]
            s_run = s_cum[:, :, -1]
            z_run = z_cum[:, :, -1]
    return out


def fmm_attention_stream(q, k, v, w_near, w_far, band_k: int, rank: int,
                         causal: bool) -> np.ndarray:
    """Same operator as fmm_attention_dense, any N."""
    return _blend(near_stream(q, k, v, band_k, causal),
                  far_stream(q, k, v, rank, causal), w_near, w_far)


# ---------------------------------------------------------------- sampled rows

def fmm_attention_rows(q, k, v, w_near, w_far, band_k: int, rank: int,
                       causal: bool, b: int, h: int, rows) -> np.ndarray:
    """The operator's output at the given rows of slice (b, h) only.

    q, k, v: [B, H, N, d]; returns [len(rows), d] in the order of `rows`.
    Used to check full-size problems where the whole output would take the
    oracle too long; the far-field state is still summed over the whole
    support F(i) of every requested row."""
    q, k, v = _check(q, k, v)
    n, d = q.shape[2], q.shape[3]
    rows = np.asarray(rows, dtype=np.int64)
    if rows.size and (rows.min() < 0 or rows.max() >= n):
        raise ValueError("row index out of range")
    qs, ks, vs = q[b, h], k[b, h], v[b, h]
    scale = 1.0 / math.sqrt(d)
    near = np.empty((rows.size, d))
    for t, i in enumerate(rows):
        lo = max(0, i - band_k)
        hi = i if causal else min(n - 1, i + band_k)
        sc = ks[lo:hi + 1] @ qs[i] * scale
        p = np.exp(sc - sc.max())
        near[t] = (p / p.sum()) @ vs[lo:hi + 1]
    far = np.zeros((rows.size, d))
    for l in range(1, rank + 1):
        pq = phi(qs[rows], l)
        pk = phi(ks, l)
        if not causal:
            s = pk.T @ vs
            z = pk.sum(axis=0)
            far += (pq @ s) / (pq @ z)[:, None]
            continue
        order = np.argsort(rows, kind="stable")
        s_run = np.zeros((d, d))
        z_run = np.zeros(d)
        done = 0  # rows [0, done) are already in the running sums
        for t in order:
            i = int(rows[t])
            if i + 1 > done:
                s_run = s_run + pk[done:i + 1].T @ vs[done:i + 1]
                z_run = z_run + pk[done:i + 1].sum(axis=0)
                done = i + 1
            far[t] += (pq[t] @ s_run) / (pq[t] @ z_run)
    a = float(sigmoid(w_near[h]))
    c = float(sigmoid(w_far[h]))
    out = np.zeros((rows.size, d))
    if a > 0:
        out += a * near
    if c > 0:
        out += c * far
    return out
