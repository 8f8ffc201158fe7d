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
      phi_3(x) = tanh(x)      (the third map of the rank-3 far field, Sec. 4.1)
  blend, Sec. 3.3, Eq. (11):
      out = sigmoid(w_near[h]) * near + sigmoid(w_far[h]) * far

Readings where the paper leaves room (each is listed with its reason in the
design notes): "bandwidth k" is a half-width; band rows are truncated at the
sequence ends; the causal band and the causal far sum both include j = i; each
feature map is normalised on its own as Eq. (9) writes it; the far sum runs over
all of F(i) (the band is not excluded); there is no epsilon in the far
denominator; the 1/sqrt(d) scale applies to the near field only; the blend
weights are raw per-head logits passed through a sigmoid.

Far-field normalisation.  norm="map" (the default) divides each map by its
own denominator, as Eq. (9) writes the sum of fractions.  norm="joint" divides
the sum of the maps' numerators by the sum of their denominators, i.e. it
normalises the rows of L = sum_l phi_l(Q) phi_l(K)^T as one matrix, the reading
of the introduction's remark that rows are normalised to sum to one (Sec. 1.2).
For rank 1 the two agree.  There is no epsilon: phi_3 = tanh can make a
denominator zero or negative, and the division is then carried out as IEEE
arithmetic gives it (no clamping).

Backward (gradients of a scalar loss L through dL/dout), written out from the
definitions above: the banded softmax of Eq. (3) (softmax derivative
p (dp - sum p dp)), the fractions of Eq. (9) (quotient rule, with the causal
sums of Eq. (7) truncated at i, so the key-side gradients become suffix sums
over the rows i >= j), the feature-map derivatives and the sigmoid of
Eq. (11) (sigma' = sigma (1 - sigma)).

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
    "phi_grad",
    "sigmoid",
    "band_mask",
    "near_dense",
    "far_dense",
    "fmm_attention_dense",
    "near_stream",
    "far_stream",
    "fmm_attention_stream",
    "fmm_attention_rows",
    "far_terms_stream",
    "fmm_attention_backward_stream",
    "fmm_layer_forward",
    "fast_weight_stream",
    "fmm_fast_weight_forward",
]


# ---------------------------------------------------------------- primitives

def _elu(x: np.ndarray) -> np.ndarray:
    """elu with alpha = 1: x for x > 0, exp(x) - 1 otherwise."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x, np.expm1(np.minimum(x, 0.0)))


def phi(x: np.ndarray, l: int) -> np.ndarray:
    """Feature map phi_l (Sec. 3.2.1): l = 1 -> elu(x)+1, l = 2 -> elu(-x)+1,
    l = 3 -> tanh(x)."""
    if l == 1:
        return _elu(x) + 1.0
    if l == 2:
        return _elu(-np.asarray(x, dtype=np.float64)) + 1.0
    if l == 3:
        return np.tanh(np.asarray(x, dtype=np.float64))
    raise ValueError(f"feature map {l} is not defined for this operator (rank 1 to 3)")


def phi_grad(x: np.ndarray, l: int) -> np.ndarray:
    """d phi_l / dx elementwise: elu'(x) = 1 for x > 0 and exp(x) otherwise, so
    phi_1' = elu'(x), phi_2' = -elu'(-x), phi_3' = 1 - tanh(x)^2."""
    x = np.asarray(x, dtype=np.float64)
    if l == 1:
        return np.where(x > 0.0, 1.0, np.exp(np.minimum(x, 0.0)))
    if l == 2:
        return -np.where(-x > 0.0, 1.0, np.exp(np.minimum(-x, 0.0)))
    if l == 3:
        return 1.0 - np.tanh(x) ** 2
    raise ValueError(f"feature map {l} is not defined for this operator (rank 1 to 3)")


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


def far_dense(q, k, v, rank: int, causal: bool, norm: str = "map") -> np.ndarray:
    """Far field, Eq. (8)-(9): for each map the explicit N x N matrix
    phi_l(Q) phi_l(K)^T (lower triangle only when causal), each row divided by
    its own sum, applied to V; the r results are added.  norm="joint": the r
    matrices are added first and the rows of the sum are divided by their
    sums."""
    q, k, v = _check(q, k, v)
    _check_norm(norm)
    n = q.shape[2]
    out = np.zeros_like(v)
    lower = np.tril(np.ones((n, n), dtype=bool))
    total = np.zeros(q.shape[:2] + (n, n))
    for l in range(1, rank + 1):
        a = np.einsum("bhic,bhjc->bhij", phi(q, l), phi(k, l))
        if causal:
            a = np.where(lower, a, 0.0)
        if norm == "joint":
            total += a
            continue
        w = a / a.sum(axis=-1, keepdims=True)
        out += np.einsum("bhij,bhjc->bhic", w, v)
    if norm == "joint":
        out = np.einsum("bhij,bhjc->bhic", total / total.sum(axis=-1, keepdims=True), v)
    return out


def _check_norm(norm: str) -> None:
    if norm not in ("map", "joint"):
        raise ValueError(f"unknown far-field normalisation {norm!r}")


def _blend(near, far, w_near, w_far):
    a = sigmoid(w_near)[None, :, None, None]
    b = sigmoid(w_far)[None, :, None, None]
    # sigmoid(-inf) = 0 must remove its part exactly, also when that part is
    # not finite, so multiply only where the weight is non-zero.
    return np.where(a > 0, a * near, 0.0) + np.where(b > 0, b * far, 0.0)


def fmm_attention_dense(q, k, v, w_near, w_far, band_k: int, rank: int,
                        causal: bool, norm: str = "map") -> np.ndarray:
    """out = sigmoid(w_near) D V + sigmoid(w_far) L V (Eq. (9), Eq. (11))."""
    return _blend(near_dense(q, k, v, band_k, causal),
                  far_dense(q, k, v, rank, causal, norm), w_near, w_far)


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


def far_terms_stream(q, k, v, rank: int, causal: bool, row_chunk: int = 512):
    """Numerator and denominator of every map of the far field (Eq. (7)-(9)),
    through associativity (Eq. (5)): a list over l = 1..rank of
    (num_l [B,H,N,d], den_l [B,H,N]) with num_l,i = phi_l(q_i)^T S_l(i) and
    den_l,i = phi_l(q_i)^T z_l(i).

    Non-causal: S_l = phi_l(K)^T V and z_l = phi_l(K)^T 1 once per slice.
    Causal: the sums are truncated at i (Sec. 3.2.1); the running sums
    S_l(i), z_l(i) are formed as explicit cumulative sums of the outer products
    phi_l(k_j) v_j^T, carried from one row block to the next."""
    q, k, v = _check(q, k, v)
    b_, h_, n, d = q.shape
    terms = []
    for l in range(1, rank + 1):
        pq = phi(q, l)
        pk = phi(k, l)
        if not causal:
            s = np.einsum("bhjc,bhje->bhce", pk, v)
            z = pk.sum(axis=2)
            num = np.einsum("bhic,bhce->bhie", pq, s)
            den = np.einsum("bhic,bhc->bhi", pq, z)
            terms.append((num, den))
            continue
        num = np.empty_like(v)
        den = np.empty((b_, h_, n))
        s_run = np.zeros((b_, h_, d, d))
        z_run = np.zeros((b_, h_, d))
        for i0 in range(0, n, row_chunk):
            i1 = min(n, i0 + row_chunk)
            outer = pk[:, :, i0:i1, :, None] * v[:, :, i0:i1, None, :]
            s_cum = s_run[:, :, None] + np.cumsum(outer, axis=2)
            z_cum = z_run[:, :, None] + np.cumsum(pk[:, :, i0:i1], axis=2)
            num[:, :, i0:i1] = np.einsum("bhic,bhice->bhie", pq[:, :, i0:i1], s_cum)
            den[:, :, i0:i1] = np.einsum("bhic,bhic->bhi", pq[:, :, i0:i1], z_cum)
            s_run = s_cum[:, :, -1]
            z_run = z_cum[:, :, -1]
        terms.append((num, den))
    return terms


def far_stream(q, k, v, rank: int, causal: bool, row_chunk: int = 512,
               norm: str = "map") -> np.ndarray:
    """Far field from the per-map terms: sum_l num_l / den_l (Eq. (9)), or
    (sum_l num_l) / (sum_l den_l) with norm="joint"."""
    _check_norm(norm)
    terms = far_terms_stream(q, k, v, rank, causal, row_chunk)
    if norm == "joint":
        num = sum(t[0] for t in terms)
        den = sum(t[1] for t in terms)
        return num / den[..., None]
    out = np.zeros_like(terms[0][0])
    for num, den in terms:
        out += num / den[..., None]
    return out


def fmm_attention_stream(q, k, v, w_near, w_far, band_k: int, rank: int,
                         causal: bool, norm: str = "map") -> np.ndarray:
    """Same operator as fmm_attention_dense, any N."""
    return _blend(near_stream(q, k, v, band_k, causal),
                  far_stream(q, k, v, rank, causal, norm=norm), w_near, w_far)


# ---------------------------------------------------------------- sampled rows

def fmm_attention_rows(q, k, v, w_near, w_far, band_k: int, rank: int,
                       causal: bool, b: int, h: int, rows, norm: str = "map") -> np.ndarray:
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
    _check_norm(norm)
    nums, dens = [], []
    for l in range(1, rank + 1):
        pq = phi(qs[rows], l)
        pk = phi(ks, l)
        if not causal:
            s = pk.T @ vs
            z = pk.sum(axis=0)
            nums.append(pq @ s)
            dens.append(pq @ z)
            continue
        num = np.zeros((rows.size, d))
        den = np.zeros(rows.size)
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
            num[t] = pq[t] @ s_run
            den[t] = pq[t] @ z_run
        nums.append(num)
        dens.append(den)
    if norm == "joint":
        far = sum(nums) / sum(dens)[:, None]
    else:
        far = np.zeros((rows.size, d))
        for num, den in zip(nums, dens):
            far += num / den[:, None]
    a = float(sigmoid(w_near[h]))
    c = float(sigmoid(w_far[h]))
    out = np.zeros((rows.size, d))
    if a > 0:
        out += a * near
    if c > 0:
        out += c * far
    return out


# ---------------------------------------------------------------- backward

def _near_backward(q, k, v, g, band_k: int, causal: bool):
    """Gradients of the near field (Eq. (3)) for the upstream gradient g of
    near.  With p_i the softmax over the band of s_ij = tau q_i.k_j:
        dv_j += sum_i p_ij g_i
        ds_ij = p_ij (g_i.v_j - g_i.near_i)          (softmax derivative)
        dq_i  = tau sum_j ds_ij k_j,  dk_j += tau sum_i ds_ij q_i
    computed per band offset o = j - i, like near_stream."""
    b_, h_, n, d = q.shape
    kk = min(band_k, n - 1)
    offs = np.arange(-kk, (0 if causal else kk) + 1)
    tau = 1.0 / math.sqrt(d)
    rows = np.arange(n)
    valid = [(rows + o >= 0) & (rows + o < n) for o in offs]
    score = np.full((b_, h_, n, len(offs)), -np.inf)
    for t, o in enumerate(offs):
        ok = valid[t]
        score[:, :, ok, t] = np.einsum("bhic,bhic->bhi", q[:, :, rows[ok]],
                                       k[:, :, rows[ok] + o]) * tau
    score = score - score.max(axis=-1, keepdims=True)
    p = np.exp(score)
    p = p / p.sum(axis=-1, keepdims=True)
    near = np.zeros_like(v)
    dp = np.zeros_like(p)
    for t, o in enumerate(offs):
        ok = valid[t]
        near[:, :, ok] += p[:, :, ok, t, None] * v[:, :, rows[ok] + o]
        dp[:, :, ok, t] = np.einsum("bhic,bhic->bhi", g[:, :, ok], v[:, :, rows[ok] + o])
    gn = np.einsum("bhic,bhic->bhi", g, near)
    ds = p * (dp - gn[..., None])
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for t, o in enumerate(offs):
        ok = valid[t]
        j = rows[ok] + o
        dq[:, :, ok] += tau * ds[:, :, ok, t, None] * k[:, :, j]
        dk[:, :, j] += tau * ds[:, :, ok, t, None] * q[:, :, rows[ok]]
        dv[:, :, j] += p[:, :, ok, t, None] * g[:, :, ok]
    return near, dq, dk, dv


def _far_backward(q, k, v, f, rank: int, causal: bool, norm: str, row_chunk: int = 512):
    """Gradients of the far field (Eq. (7)-(9)) for the upstream gradient f of
    far.  Per map, num_i = phi(q_i)^T S(i), den_i = phi(q_i)^T z(i):
      norm="map":   dnum_i = f_i / den_i,   dden_i = -(f_i.num_i) / den_i^2
      norm="joint": dnum_i = f_i / Den_i,   dden_i = -(f_i.far_i) / Den_i
                    (Den_i = sum_l den_l,i; the same for every map)
      dphi(q_i) = S(i) dnum_i + z(i) dden_i
      dS(j) = sum_{i in G(j)} phi(q_i) dnum_i^T,  dz(j) = sum_{i in G(j)} phi(q_i) dden_i
              G(j) = all rows (non-causal), rows i >= j (causal: suffix sums)
      dphi(k_j) = dS(j) v_j + dz(j),  dv_j += dS(j)^T phi(k_j)
    and dq, dk through phi_l'."""
    b_, h_, n, d = q.shape
    terms = far_terms_stream(q, k, v, rank, causal, row_chunk)
    if norm == "joint":
        den_all = sum(t[1] for t in terms)
        far = sum(t[0] for t in terms) / den_all[..., None]
    else:
        far = np.zeros_like(v)
        for num, den in terms:
            far += num / den[..., None]
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for l in range(1, rank + 1):
        num, den = terms[l - 1]
        if norm == "joint":
            dnum = f / den_all[..., None]
            dden = -np.einsum("bhic,bhic->bhi", f, far) / den_all
        else:
            dnum = f / den[..., None]
            dden = -np.einsum("bhic,bhic->bhi", f, num) / den ** 2
        pq = phi(q, l)
        pk = phi(k, l)
        if not causal:
            state = np.einsum("bhjc,bhje->bhce", pk, v)
            zsum = pk.sum(axis=2)
            dpq = (np.einsum("bhce,bhie->bhic", state, dnum)
                   + zsum[:, :, None, :] * dden[..., None])
            ds = np.einsum("bhic,bhie->bhce", pq, dnum)
            dz = np.einsum("bhic,bhi->bhc", pq, dden)
            dpk = np.einsum("bhce,bhje->bhjc", ds, v) + dz[:, :, None, :]
            dv += np.einsum("bhjc,bhce->bhje", pk, ds)
        else:
            # prefix sums S(i), z(i) over keys j <= i, as in the forward
            dpq = np.empty_like(q)
            s_pre = np.zeros((b_, h_, d, d))
            z_pre = np.zeros((b_, h_, d))
            for i0 in range(0, n, row_chunk):
                i1 = min(n, i0 + row_chunk)
                kv = pk[:, :, i0:i1, :, None] * v[:, :, i0:i1, None, :]
                s_i = s_pre[:, :, None] + np.cumsum(kv, axis=2)
                z_i = z_pre[:, :, None] + np.cumsum(pk[:, :, i0:i1], axis=2)
                dpq[:, :, i0:i1] = (np.einsum("bhice,bhie->bhic", s_i, dnum[:, :, i0:i1])
                                    + z_i * dden[:, :, i0:i1, None])
                s_pre = s_i[:, :, -1]
                z_pre = z_i[:, :, -1]
            # suffix sums over rows i >= j, walked from the end
            dpk = np.empty_like(k)
            ds_run = np.zeros((b_, h_, d, d))
            dz_run = np.zeros((b_, h_, d))
            for i1 in range(n, 0, -row_chunk):
                i0 = max(0, i1 - row_chunk)
                outer = pq[:, :, i0:i1, :, None] * dnum[:, :, i0:i1, None, :]
                ds_suf = ds_run[:, :, None] + np.cumsum(outer[:, :, ::-1], axis=2)[:, :, ::-1]
                dz_suf = dz_run[:, :, None] + np.cumsum(
                    (pq[:, :, i0:i1] * dden[:, :, i0:i1, None])[:, :, ::-1], axis=2)[:, :, ::-1]
                dpk[:, :, i0:i1] = (np.einsum("bhjce,bhje->bhjc", ds_suf, v[:, :, i0:i1])
                                    + dz_suf)
                dv[:, :, i0:i1] += np.einsum("bhjc,bhjce->bhje", pk[:, :, i0:i1], ds_suf)
                ds_run = ds_suf[:, :, 0]
                dz_run = dz_suf[:, :, 0]
        dq += phi_grad(q, l) * dpq
        dk += phi_grad(k, l) * dpk
    return far, dq, dk, dv


def fmm_attention_backward_stream(q, k, v, w_near, w_far, dout, band_k: int, rank: int,
                                  causal: bool, norm: str = "map", row_chunk: int = 512):
    """Gradients of sum(dout * out) with out = fmm_attention_stream(...):
    returns (dq, dk, dv, dw_near, dw_far).  Eq. (11): out = a near + c far with
    a = sigmoid(w_near[h]), c = sigmoid(w_far[h]); so near and far receive
    a dout and c dout, and dw = sigmoid'(w) sum over (b, i, channel) of
    dout * part, with sigmoid' = sigmoid (1 - sigmoid)."""
    q, k, v = _check(q, k, v)
    _check_norm(norm)
    dout = np.asarray(dout, dtype=np.float64)
    a = sigmoid(w_near)[None, :, None, None]
    c = sigmoid(w_far)[None, :, None, None]
    near, dq, dk, dv = _near_backward(q, k, v, a * dout, band_k, causal)
    far, dqf, dkf, dvf = _far_backward(q, k, v, c * dout, rank, causal, norm, row_chunk)
    dq += dqf
    dk += dkf
    dv += dvf
    sa, sc = sigmoid(w_near), sigmoid(w_far)
    dw_near = sa * (1.0 - sa) * np.einsum("bhic,bhic->h", dout, near)
    dw_far = sc * (1.0 - sc) * np.einsum("bhic,bhic->h", dout, far)
    return dq, dk, dv, dw_near, dw_far


# ---------------------------------------------------------------- attention layer

def _layer_heads(x, w_qkv, w_out, heads: int):
    """q, k, v [B, heads, N, d] of the layer's input projection qkv = x W_qkv
    (within each of q, k, v the heads in order, d columns each)."""
    x = np.asarray(x, dtype=np.float64)
    w_qkv = np.asarray(w_qkv, dtype=np.float64)
    b_, n, e = x.shape
    if e % heads or w_qkv.shape != (e, 3 * e) or np.shape(w_out) != (e, e):
        raise ValueError("x [B, N, E], w_qkv [E, 3E], w_out [E, E], E divisible by heads")
    d = e // heads
    qkv = (x @ w_qkv).reshape(b_, n, 3, heads, d)
    return tuple(np.ascontiguousarray(qkv[:, :, p].transpose(0, 2, 1, 3)) for p in range(3))


def fmm_layer_forward(x, w_qkv, w_out, heads: int, w_near, w_far, band_k: int, rank: int,
                      causal: bool, norm: str = "map") -> np.ndarray:
    """The attention layer around the operator (Sec. 1.1, Step 1, and the
    output projection): per token t, [q_t | k_t | v_t] = x_t W_qkv (W_qkv of
    shape [E, 3E]; within each of q, k, v the E = heads * d columns are the
    heads in order, d columns each); the operator runs per head on
    [B, heads, N, d]; the heads' outputs are concatenated per token (head
    order) and multiplied by W_out [E, E].  x: [B, N, E]; returns [B, N, E]."""
    x = np.asarray(x, dtype=np.float64)
    w_out = np.asarray(w_out, dtype=np.float64)
    b_, n, e = x.shape
    q, k, v = _layer_heads(x, w_qkv, w_out, heads)
    o = fmm_attention_stream(q, k, v, w_near, w_far, band_k, rank, causal, norm)
    merged = o.transpose(0, 2, 1, 3).reshape(b_, n, e)
    return merged @ w_out



def fmm_layer_backward(x, w_qkv, w_out, heads: int, w_near, w_far, dy, band_k: int, rank: int,
                       causal: bool, norm: str = "map"):
    """Gradients of sum(dy * y) with y = fmm_layer_forward(...): returns
    (dx, dw_qkv, dw_out, dw_near, dw_far).  With m the concatenated heads'
    outputs and qkv = x W_qkv:
        dm = dy W_out^T,  dW_out = m^T dy   (summed over every token)
        the operator's backward for the heads' share of dm gives dq, dk, dv
        dqkv = [dq | dk | dv] per token,  dx = dqkv W_qkv^T,  dW_qkv = x^T dqkv."""
    x = np.asarray(x, dtype=np.float64)
    w_qkv = np.asarray(w_qkv, dtype=np.float64)
    w_out = np.asarray(w_out, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    b_, n, e = x.shape
    d = e // heads
    q, k, v = _layer_heads(x, w_qkv, w_out, heads)
    o = fmm_attention_stream(q, k, v, w_near, w_far, band_k, rank, causal, norm)
    m = o.transpose(0, 2, 1, 3).reshape(b_ * n, e)
    dyf = dy.reshape(b_ * n, e)
    dw_out = m.T @ dyf
    do = (dyf @ w_out.T).reshape(b_, n, heads, d).transpose(0, 2, 1, 3)
    dq, dk, dv, dw_near, dw_far = fmm_attention_backward_stream(q, k, v, w_near, w_far, do,
                                                                band_k, rank, causal, norm)
    dqkv = np.stack([g.transpose(0, 2, 1, 3).reshape(b_ * n, e) for g in (dq, dk, dv)], axis=1)
    dqkv = dqkv.reshape(b_ * n, 3 * e)
    dx = (dqkv @ w_qkv.T).reshape(b_, n, e)
    dw_qkv = x.reshape(b_ * n, e).T @ dqkv
    return dx, dw_qkv, dw_out, dw_near, dw_far

# ---------------------------------------------------------------- fast-weight far field

def fast_weight_stream(q, k, v, beta) -> np.ndarray:
    """The fast-weight far field (Appendix D: a linear transformer with the
    fast weight update of the cited fast-weight-programmer work), causal, per
    (b, h), with phi = elu(x) + 1 normalised by its sum over the channels,
    p(x) = phi(x) / sum_c phi(x)_c:
        u_i = W_{i-1} p(k_i)                          (value read at key i)
        W_i = W_{i-1} + beta_i (v_i - u_i) p(k_i)^T   (delta-rule write)
        z_i = z_{i-1} + p(k_i)
        fw_i = W_i p(q_i) / (z_i . p(q_i))            (attention normalisation)
    with W_{-1} = 0, z_{-1} = 0.  beta: [B, H, N] write strengths.  A plain
    sequential loop over i."""
    q, k, v = _check(q, k, v)
    beta = np.asarray(beta, dtype=np.float64)
    b_, h_, n, d = q.shape
    if beta.shape != (b_, h_, n):
        raise ValueError("beta must be [B, H, N]")
    pk = phi(k, 1)
    pk = pk / pk.sum(axis=-1, keepdims=True)
    pq = phi(q, 1)
    pq = pq / pq.sum(axis=-1, keepdims=True)
    out = np.empty_like(v)
    for bb in range(b_):
        for hh in range(h_):
            w = np.zeros((d, d))
            z = np.zeros(d)
            for i in range(n):
                u = w @ pk[bb, hh, i]
                w = w + beta[bb, hh, i] * np.outer(v[bb, hh, i] - u, pk[bb, hh, i])
                z = z + pk[bb, hh, i]
                out[bb, hh, i] = (w @ pq[bb, hh, i]) / (z @ pq[bb, hh, i])
    return out


def _normalised_phi(x):
    """p = phi_1(x) / sum_c phi_1(x)_c over the last axis, and that sum."""
    f = phi(x, 1)
    s = f.sum(axis=-1, keepdims=True)
    return f / s, s


def fast_weight_backward_stream(q, k, v, beta, f):
    """Gradients of sum(f * fw) with fw = fast_weight_stream(q, k, v, beta):
    returns (fw, dq, dk, dv, dbeta).  The recurrence differentiated and run
    backwards, per (b, h), with G_i the gradient with respect to W_i and Zs_i
    the one with respect to z_i (both including every later use):
        n_i = W_i pq_i,  s_i = z_i . pq_i,  fw_i = n_i / s_i
        dn_i = f_i / s_i,  ds_i = -(f_i . fw_i) / s_i
        G_i = dn_i pq_i^T + G_{i+1} (I - beta_{i+1} pk_{i+1} pk_{i+1}^T),  G_N = 0
        Zs_i = ds_i pq_i + Zs_{i+1},  Zs_N = 0
        dpq_i = W_i^T dn_i + ds_i z_i
        e_i = v_i - u_i,  gp_i = G_i pk_i
        dv_i = beta_i gp_i,  dbeta_i = e_i . gp_i
        dpk_i = beta_i (G_i^T e_i - W_{i-1}^T gp_i) + Zs_i
    and through p = phi / sum(phi): dphi = (dp - dp . p) / sum(phi), then
    dx = phi_1'(x) dphi.  The forward states W_i are kept from a forward
    sweep (plain loops)."""
    q, k, v = _check(q, k, v)
    beta = np.asarray(beta, dtype=np.float64)
    f = np.asarray(f, dtype=np.float64)
    b_, h_, n, d = q.shape
    pk, sk = _normalised_phi(k)
    pq, sq = _normalised_phi(q)
    fw = np.empty_like(v)
    dpq = np.zeros_like(q)
    dpk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dbeta = np.zeros_like(beta)
    for bb in range(b_):
        for hh in range(h_):
            ws = [np.zeros((d, d))]          # ws[i + 1] = W_i, ws[0] = W_{-1}
            zs = [np.zeros(d)]
            us = []
            for i in range(n):
                p = pk[bb, hh, i]
                u = ws[-1] @ p
                us.append(u)
                ws.append(ws[-1] + beta[bb, hh, i] * np.outer(v[bb, hh, i] - u, p))
                zs.append(zs[-1] + p)
                fw[bb, hh, i] = (ws[-1] @ pq[bb, hh, i]) / (zs[-1] @ pq[bb, hh, i])
            g_w = np.zeros((d, d))
            z_s = np.zeros(d)
            for i in range(n - 1, -1, -1):
                if i + 1 < n:  # carry G_{i+1} back through W_{i+1}'s update
                    p1 = pk[bb, hh, i + 1]
                    g_w = g_w - beta[bb, hh, i + 1] * np.outer(g_w @ p1, p1)
                wi, wprev, zi = ws[i + 1], ws[i], zs[i + 1]
                pqi, p = pq[bb, hh, i], pk[bb, hh, i]
                s_i = zi @ pqi
                dn = f[bb, hh, i] / s_i
                ds = -(f[bb, hh, i] @ fw[bb, hh, i]) / s_i
                g_w = g_w + np.outer(dn, pqi)
                z_s = z_s + ds * pqi
                dpq[bb, hh, i] = wi.T @ dn + ds * zi
                e = v[bb, hh, i] - us[i]
                gp = g_w @ p
                dv[bb, hh, i] = beta[bb, hh, i] * gp
                dbeta[bb, hh, i] = e @ gp
                dpk[bb, hh, i] = beta[bb, hh, i] * (g_w.T @ e - wprev.T @ gp) + z_s
    dq = phi_grad(q, 1) * (dpq - (dpq * pq).sum(axis=-1, keepdims=True)) / sq
    dk = phi_grad(k, 1) * (dpk - (dpk * pk).sum(axis=-1, keepdims=True)) / sk
    return fw, dq, dk, dv, dbeta


def fmm_fast_weight_backward(q, k, v, beta, w_near, w_far, dout, band_k: int, n_linear: int):
    """Gradients of sum(dout * out) with out = fmm_fast_weight_forward(...):
    returns (dq, dk, dv, dbeta, dw_near, dw_far).  With a = sigmoid(w_near),
    c = sigmoid(w_far): the near field receives a dout, the fast-weight far
    field and (n_linear = 1) the linear far part c dout, and
    dw_near = a (1 - a) sum dout . near, dw_far = c (1 - c) sum dout . far."""
    if n_linear not in (0, 1):
        raise ValueError("n_linear must be 0 or 1")
    q, k, v = _check(q, k, v)
    dout = np.asarray(dout, dtype=np.float64)
    a = sigmoid(w_near)[None, :, None, None]
    c = sigmoid(w_far)[None, :, None, None]
    near, dq, dk, dv = _near_backward(q, k, v, a * dout, band_k, True)
    far, dqf, dkf, dvf, dbeta = fast_weight_backward_stream(q, k, v, beta, c * dout)
    dq, dk, dv = dq + dqf, dk + dkf, dv + dvf
    if n_linear:
        lin, dql, dkl, dvl = _far_backward(q, k, v, c * dout, 1, True, "map")
        far = far + lin
        dq, dk, dv = dq + dql, dk + dkl, dv + dvl
    s_near, s_far = sigmoid(w_near), sigmoid(w_far)
    dw_near = s_near * (1.0 - s_near) * np.einsum("bhic,bhic->h", dout, near)
    dw_far = s_far * (1.0 - s_far) * np.einsum("bhic,bhic->h", dout, far)
    return dq, dk, dv, dbeta, dw_near, dw_far


def fmm_fast_weight_forward(q, k, v, beta, w_near, w_far, band_k: int,
                            n_linear: int) -> np.ndarray:
    """FMMformer with the fast-weight far field (Appendix D), causal:
    out = sigmoid(w_near) near + sigmoid(w_far) (fw + [n_linear = 1] lin),
    near the causal banded softmax (Eq. (3)), fw the fast-weight far field
    above, lin the causal linear attention of phi_1 (Eq. (8)) -- the
    2-kernel variant pairs one fast-weight kernel with one linear kernel,
    both with elu(x) + 1."""
    if n_linear not in (0, 1):
        raise ValueError("n_linear must be 0 or 1")
    far = fast_weight_stream(q, k, v, beta)
    if n_linear:
        far = far + far_stream(q, k, v, 1, True)
    return _blend(near_stream(q, k, v, band_k, True), far, w_near, w_far)
