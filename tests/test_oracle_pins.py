"""Pins for the float64 oracle (CPU only).

Every check here ties the oracle to something other than itself: closed forms
derived by hand from the paper's definitions, torch's float64
scaled_dot_product_attention (a library routine the banded softmax reduces to),
scalar brute-force loops written independently of the vectorised oracle,
invariants the definitions imply, and the one number the paper prints about
the band (Sec. 4.2).  A dropped term, a wrong sign or index, or a transposed
operand in the oracle fails at least one of them.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import fmm_ref as ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rnd(shape, seed, std=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * std


def sig(x):
    return 1.0 / (1.0 + math.exp(-x))


# ------------------------------------------------------------------ brute force
# Scalar loops, written from the definitions with the math module only.

def bf_elu(x):
    return x if x > 0 else math.exp(x) - 1.0


def bf_phi(x, l):
    if l == 3:
        return math.tanh(x)
    return bf_elu(x) + 1.0 if l == 1 else bf_elu(-x) + 1.0


def bf_near(qs, ks, vs, kw, causal):
    n, d = len(qs), len(qs[0])
    out = []
    for i in range(n):
        js = [j for j in range(n) if (i - kw <= j <= i if causal else abs(i - j) <= kw)]
        sc = [sum(qs[i][c] * ks[j][c] for c in range(d)) / math.sqrt(d) for j in js]
        m = max(sc)
        w = [math.exp(s - m) for s in sc]
        tot = sum(w)
        out.append([sum(w[t] * vs[j][c] for t, j in enumerate(js)) / tot for c in range(d)])
    return np.array(out)


def bf_far(qs, ks, vs, rank, causal, joint=False):
    n, d = len(qs), len(qs[0])
    out = np.zeros((n, d))
    for i in range(n):
        js = range(i + 1) if causal else range(n)
        nums, dens = [], []
        for l in range(1, rank + 1):
            a = {j: sum(bf_phi(qs[i][c], l) * bf_phi(ks[j][c], l) for c in range(d)) for j in js}
            nums.append([sum(a[j] * vs[j][c] for j in js) for c in range(d)])
            dens.append(sum(a.values()))
        for c in range(d):
            if joint:
                out[i, c] = sum(nm[c] for nm in nums) / sum(dens)
            else:
                out[i, c] = sum(nm[c] / dn for nm, dn in zip(nums, dens))
    return out


# ------------------------------------------------------------------ primitives

def test_phi_closed_forms():
    e = math.exp
    assert ref.phi(np.array(1.5), 1) == pytest.approx(2.5)
    assert ref.phi(np.array(-1.0), 1) == pytest.approx(e(-1.0))
    assert ref.phi(np.array(0.0), 1) == pytest.approx(1.0)
    assert ref.phi(np.array(1.0), 2) == pytest.approx(e(-1.0))
    assert ref.phi(np.array(-2.0), 2) == pytest.approx(3.0)
    assert ref.phi(np.array(0.0), 2) == pytest.approx(1.0)
    # phi_2(x) = phi_1(-x) and both are strictly positive
    x = rnd(1000, 0) * 5
    assert np.array_equal(ref.phi(x, 2), ref.phi(-x, 1))
    assert (ref.phi(x, 1) > 0).all() and (ref.phi(x, 2) > 0).all()
    # phi_3 = tanh: odd, tanh(ln 3) = (9 - 1) / (9 + 1)
    assert ref.phi(np.array(0.0), 3) == 0.0
    assert ref.phi(np.array(math.log(3.0)), 3) == pytest.approx(0.8, rel=1e-15)
    assert np.array_equal(ref.phi(-x, 3), -ref.phi(x, 3))
    with pytest.raises(ValueError):
        ref.phi(x, 4)


def test_phi_grad_closed_forms_and_differences():
    e = math.exp
    g = lambda x, l: float(ref.phi_grad(np.array(x), l))
    assert g(1.0, 1) == 1.0 and g(-1.0, 1) == pytest.approx(e(-1.0))
    assert g(1.0, 2) == pytest.approx(-e(-1.0)) and g(-2.0, 2) == -1.0
    assert g(math.log(3.0), 3) == pytest.approx(1.0 - 0.64, rel=1e-14)
    x = rnd(200, 1) * 3
    x = x[np.abs(x) > 1e-3]  # away from the kink-free but piecewise point 0
    for l in (1, 2, 3):
        fd = (ref.phi(x + 1e-6, l) - ref.phi(x - 1e-6, l)) / 2e-6
        np.testing.assert_allclose(ref.phi_grad(x, l), fd, rtol=1e-7, atol=1e-9)


def test_sigmoid_closed_forms():
    assert ref.sigmoid(0.0) == 0.5
    assert ref.sigmoid(math.log(3.0)) == pytest.approx(0.75)
    assert ref.sigmoid(np.inf) == 1.0
    assert ref.sigmoid(-np.inf) == 0.0


def test_band_coverage_matches_paper():
    g = json.load(open(os.path.join(GOLDEN, "band_coverage.json")))
    n, k = g["n"], g["half_width_k"]
    mask = ref.band_mask(n, k, causal=False)
    assert mask.sum(axis=1).max() == g["paper_bandwidth"]
    pct = 100.0 * mask.sum() / n ** 2
    assert round(pct, g["printed_digits"]) == g["fraction_percent"]


# ------------------------------------------------------------------ near field

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("form", ["dense", "stream"])
def test_near_full_band_is_softmax_attention(causal, form):
    # k >= N-1: the band is the whole (causal) matrix, so Eq. (3) is Eq. (1).
    b, h, n, d = 2, 3, 37, 8
    q, k, v = (rnd((b, h, n, d), s) for s in (1, 2, 3))
    fn = ref.near_dense if form == "dense" else ref.near_stream
    for kw in (n - 1, n, n + 5):
        got = fn(q, k, v, kw, causal)
        want = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
            is_causal=causal).numpy()
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("kw", [0, 1, 3, 6])
def test_near_band_is_masked_softmax_attention(causal, kw):
    b, h, n, d = 1, 2, 29, 5
    q, k, v = (rnd((b, h, n, d), s) for s in (4, 5, 6))
    allowed = np.zeros((n, n), dtype=bool)
    for i in range(n):
        for j in range(n):
            allowed[i, j] = (i - kw <= j <= i) if causal else (i - kw <= j <= i + kw)
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=torch.from_numpy(allowed)).numpy()
    for fn in (ref.near_dense, ref.near_stream):
        np.testing.assert_allclose(fn(q, k, v, kw, causal), want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_near_brute_force(causal):
    n, d = 11, 3
    q, k, v = (rnd((1, 1, n, d), s) for s in (7, 8, 9))
    for kw in (0, 1, 2, 4, 20):
        want = bf_near(q[0, 0].tolist(), k[0, 0].tolist(), v[0, 0].tolist(), kw, causal)
        np.testing.assert_allclose(ref.near_stream(q, k, v, kw, causal)[0, 0], want,
                                   rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_near_zero_width_is_v(causal):
    q, k, v = (rnd((2, 2, 17, 4), s) for s in (10, 11, 12))
    for fn in (ref.near_dense, ref.near_stream):
        np.testing.assert_array_equal(fn(q, k, v, 0, causal), v)


@pytest.mark.parametrize("causal", [False, True])
def test_near_zero_queries_average_the_band(causal):
    n, d, kw = 23, 4, 3
    k, v = rnd((1, 1, n, d), 13), rnd((1, 1, n, d), 14)
    q = np.zeros_like(k)
    got = ref.near_stream(q, k, v, kw, causal)[0, 0]
    for i in range(n):
        lo, hi = max(0, i - kw), (i if causal else min(n - 1, i + kw))
        np.testing.assert_allclose(got[i], v[0, 0, lo:hi + 1].mean(axis=0), rtol=1e-12)


def test_near_translation_equivariance_interior():
    # Shifting the whole sequence by one position shifts interior near rows.
    n, d, kw = 30, 4, 3
    q, k, v = (rnd((1, 1, n + 1, d), s) for s in (15, 16, 17))
    a = ref.near_stream(q[:, :, :n], k[:, :, :n], v[:, :, :n], kw, False)
    b = ref.near_stream(q[:, :, 1:], k[:, :, 1:], v[:, :, 1:], kw, False)
    np.testing.assert_allclose(a[0, 0, kw + 1:n - kw], b[0, 0, kw:n - kw - 1], rtol=1e-12)


# ------------------------------------------------------------------ far field

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("rank", [1, 2, 3])
@pytest.mark.parametrize("norm", ["map", "joint"])
def test_far_brute_force(causal, rank, norm):
    n, d = 9, 3
    q, k, v = (rnd((1, 1, n, d), s) for s in (20, 21, 22))
    if rank == 3:  # keep tanh's denominator away from zero
        q, k = q + 1.5, k + 1.5
    want = bf_far(q[0, 0].tolist(), k[0, 0].tolist(), v[0, 0].tolist(), rank, causal,
                  joint=norm == "joint")
    for fn in (ref.far_dense, ref.far_stream):
        np.testing.assert_allclose(fn(q, k, v, rank, causal, norm=norm)[0, 0], want,
                                   rtol=1e-11, atol=1e-12)


def test_far_joint_rows_sum_to_one():
    # joint normalisation: the rows of the whole far matrix sum to one (per map
    # they sum to one each, so the per-map far matrix rows sum to the rank);
    # rank 1 is the same under both readings
    n, d = 13, 3
    q, k = rnd((1, 1, n, d), 70) + 1.0, rnd((1, 1, n, d), 71) + 1.0
    c = rnd(d, 72)
    v = np.broadcast_to(c, (1, 1, n, d)).copy()
    for causal in (False, True):
        for rank in (1, 2, 3):
            np.testing.assert_allclose(ref.far_stream(q, k, v, rank, causal, norm="joint"),
                                       np.broadcast_to(c, v.shape), rtol=1e-12)
            np.testing.assert_allclose(ref.far_stream(q, k, v, rank, causal, norm="map"),
                                       rank * np.broadcast_to(c, v.shape), rtol=1e-12)
        v2 = rnd((1, 1, n, d), 73)
        np.testing.assert_array_equal(ref.far_stream(q, k, v2, 1, causal, norm="joint"),
                                      ref.far_stream(q, k, v2, 1, causal, norm="map"))


def test_far_rank3_closed_form():
    # d = 1, one key k = ln 3 (phi_1 = 1 + ln 3, phi_2 = 1/3, phi_3 = 0.8), value 2,
    # query ln 3 too: every map's weight matrix is the 1 x 1 matrix [1], so per
    # map far = 3 * 2, joint far = 2.  A second key 0 (phi = 1, 1, 0) with value
    # 0 and the same query: map 3's weight on key 0 is 0, so its term is 2 again.
    x = math.log(3.0)
    q = np.array([x, x]).reshape(1, 1, 2, 1)
    k = np.array([x, 0.0]).reshape(1, 1, 2, 1)
    v = np.array([2.0, 0.0]).reshape(1, 1, 2, 1)
    p1, p2 = (1.0 + x), 1.0 / 3.0
    want = 2.0 * (p1 * p1 / (p1 * p1 + p1) + p2 * p2 / (p2 * p2 + p2) + 1.0)
    got = ref.far_stream(q, k, v, 3, False)[0, 0, :, 0]
    np.testing.assert_allclose(got, [want, want], rtol=1e-14)
    den = p1 * p1 + p1 + p2 * p2 + p2 + 0.64
    num = 2.0 * (p1 * p1 + p2 * p2 + 0.64)
    np.testing.assert_allclose(ref.far_stream(q, k, v, 3, False, norm="joint")[0, 0, :, 0],
                               [num / den] * 2, rtol=1e-14)


def test_far_rank2_closed_form():
    # d = 1, keys (1, -1), values (1, 0).  phi_1(k) = (2, 1/e), phi_2(k) = (1/e, 2),
    # and with d = 1 the query factor cancels in each map, so every row is
    # 2/(2 + 1/e) + (1/e)/(1/e + 2) = 1.  Using elu(x)+1 for both maps, or
    # dropping a denominator, gives a different value.
    k = np.array([1.0, -1.0]).reshape(1, 1, 2, 1)
    v = np.array([1.0, 0.0]).reshape(1, 1, 2, 1)
    q = np.array([0.3, -2.0]).reshape(1, 1, 2, 1)
    for fn in (ref.far_dense, ref.far_stream):
        np.testing.assert_allclose(fn(q, k, v, 2, False)[0, 0, :, 0], [1.0, 1.0], rtol=1e-14)
        one = fn(q, k, v, 1, False)[0, 0, :, 0]
        np.testing.assert_allclose(one, [2.0 / (2.0 + math.exp(-1))] * 2, rtol=1e-14)
    # causal row 0 sees only key 0, row 1 sees both
    c = ref.far_stream(q, k, v, 2, True)[0, 0, :, 0]
    np.testing.assert_allclose(c, [2.0, 1.0], rtol=1e-14)


def test_far_two_dim_closed_form():
    # d = 2 so that the query does not cancel: one query (0, 1), keys (0, 0) and
    # (1, 0), values (1, 0) and (0, 1), rank 1.  phi_1(q) = (1, 2),
    # phi_1(k_0) = (1, 1), phi_1(k_1) = (2, 1); a_0 = 1 + 2 = 3, a_1 = 2 + 2 = 4;
    # far = (3 v_0 + 4 v_1) / 7.
    q = np.array([[0.0, 1.0], [0.0, 1.0]]).reshape(1, 1, 2, 2)
    k = np.array([[0.0, 0.0], [1.0, 0.0]]).reshape(1, 1, 2, 2)
    v = np.array([[1.0, 0.0], [0.0, 1.0]]).reshape(1, 1, 2, 2)
    for fn in (ref.far_dense, ref.far_stream):
        np.testing.assert_allclose(fn(q, k, v, 1, False)[0, 0, 0], [3 / 7, 4 / 7], rtol=1e-14)
    np.testing.assert_allclose(ref.far_stream(q, k, v, 1, True)[0, 0, 1], [3 / 7, 4 / 7],
                               rtol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_far_zero_qk_is_mean(causal):
    n, d = 19, 3
    v = rnd((1, 2, n, d), 23)
    z = np.zeros_like(v)
    for rank in (1, 2):
        got = ref.far_stream(z, z, v, rank, causal)
        if causal:
            want = np.cumsum(v, axis=2) / np.arange(1, n + 1)[None, None, :, None]
        else:
            want = np.broadcast_to(v.mean(axis=2, keepdims=True), v.shape)
        np.testing.assert_allclose(got, rank * want, rtol=1e-12, atol=1e-14)


def test_far_permutation_invariance_noncausal():
    n, d = 21, 4
    q, k, v = (rnd((1, 1, n, d), s) for s in (24, 25, 26))
    p = np.random.default_rng(0).permutation(n)
    a = ref.far_stream(q, k, v, 2, False)
    b = ref.far_stream(q, k[:, :, p], v[:, :, p], 2, False)
    np.testing.assert_allclose(a, b, rtol=1e-12)


def test_far_rank_bounded_by_feature_width():
    # Prop. 1 analogue (Eq. (10)): each phi_l(Q) phi_l(K)^T has rank <= d, so the
    # row-normalised far map of r feature maps has rank <= r d.
    n, d = 39, 3
    q, k = rnd((1, 1, n, d), 27), rnd((1, 1, n, d), 28)
    eye = np.eye(n)
    for rank in (1, 2):
        # far applied to unit value vectors, d columns at a time, exposes the
        # N x N far matrix itself
        cols = []
        for j0 in range(0, n, d):
            v = eye[:, j0:j0 + d].reshape(1, 1, n, d)
            cols.append(ref.far_dense(q, k, v, rank, False)[0, 0])
        m = np.concatenate(cols, axis=1)
        np.testing.assert_allclose(m.sum(axis=1), rank, rtol=1e-12)
        s = np.linalg.svd(m, compute_uv=False)
        assert (s > 1e-10 * s[0]).sum() <= rank * d
        assert (s > 1e-10 * s[0]).sum() > (rank - 1) * d


# ------------------------------------------------------------------ blend / whole op

@pytest.mark.parametrize("causal", [False, True])
def test_equal_value_rows_give_weighted_sum(causal):
    b, h, n, d = 1, 3, 16, 4
    q, k = rnd((b, h, n, d), 29), rnd((b, h, n, d), 30)
    c = rnd(d, 31)
    v = np.broadcast_to(c, (b, h, n, d)).copy()
    wn, wf = rnd(h, 32), rnd(h, 33)
    for rank in (1, 2):
        out = ref.fmm_attention_stream(q, k, v, wn, wf, 3, rank, causal)
        for hh in range(h):
            coef = sig(wn[hh]) + rank * sig(wf[hh])
            np.testing.assert_allclose(out[0, hh], np.broadcast_to(coef * c, (n, d)),
                                       rtol=1e-12)


def test_causal_first_row():
    q, k, v = (rnd((2, 2, 12, 4), s) for s in (34, 35, 36))
    wn, wf = rnd(2, 37), rnd(2, 38)
    for rank in (1, 2):
        out = ref.fmm_attention_stream(q, k, v, wn, wf, 5, rank, True)
        for hh in range(2):
            coef = sig(wn[hh]) + rank * sig(wf[hh])
            np.testing.assert_allclose(out[:, hh, 0], coef * v[:, hh, 0], rtol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_blend_isolates_parts(causal):
    q, k, v = (rnd((1, 2, 14, 4), s) for s in (39, 40, 41))
    inf = np.inf
    near = ref.fmm_attention_stream(q, k, v, np.array([inf, inf]), np.array([-inf, -inf]),
                                    3, 2, causal)
    far = ref.fmm_attention_stream(q, k, v, np.array([-inf, -inf]), np.array([inf, inf]),
                                   3, 2, causal)
    np.testing.assert_array_equal(near, ref.near_stream(q, k, v, 3, causal))
    np.testing.assert_array_equal(far, ref.far_stream(q, k, v, 2, causal))
    half = ref.fmm_attention_stream(q, k, v, np.zeros(2), np.zeros(2), 3, 2, causal)
    np.testing.assert_allclose(half, 0.5 * near + 0.5 * far, rtol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_each_part_is_convex_combination(causal):
    n, d, kw = 25, 3, 4
    q, k, v = (rnd((1, 1, n, d), s, 2.0) for s in (42, 43, 44))
    near = ref.near_stream(q, k, v, kw, causal)[0, 0]
    vs = v[0, 0]
    for i in range(n):
        lo, hi = max(0, i - kw), (i if causal else min(n - 1, i + kw))
        assert (near[i] >= vs[lo:hi + 1].min(axis=0) - 1e-12).all()
        assert (near[i] <= vs[lo:hi + 1].max(axis=0) + 1e-12).all()
    for rank in (1, 2):
        far = ref.far_stream(q, k, v, rank, causal)[0, 0] / rank
        for i in range(n):
            hi = i if causal else n - 1
            assert (far[i] >= vs[:hi + 1].min(axis=0) - 1e-12).all()
            assert (far[i] <= vs[:hi + 1].max(axis=0) + 1e-12).all()


def test_linear_in_values():
    q, k, v1, v2 = (rnd((1, 2, 18, 4), s) for s in (45, 46, 47, 48))
    wn, wf = rnd(2, 49), rnd(2, 50)
    for causal in (False, True):
        f = lambda v: ref.fmm_attention_stream(q, k, v, wn, wf, 2, 2, causal)
        np.testing.assert_allclose(f(2.0 * v1 - 3.0 * v2), 2.0 * f(v1) - 3.0 * f(v2),
                                   rtol=1e-10, atol=1e-12)


# ------------------------------------------------------------------ forms agree

@pytest.mark.parametrize("shape", [(1, 1, 1, 4), (2, 3, 17, 8), (1, 2, 64, 16), (1, 1, 130, 4)])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("rank", [1, 2])
def test_dense_equals_stream(shape, causal, rank):
    q, k, v = (rnd(shape, s) for s in (51, 52, 53))
    wn, wf = rnd(shape[1], 54), rnd(shape[1], 55)
    for kw in (0, 2, 7, shape[2] + 3):
        a = ref.fmm_attention_dense(q, k, v, wn, wf, kw, rank, causal)
        b = ref.fmm_attention_stream(q, k, v, wn, wf, kw, rank, causal)
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("rank,norm", [(3, "map"), (2, "joint"), (3, "joint")])
def test_dense_equals_stream_extended_maps(causal, rank, norm):
    q, k, v = (rnd((2, 2, 33, 8), s) + 0.7 for s in (74, 75, 76))
    wn, wf = rnd(2, 77), rnd(2, 78)
    a = ref.fmm_attention_dense(q, k, v, wn, wf, 4, rank, causal, norm)
    b = ref.fmm_attention_stream(q, k, v, wn, wf, 4, rank, causal, norm)
    np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-12)
    rows = [32, 0, 5, 17]
    for bb in range(2):
        for hh in range(2):
            got = ref.fmm_attention_rows(q, k, v, wn, wf, 4, rank, causal, bb, hh, rows, norm)
            np.testing.assert_allclose(got, b[bb, hh, rows], rtol=1e-11, atol=1e-12)


def test_stream_chunking_is_invisible():
    q, k, v = (rnd((1, 2, 300, 4), s) for s in (56, 57, 58))
    for causal in (False, True):
        a = ref.far_stream(q, k, v, 2, causal, row_chunk=7)
        b = ref.far_stream(q, k, v, 2, causal, row_chunk=512)
        np.testing.assert_allclose(a, b, rtol=1e-12)
        c = ref.near_stream(q, k, v, 9, causal, row_chunk=13)
        e = ref.near_stream(q, k, v, 9, causal)
        np.testing.assert_allclose(c, e, rtol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_rows_form_equals_stream(causal):
    b, h, n, d = 2, 2, 150, 8
    q, k, v = (rnd((b, h, n, d), s) for s in (59, 60, 61))
    wn, wf = rnd(h, 62), rnd(h, 63)
    full = ref.fmm_attention_stream(q, k, v, wn, wf, 6, 2, causal)
    rows = [149, 0, 3, 77, 77, 6, 148]
    for bb in range(b):
        for hh in range(h):
            got = ref.fmm_attention_rows(q, k, v, wn, wf, 6, 2, causal, bb, hh, rows)
            np.testing.assert_allclose(got, full[bb, hh, rows], rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ backward
# The gradients of sum(dout * out) are pinned by central finite differences
# of the forward oracle and by torch float64 autograd of a dense forward
# written with torch's own softmax, masking and sigmoid.

def _fd_grads(q, k, v, wn, wf, dout, kw, rank, causal, norm, eps=1e-6):
    f = lambda *a: float((ref.fmm_attention_stream(*a, kw, rank, causal, norm) * dout).sum())
    args = [q, k, v, wn, wf]
    out = []
    for ai, x in enumerate(args):
        g = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            a1, a2 = list(args), list(args)
            a1[ai], a2[ai] = xp, xm
            g[idx] = (f(*a1) - f(*a2)) / (2 * eps)
        out.append(g)
    return out


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("rank,norm", [(1, "map"), (2, "map"), (3, "map"), (2, "joint"),
                                       (3, "joint")])
def test_backward_finite_differences(causal, rank, norm):
    b, h, n, d, kw = 1, 2, 8, 3, 2
    q, k, v, dout = (rnd((b, h, n, d), s) for s in (80, 81, 82, 83))
    if rank == 3:
        q, k = q + 1.0, k + 1.0
    wn, wf = rnd(h, 84), rnd(h, 85)
    got = ref.fmm_attention_backward_stream(q, k, v, wn, wf, dout, kw, rank, causal, norm)
    want = _fd_grads(q, k, v, wn, wf, dout, kw, rank, causal, norm)
    for g, w in zip(got, want):
        np.testing.assert_allclose(g, w, rtol=1e-6, atol=1e-7 * np.abs(w).max())


def _torch_dense_forward(q, k, v, wn, wf, kw, rank, causal, norm):
    n, d = q.shape[-2], q.shape[-1]
    i = torch.arange(n)[:, None]
    j = torch.arange(n)[None, :]
    band = ((j <= i) & (j >= i - kw)) if causal else ((i - j).abs() <= kw)
    s = (q @ k.transpose(-1, -2)) / math.sqrt(d)
    p = torch.softmax(s.masked_fill(~band, float("-inf")), dim=-1)
    near = p @ v
    maps = [lambda x: torch.nn.functional.elu(x) + 1, lambda x: torch.nn.functional.elu(-x) + 1,
            torch.tanh]
    lower = torch.ones(n, n, dtype=torch.bool).tril()
    mats = []
    for l in range(rank):
        a = maps[l](q) @ maps[l](k).transpose(-1, -2)
        mats.append(a.masked_fill(~lower, 0.0) if causal else a)
    if norm == "joint":
        tot = sum(mats)
        far = (tot / tot.sum(-1, keepdim=True)) @ v
    else:
        far = sum((a / a.sum(-1, keepdim=True)) @ v for a in mats)
    return (torch.sigmoid(wn)[None, :, None, None] * near
            + torch.sigmoid(wf)[None, :, None, None] * far)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("rank,norm", [(1, "map"), (2, "map"), (3, "map"), (2, "joint"),
                                       (3, "joint")])
def test_backward_matches_torch_autograd(causal, rank, norm):
    b, h, n, d, kw = 2, 2, 21, 5, 3
    q, k, v, dout = (rnd((b, h, n, d), s) for s in (86, 87, 88, 89))
    if rank == 3:
        q, k = q + 1.0, k + 1.0
    wn, wf = rnd(h, 90), rnd(h, 91)
    ts = [torch.tensor(x, requires_grad=True) for x in (q, k, v, wn, wf)]
    out = _torch_dense_forward(*ts, kw, rank, causal, norm)
    (out * torch.tensor(dout)).sum().backward()
    got = ref.fmm_attention_backward_stream(q, k, v, wn, wf, dout, kw, rank, causal, norm)
    for g, t in zip(got, ts):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_backward_zero_band_without_far_part():
    # k = 0 makes near = v and w_far = -inf removes the far part: out =
    # sigmoid(w_near) v, so dq = dk = 0, dv = sigmoid(w_near) dout,
    # dw_near = sigmoid' sum(dout * v), dw_far = 0
    q, k, v, dout = (rnd((2, 2, 10, 4), s) for s in (92, 93, 94, 95))
    wn = rnd(2, 96)
    wf = np.array([-np.inf, -np.inf])
    for causal in (False, True):
        dq, dk, dv, dwn, dwf = ref.fmm_attention_backward_stream(q, k, v, wn, wf, dout, 0, 2,
                                                                 causal)
        np.testing.assert_array_equal(dq, 0.0)
        np.testing.assert_array_equal(dk, 0.0)
        sn = 1.0 / (1.0 + np.exp(-wn))
        np.testing.assert_allclose(dv, sn[None, :, None, None] * dout, rtol=1e-14)
        np.testing.assert_allclose(dwn, sn * (1 - sn) * np.einsum("bhic,bhic->h", dout, v),
                                   rtol=1e-13)
        np.testing.assert_array_equal(dwf, 0.0)


def test_backward_chunking_is_invisible():
    # the causal prefix and suffix sums are carried across row blocks
    q, k, v, dout = (rnd((1, 2, 70, 4), s) for s in (97, 98, 99, 100))
    wn, wf = rnd(2, 101), rnd(2, 102)
    for causal in (False, True):
        a = ref.fmm_attention_backward_stream(q, k, v, wn, wf, dout, 3, 2, causal, row_chunk=9)
        b = ref.fmm_attention_backward_stream(q, k, v, wn, wf, dout, 3, 2, causal)
        for x, y in zip(a, b):
            np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ attention layer

def test_layer_with_identity_projections_is_the_operator():
    # W_qkv = [I | I | I], W_out = I: the layer is the operator applied to the
    # token vectors split into heads (head h = columns h*d .. h*d + d - 1)
    b, n, h, d = 2, 37, 3, 4
    e = h * d
    x = rnd((b, n, e), 110)
    eye = np.eye(e)
    wn, wf = rnd(h, 111), rnd(h, 112)
    for causal in (False, True):
        got = ref.fmm_layer_forward(x, np.concatenate([eye, eye, eye], axis=1), eye, h, wn, wf,
                                    3, 2, causal)
        heads = np.ascontiguousarray(x.reshape(b, n, h, d).transpose(0, 2, 1, 3))
        op = ref.fmm_attention_stream(heads, heads, heads, wn, wf, 3, 2, causal)
        np.testing.assert_allclose(got, op.transpose(0, 2, 1, 3).reshape(b, n, e), rtol=1e-13,
                                   atol=1e-14)


def test_layer_projections_by_brute_force():
    # distinct q, k, v projections and an output projection, checked against
    # per-token loops over the weight matrices and the per-head operator
    b, n, h, d = 1, 9, 2, 3
    e = h * d
    x = rnd((b, n, e), 113)
    wqkv, wo = rnd((e, 3 * e), 114), rnd((e, e), 115)
    wn, wf = rnd(h, 116), rnd(h, 117)
    got = ref.fmm_layer_forward(x, wqkv, wo, h, wn, wf, 2, 1, False)
    q = np.zeros((b, h, n, d)); k = np.zeros_like(q); v = np.zeros_like(q)
    for t in range(n):
        for hh in range(h):
            for c in range(d):
                col = hh * d + c
                q[0, hh, t, c] = sum(x[0, t, i] * wqkv[i, col] for i in range(e))
                k[0, hh, t, c] = sum(x[0, t, i] * wqkv[i, e + col] for i in range(e))
                v[0, hh, t, c] = sum(x[0, t, i] * wqkv[i, 2 * e + col] for i in range(e))
    o = ref.fmm_attention_stream(q, k, v, wn, wf, 2, 1, False)
    want = np.zeros((b, n, e))
    for t in range(n):
        for j in range(e):
            want[0, t, j] = sum(o[0, hh, t, c] * wo[hh * d + c, j]
                                for hh in range(h) for c in range(d))
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ fast-weight far field

def _bf_fast_weight(qs, ks, vs, betas):
    # scalar loops over the same recurrence, written with lists only
    n, d = len(qs), len(qs[0])
    def p(x):
        f = [bf_phi(c, 1) for c in x]
        s = sum(f)
        return [c / s for c in f]
    w = [[0.0] * d for _ in range(d)]
    z = [0.0] * d
    out = []
    for i in range(n):
        pk, pq = p(ks[i]), p(qs[i])
        u = [sum(w[r][c] * pk[c] for c in range(d)) for r in range(d)]
        for r in range(d):
            for c in range(d):
                w[r][c] += betas[i] * (vs[i][r] - u[r]) * pk[c]
        z = [z[c] + pk[c] for c in range(d)]
        den = sum(z[c] * pq[c] for c in range(d))
        out.append([sum(w[r][c] * pq[c] for c in range(d)) / den for r in range(d)])
    return np.array(out)


def test_fast_weight_brute_force():
    n, d = 11, 3
    q, k, v = (rnd((1, 1, n, d), s) for s in (120, 121, 122))
    beta = np.random.default_rng(123).uniform(0.0, 1.0, (1, 1, n))
    want = _bf_fast_weight(q[0, 0].tolist(), k[0, 0].tolist(), v[0, 0].tolist(),
                           beta[0, 0].tolist())
    np.testing.assert_allclose(ref.fast_weight_stream(q, k, v, beta)[0, 0], want, rtol=1e-12,
                               atol=1e-13)


def test_fast_weight_closed_forms():
    # row 0: W_0 = beta_0 v_0 p(k_0)^T, z_0 = p(k_0), so fw_0 = beta_0 v_0
    q, k, v = (rnd((2, 2, 6, 4), s) for s in (124, 125, 126))
    beta = np.random.default_rng(127).uniform(0.0, 1.0, (2, 2, 6))
    fw = ref.fast_weight_stream(q, k, v, beta)
    np.testing.assert_allclose(fw[:, :, 0], beta[:, :, 0, None] * v[:, :, 0], rtol=1e-13)
    # d = 1: p = 1 always, so W is the running average W_i = W_{i-1} + beta_i (v_i - W_{i-1})
    # and fw_i = W_i / (i + 1)
    n = 9
    q1, k1, v1 = (rnd((1, 1, n, 1), s) for s in (128, 129, 130))
    b1 = np.random.default_rng(131).uniform(0.0, 1.0, (1, 1, n))
    w, want = 0.0, []
    for i in range(n):
        w = w + b1[0, 0, i] * (v1[0, 0, i, 0] - w)
        want.append(w / (i + 1))
    np.testing.assert_allclose(ref.fast_weight_stream(q1, k1, v1, b1)[0, 0, :, 0], want,
                               rtol=1e-13)
    # beta = 0: nothing is ever written
    np.testing.assert_array_equal(ref.fast_weight_stream(q, k, v, np.zeros((2, 2, 6))), 0.0)


def test_fast_weight_operator_composition():
    q, k, v = (rnd((1, 2, 20, 4), s) for s in (132, 133, 134))
    beta = np.random.default_rng(135).uniform(0.0, 1.0, (1, 2, 20))
    wn, wf = rnd(2, 136), rnd(2, 137)
    sn, sf = 1 / (1 + np.exp(-wn)), 1 / (1 + np.exp(-wf))
    fw = ref.fast_weight_stream(q, k, v, beta)
    near = ref.near_stream(q, k, v, 3, True)
    lin = ref.far_stream(q, k, v, 1, True)
    for nl in (0, 1):
        got = ref.fmm_fast_weight_forward(q, k, v, beta, wn, wf, 3, nl)
        want = sn[None, :, None, None] * near + sf[None, :, None, None] * (fw + nl * lin)
        np.testing.assert_allclose(got, want, rtol=1e-13)


# ------------------------------------------------------------------ fast-weight backward
# The gradients of the fast-weight far field and of the whole fast-weight
# operator are pinned by central finite differences of the forward oracle and
# by torch float64 autograd of the recurrence written in torch.

def _fd(fn, args, eps=1e-6):
    out = []
    for ai, x in enumerate(args):
        g = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            a1, a2 = list(args), list(args)
            a1[ai], a2[ai] = xp, xm
            g[idx] = (fn(*a1) - fn(*a2)) / (2 * eps)
        out.append(g)
    return out


def test_fast_weight_backward_finite_differences():
    b, h, n, d = 1, 2, 7, 3
    q, k, v, f = (rnd((b, h, n, d), s) for s in (700, 701, 702, 703))
    beta = np.random.default_rng(704).uniform(0.0, 1.0, (b, h, n))
    fw, dq, dk, dv, dbeta = ref.fast_weight_backward_stream(q, k, v, beta, f)
    np.testing.assert_array_equal(fw, ref.fast_weight_stream(q, k, v, beta))
    loss = lambda q_, k_, v_, b_: float((ref.fast_weight_stream(q_, k_, v_, b_) * f).sum())
    want = _fd(loss, [q, k, v, beta])
    for g, w in zip((dq, dk, dv, dbeta), want):
        np.testing.assert_allclose(g, w, rtol=1e-6, atol=1e-8 * max(1.0, np.abs(w).max()))


def _torch_fast_weight(q, k, v, beta):
    def p(x):
        f = torch.nn.functional.elu(x) + 1
        return f / f.sum(-1, keepdim=True)
    pk, pq = p(k), p(q)
    b, h, n, d = q.shape
    w = torch.zeros(b, h, d, d, dtype=q.dtype)
    z = torch.zeros(b, h, d, dtype=q.dtype)
    outs = []
    for i in range(n):
        ki, qi = pk[:, :, i], pq[:, :, i]
        u = (w @ ki[..., None])[..., 0]
        w = w + beta[:, :, i, None, None] * (v[:, :, i] - u)[..., None] * ki[..., None, :]
        z = z + ki
        outs.append((w @ qi[..., None])[..., 0] / (z * qi).sum(-1, keepdim=True))
    return torch.stack(outs, dim=2)


def test_fast_weight_backward_matches_torch_autograd():
    b, h, n, d = 2, 2, 13, 4
    q, k, v, f = (rnd((b, h, n, d), s) for s in (710, 711, 712, 713))
    beta = np.random.default_rng(714).uniform(0.0, 1.0, (b, h, n))
    ts = [torch.tensor(x, requires_grad=True) for x in (q, k, v, beta)]
    (_torch_fast_weight(*ts) * torch.tensor(f)).sum().backward()
    got = ref.fast_weight_backward_stream(q, k, v, beta, f)[1:]
    for g, t in zip(got, ts):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("n_linear", [0, 1])
def test_fast_weight_operator_backward_finite_differences(n_linear):
    b, h, n, d, kw = 1, 2, 6, 3, 2
    q, k, v, g = (rnd((b, h, n, d), s) for s in (720, 721, 722, 723))
    beta = np.random.default_rng(724).uniform(0.0, 1.0, (b, h, n))
    wn, wf = rnd(h, 725), rnd(h, 726)
    got = ref.fmm_fast_weight_backward(q, k, v, beta, wn, wf, g, kw, n_linear)
    loss = lambda q_, k_, v_, b_, wn_, wf_: float(
        (ref.fmm_fast_weight_forward(q_, k_, v_, b_, wn_, wf_, kw, n_linear) * g).sum())
    want = _fd(loss, [q, k, v, beta, wn, wf])
    # got: dq, dk, dv, dbeta, dw_near, dw_far (the inputs' order)
    for gg, w in zip(got, want):
        np.testing.assert_allclose(gg, w, rtol=1e-6, atol=1e-8 * max(1.0, np.abs(w).max()))


# ------------------------------------------------------------------ layer backward
# Pinned by central finite differences of the layer's forward oracle and by
# torch float64 autograd of the layer written with the dense torch forward.

@pytest.mark.parametrize("causal", [False, True])
def test_layer_backward_finite_differences(causal):
    b, n, e, heads, kw, rank = 1, 5, 4, 2, 2, 2
    x = rnd((b, n, e), 730)
    wq, wo = rnd((e, 3 * e), 731, 0.5), rnd((e, e), 732, 0.5)
    wn, wf, dy = rnd(heads, 733), rnd(heads, 734), rnd((b, n, e), 735)
    got = ref.fmm_layer_backward(x, wq, wo, heads, wn, wf, dy, kw, rank, causal)
    loss = lambda x_, wq_, wo_, wn_, wf_: float(
        (ref.fmm_layer_forward(x_, wq_, wo_, heads, wn_, wf_, kw, rank, causal) * dy).sum())
    want = _fd(loss, [x, wq, wo, wn, wf])
    for g, w in zip(got, want):
        np.testing.assert_allclose(g, w, rtol=1e-6, atol=1e-8 * max(1.0, np.abs(w).max()))


@pytest.mark.parametrize("causal", [False, True])
def test_layer_backward_matches_torch_autograd(causal):
    b, n, e, heads, kw, rank = 2, 9, 6, 2, 2, 2
    d = e // heads
    x = rnd((b, n, e), 740)
    wq, wo = rnd((e, 3 * e), 741, 0.5), rnd((e, e), 742, 0.5)
    wn, wf, dy = rnd(heads, 743), rnd(heads, 744), rnd((b, n, e), 745)
    ts = [torch.tensor(a, requires_grad=True) for a in (x, wq, wo, wn, wf)]
    qkv = (ts[0] @ ts[1]).reshape(b, n, 3, heads, d)
    q, k, v = (qkv[:, :, p].permute(0, 2, 1, 3) for p in range(3))
    o = _torch_dense_forward(q, k, v, ts[3], ts[4], kw, rank, causal, "map")
    y = o.permute(0, 2, 1, 3).reshape(b, n, e) @ ts[2]
    (y * torch.tensor(dy)).sum().backward()
    got = ref.fmm_layer_backward(x, wq, wo, heads, wn, wf, dy, kw, rank, causal)
    for g, t in zip(got, ts):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-9, atol=1e-12)
