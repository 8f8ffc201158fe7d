"""Parity of the general apply path with the float64 oracle: head width 128,
the third feature map (phi_3 = tanh) and the joint far-field normalisation,
in both forms and both storage types.

Tolerance.  Joint normalisation and inputs that keep phi_3's denominator away
from zero use the same worst-slice bound as the other tests.  With per-map
normalisation (Eq. (9)) phi_3(q)^T z_3 has no fixed sign and comes arbitrarily
close to zero for N(0, 1) inputs, so the quotient is ill-conditioned there; on
such inputs each element is held to a bound from the arithmetic: the numerator
and denominator of map l carry errors up to eta * A and eta * B (A, B the sums
of absolute products that form them, eta = the dtype's tolerance), which
divide into |far| as eta * (B / |den| + |num| A / den^2)."""

import numpy as np
import pytest
import torch

from fmm_testlib import TOL, check_full, floored_mean_rel_error, log, slice_errors, upload
from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu


def run(q, k, v, wn, wf, kw, rank, causal, dtype, joint):
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, dtype)
    out = binding.forward(tq, tk, tv, twn, twf, kw, rank, causal, joint=joint)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


def check(B, H, N, d, kw, rank, causal, dtype, joint, seed, shift=0.0, std=1.0):
    q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, std, seed)
    if shift:
        # shifted queries and keys (rounded to the storage type again)
        from paper_2108_02347_amd.inputs import to_dtype
        q, k = to_dtype(q + shift, dtype), to_dtype(k + shift, dtype)
    log(f"case B={B} H={H} N={N} d={d} k={kw} r={rank} causal={causal} {dtype} "
        f"joint={joint} shift={shift}")
    got = run(q, k, v, wn, wf, kw, rank, causal, dtype, joint)
    want = ref.fmm_attention_stream(q, k, v, wn, wf, kw, rank, bool(causal),
                                    norm="joint" if joint else "map")
    assert np.isfinite(got).all()
    err = slice_errors(got, want).max()
    log(f"  max slice error {err:.3e}, floored mean relative "
        f"{floored_mean_rel_error(got, want):.3e}")
    assert err <= TOL[dtype]
    return err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
def test_width_128(dtype, causal):
    # several tiles and state segments per slice, bands narrower and wider
    # than a staging round, a ragged tail
    worst = 0.0
    for B, H, N, kw, rank in ((2, 2, 2000, 64, 2), (1, 3, 777, 5, 1), (1, 1, 1500, 300, 2),
                              (3, 1, 64, 0, 2)):
        worst = max(worst, check(B, H, N, 128, kw, rank, causal, dtype, False, 900 + N + kw,
                                 std=1.0 / np.sqrt(128)))
    log(f"d=128 {dtype} causal={causal}: worst {worst:.3e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
@pytest.mark.parametrize("d", [16, 32, 64, 128])
def test_joint_normalisation(d, causal, dtype):
    worst = 0.0
    for rank in (1, 2, 3):
        for N, kw in ((300, 7), (1100, 40)):
            worst = max(worst, check(2, 2, N, d, kw, rank, causal, dtype, True,
                                     1000 + d + 10 * rank + N))
    log(f"joint d={d} {dtype} causal={causal}: worst {worst:.3e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
@pytest.mark.parametrize("d", [16, 32, 64, 128])
def test_rank3_well_conditioned(d, causal, dtype):
    # queries and keys with mean 1: phi_3's denominator keeps one sign
    worst = 0.0
    for N, kw in ((300, 7), (1100, 40)):
        worst = max(worst, check(2, 2, N, d, kw, 3, causal, dtype, False, 1200 + d + N,
                                 shift=1.0))
    log(f"rank 3 d={d} {dtype} causal={causal}: worst {worst:.3e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [0, 1])
def test_rank3_standard_normal_conditioned_bound(causal, dtype):
    # N(0, 1) inputs: elementwise bound scaled by the conditioning of each map
    B, H, N, d, kw = 2, 2, 1500, 32, 20
    q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, 1.0, 1300 + causal)
    got = run(q, k, v, wn, wf, kw, 3, causal, dtype, False)
    want = ref.fmm_attention_stream(q, k, v, wn, wf, kw, 3, bool(causal))
    terms = ref.far_terms_stream(q, k, v, 3, bool(causal))
    absq = np.abs(q)
    bound = np.zeros_like(want)
    for l, (num, den) in enumerate(terms, start=1):
        aq = np.abs(ref.phi(q, l))
        ak, av = np.abs(ref.phi(k, l)), np.abs(v)
        if causal:
            za = np.cumsum(ak, axis=2)
            sa = np.cumsum(ak[..., :, None] * av[..., None, :], axis=2)
            A = np.einsum("bhic,bhic->bhi", aq, za)
            Bm = np.einsum("bhic,bhice->bhie", aq, sa)
        else:
            A = np.einsum("bhic,bhc->bhi", aq, ak.sum(axis=2))
            Bm = np.einsum("bhic,bhce->bhie", aq, np.einsum("bhjc,bhje->bhce", ak, av))
        bound += Bm / np.abs(den)[..., None] + np.abs(num) * (A / den ** 2)[..., None]
    sf = 1.0 / (1.0 + np.exp(-wf))
    eta = TOL[dtype]
    scale = np.abs(want).max(axis=(2, 3), keepdims=True)
    allowed = eta * scale + eta * sf[None, :, None, None] * bound
    excess = (np.abs(got - want) / allowed).max()
    worst_den = min(np.abs(t[1]).min() for t in terms)
    log(f"rank 3 N(0,1) causal={causal} {dtype}: max error / bound {excess:.3e}, "
        f"smallest |den| {worst_den:.3e}")
    assert np.isfinite(got).all()
    assert excess <= 1.0
