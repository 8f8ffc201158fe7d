"""The operator as a torch.autograd function (binding.fmm_attention): its
output is the forward entry point's and the gradients that autograd hands to
q, k, v and the two blend logits are the backward entry point's, bit for bit
(the entry points themselves are checked against the float64 oracle in the
forward and backward tests)."""

import numpy as np
import pytest
import torch

from fmm_testlib import log, upload
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,d,causal", [("bf16", 64, 0), ("bf16", 64, 1), ("f32", 32, 1),
                                            ("bf16", 32, 0)])
def test_autograd_matches_entry_points(dtype, d, causal):
    B, H, N, kw, rank = 2, 2, 1000, 32, 2
    log(f"autograd B={B} H={H} N={N} d={d} k={kw} r={rank} causal={causal} {dtype}")
    q, k, v, wn, wf = make_inputs(B, H, N, d, dtype, 1.0 / np.sqrt(d), 1600 + d + causal)
    t = upload(q, k, v, wn, wf, dtype)
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(1601)
    g = torch.randn(t[0].shape, generator=gen, device="cuda:0").to(t[0].dtype)
    leaves = [x.clone().requires_grad_(True) for x in t]
    out = binding.fmm_attention(*leaves, kw, rank, causal)
    # the loss sum(out * g): its gradient with respect to out is g
    (out.float() * g.float()).sum().backward()
    want_out = binding.forward(*t, kw, rank, causal)
    want = binding.backward(t[0], t[1], t[2], g, t[3], t[4], kw, rank, causal)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), want_out)
    for name, leaf, w in zip(("q", "k", "v", "w_near", "w_far"), leaves, want):
        assert leaf.grad is not None and leaf.grad.shape == leaf.shape, name
        assert torch.equal(leaf.grad, w), name


@pytest.mark.parametrize("causal", [0, 1])
def test_autograd_joint_normalisation(causal):
    B, H, N, d, kw, rank = 1, 2, 800, 64, 24, 3
    q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 1620 + causal)
    t = upload(q, k, v, wn, wf, "bf16")
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(1621)
    g = torch.randn(t[0].shape, generator=gen, device="cuda:0").to(t[0].dtype)
    leaves = [x.clone().requires_grad_(True) for x in t]
    out = binding.fmm_attention(*leaves, kw, rank, causal, joint=True)
    (out.float() * g.float()).sum().backward()
    want_out = binding.forward(*t, kw, rank, causal, joint=True)
    want = binding.backward(t[0], t[1], t[2], g, t[3], t[4], kw, rank, causal, joint=True)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), want_out)
    for name, leaf, w in zip(("q", "k", "v", "w_near", "w_far"), leaves, want):
        assert torch.equal(leaf.grad, w), name


def test_autograd_only_where_asked():
    # inputs without requires_grad get no gradient; the others still do
    B, H, N, d, kw, rank = 1, 2, 700, 32, 16, 2
    q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 1650)
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, "bf16")
    tq.requires_grad_(True)
    twf.requires_grad_(True)
    out = binding.fmm_attention(tq, tk, tv, twn, twf, kw, rank, 0)
    out.float().sum().backward()
    torch.cuda.synchronize()
    assert tq.grad is not None and twf.grad is not None
    assert tk.grad is None and tv.grad is None and twn.grad is None
    want = binding.backward(tq.detach(), tk, tv, torch.ones_like(out), twn, twf.detach(), kw,
                            rank, 0)
    assert torch.equal(tq.grad, want[0]) and torch.equal(twf.grad, want[4])


@pytest.mark.parametrize("n_linear", [0, 1])
def test_fast_weight_autograd_matches_entry_points(n_linear):
    B, H, N, d, kw = 2, 2, 200, 16, 20
    q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0, 1660 + n_linear)
    t = list(upload(q, k, v, wn, wf, "bf16"))
    beta = torch.from_numpy(np.random.default_rng(1661).uniform(0, 1, (B, H, N))
                            .astype(np.float32)).to("cuda:0")
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(1662)
    g = torch.randn(t[0].shape, generator=gen, device="cuda:0").to(t[0].dtype)
    ins = [t[0], t[1], t[2], beta, t[3], t[4]]
    leaves = [x.clone().requires_grad_(True) for x in ins]
    out = binding.fmm_fast_weight_attention(*leaves, kw, n_linear)
    (out.float() * g.float()).sum().backward()
    want_out = binding.forward_fastweight(t[0], t[1], t[2], beta, t[3], t[4], kw, n_linear)
    want = binding.backward_fastweight(t[0], t[1], t[2], beta, g, t[3], t[4], kw, n_linear)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), want_out)
    for name, leaf, w in zip(("q", "k", "v", "beta", "w_near", "w_far"), leaves, want):
        assert torch.equal(leaf.grad, w), name


def test_training_steps_through_the_operator():
    # a small attention layer trained through the operator: projections in
    # torch, the operator through fmm_attention (bf16, causal, rank 2), SGD
    # on a fixed synthetic regression target; the loss must fall, and every
    # gradient that reaches the layer's parameters must be finite
    torch.manual_seed(1700)
    B, N, E, H, kw, rank = 2, 512, 64, 2, 32, 2
    d = E // H
    dev = "cuda:0"
    w_qkv = (torch.randn(E, 3 * E, device=dev) / np.sqrt(E)).requires_grad_(True)
    w_out = (torch.randn(E, E, device=dev) / np.sqrt(E)).requires_grad_(True)
    w_near = torch.zeros(H, device=dev, requires_grad=True)
    w_far = torch.zeros(H, device=dev, requires_grad=True)
    x = torch.randn(B, N, E, device=dev)
    target = torch.roll(x, 1, dims=1) * 0.5  # a causal target: the previous token

    def layer(x):
        qkv = (x @ w_qkv).to(torch.bfloat16)
        q, k, v = (t.reshape(B, N, H, d).permute(0, 2, 1, 3).contiguous()
                   for t in qkv.split(E, dim=-1))
        o = binding.fmm_attention(q, k, v, w_near, w_far, kw, rank, True)
        return o.permute(0, 2, 1, 3).reshape(B, N, E).float() @ w_out

    losses = []
    params = [w_qkv, w_out, w_near, w_far]
    for step in range(30):
        loss = ((layer(x) - target) ** 2).mean()
        for p in params:
            p.grad = None
        loss.backward()
        for p in params:
            assert p.grad is not None and torch.isfinite(p.grad).all()
        with torch.no_grad():
            for p in params:
                p -= 0.5 * p.grad
        losses.append(float(loss.detach()))
    log(f"training loss {losses[0]:.4f} -> {losses[10]:.4f} -> {losses[-1]:.4f}")
    assert losses[-1] < losses[10] < losses[0]
    assert losses[-1] < 0.95 * losses[0]
