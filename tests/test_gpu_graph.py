"""Graph capture of the forward: a call captured into a HIP graph (through
torch.cuda.CUDAGraph) and replayed with new inputs copied into the captured
tensors, with eager calls and synchronisations between the replays, must give
exactly the bits of an eager call on the same inputs.

The one-launch path is the case that needs care: its workgroups exchange
partial far-field states through stamps in memory, and the kernel arguments
of a captured launch are frozen, so a replay must not take the stamps left by
the previous replay (same workspace, same slots) for its own.  Back-to-back
replays with different inputs are the sharpest form of that, and each case
runs them.  The three-launch causal path is covered too (it must enqueue
nothing that a graph cannot replay)."""

import numpy as np
import pytest
import torch

from fmm_testlib import TOL, log, slice_errors, upload
from oracle import fmm_ref as ref
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu

# (entry point, (B, H, N, d, band_k, rank), causal)
CASES = [
    ("noalloc", (8, 2, 4096, 32, 20, 2), 0),  # one launch: the 4K retrieval shape
    ("ws", (4, 2, 1000, 64, 64, 2), 0),       # one launch, ragged tail, caller workspace
    ("noalloc", (2, 4, 3000, 64, 40, 2), 1),  # causal: state, scan and apply launches
]


def _ids(c):
    e, (B, H, N, d, kw, r), causal = c
    return f"{e}-B{B}H{H}N{N}d{d}k{kw}r{r}c{causal}"


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_graph_replays_match_eager(case):
    entry, (B, H, N, d, kw, rank), causal = case
    log(f"graph case {_ids(case)} bf16")
    sets = []
    for i in range(4):
        q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 1200 + 7 * i)
        sets.append(((q, k, v, wn, wf), upload(q, k, v, wn, wf, "bf16")))
    _, (q0, k0, v0, twn, twf) = sets[0]
    sq, sk, sv = q0.clone(), k0.clone(), v0.clone()
    out = torch.empty_like(sq)
    ws = None
    if entry == "ws":
        nbytes = binding.workspace_bytes(B, H, N, d, rank, causal)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")

    def call(q, k, v, o):
        if entry == "ws":
            return binding.forward_ws(q, k, v, twn, twf, kw, rank, causal, ws, out=o)
        return binding.forward_noalloc(q, k, v, twn, twf, kw, rank, causal, out=o)

    prev = binding.set_one_launch(1)
    try:
        call(sq, sk, sv, out)  # first call outside the capture (one-time set-up)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            call(sq, sk, sv, out)
        torch.cuda.synchronize()
        for rep in range(3):
            i, j = rep % 4, (rep + 1) % 4
            # two replays back to back with different inputs, then eager calls
            sq.copy_(sets[i][1][0]), sk.copy_(sets[i][1][1]), sv.copy_(sets[i][1][2])
            g.replay()
            r1 = out.clone()
            sq.copy_(sets[j][1][0]), sk.copy_(sets[j][1][1]), sv.copy_(sets[j][1][2])
            g.replay()
            r2 = out.clone()
            e1 = call(*sets[i][1][:3], torch.empty_like(out))
            e2 = call(*sets[j][1][:3], torch.empty_like(out))
            torch.cuda.synchronize()
            assert torch.equal(r1.view(torch.int16), e1.view(torch.int16)), (rep, i)
            assert torch.equal(r2.view(torch.int16), e2.view(torch.int16)), (rep, j)
            if rep == 0:
                q, k, v = sets[i][0][:3]
                wn, wf = sets[0][0][3:]  # the captured weights
                want = ref.fmm_attention_stream(q, k, v, wn, wf, kw, rank, bool(causal))
                err = slice_errors(r1.float().cpu().numpy().astype(np.float64), want).max()
                log(f"  replay against the oracle: {err:.3e}")
                assert err <= TOL["bf16"]
        del g
    finally:
        binding.set_one_launch(prev)


def test_capture_needing_a_new_workspace_is_rejected():
    # a stream without a library-owned workspace cannot get one while it is
    # under capture: the call must fail with nothing enqueued
    B, H, N, d, kw, rank = 2, 2, 700, 32, 9, 2
    q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 1300)
    tq, tk, tv, twn, twf = upload(q, k, v, wn, wf, "bf16")
    # one call first (one-time kernel set-up), then every workspace freed, so
    # that the stream below has none whichever stream of torch's pool it is
    binding.forward(tq, tk, tv, twn, twf, kw, rank, 1)
    torch.cuda.synchronize()
    binding.release_workspace()
    out = torch.full_like(tq, 3.0)
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    status = None
    with torch.cuda.graph(g, stream=s):
        try:
            binding.forward(tq, tk, tv, twn, twf, kw, rank, 1, out=out)
        except binding.FmmError as e:
            status = e.status
    torch.cuda.synchronize()
    assert status == binding.FMM_ERR_UNSUPPORTED
    assert bool((out == 3.0).all())
    del g
    # after one call on that stream outside the capture, capturing works
    with torch.cuda.stream(s):
        want = binding.forward(tq, tk, tv, twn, twf, kw, rank, 1)
    torch.cuda.synchronize()
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=s):
        binding.forward(tq, tk, tv, twn, twf, kw, rank, 1, out=out)
    g2.replay()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), want.view(torch.int16))


def test_backward_graph_replays_match_eager():
    # the backward enqueues kernels only: captured once (after an eager call
    # that sets up its workspace) and replayed with new inputs, it must give
    # the eager call's bits
    B, H, N, d, kw, rank, causal = 2, 2, 1500, 64, 32, 2, 1
    sets = []
    for i in range(3):
        q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 1700 + i)
        t = upload(q, k, v, wn, wf, "bf16")
        g = upload(make_inputs(B, H, N, d, "bf16", 1.0, 1710 + i)[0], q, q, wn, wf, "bf16")[0]
        sets.append((t, g))
    (tq, tk, tv, twn, twf), tg = sets[0]
    sq, sk, sv, sg = tq.clone(), tk.clone(), tv.clone(), tg.clone()
    # the library's workspace is per stream: one eager call on the stream that
    # will capture sets it up
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        binding.backward(sq, sk, sv, sg, twn, twf, kw, rank, causal)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        outs = binding.backward(sq, sk, sv, sg, twn, twf, kw, rank, causal)
    torch.cuda.synchronize()
    for rep in range(3):
        (q_, k_, v_, _, _), g_ = sets[rep]
        sq.copy_(q_), sk.copy_(k_), sv.copy_(v_), sg.copy_(g_)
        graph.replay()
        got = [o.clone() for o in outs]
        want = binding.backward(q_, k_, v_, g_, twn, twf, kw, rank, causal)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv", "dw_near", "dw_far"), got, want):
            assert torch.equal(a, b), (rep, name)
    del graph
