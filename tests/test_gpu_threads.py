"""Calls from several host threads at once, each on its own stream: the
library keeps one workspace per (device, stream) and holds its workspace lock
from the workspace lookup until the call's kernels are enqueued, so calls on
different streams must neither share nor free each other's workspace.  Each
thread repeats its calls and compares every output bit for bit with the same
call made alone beforehand."""

import threading

import numpy as np
import pytest
import torch

from fmm_testlib import log, upload
from paper_2108_02347_amd import binding
from paper_2108_02347_amd.inputs import make_inputs

pytestmark = pytest.mark.gpu

# (B, H, N, d, band_k, rank, causal): the one-launch path, the three-launch
# causal path, and a shape whose workspace is larger than the others' (so a
# stream's workspace grows while another thread uses its own)
SHAPES = [
    (8, 2, 4096, 32, 20, 2, 0),
    (2, 4, 3000, 64, 40, 2, 1),
    (1, 8, 16384, 64, 64, 2, 0),
]


def test_concurrent_calls_on_separate_streams():
    cases = []
    for i, (B, H, N, d, kw, rank, causal) in enumerate(SHAPES):
        q, k, v, wn, wf = make_inputs(B, H, N, d, "bf16", 1.0 / np.sqrt(d), 1500 + i)
        t = upload(q, k, v, wn, wf, "bf16")
        want = binding.forward(*t, kw, rank, causal)
        cases.append((t, kw, rank, causal, want))
    torch.cuda.synchronize()
    errors = []
    rounds = 15

    def worker(tid):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                outs = [torch.empty_like(c[0][0]) for c in cases]
                for r in range(rounds):
                    # each thread walks the shapes in its own order
                    for j in range(len(cases)):
                        ci = (j + tid + r) % len(cases)
                        t, kw, rank, causal, want = cases[ci]
                        outs[ci].fill_(7.0)
                        binding.forward(*t, kw, rank, causal, out=outs[ci])
                        s.synchronize()
                        if not torch.equal(outs[ci].view(torch.int16), want.view(torch.int16)):
                            errors.append((tid, r, ci))
                            return
        except Exception as e:  # reported below, in the main thread
            errors.append((tid, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(3)]
    log(f"3 threads x {rounds} rounds x {len(cases)} shapes, one stream each")
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads), "a thread did not finish"
    assert not errors, errors
