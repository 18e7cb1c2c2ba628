"""Decode steps captured in a HIP graph (a serving loop without a host
launch per token): every replay, with the program's own eager work and
synchronisations between replays, equals the eager launches bit for bit."""
import numpy as np
import pytest
import torch

from paper_2606_08804_amd import qdelta, synth

pytestmark = pytest.mark.gpu


def test_captured_decode_steps_equal_eager():
    N, H, D, steps = 16, 4, 128, 12
    d = synth.make_decode(N, H, D, steps)
    q, k, v = d["q"].cuda(), d["k"].cuda(), d["v"].cuda()
    beta, lam, la = d["beta"].cuda(), d["lam"].cuda(), d["log_alpha"].cuda()
    S0 = d["initial_state"].cuda()
    S = S0.clone()
    outs = torch.empty((steps, N, H, D), dtype=torch.bfloat16, device="cuda")

    def decode_all():
        for s in range(steps):
            qdelta.recurrent_step(q[s], k[s], v[s], beta[s], lam[s], la[s], S, out=outs[s])

    decode_all()
    torch.cuda.synchronize()
    o_ref, S_ref = outs.clone(), S.clone()

    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        S.copy_(S0)
        decode_all()
        torch.cuda.synchronize()
        S.copy_(S0)
        with torch.cuda.graph(graph, stream=cap):
            decode_all()
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()
    for rep in range(4):
        outs.zero_()
        S.copy_(S0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs, o_ref), f"replay {rep}: outputs differ from the eager launches"
        assert torch.equal(S, S_ref), f"replay {rep}: state differs from the eager launches"
        # eager work between replays
        scratch = torch.randn(1 << 16, device="cuda").sum()
        assert torch.isfinite(scratch)
