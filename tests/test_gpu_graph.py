"""The library under HIP graph capture: every entry point the block runs is a
plain sequence of kernel launches on the caller's stream (no allocation, no
memset, no synchronisation), so a captured graph replays it.  Each replay is
checked against the eager result, with eager work and synchronisations
between the replays, and after the input is changed in place (the graph reads
the input buffer, not a copy)."""
import numpy as np
import pytest

import synth
from tests.gpu_util import dev, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _capture(torch, fn):
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()  # warm-up outside the graph
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _replays_match(torch, g, out, eager_fn, x, n=3):
    for i in range(n):
        out.fill_(float("nan"))          # eager work between replays
        if i == 2:
            x.mul_(0.5)                   # the graph must see the new input
        want = eager_fn().clone()
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want), f"replay {i}"


def test_tiny_chain_graph(torch):
    import paper_2403_10266_amd as dsp
    wl = synth.WORKLOADS["tiny_chain_f32"]
    x, p = synth.chain_inputs(wl)
    xd = dev(x, "f32")
    wd = {n: dev(v, "f32") for n, v in p.items()}
    out = torch.empty((wl.B, wl.S, wl.T, wl.C), dtype=torch.float32, device="cuda")
    ws = torch.empty(dsp.block_workspace_bytes(wl.B, wl.T, wl.S, wl.C, wl.H, 0, dsp.DSP_F32),
                     dtype=torch.uint8, device="cuda")
    run = lambda: dsp.dsp_st_block_forward(xd, wd, wl.H, flags=dsp.DSP_BLOCK_ATTN_ONLY, out=out, workspace=ws)
    say("tiny chain under graph capture")
    g = _capture(torch, run)
    _replays_match(torch, g, out, run, xd)


@pytest.mark.parametrize("flags", [0, 5])
def test_block_graph_bf16(torch, flags):
    import paper_2403_10266_amd as dsp
    w = synth.Workload("block_graph", "block", "bf16", B=1, T=6, S=80, C=144, H=2, F=576, seed=31)
    x, p = synth.block_inputs(w, with_bias=True)
    xd = dev(x, "f32")
    wd = {n: (None if v is None else dev(v, "bf16")) for n, v in p.items()}
    out = torch.empty((w.B, w.S, w.T, w.C), dtype=torch.float32, device="cuda")
    ws = torch.empty(dsp.block_workspace_bytes(w.B, w.T, w.S, w.C, w.H, w.F, dsp.DSP_BF16),
                     dtype=torch.uint8, device="cuda")
    run = lambda: dsp.dsp_st_block_forward(xd, wd, w.H, flags=flags, out=out, workspace=ws)
    say(f"bf16 block flags={flags} under graph capture")
    g = _capture(torch, run)
    _replays_match(torch, g, out, run, xd)
    assert bool(torch.isfinite(out).all())
