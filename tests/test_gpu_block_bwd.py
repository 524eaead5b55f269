"""Training the block on the GPU: dsp_st_block_forward_train and
dsp_st_block_backward against the oracle's chain rule (oracle.st_block_bwd).

The GPU gets the exact bf16 weights and fp32 inputs the oracle uses; dy is
N(0, 1) in fp32.  Bars, after dividing each gradient by its largest magnitude
in the oracle: fp32 1e-4 max-abs and 1e-5 relative L2 (every step in fp32).
bf16: the forward's bar, 2e-2 max-abs and 1e-2 relative L2.  The gradient
passes through about a dozen products whose operands are rounded to bf16 (the
upstream gradient at every GEMM and attention input, the saved activations,
the probabilities and dZ), each contributing ~2^-9 relative; the measured
errors are ~4e-3.  ReLU's derivative decides on the sign of its input, so the
ReLU cases keep that input away from zero (see _train_case)."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import assert_close, dev, host, say, errors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _oracle_params(stored):
    return {n: (None if v is None else (v.T if n.startswith("w") else v)) for n, v in stored.items()}


def _grad_close(got, want, dtype, what):
    mx = float(np.abs(want).max())
    assert mx > 0, what
    a, r = errors(got / mx, want / mx)
    ta, tr = (1e-4, 1e-5) if dtype == "f32" else (2e-2, 1e-2)
    say(f"  {what}: max_abs/max={a:.2e} rel_l2={r:.2e} (tol {ta:g}/{tr:g})")
    assert a <= ta and r <= tr, what


def _train_case(torch, w, with_bias, flags):
    import paper_2403_10266_amd as dsp
    x, p = synth.block_inputs(w, with_bias=with_bias)
    if flags & dsp.DSP_BLOCK_RELU:
        # ReLU's derivative is a decision on the sign of u.  Where |u| is within the
        # rounding of the bf16 operands of 0, the GPU (bf16 operands) and the oracle
        # (fp64) may decide differently; a bias of +-3 on the first MLP layer keeps
        # |u| far from 0 (|h3 W1| stays below ~1.2 here, also without the MLP's LN)
        # while still masking about half of the units.
        signs = np.where(np.random.default_rng(w.seed + 2).random(w.F) < 0.5, -3.0, 3.0).astype(np.float32)
        p["b1"] = signs
    dy = np.random.default_rng(w.seed + 1).standard_normal((w.B, w.S, w.T, w.C), dtype=np.float32)
    say(f"block train {w.name} {x.shape} bias={with_bias} flags={flags}")
    wd = {n: (None if v is None else dev(v, w.dtype)) for n, v in p.items()}
    xd = dev(x, "f32")
    y, saved = dsp.dsp_st_block_forward_train(xd, wd, w.H, flags=flags)
    dx, g = dsp.dsp_st_block_backward(xd, dev(dy, "f32"), wd, saved, w.H, flags=flags, with_bias=True)
    torch.cuda.synchronize()
    po = _oracle_params(p)
    assert_close(host(y), oracle.st_block(x, po, w.H, flags=flags), w.dtype, "forward (training) output")
    want_dx, want_g = oracle.st_block_bwd(x, po, w.H, dy, flags=flags)
    _grad_close(host(dx), want_dx, w.dtype, "dx")
    for n, v in want_g.items():
        # the oracle's weight gradients are [in, out]; the library's follow the stored [out][in]
        _grad_close(host(g[n]), v.T if n.startswith("w") else v, w.dtype, n)
    if not with_bias:
        # bias gradients exist whether or not the forward used biases: the row sums of
        # the gradient at each linear map's output
        C = w.C
        for n in ("bo_s", "bo_t", "b2"):
            assert g[n].shape == (C,)
    return dx, g


@pytest.mark.parametrize("with_bias", [False, True])
@pytest.mark.parametrize("flags", [0, 1, 8, 9, 4, 5, 12, 13])
def test_block_train_bf16(torch, with_bias, flags):
    """Pre-LN (flags 0, 1, 8, 9) and the paper's post-LN block (4, 5, 12, 13:
    LN after each residual add), GELU or ReLU, with or without the MLP's LN."""
    w = synth.Workload("block_small", "block", "bf16", B=2, T=5, S=24, C=144, H=2, F=576, seed=21)
    _train_case(torch, w, with_bias, flags)


@pytest.mark.parametrize("flags", [0, 9, 4, 13])
def test_block_train_f32(torch, flags):
    w = synth.Workload("block_small_f32", "block", "f32", B=1, T=4, S=9, C=64, H=4, F=128, seed=22)
    _train_case(torch, w, True, flags)


@pytest.mark.parametrize("flags,T", [(0, 16), (4, 8)])
def test_block_train_full_width_bf16(torch, flags, T):
    """The 720M model's widths (C = 1152, 16 heads of 72, MLP 4608) on 4096 and
    2048 tokens; at 4096 the MLP's first GEMM (with the pre-activation kept)
    runs on the large-tile kernel."""
    w = synth.Workload("block_wide", "block", "bf16", B=1, T=T, S=256, C=1152, H=16, F=4608, seed=23)
    _train_case(torch, w, False, flags)


def test_block_train_large_tiles_partial_bf16(torch):
    """Widths that are not multiples of 64 (C = 864, 12 heads of 72; MLP 3464)
    on 5120 tokens: the MLP's second weight takes the large-tile input gradient,
    so its transpose has partial 64 x 64 tiles in both dimensions, and the first
    GEMM keeps GELU' over a ragged last tile column."""
    w = synth.Workload("block_ragged", "block", "bf16", B=1, T=20, S=256, C=864, H=12, F=3464, seed=24)
    _train_case(torch, w, True, 0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("flags", [0, 1, 4, 5, 12, 13])
def test_forward_train_output_matches_forward(torch, dtype, flags):
    """The training forward writes the bits dsp_st_block_forward writes."""
    import paper_2403_10266_amd as dsp
    w = synth.Workload("block_bits", "block", dtype, B=1, T=6, S=40, C=144, H=2, F=576, seed=24)
    x, p = synth.block_inputs(w, with_bias=True)
    wd = {n: (None if v is None else dev(v, dtype)) for n, v in p.items()}
    xd = dev(x, "f32")
    y_train, _ = dsp.dsp_st_block_forward_train(xd, wd, w.H, flags=flags)
    y = dsp.dsp_st_block_forward(xd, wd, w.H, flags=flags)
    torch.cuda.synchronize()
    assert torch.equal(y_train, y), flags


@pytest.mark.parametrize("flags", [0, 5])
def test_forward_train_matches_forward_full_size(torch, flags):
    """The bench workload (B1 T32 S1024, 32768 tokens: every GEMM on the
    large-tile kernel): the training forward writes the inference forward's bits."""
    import paper_2403_10266_amd as dsp
    w = synth.WORKLOADS["block_bf16_B1_T32_S1024"]
    x, p = synth.block_inputs(w)
    wd = {n: (None if v is None else dev(v, "bf16")) for n, v in p.items()}
    xd = dev(x, "f32")
    y_train, saved = dsp.dsp_st_block_forward_train(xd, wd, w.H, flags=flags)
    del saved
    y = dsp.dsp_st_block_forward(xd, wd, w.H, flags=flags)
    torch.cuda.synchronize()
    assert torch.equal(y_train, y)


def test_block_backward_deterministic_and_finite_full_size(torch):
    """The bench workload (B1 T32 S1024): two backward calls give identical bits."""
    import paper_2403_10266_amd as dsp
    w = synth.WORKLOADS["block_bf16_B1_T32_S1024"]
    x, p = synth.block_inputs(w)
    wd = {n: (None if v is None else dev(v, "bf16")) for n, v in p.items()}
    xd = dev(x, "f32")
    dy = torch.randn((w.B, w.S, w.T, w.C), generator=torch.Generator(device="cuda").manual_seed(3),
                     device="cuda")
    _, saved = dsp.dsp_st_block_forward_train(xd, wd, w.H)
    dx1, g1 = dsp.dsp_st_block_backward(xd, dy, wd, saved, w.H)
    dx2, g2 = dsp.dsp_st_block_backward(xd, dy, wd, saved, w.H)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(dx1).all())
    assert torch.equal(dx1, dx2)
    for n in g1:
        assert bool(torch.isfinite(g1[n]).all()) and torch.equal(g1[n], g2[n]), n


def test_block_backward_homogeneous_full_size(torch):
    """The bench workload: the backward is linear in dy, and every step of it
    (bf16 rounding of an operand, fp32 sums in a fixed order, the LayerNorm
    backward, dZ = P * (dP - Delta) with Delta's hi/lo split, the split-K
    reductions) commutes exactly with scaling by a power of two, so
    backward(2 dy) has exactly twice the bits of backward(dy): a property of
    the whole chain that holds at any size."""
    import paper_2403_10266_amd as dsp
    w = synth.WORKLOADS["block_bf16_B1_T32_S1024"]
    x, p = synth.block_inputs(w)
    wd = {n: (None if v is None else dev(v, "bf16")) for n, v in p.items()}
    xd = dev(x, "f32")
    dy = torch.randn((w.B, w.S, w.T, w.C), generator=torch.Generator(device="cuda").manual_seed(5),
                     device="cuda")
    _, saved = dsp.dsp_st_block_forward_train(xd, wd, w.H)
    dx1, g1 = dsp.dsp_st_block_backward(xd, dy, wd, saved, w.H, with_bias=True)
    dx2, g2 = dsp.dsp_st_block_backward(xd, dy * 2.0, wd, saved, w.H, with_bias=True)
    torch.cuda.synchronize()
    assert torch.equal(dx2, dx1 * 2.0)
    for n in g1:
        assert torch.equal(g2[n], g1[n] * 2.0), n



def test_block_backward_full_size_sampled_against_oracle(torch):
    """The bench workload (B1 T32 S1024, C 1152, 16 heads, MLP 4608, the
    split-K weight-gradient counts chosen at 32768 tokens) against the fp64
    oracle's chain rule: 8 whole rows of dx and 128 entries of every weight
    gradient, stored by tests/golden/make_block_bwd_samples.py (oracle only).
    Errors are taken relative to each tensor's largest magnitude, as in the
    smaller cases above."""
    import json
    from pathlib import Path
    import paper_2403_10266_amd as dsp
    gold = json.loads((Path(__file__).parent / "golden" / "block_bwd_B1_T32_S1024_samples.json").read_text())
    w = synth.WORKLOADS["block_bf16_B1_T32_S1024"]
    x, p = synth.block_inputs(w)
    dy = np.random.default_rng(w.seed + 1).standard_normal((w.B, w.S, w.T, w.C), dtype=np.float32)
    say(f"block backward sampled {w.name}")
    wd = {n: (None if v is None else dev(v, "bf16")) for n, v in p.items()}
    xd = dev(x, "f32")
    _, saved = dsp.dsp_st_block_forward_train(xd, wd, w.H)
    dx, g = dsp.dsp_st_block_backward(xd, dev(dy, "f32"), wd, saved, w.H)
    torch.cuda.synchronize()
    dxh = host(dx)
    # dx is returned in the input's (B, T, S, C) order
    got = np.stack([dxh[b, t, s] for b, t, s in gold["dx_rows"]])
    mx = gold["dx_max_abs"]
    a, r = errors(got / mx, np.asarray(gold["dx"]) / mx)
    say(f"  dx rows: max_abs/max={a:.2e} rel_l2={r:.2e}")
    assert a <= 2e-2 and r <= 1e-2, "dx"
    for n, e in gold["grads"].items():
        gh = host(g[n])
        got = np.array([gh[i, j] for i, j in e["pos"]])
        mx = e["max_abs"]
        a, r = errors(got / mx, np.asarray(e["val"]) / mx)
        say(f"  {n} ({len(got)} entries): max_abs/max={a:.2e} rel_l2={r:.2e}")
        assert a <= 2e-2 and r <= 1e-2, n
