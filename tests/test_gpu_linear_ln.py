"""LayerNorm and the linear maps (with their epilogues) on the GPU against the oracle."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import assert_close, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


@pytest.mark.parametrize("rows,C", [(1, 64), (37, 1152), (5, 100), (3, 3000)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_layernorm(torch, rows, C, out):
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(rows + C)
    x = (rng.standard_normal((rows, C), dtype=np.float32) * 2 + 0.5).astype(np.float32)
    xd = dev(x, "f32")
    y = dsp.dsp_layernorm(xd, 1e-6, out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    torch.cuda.synchronize()
    say(f"layernorm rows={rows} C={C} -> {out}")
    assert_close(host(y), oracle.layernorm(x, 1e-6), out, "layernorm")


# ragged M, N and K tails, a single partial K slice, and the block's own N = 3C
@pytest.mark.parametrize("M,N,K", [(1, 8, 8), (300, 200, 72), (513, 1152, 1152), (64, 4608, 1152),
                                   (257, 136, 4608), (256, 192, 8), (777, 385, 104),
                                   (512, 3456, 1152)])
@pytest.mark.parametrize("epi", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("bias", [False, True])
def test_linear_bf16(torch, M, N, K, epi, bias):
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(M * 7 + N + K)
    a = synth.bf16_round(rng.standard_normal((M, K), dtype=np.float32))
    w = synth.bf16_round(rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02))
    b = synth.bf16_round(rng.standard_normal(N, dtype=np.float32) * np.float32(0.02)) if bias else None
    r = rng.standard_normal((M, N), dtype=np.float32)
    say(f"linear bf16 M={M} N={N} K={K} epi={epi} bias={bias}")
    out = dsp.dsp_linear(dev(a, "bf16"), dev(w, "bf16"), dev(b, "bf16") if bias else None,
                         dev(r, "f32") if epi == 2 else None, epi)
    torch.cuda.synchronize()
    want = oracle.linear(a, w.T, b)
    if epi == 1:
        want = oracle.gelu(want)
    if epi == 4:
        want = oracle.relu(want)
    if epi == 2:
        want = want + r
    # bf16 outputs carry a bf16 rounding; fp32 outputs only accumulation error
    assert_close(host(out), want, "bf16", f"linear epi={epi}")


# Problems of at least 256 output tiles of 256 x 192 (N < 2048) or 256 x 256
# run the large-tile kernel: ragged M, N and K (a partial last 64-wide slice).
LARGE = [(16421, 1000, 1176), (8292, 2056, 136), (8292, 1004, 136)]


@pytest.mark.parametrize("M,N,K", LARGE)
@pytest.mark.parametrize("epi", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("bias", [False, True])
def test_linear_bf16_large_tiles(torch, M, N, K, epi, bias):
    test_linear_bf16(torch, M, N, K, epi, bias)


@pytest.mark.parametrize("M,N,K", LARGE + [(32768, 1152, 4608), (32768, 3456, 1152)])
@pytest.mark.parametrize("epi", [0, 1, 2, 3, 4])
def test_linear_large_tiles_match_small(torch, M, N, K, epi):
    """Rows are independent, so rows computed by a call too small for the
    large-tile kernel must have the bits of the same rows of the large call
    (both kernels accumulate in the same k order)."""
    import paper_2403_10266_amd as dsp
    gen = torch.Generator(device="cuda").manual_seed(M + N + K + epi)
    a = torch.randn((M, K), device="cuda", generator=gen).to(torch.bfloat16)
    w = (torch.randn((N, K), device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    b = (torch.randn((N,), device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    r = torch.randn((M, N), device="cuda", generator=gen) if epi == 2 else None
    say(f"linear large vs small tiles M={M} N={N} K={K} epi={epi}")
    full = dsp.dsp_linear(a, w, b, r, epi)
    for r0 in (0, 4096, M - 200):
        rows = slice(r0, r0 + 200)
        part = dsp.dsp_linear(a[rows].contiguous(), w, b, r[rows].contiguous() if r is not None else None, epi)
        torch.cuda.synchronize()
        assert torch.equal(part.view(torch.int16) if part.dtype == torch.bfloat16 else part,
                           full[rows].view(torch.int16) if full.dtype == torch.bfloat16 else full[rows]), r0


@pytest.mark.parametrize("M,N,K", [(130, 96, 64), (300, 200, 72)])
def test_linear_resid_in_place(torch, M, N, K):
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(1)
    a = synth.bf16_round(rng.standard_normal((M, K), dtype=np.float32))
    w = synth.bf16_round(rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.1))
    r = rng.standard_normal((M, N), dtype=np.float32)
    rd = dev(r, "f32")
    dsp.dsp_linear(dev(a, "bf16"), dev(w, "bf16"), None, rd, 2, out=rd)
    torch.cuda.synchronize()
    assert_close(host(rd), oracle.linear(a, w.T) + r, "bf16", "in-place residual")


@pytest.mark.parametrize("M,N,K", [(3, 5, 7), (100, 70, 64), (65, 192, 64)])
@pytest.mark.parametrize("epi", [0, 1, 2, 4])
def test_linear_f32(torch, M, N, K, epi):
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(M + N + K)
    a = rng.standard_normal((M, K), dtype=np.float32)
    w = rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.1)
    b = rng.standard_normal(N, dtype=np.float32) * np.float32(0.1)
    r = rng.standard_normal((M, N), dtype=np.float32)
    out = dsp.dsp_linear(dev(a, "f32"), dev(w, "f32"), dev(b, "f32"), dev(r, "f32") if epi == 2 else None, epi)
    torch.cuda.synchronize()
    want = oracle.linear(a, w.T, b)
    if epi == 1:
        want = oracle.gelu(want)
    if epi == 4:
        want = oracle.relu(want)
    if epi == 2:
        want = want + r
    assert_close(host(out), want, "f32", f"linear f32 epi={epi}")
