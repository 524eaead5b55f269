"""Gradients of the linear maps on the GPU against the fp64 oracle
(oracle.linear_bwd, oracle.gelu_bwd, oracle.relu_bwd).

The GPU gets the exact bf16 (or fp32) values the oracle uses, so the only
differences are fp32 accumulation order and, for bf16 outputs, the final
rounding.  Bars, after dividing by the largest magnitude of the oracle's
result: fp32 outputs 1e-4 max-abs and 1e-5 relative L2; bf16 outputs (one
rounding, 2^-9 relative) 1e-2 max-abs and 4e-3 relative L2."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import dev, host, say, errors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _close(got, want, kind, what):
    mx = float(np.abs(want).max())
    assert mx > 0
    a, r = errors(got / mx, want / mx)
    ta, tr = (1e-4, 1e-5) if kind == "f32" else (1e-2, 4e-3)
    say(f"  {what}: max_abs/max={a:.2e} rel_l2={r:.2e} (tol {ta:g}/{tr:g})")
    assert a <= ta and r <= tr, what


def _draw(shape, dtype, seed, scale=1.0):
    a = np.random.default_rng(seed).standard_normal(shape, dtype=np.float32) * scale
    return synth.bf16_round(a) if dtype == "bf16" else a


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,N,K", [(1, 8, 8), (300, 72, 136), (257, 1152, 264), (64, 3456, 1152),
                                    (1000, 40, 16)])
def test_linear_bwd_data(torch, dtype, M, N, K):
    import paper_2403_10266_amd as dsp
    dy, w = _draw((M, N), dtype, M + N), _draw((N, K), dtype, K, 0.05)
    say(f"bwd_data {dtype} M={M} N={N} K={K}")
    # dsp_linear stores W as [out][in] = [N][K]; the oracle's W is [in][out] = w.T
    want = oracle.linear_bwd(np.zeros((M, K)), w.T, dy)[0]
    got = dsp.dsp_linear_bwd_data(dev(dy, dtype), dev(w, dtype), epilogue=dsp.DSP_GRAD_EPI_F32)
    _close(host(got), want, "f32", "dx fp32")
    if dtype == "bf16":
        got = dsp.dsp_linear_bwd_data(dev(dy, dtype), dev(w, dtype), epilogue=dsp.DSP_GRAD_EPI_BF16)
        _close(host(got), want, "bf16", "dx bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("act", ["gelu", "relu"])
def test_linear_bwd_data_activation(torch, dtype, act):
    """dx = (dy W) * act'(u): the backward through the MLP's activation (Eq. 5)."""
    import paper_2403_10266_amd as dsp
    M, N, K = 330, 1152, 4608 // 8
    dy, w, u = _draw((M, N), dtype, 5), _draw((N, K), dtype, 6, 0.05), _draw((M, K), dtype, 7, 1.5)
    dg = oracle.linear_bwd(np.zeros((M, K)), w.T, dy)[0]
    want = oracle.gelu_bwd(u, dg) if act == "gelu" else oracle.relu_bwd(u, dg)
    epi = dsp.DSP_GRAD_EPI_GELU_BWD if act == "gelu" else dsp.DSP_GRAD_EPI_RELU_BWD
    got = dsp.dsp_linear_bwd_data(dev(dy, dtype), dev(w, dtype), u=dev(u, dtype), epilogue=epi)
    _close(host(got), want, "f32" if dtype == "f32" else "bf16", f"{act} backward")


_SMALL_W = [(1, 8, 8), (300, 72, 136), (1000, 1152, 264)]
# bf16 only (the fp32 path is for small problems): the 256 x 128 gradient
# kernel, then the large-tile one with ragged tiles in both output dimensions
# and in the token reduction, and split-K partials
_LARGE_W = [(4100, 3456, 1152), (4100, 1160, 520), (12000, 1152, 4608)]


@pytest.mark.parametrize("dtype,M,N,K", [(d, *m) for d in ("f32", "bf16") for m in _SMALL_W] +
                         [("bf16", *m) for m in _LARGE_W])
def test_linear_bwd_weight(torch, dtype, M, N, K):
    import paper_2403_10266_amd as dsp
    x, dy = _draw((M, K), dtype, M + K), _draw((M, N), dtype, N)
    say(f"bwd_weight {dtype} M={M} N={N} K={K}")
    _, dw_paper, db = oracle.linear_bwd(x, np.zeros((K, N)), dy)
    dw, dbg = dsp.dsp_linear_bwd_weight(dev(dy, dtype), dev(x, dtype), with_bias=True)
    _close(host(dw), dw_paper.T, "f32", "dW")
    _close(host(dbg), db, "f32", "db")


def test_linear_bwd_weight_split_deterministic(torch):
    """The split reduction adds its partial sums in a fixed order."""
    import paper_2403_10266_amd as dsp
    M, N, K = 32768, 1152, 1152
    assert dsp.lib().dsp_linear_bwd_weight_workspace_bytes(M, N, K, dsp.DSP_BF16) > 0
    x, dy = _draw((M, K), "bf16", 1), _draw((M, N), "bf16", 2)
    xd, dyd = dev(x, "bf16"), dev(dy, "bf16")
    a, _ = dsp.dsp_linear_bwd_weight(dyd, xd)
    b, _ = dsp.dsp_linear_bwd_weight(dyd, xd)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    rng = np.random.default_rng(3)
    rows, cols = rng.integers(N, size=24), rng.integers(K, size=24)
    want = np.array([np.dot(dy[:, r].astype(np.float64), x[:, c].astype(np.float64)) for r, c in zip(rows, cols)])
    got = host(a)[rows, cols]
    _close(got, want, "f32", "sampled dW at the block's token count")


@pytest.mark.parametrize("x_dtype,dy_dtype", [("f32", "f32"), ("f32", "bf16"), ("bf16", "bf16")])
@pytest.mark.parametrize("rows,C", [(1, 64), (37, 1152), (300, 72), (5, 3000)])
def test_layernorm_bwd(torch, x_dtype, dy_dtype, rows, C):
    """dx = dres + LN backward (oracle.layernorm_bwd) with fp32 statistics."""
    import paper_2403_10266_amd as dsp
    x = _draw((rows, C), x_dtype, rows + C, 2.0) + 0.5
    x = synth.bf16_round(x) if x_dtype == "bf16" else x
    dy, dres = _draw((rows, C), dy_dtype, C), _draw((rows, C), "f32", 9)
    want = oracle.layernorm_bwd(x, dy, 1e-6)
    got = dsp.dsp_layernorm_bwd(dev(x, x_dtype), dev(dy, dy_dtype), 1e-6)
    _close(host(got), want, "f32", f"LN bwd rows={rows} C={C}")
    acc = dev(dres, "f32")
    dsp.dsp_layernorm_bwd(dev(x, x_dtype), dev(dy, dy_dtype), 1e-6, dres=acc, out=acc)   # in place
    _close(host(acc), want + dres, "f32", "LN bwd + residual gradient, in place")
