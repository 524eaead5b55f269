"""Grouped-query / multi-query attention and cross-attention on the GPU
(dsp_attn_general, dsp_attn_general_bwd) against the oracle's
attention_grouped and attention_grouped_bwd.  Bars as for attention: the
forward 2e-2 max-abs / 1e-2 relative L2 in bf16 and 1e-5 in fp32; gradients
the same after dividing by their largest magnitude in the oracle."""
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


def _draw(shape, dtype, seed):
    a = np.random.default_rng(seed).standard_normal(shape, dtype=np.float32)
    return synth.bf16_round(a) if dtype == "bf16" else a


def _grad_close(got, want, dtype, what):
    mx = float(np.abs(want).max())
    assert mx > 0, what
    assert_close(got / mx, want / mx, dtype, f"{what} (/max {mx:.3e})")


CASES = [
    # B, X, Lq, Lk, H, Hkv, D
    (1, 2, 100, 100, 4, 1, 72),      # multi-query attention
    (2, 2, 70, 70, 4, 2, 72),        # grouped-query attention
    (1, 2, 300, 77, 4, 4, 72),       # cross-attention: many queries, few keys (a text sequence)
    (1, 3, 33, 200, 4, 2, 72),       # cross + grouped, more keys than queries
    (1, 2, 128, 128, 8, 2, 64),
    (1, 2, 50, 20, 2, 1, 80),
    (2, 1, 1, 5, 2, 2, 72),          # one query
    (1, 1, 8, 1, 2, 1, 72),          # one key: the output is v
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,X,Lq,Lk,H,Hkv,D", CASES)
def test_attention_general(torch, dtype, B, X, Lq, Lk, H, Hkv, D):
    import paper_2403_10266_amd as dsp
    q = _draw((B, X, Lq, H * D), dtype, Lq + H)
    k, v = _draw((B, X, Lk, Hkv * D), dtype, Lk + 1), _draw((B, X, Lk, Hkv * D), dtype, Lk + 2)
    do = _draw((B, X, Lq, H * D), dtype, 9)
    say(f"general attn {dtype} B={B} X={X} Lq={Lq} Lk={Lk} H={H} Hkv={Hkv} D={D}")
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    o, lse = dsp.dsp_attn_general(qd, kd, vd, H, Hkv, with_lse=True)
    dq, dk, dv = dsp.dsp_attn_general_bwd(qd, kd, vd, o, dev(do, dtype), lse, H, Hkv)
    torch.cuda.synchronize()
    assert_close(host(o), oracle.attention_grouped(q, k, v, H, Hkv), dtype, "o")
    want = oracle.attention_grouped_bwd(q, k, v, do, H, Hkv)
    for got, w, name in zip((dq, dk, dv), want, ("dq", "dk", "dv")):
        if np.abs(w).max() == 0.0:      # one key: dq = dk = 0 up to fp32 rounding
            assert float(np.abs(host(got)).max()) <= 1e-4, name
            continue
        _grad_close(host(got), w, dtype, name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_cross_attention_broadcast_keys(torch, dtype):
    """One key/value sequence shared by every frame (x stride 0): the forward
    reads it broadcast; equal to the oracle with the sequence repeated."""
    import paper_2403_10266_amd as dsp
    B, X, Lq, Lk, H, D = 1, 6, 64, 30, 4, 72
    q = _draw((B, X, Lq, H * D), dtype, 1)
    k1, v1 = _draw((B, 1, Lk, H * D), dtype, 2), _draw((B, 1, Lk, H * D), dtype, 3)
    kd, vd = dev(k1, dtype).expand(B, X, Lk, H * D), dev(v1, dtype).expand(B, X, Lk, H * D)
    o = dsp.dsp_attn_general(dev(q, dtype), kd, vd, H, H)
    torch.cuda.synchronize()
    rep = lambda a: np.repeat(a, X, axis=1)
    assert_close(host(o), oracle.attention_grouped(q, rep(k1), rep(v1), H, H), dtype, "broadcast kv")


def test_general_equals_strided_self_attention(torch):
    """Hkv = H, Lq = Lk, one layout: the same kernels as dsp_attn_strided, the same bits."""
    import paper_2403_10266_amd as dsp
    q, k, v = (dev(_draw((1, 2, 300, 1152), "bf16", s), "bf16") for s in (4, 5, 6))
    a = dsp.dsp_attn_general(q, k, v, 16, 16)
    b = dsp.dsp_attn_strided(q, k, v, 16)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
