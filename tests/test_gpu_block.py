"""The spatial-temporal block composite on the GPU against the fp64 oracle."""
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


def _oracle_params(stored):
    """Stored [out][in] weights -> the paper's [in, out] matrices for the oracle."""
    return {n: (None if v is None else (v.T if n.startswith("w") else v)) for n, v in stored.items()}


def test_tiny_chain_fp32(torch):
    import paper_2403_10266_amd as dsp
    w = synth.WORKLOADS["tiny_chain_f32"]
    x, p = synth.chain_inputs(w)
    say(f"tiny chain {x.shape}")
    wd = {n: dev(v, "f32") for n, v in p.items()}
    y = dsp.dsp_st_block_forward(dev(x, "f32"), wd, w.H, flags=dsp.DSP_BLOCK_ATTN_ONLY)
    torch.cuda.synchronize()
    want = oracle.tiny_chain(x, _oracle_params(p), w.H)
    assert_close(host(y), want, "f32", "tiny chain")


@pytest.mark.parametrize("B,T,S,C,H,bias", [
    (1, 4, 16, 64, 4, False),    # the tiny configuration (one kernel per sublayer)
    (2, 3, 20, 32, 2, True),     # biases, B > 1
    (1, 7, 5, 48, 3, True),      # C not a divisor of the work-group: partial row bands
    (1, 64, 64, 64, 8, True),    # the largest one-kernel shape
    (1, 2, 70, 64, 4, True),     # S > 64: the general path (GEMM and attention launches)
    (1, 3, 8, 96, 4, True),      # C > 64: the general path
])
def test_projection_chain_fp32(torch, B, T, S, C, H, bias):
    """The projection-only chain (DSP_BLOCK_ATTN_ONLY) in fp32 against the
    oracle's pieces: Wqkv_s, spatial attention, Wo_s, the switch, Wqkv_t,
    temporal attention, Wo_t, each linear map with its bias when given."""
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(B * 1000 + T * 100 + S + C)
    x = rng.standard_normal((B, T, S, C), dtype=np.float32)
    p = {"wqkv_s": 0.05 * rng.standard_normal((3 * C, C), dtype=np.float32),
         "wo_s": 0.05 * rng.standard_normal((C, C), dtype=np.float32),
         "wqkv_t": 0.05 * rng.standard_normal((3 * C, C), dtype=np.float32),
         "wo_t": 0.05 * rng.standard_normal((C, C), dtype=np.float32)}
    if bias:
        for n, k in (("bqkv_s", 3 * C), ("bo_s", C), ("bqkv_t", 3 * C), ("bo_t", C)):
            p[n] = 0.1 * rng.standard_normal(k, dtype=np.float32)
    p = {n: v.astype(np.float32) for n, v in p.items()}
    say(f"projection chain fp32 B={B} T={T} S={S} C={C} H={H} bias={bias}")
    y = dsp.dsp_st_block_forward(dev(x, "f32"), {n: dev(v, "f32") for n, v in p.items()}, H,
                                 flags=dsp.DSP_BLOCK_ATTN_ONLY)
    torch.cuda.synchronize()

    def sub(h, tag, attn):
        qkv = oracle.linear(h, p["wqkv_" + tag].T, p.get("bqkv_" + tag))
        o = attn(qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:], H)
        return oracle.linear(o, p["wo_" + tag].T, p.get("bo_" + tag))

    ys = sub(x.astype(np.float64), "s", oracle.spatial_attention)
    want = sub(np.ascontiguousarray(ys.transpose(0, 2, 1, 3)), "t", oracle.temporal_attention)
    assert_close(host(y), want, "f32", "projection chain")


def _block_case(torch, w, with_bias, flags=0):
    import paper_2403_10266_amd as dsp
    x, p = synth.block_inputs(w, with_bias=with_bias)
    say(f"block {w.name} {x.shape} bias={with_bias} flags={flags}")
    wd = {n: (None if v is None else dev(v, w.dtype)) for n, v in p.items()}
    y = dsp.dsp_st_block_forward(dev(x, "f32"), wd, w.H, flags=flags)
    torch.cuda.synchronize()
    want = oracle.st_block(x, _oracle_params(p), w.H, flags=flags)
    assert_close(host(y), want, w.dtype, w.name)


# flags: 0 pre-LN GELU, 1 no MLP LayerNorm, 4 post-LN (Eq. 4, 6), 8 ReLU FFN
# (Eq. 5), 12 the paper's post-LN ReLU block, 13 post-LN without the last LN
@pytest.mark.parametrize("with_bias", [False, True])
@pytest.mark.parametrize("flags", [0, 1, 4, 8, 12, 13])
def test_small_block_bf16(torch, with_bias, flags):
    w = synth.Workload("block_small", "block", "bf16", B=2, T=5, S=24, C=144, H=2, F=576, seed=11)
    _block_case(torch, w, with_bias, flags)


@pytest.mark.parametrize("flags", [0, 12, 13])
def test_small_block_f32(torch, flags):
    w = synth.Workload("block_small_f32", "block", "f32", B=1, T=4, S=9, C=64, H=4, F=128, seed=12)
    _block_case(torch, w, True, flags)


def test_full_block_bf16(torch):
    """The 720M-model block at B=1, T=32, S=1024 (C=1152, 16 heads, MLP 4608)."""
    _block_case(torch, synth.WORKLOADS["block_bf16_B1_T32_S1024"], False)


def test_full_block_bf16_post_ln_relu(torch):
    """The same block in the paper's post-LN form with a ReLU FFN."""
    import paper_2403_10266_amd as dsp
    _block_case(torch, synth.WORKLOADS["block_bf16_B1_T32_S1024"], False,
                dsp.DSP_BLOCK_POST_LN | dsp.DSP_BLOCK_RELU)
