"""dsp_attn_bwd_noalloc -- the attention backward whose Delta rows live in a
library-owned static device array -- against dsp_attn_bwd on the same
inputs.  Both run the same kernels, so dq, dk and dv must agree bit for bit.
Two calls in a row, the second with a smaller input (the array keeps the
first call's contents), on the two-kernel bf16 path (L > 128), the fused
short-unit path (L <= 128) and fp32."""
import ctypes

import numpy as np
import pytest

import synth
from tests.gpu_util import bits16, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _case(torch, dsp, B, X, L, H, D, dtype, seed):
    rng = np.random.default_rng(seed)
    C = H * D
    arrs = [rng.standard_normal((B, X, L, C), dtype=np.float32) for _ in range(4)]
    if dtype == "bf16":
        arrs = [synth.bf16_round(a) for a in arrs]
    q, k, v, do = (dev(a, dtype) for a in arrs)
    o, lse = dsp.dsp_attn_fwd_lse(q, k, v, H)
    want = dsp.dsp_attn_bwd(q, k, v, o, do, lse, H)
    got = tuple(torch.full_like(q, float("nan")) for _ in range(3))
    dsp.dsp_attn_bwd_noalloc(q, k, v, o, do, lse, H, *got)
    torch.cuda.synchronize()
    for g, w, name in zip(got, want, ("dq", "dk", "dv")):
        if dtype == "bf16":
            same = np.array_equal(bits16(g), bits16(w))
        else:
            same = np.array_equal(host(g).astype(np.float32).view(np.int32),
                                  host(w).astype(np.float32).view(np.int32))
        say(f"  {dtype} B={B} X={X} L={L} H={H} D={D} {name}: identical bits {same}")
        assert same, name


@pytest.mark.parametrize("first,second", [
    ((2, 8, 1024, 16, 72, "bf16"), (1, 3, 300, 4, 72, "bf16")),     # two-kernel path, then smaller
    ((1, 64, 128, 16, 72, "bf16"), (1, 5, 40, 2, 72, "bf16")),      # fused short-unit path
    ((1, 4, 200, 4, 64, "f32"), (1, 2, 33, 2, 64, "f32")),          # fp32
])
def test_noalloc_matches_workspace_entry(torch, first, second):
    import paper_2403_10266_amd as dsp
    for i, (B, X, L, H, D, dtype) in enumerate((first, second)):
        assert B * X * L * H <= dsp.attn_bwd_noalloc_max_rows()
        say(f"call {i + 1}: B={B} X={X} L={L} H={H} D={D} {dtype}")
        _case(torch, dsp, B, X, L, H, D, dtype, seed=40 + i + 7 * L)


def test_noalloc_rejects_more_rows_than_its_array(torch):
    """Checked on the host before anything is touched: DSP_ERR_WORKSPACE."""
    import paper_2403_10266_amd as dsp
    L = dsp.attn_bwd_noalloc_max_rows() // 16 + 1
    st = (ctypes.c_int64 * 3)(L * 1152, L * 1152, 1152)
    status = dsp.lib().dsp_attn_bwd_noalloc(None, None, None, None, None, None, None, None, None, 1, 1, L, 16,
                                            72, st, st, 0.0, dsp.DSP_BF16, None)
    assert status == dsp.DSP_ERR_WORKSPACE
