"""Spatial and temporal attention on the GPU against the fp64 oracle."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import assert_close, dev, host, say, bits16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _inputs(shape, dtype, seed):
    rng = np.random.default_rng(seed)
    arrs = [rng.standard_normal(shape, dtype=np.float32) for _ in range(3)]
    if dtype == "bf16":
        arrs = [synth.bf16_round(a) for a in arrs]
    return arrs


@pytest.mark.parametrize("kind", ["spatial", "temporal"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,X,L,H,D", [
    (1, 4, 16, 4, 16),      # the tiny configuration's shape
    (2, 3, 1, 2, 72),       # L = 1
    (1, 2, 7, 3, 72),       # L below one tile
    (1, 2, 64, 2, 72),      # exactly one tile
    (2, 2, 65, 2, 72),      # one past a tile
    (1, 1, 300, 4, 72),     # several tiles + ragged tail, several query blocks
    (1, 2, 130, 2, 64),     # D a multiple of 32: VALU row sums
    (1, 2, 97, 2, 80),
    (1, 2, 50, 2, 96),
    (1, 2, 33, 2, 32),
])
def test_attention_small(torch, kind, dtype, B, X, L, H, D):
    import paper_2403_10266_amd as dsp
    C = H * D
    q, k, v = _inputs((B, X, L, C), dtype, seed=B * 1000 + L * 7 + D)
    say(f"{kind} {dtype} B={B} X={X} L={L} H={H} D={D}")
    fn = dsp.dsp_spatial_attn if kind == "spatial" else dsp.dsp_temporal_attn
    o = fn(dev(q, dtype), dev(k, dtype), dev(v, dtype), H)
    torch.cuda.synchronize()
    want = (oracle.spatial_attention if kind == "spatial" else oracle.temporal_attention)(q, k, v, H)
    assert_close(host(o), want, dtype, f"{kind} L={L} D={D}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_packed_qkv_and_scale(torch, dtype):
    """q/k/v as column slices of one packed [Q|K|V] buffer (row stride 3C) and an
    explicit softmax scale."""
    import paper_2403_10266_amd as dsp
    B, T, S, H, D = 1, 3, 70, 4, 72
    C = H * D
    rng = np.random.default_rng(42)
    qkv = rng.standard_normal((B, T, S, 3 * C), dtype=np.float32)
    if dtype == "bf16":
        qkv = synth.bf16_round(qkv)
    t = dev(qkv, dtype)
    q, k, v = t[..., :C], t[..., C:2 * C], t[..., 2 * C:]
    o = dsp.dsp_spatial_attn(q, k, v, H, C=C, ld_in=3 * C, scale=0.05)
    torch.cuda.synchronize()
    want = oracle.spatial_attention(qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:], H, scale=0.05)
    assert_close(host(o), want, dtype, "packed qkv")


def test_l1_returns_v_exactly(torch):
    import paper_2403_10266_amd as dsp
    q, k, v = _inputs((2, 5, 1, 1152), "bf16", seed=9)
    o = dsp.dsp_temporal_attn(dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), 16)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(o), bits16(dev(v, "bf16")))


@pytest.mark.parametrize("B,X,L,H,D", [
    (1, 150, 128, 4, 72),   # 600 units: several per persistent work-group, count not a multiple of 8
    (2, 37, 100, 3, 72),    # ragged L, 222 units
    (1, 3, 128, 1, 72),     # 3 units: most XCD ranges empty
    (1, 64, 128, 2, 64),    # D a multiple of 32: VALU row sums
    (1, 40, 77, 2, 16),
    (1, 40, 127, 2, 96),
    (1, 300, 32, 4, 72),    # 32-key variant: 1200 units, one wave per work-group
    (2, 150, 20, 3, 72),    # 32-key variant, ragged L
    (1, 260, 64, 2, 72),    # 64-key variant: 520 units
    (3, 50, 45, 2, 80),     # 64-key variant, ragged L, VALU-free row sums from a 32-row tile
    (1, 70, 33, 2, 32),
    (1, 300, 32, 8, 72),    # 32 keys, 4-head groups: 600 groups
    (2, 100, 64, 4, 72),    # 64 keys, 4-head groups
    (1, 64, 50, 8, 80),     # 64 keys, 4-head groups, ragged L
    (1, 64, 128, 4, 96),    # 128 keys, 2-head groups at the LDS limit (160 KB)
    (1, 90, 111, 6, 72),    # 128 keys, 2-head groups, ragged L
])
def test_temporal_stream_many_units(torch, B, X, L, H, D):
    """L <= 128 runs the persistent single-tile kernel: many units per work-group,
    unit counts that are and are not multiples of the XCD count."""
    import paper_2403_10266_amd as dsp
    C = H * D
    q, k, v = _inputs((B, X, L, C), "bf16", seed=B * 77 + X + L * 3 + D)
    say(f"temporal stream B={B} X={X} L={L} H={H} D={D}")
    o = dsp.dsp_temporal_attn(dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), H)
    torch.cuda.synchronize()
    want = oracle.temporal_attention(q, k, v, H)
    assert_close(host(o), want, "bf16", f"temporal stream L={L} D={D}")


def _sampled_check(torch, kind, w, n_units, n_rows, seed):
    import paper_2403_10266_amd as dsp
    layout = "BTSC" if kind == "spatial" else "BSTC"
    q, k, v = synth.qkv_inputs(w, layout)
    X, L = (w.T, w.S) if kind == "spatial" else (w.S, w.T)
    say(f"{kind} full size {q.shape} H={w.H}")
    fn = dsp.dsp_spatial_attn if kind == "spatial" else dsp.dsp_temporal_attn
    o = fn(dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), w.H)
    torch.cuda.synchronize()
    o = o.float().cpu().numpy()
    rng = np.random.default_rng(seed)
    D = w.D
    got, want = [], []
    for _ in range(n_units):
        b, x, h = rng.integers(w.B), rng.integers(X), rng.integers(w.H)
        rows = rng.choice(L, size=min(n_rows, L), replace=False)
        cs = slice(h * D, (h + 1) * D)
        want.append(oracle.attention_rows(q[b, x, rows, cs], k[b, x, :, cs], v[b, x, :, cs]))
        got.append(o[b, x, rows, cs])
    assert_close(np.concatenate(got), np.concatenate(want), "bf16", f"{kind} sampled")
    assert np.isfinite(o).all()
    return o


def test_spatial_full_size_sampled(torch):
    _sampled_check(torch, "spatial", synth.WORKLOADS["spatial_bf16_B2_T16_S4096"], 24, 96, 1)


def test_temporal_full_size_sampled(torch):
    _sampled_check(torch, "temporal", synth.WORKLOADS["temporal_bf16_B2_S512_T128"], 256, 128, 2)


def test_deterministic(torch):
    import paper_2403_10266_amd as dsp
    q, k, v = _inputs((1, 2, 200, 1152), "bf16", seed=3)
    a = dsp.dsp_spatial_attn(dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), 16)
    b = dsp.dsp_spatial_attn(dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), 16)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(a), bits16(b))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,S,H,D", [(1, 40, 12, 2, 72), (2, 130, 6, 3, 72), (1, 17, 9, 2, 64),
                                       (1, 300, 4, 1, 72), (1, 100, 6, 4, 72), (2, 24, 5, 8, 72)])
def test_temporal_attention_on_unswitched_layout(torch, dtype, B, T, S, H, D):
    """dsp_attn_strided reads (B, T, S, C) directly (no switch): equal to the
    oracle's strided temporal attention, output also written in (B, T, S, C)."""
    import paper_2403_10266_amd as dsp
    C = H * D
    q, k, v = _inputs((B, T, S, C), dtype, seed=T * 11 + S + D)
    say(f"temporal strided {dtype} B={B} T={T} S={S} H={H} D={D}")
    qd, kd, vd = (dev(a, dtype).permute(0, 2, 1, 3) for a in (q, k, v))     # views (B, S, T, C)
    out_full = torch.zeros((B, T, S, C), dtype=qd.dtype, device=qd.device)
    o = dsp.dsp_attn_strided(qd, kd, vd, H, out=out_full.permute(0, 2, 1, 3))
    torch.cuda.synchronize()
    want = oracle.temporal_attention_strided(q, k, v, H)
    assert_close(host(out_full), want, dtype, f"temporal strided T={T}")
    assert o.data_ptr() == out_full.data_ptr()


def test_strided_equals_dense_temporal(torch):
    """Reading the unswitched layout gives bit-identical results to switching
    first and reading the dense (B, S, T, C) layout (same kernel, same order)."""
    import paper_2403_10266_amd as dsp
    B, T, S, H, D = 1, 128, 8, 16, 72
    C = H * D
    q, k, v = _inputs((B, T, S, C), "bf16", seed=7)
    qd, kd, vd = (dev(a, "bf16") for a in (q, k, v))
    a = dsp.dsp_attn_strided(qd.permute(0, 2, 1, 3), kd.permute(0, 2, 1, 3), vd.permute(0, 2, 1, 3), H)
    dense = [t.permute(0, 2, 1, 3).contiguous() for t in (qd, kd, vd)]
    b = dsp.dsp_temporal_attn(*dense, H)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(a), bits16(b))


def test_temporal_strided_full_size_sampled(torch):
    """The temporal workload (B2 S512 T128 H16 D72) read straight from (B, T, S, C)."""
    import paper_2403_10266_amd as dsp
    w = synth.WORKLOADS["temporal_bf16_B2_S512_T128"]
    q, k, v = synth.qkv_inputs(w, "BSTC")
    q, k, v = (np.ascontiguousarray(a.transpose(0, 2, 1, 3)) for a in (q, k, v))     # (B, T, S, C)
    say(f"temporal strided full size {q.shape}")
    o = dsp.dsp_attn_strided(*(dev(a, "bf16").permute(0, 2, 1, 3) for a in (q, k, v)), w.H)
    torch.cuda.synchronize()
    o = o.float().cpu().numpy()                                                        # (B, S, T, C)
    rng = np.random.default_rng(4)
    D = w.D
    got, want = [], []
    for _ in range(128):
        b, s, h = rng.integers(w.B), rng.integers(w.S), rng.integers(w.H)
        cs = slice(h * D, (h + 1) * D)
        want.append(oracle.attention_rows(q[b, :, s, cs], k[b, :, s, cs], v[b, :, s, cs]))
        got.append(o[b, s, :, cs])
    assert_close(np.concatenate(got), np.concatenate(want), "bf16", "temporal strided sampled")
