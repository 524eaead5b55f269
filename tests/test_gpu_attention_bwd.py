"""Attention backward on the GPU against the fp64 oracle: the forward's row
log-sum-exp (dsp_attn_fwd_lse) and the gradients dq, dk, dv (dsp_attn_bwd).

The oracle computes the exact gradients from q, k, v and dout in float64.
The GPU backward recomputes the probabilities from its own forward's lse and
bf16 output o, so the comparison covers the whole training path.
Tolerances: fp32 1e-5 (max-abs and relative L2), as for the forward.  bf16:
relative L2 <= 1e-2 and max-abs <= 2e-2 -- the forward's bar, whose outputs
are of order one -- applied to each gradient after dividing by that
gradient's largest magnitude in the oracle, so that the bar means the same for
gradients of different scale (dv ~ 1/sqrt(L), dq ~ scale * |dP| / sqrt(L)).
Rounding of the bf16 inputs, of Q * scale * log2(e), of the probabilities and
of dZ to bf16 each contributes ~2^-9 relative."""
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


def _inputs(shape, dtype, seed, n=4):
    rng = np.random.default_rng(seed)
    arrs = [rng.standard_normal(shape, dtype=np.float32) for _ in range(n)]
    if dtype == "bf16":
        arrs = [synth.bf16_round(a) for a in arrs]
    return arrs


def _assert_grad(got, want, dtype, what):
    if dtype == "f32":
        assert_close(got, want, "f32", what)
        return
    mx = float(np.abs(want).max())
    if mx == 0.0:   # an exactly zero gradient (one key): only fp32 rounding residue allowed
        err = float(np.abs(got).max())
        say(f"  {what}: zero gradient, max |got| {err:.3e}")
        assert err <= 1e-4, what
        return
    assert_close(got / mx, want / mx, "bf16", f"{what} (/max {mx:.3e})")


def _run(torch, q, k, v, do, H, dtype, scale=0.0):
    import paper_2403_10266_amd as dsp
    qd, kd, vd, dd = (dev(a, dtype) for a in (q, k, v, do))
    o, lse = dsp.dsp_attn_fwd_lse(qd, kd, vd, H, scale=scale)
    dq, dk, dv = dsp.dsp_attn_bwd(qd, kd, vd, o, dd, lse, H, scale=scale)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,X,L,H,D", [
    (1, 2, 16, 4, 16),      # the tiny configuration's head width
    (2, 3, 1, 2, 72),       # L = 1: dq = dk = 0, dv = dout
    (1, 2, 7, 3, 72),       # below one tile
    (1, 2, 64, 2, 72),      # exactly one tile
    (2, 2, 65, 2, 72),      # one past a tile
    (1, 1, 300, 4, 72),     # several tiles + ragged tail, several blocks of keys and queries
    (1, 3, 128, 2, 72),     # the temporal length
    (1, 2, 130, 2, 64),
    (1, 2, 97, 2, 80),
    (1, 2, 50, 2, 96),
    (1, 2, 33, 2, 32),
])
def test_attention_bwd_small(torch, dtype, B, X, L, H, D):
    C = H * D
    q, k, v, do = _inputs((B, X, L, C), dtype, seed=B * 1000 + L * 7 + D)
    say(f"attn bwd {dtype} B={B} X={X} L={L} H={H} D={D}")
    o, lse, dq, dk, dv = _run(torch, q, k, v, do, H, dtype)
    # forward pieces: o as dsp_attn_strided would give, lse against the oracle
    assert_close(host(o), oracle.spatial_attention(q, k, v, H), dtype, "o")
    want_lse = oracle.attention_lse_units(q, k, H).reshape(B, X, H, L)
    tol = 1e-5 if dtype == "f32" else 2e-2
    err = float(np.abs(host(lse) - want_lse).max())
    say(f"  lse max-abs {err:.3e} (tol {tol:g})")
    assert err <= tol
    want = oracle.attention_bwd_units(q, k, v, do, H)
    for got, w, name in zip((dq, dk, dv), want, ("dq", "dk", "dv")):
        _assert_grad(host(got), w, dtype, name)


def test_l1_gradients(torch):
    """One key: the softmax is constant, so dv = dout exactly and dq = dk = 0
    up to the fp32 rounding of dP - Delta (P = 1 to within 1e-6)."""
    q, k, v, do = _inputs((2, 5, 1, 1152), "bf16", seed=9)
    o, lse, dq, dk, dv = _run(torch, q, k, v, do, 16, "bf16")
    assert np.array_equal(bits16(dv), bits16(dev(do, "bf16")))
    assert float(np.abs(host(dq)).max()) <= 1e-4
    assert float(np.abs(host(dk)).max()) <= 1e-4


def test_fwd_lse_output_matches_forward(torch):
    """The forward with lse writes the same bits of o as dsp_attn_strided."""
    import paper_2403_10266_amd as dsp
    for L in (50, 128, 300):
        q, k, v = _inputs((1, 2, L, 1152), "bf16", seed=L, n=3)
        qd, kd, vd = (dev(a, "bf16") for a in (q, k, v))
        a, _ = dsp.dsp_attn_fwd_lse(qd, kd, vd, 16)
        b = dsp.dsp_attn_strided(qd, kd, vd, 16)
        torch.cuda.synchronize()
        assert np.array_equal(bits16(a), bits16(b)), L


def test_bwd_deterministic(torch):
    import paper_2403_10266_amd as dsp
    q, k, v, do = _inputs((1, 2, 200, 1152), "bf16", seed=3)
    qd, kd, vd, dd = (dev(a, "bf16") for a in (q, k, v, do))
    o, lse = dsp.dsp_attn_fwd_lse(qd, kd, vd, 16)
    g1 = dsp.dsp_attn_bwd(qd, kd, vd, o, dd, lse, 16)
    g2 = dsp.dsp_attn_bwd(qd, kd, vd, o, dd, lse, 16)
    torch.cuda.synchronize()
    for a, b in zip(g1, g2):
        assert np.array_equal(bits16(a), bits16(b))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bwd_packed_qkv_and_scale(torch, dtype):
    """q/k/v as column slices of one packed [Q|K|V] buffer (row stride 3C), the
    gradients into the matching slices of a packed gradient buffer, explicit scale."""
    import paper_2403_10266_amd as dsp
    B, T, S, H, D = 1, 3, 70, 4, 72
    C = H * D
    rng = np.random.default_rng(42)
    qkv = rng.standard_normal((B, T, S, 3 * C), dtype=np.float32)
    do = rng.standard_normal((B, T, S, C), dtype=np.float32)
    if dtype == "bf16":
        qkv, do = synth.bf16_round(qkv), synth.bf16_round(do)
    t = dev(qkv, dtype)
    q, k, v = t[..., :C], t[..., C:2 * C], t[..., 2 * C:]
    o, lse = dsp.dsp_attn_fwd_lse(q, k, v, H, scale=0.05)
    g = torch.zeros_like(t)
    dsp.dsp_attn_bwd(q, k, v, o, dev(do, dtype), lse, H, dq=g[..., :C], dk=g[..., C:2 * C],
                     dv=g[..., 2 * C:], scale=0.05)
    torch.cuda.synchronize()
    want = oracle.attention_bwd_units(qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:], do, H, scale=0.05)
    gh = host(g)
    for i, (w, name) in enumerate(zip(want, ("dq", "dk", "dv"))):
        _assert_grad(gh[..., i * C:(i + 1) * C], w, dtype, f"packed {name}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bwd_temporal_on_unswitched_layout(torch, dtype):
    """Temporal attention's gradients read and written in (B, T, S, C) directly."""
    import paper_2403_10266_amd as dsp
    B, T, S, H, D = 1, 40, 6, 4, 72
    C = H * D
    q, k, v, do = _inputs((B, T, S, C), dtype, seed=77)
    qd, kd, vd, dd = (dev(a, dtype).permute(0, 2, 1, 3) for a in (q, k, v, do))   # (B, S, T, C) views
    o_full = torch.empty((B, T, S, C), dtype=qd.dtype, device=qd.device)
    o, lse = dsp.dsp_attn_fwd_lse(qd, kd, vd, H, out=o_full.permute(0, 2, 1, 3))
    grads = [torch.empty((B, T, S, C), dtype=qd.dtype, device=qd.device) for _ in range(3)]
    dsp.dsp_attn_bwd(qd, kd, vd, o, dd, lse, H, *(x.permute(0, 2, 1, 3) for x in grads))
    torch.cuda.synchronize()
    tr = lambda a: np.ascontiguousarray(a.transpose(0, 2, 1, 3))
    want = oracle.attention_bwd_units(tr(q), tr(k), tr(v), tr(do), H)
    for x, w, name in zip(grads, want, ("dq", "dk", "dv")):
        _assert_grad(tr(host(x)), w, dtype, f"strided {name}")


def _sampled_bwd(torch, w, layout, n_units, seed):
    """Full-size workload: gradients of a few sampled units against the oracle
    (the units are independent), every output finite."""
    import paper_2403_10266_amd as dsp
    q, k, v = synth.qkv_inputs(w, layout)
    rng = np.random.default_rng(seed)
    do = synth.bf16_round(rng.standard_normal(q.shape, dtype=np.float32))
    X, L = (w.T, w.S) if layout == "BTSC" else (w.S, w.T)
    say(f"attn bwd full size {q.shape} H={w.H}")
    qd, kd, vd, dd = (dev(a, "bf16") for a in (q, k, v, do))
    o, lse = dsp.dsp_attn_fwd_lse(qd, kd, vd, w.H)
    dq, dk, dv = dsp.dsp_attn_bwd(qd, kd, vd, o, dd, lse, w.H)
    torch.cuda.synchronize()
    del qd, kd, vd
    D = w.D
    for _ in range(n_units):
        b, x, h = rng.integers(w.B), rng.integers(X), rng.integers(w.H)
        cs = slice(h * D, (h + 1) * D)
        want = oracle.attention_bwd(q[b, x, :, cs], k[b, x, :, cs], v[b, x, :, cs], do[b, x, :, cs])
        for got, wg, name in zip((dq, dk, dv), want, ("dq", "dk", "dv")):
            _assert_grad(host(got[b, x, :, cs]), wg, "bf16", f"unit ({b},{x},{h}) {name}")
    for t in (dq, dk, dv):
        assert bool(torch.isfinite(t).all())


def test_bwd_spatial_full_size_sampled(torch):
    _sampled_bwd(torch, synth.WORKLOADS["spatial_bf16_B2_T16_S4096"], "BTSC", 3, 5)


def test_bwd_temporal_full_size_sampled(torch):
    _sampled_bwd(torch, synth.WORKLOADS["temporal_bf16_B2_S512_T128"], "BSTC", 48, 6)
