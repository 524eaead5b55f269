"""The K = 3 switch and the Split / Gather primitives on the GPU against the
oracle: bit-exact on raw bit patterns."""
import itertools

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _to_dev(torch, x):
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(x.view(np.float32)).cuda()


def _to_host(torch, t, dt):
    if dt == np.uint16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy().view(np.uint32)


def _rand(shape, dt, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2 ** 16 if dt == np.uint16 else 2 ** 31, size=shape).astype(dt)


@pytest.mark.parametrize("shape,dt", [
    ((2, 3, 4, 6, 8), np.uint16),       # 16-byte rows
    ((1, 4, 6, 2, 3), np.uint16),       # 6-byte rows: 2-byte units
    ((2, 3, 4, 6, 5), np.uint32),       # 20-byte fp32 rows: 4-byte units
    ((1, 5, 7, 9, 72), np.uint16),      # ragged sizes, 144-byte rows
])
def test_switch_k3_all_pairs(torch, shape, dt):
    import paper_2403_10266_amd as dsp
    x = _rand(shape, dt, 21)
    xt = _to_dev(torch, x)
    for f, t in itertools.product((1, 2, 3), repeat=2):
        for n in [d for d in (1, 2, 3, 4) if shape[t] % d == 0]:
            say(f"switch K=3 {shape} {f}->{t} n={n} {np.dtype(dt).name}")
            y = dsp.dsp_switch(xt, f, t, n)
            torch.cuda.synchronize()
            want = oracle.switch(x, f, t, n)
            got = _to_host(torch, y, dt)
            assert got.shape == want.shape and np.array_equal(got, want)


def test_switch_k3_full_size(torch):
    """A K = 3 video shard: 64 local frames of 64 x 64 latent tokens, C = 1152
    bf16 (604 MB), switched to each other dimension in 8 chunks."""
    import paper_2403_10266_amd as dsp
    w = synth.WORKLOADS["switch_bf16_T64_S4096"]
    x = synth.f32_to_bf16_bits(synth.switch_input(w)).reshape(w.B, w.T, 64, 64, w.C)
    xt = _to_dev(torch, x)
    for f, t in [(1, 2), (1, 3), (2, 3), (3, 1)]:
        say(f"switch K=3 full {x.shape} {f}->{t} n=8")
        y = dsp.dsp_switch(xt, f, t, 8)
        torch.cuda.synchronize()
        assert np.array_equal(_to_host(torch, y, np.uint16), oracle.switch(x, f, t, 8))
        del y


def test_switch_k3_nrank_simulation(torch):
    """N ranks on one GPU: switch + exchange/unpack of K = 3 shards leave rank n
    with shard n of the to-dim of the whole tensor, the from-dim next to C."""
    import paper_2403_10266_amd as dsp
    X = _rand((2, 4, 6, 8, 24), np.uint16, 22)
    for f, t, N in [(1, 3, 2), (3, 2, 2), (2, 1, 2), (3, 1, 4)]:
        say(f"K=3 N-rank simulation {f}->{t} N={N}")
        shards = [np.ascontiguousarray(s) for s in np.split(X, N, axis=f)]
        packed = [dsp.dsp_switch(_to_dev(torch, s), f, t, N) for s in shards]
        out = dsp.dsp_exchange_unpack([p.reshape(N, p.shape[1], -1, p.shape[-2], p.shape[-1])
                                       for p in packed])
        torch.cuda.synchronize()
        want = np.split(np.moveaxis(X, f, -2), N, axis=t if t < f else t - 1)
        for n in range(N):
            got = _to_host(torch, out[n], np.uint16).reshape(want[n].shape)
            assert np.array_equal(got, want[n])


@pytest.mark.parametrize("shape,dt", [
    ((2, 8, 12, 8), np.uint16), ((3, 6, 4, 5), np.uint32), ((1, 4, 6, 3), np.uint16),
    ((2, 4, 6, 8, 16), np.uint16), ((1, 6, 2, 4, 3), np.uint32), ((1, 64, 4096 // 8, 1152), np.uint16),
])
def test_split_gather(torch, shape, dt):
    import paper_2403_10266_amd as dsp
    x = _rand(shape, dt, 23)
    xt = _to_dev(torch, x)
    for dim in range(1, len(shape) - 1):
        for N in [d for d in (1, 2, 3, 4, 8) if shape[dim] % d == 0]:
            say(f"split/gather {shape} dim={dim} N={N} {np.dtype(dt).name}")
            parts = [dsp.dsp_split(xt, dim, N, r) for r in range(N)]
            torch.cuda.synchronize()
            for r in range(N):
                assert np.array_equal(_to_host(torch, parts[r], dt), oracle.split(x, dim, N, r))
            y = dsp.dsp_gather(parts, dim)
            torch.cuda.synchronize()
            want = oracle.gather([oracle.split(x, dim, N, r) for r in range(N)], dim)
            assert np.array_equal(_to_host(torch, y, dt), want)
            assert np.array_equal(want, x)


def test_gather_unaligned_and_aliased_shards(torch):
    """Shards at 2-byte offsets (narrow units) and one buffer given twice."""
    import paper_2403_10266_amd as dsp
    base = torch.zeros(4 * 3 * 5 * 7 + 8, dtype=torch.bfloat16, device="cuda")
    a = _rand((1, 3, 5, 7), np.uint16, 24)
    b = _rand((1, 3, 5, 7), np.uint16, 25)
    sa = base[1:1 + a.size].view(1, 3, 5, 7)
    sb = base[2 + a.size:2 + 2 * a.size].view(1, 3, 5, 7)
    sa.copy_(_to_dev(torch, a))
    sb.copy_(_to_dev(torch, b))
    for dim in (1, 2):
        y = dsp.dsp_gather([sa, sb, sa], dim)
        torch.cuda.synchronize()
        assert np.array_equal(_to_host(torch, y, np.uint16), oracle.gather([a, b, a], dim))


def test_split_gather_empty(torch):
    import paper_2403_10266_amd as dsp
    x = torch.zeros((0, 4, 6, 8), dtype=torch.bfloat16, device="cuda")
    assert dsp.dsp_split(x, 1, 2, 1).numel() == 0
    assert dsp.dsp_gather([x, x], 2).numel() == 0
