"""dsp_switch on the GPU against the oracle: bit-exact on raw bit patterns."""
import json

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


def _run(torch, x_np, from_dim, to_dim, n, variant, np_dtype):
    import paper_2403_10266_amd as dsp
    if np_dtype == np.uint16:
        xt = torch.from_numpy(x_np.view(np.int16)).cuda().view(torch.bfloat16)
    else:
        xt = torch.from_numpy(x_np.view(np.float32)).cuda()
    y = dsp.dsp_switch(xt, from_dim, to_dim, n, variant=variant)
    torch.cuda.synchronize()
    if np_dtype == np.uint16:
        return y.view(torch.int16).cpu().numpy().view(np.uint16)
    return y.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("variant", [0, 1, 2])
def test_golden_fixtures(torch, variant):
    from tests.oracle_pins import GOLDEN
    for f in sorted(GOLDEN.glob("switch_*.json")):
        g = json.loads(f.read_text())
        x = np.array(g["x"], dtype=np.float32).reshape(g["shape"])
        if variant == 1 and (g["shape"][3] * 4) % 16:
            continue
        say(f"golden {f.name} variant {variant}")
        y = _run(torch, x.view(np.uint32), g["from_dim"], g["to_dim"], g["n_chunks"], variant, np.uint32)
        assert np.array_equal(y.view(np.float32).ravel(), np.array(g["y"], np.float32))


@pytest.mark.parametrize("variant", [1, 2])
def test_full_size_switch_and_inverse(torch, variant):
    """1 x 64 x 4096 x 1152 bf16 shard -> 8 chunks, and the inverse switch back."""
    w = synth.WORKLOADS["switch_bf16_T64_S4096"]
    x = synth.f32_to_bf16_bits(synth.switch_input(w))
    say(f"switch {x.shape} n={w.n_chunks} variant {variant}")
    y = _run(torch, x, 1, 2, w.n_chunks, variant, np.uint16)
    want = oracle.switch(x, 1, 2, w.n_chunks)
    assert y.shape == want.shape and np.array_equal(y, want)
    # inverse: the permuted (B,S,T,C) tensor switched back S -> T
    yt = want.transpose(1, 0, 2, 3, 4).reshape(w.B, w.S, w.T, w.C)
    yt = np.ascontiguousarray(yt)
    z = _run(torch, yt, 1, 2, w.n_chunks, variant, np.uint16)
    assert np.array_equal(z, oracle.switch(yt, 1, 2, w.n_chunks))
    # and with one chunk the round trip is the identity
    z1 = _run(torch, yt, 1, 2, 1, variant, np.uint16)[0]
    assert np.array_equal(z1, x)


@pytest.mark.parametrize("shape,fd,td,n,dt", [
    ((3, 5, 12, 8), 1, 2, 4, np.uint16),      # B > 1, ragged sizes, 16-byte rows
    ((2, 7, 6, 3), 1, 2, 3, np.uint16),       # 6-byte rows (tile kernel, 2-byte units)
    ((2, 7, 6, 3), 1, 2, 2, np.uint32),       # 12-byte fp32 rows
    ((1, 33, 65, 64), 1, 2, 5, np.uint32),    # tails in both tile dimensions
    ((2, 6, 5, 16), 2, 1, 3, np.uint16),      # from=2, to=1 (slice only)
    ((2, 3, 4, 24), 1, 1, 1, np.uint16),      # from == to: copy
    ((1, 1, 1, 1152), 1, 2, 1, np.uint16),    # single row
    ((2, 8, 64, 32), 1, 2, 2, np.uint16),     # row kernel in 4 x 16 tiles, B > 1, 2 chunks
    ((2, 40, 24, 32), 1, 2, 3, np.uint16),    # local to-extent 8: plain row order
    ((2, 64, 12, 32), 2, 1, 4, np.uint16),    # from=2, to=1 in tiles
])
def test_small_and_ragged(torch, shape, fd, td, n, dt):
    rng = np.random.default_rng(5)
    x = rng.integers(0, 2 ** 16 if dt == np.uint16 else 2 ** 31, size=shape).astype(dt)
    want = oracle.switch(x, fd, td, n)
    for variant in (0, 1, 2):
        if variant == 1 and (shape[3] * np.dtype(dt).itemsize) % 16:
            continue
        say(f"switch {shape} {fd}->{td} n={n} {np.dtype(dt).name} variant {variant}")
        y = _run(torch, x, fd, td, n, variant, dt)
        assert np.array_equal(y.reshape(want.shape), want)


def test_bit_patterns_survive(torch):
    pats = np.array([0x7FC1, 0xFFC3, 0x8000, 0x0000, 0x7F80, 0xFF80, 0x0001, 0x8001], np.uint16)
    x = np.tile(pats, 64).reshape(2, 4, 8, 8)
    for variant in (1, 2):
        y = _run(torch, x, 1, 2, 2, variant, np.uint16)
        assert np.array_equal(y, oracle.switch(x, 1, 2, 2))


def test_empty_is_noop(torch):
    import paper_2403_10266_amd as dsp
    x = torch.zeros((0, 4, 8, 16), dtype=torch.bfloat16, device="cuda")
    y = dsp.dsp_switch(x, 1, 2, 2)
    torch.cuda.synchronize()
    assert y.numel() == 0


def test_deterministic(torch):
    rng = np.random.default_rng(6)
    x = rng.integers(0, 2 ** 16, size=(2, 16, 32, 72)).astype(np.uint16)
    a = _run(torch, x, 1, 2, 4, 0, np.uint16)
    b = _run(torch, x, 1, 2, 4, 0, np.uint16)
    assert np.array_equal(a, b)
