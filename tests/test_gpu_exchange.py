"""The N-rank exchange + unpack of the switch, run on one GPU with one buffer
per rank, against the oracle (bit-exact), and the full N-rank switch
simulation: T-shards -> dsp_switch -> dsp_exchange_unpack -> S-shards of the
permuted tensor."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _dev(torch, a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a.view(np.float32)).cuda()


def _host(t, dt):
    import torch
    if dt == np.uint16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("N,B,P,F,C,dt", [
    (1, 1, 3, 2, 8, np.uint16),      # one rank: a plain copy
    (2, 1, 4, 3, 8, np.uint16),      # 16-byte runs
    (3, 2, 5, 7, 3, np.uint16),      # 42-byte runs: 2-byte units
    (4, 2, 3, 5, 6, np.uint32),      # 120-byte runs: 8-byte aligned only -> 4-byte units
    (5, 1, 2, 4, 1152, np.uint16),   # the model's rows, 5 ranks
    (8, 1, 8, 8, 1152, np.uint16),   # 8 ranks
])
def test_exchange_unpack_matches_oracle(torch, N, B, P, F, C, dt):
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(N * 100 + F)
    hi = 2 ** 16 if dt == np.uint16 else 2 ** 32
    packed = [rng.integers(0, hi, size=(N, B, P, F, C), dtype=np.uint64).astype(dt) for _ in range(N)]
    say(f"exchange N={N} B={B} P={P} F={F} C={C} {np.dtype(dt).name}")
    got = dsp.dsp_exchange_unpack([_dev(torch, a) for a in packed])
    torch.cuda.synchronize()
    want = oracle.exchange_unpack(packed)
    for n in range(N):
        assert np.array_equal(_host(got[n], dt), want[n]), f"rank {n}"


def test_exchange_unaligned_buffers(torch):
    """Buffers that are only 2-byte aligned (views one element into larger
    allocations) take the narrow path and stay bit-exact."""
    import paper_2403_10266_amd as dsp
    N, B, P, F, C = 3, 1, 4, 2, 5
    rng = np.random.default_rng(3)
    packed = [rng.integers(0, 2 ** 16, size=(N, B, P, F, C), dtype=np.uint64).astype(np.uint16)
              for _ in range(N)]
    n_el = N * B * P * F * C
    big_in = [torch.zeros(n_el + 1, dtype=torch.bfloat16, device="cuda") for _ in range(N)]
    srcs = []
    for i in range(N):
        big_in[i][1:] = _dev(torch, packed[i].ravel())
        srcs.append(big_in[i][1:].view(N, B, P, F, C))
    big_out = [torch.zeros(n_el + 1, dtype=torch.bfloat16, device="cuda") for _ in range(N)]
    outs = [o[1:].view(B, P, N * F, C) for o in big_out]
    dsp.dsp_exchange_unpack(srcs, outs)
    torch.cuda.synchronize()
    want = oracle.exchange_unpack(packed)
    for n in range(N):
        assert np.array_equal(_host(outs[n], np.uint16), want[n])
        assert _host(big_out[n][:1], np.uint16)[0] == 0          # nothing written before the view


@pytest.mark.parametrize("B,T,S,C,N", [(1, 64, 512, 1152, 8), (2, 12, 18, 24, 3)])
def test_nrank_switch_simulation(torch, B, T, S, C, N):
    """N ranks hold T-shards; switch + exchange + unpack leaves rank n with
    S-shard n of the (B, S, T, C) permutation of the whole tensor."""
    import paper_2403_10266_amd as dsp
    rng = np.random.default_rng(B + T + S)
    X = rng.integers(0, 2 ** 16, size=(B, T, S, C), dtype=np.uint64).astype(np.uint16)
    say(f"N-rank switch simulation X={X.shape} N={N}")
    shards = [np.ascontiguousarray(s) for s in np.split(X, N, axis=1)]
    packed = [dsp.dsp_switch(_dev(torch, s), 1, 2, N) for s in shards]
    got = dsp.dsp_exchange_unpack(packed)
    torch.cuda.synchronize()
    G = np.ascontiguousarray(X.transpose(0, 2, 1, 3))
    want = np.split(G, N, axis=1)
    for n in range(N):
        assert np.array_equal(_host(got[n], np.uint16), want[n]), f"rank {n}"
