"""Pins of the CPU oracle: checks against closed forms, invariants, hand-worked
fixtures and brute force.  Each pin takes the implementation under test as an
argument, so the same pins run against the oracle (they must pass) and
against deliberately broken copies of it (each must be caught by some pin).
"""
from __future__ import annotations

import itertools
import json
import math
from pathlib import Path

import numpy as np
from scipy.stats import norm

GOLDEN = Path(__file__).resolve().parent / "golden"


# ----------------------------------------------------------------------------- switch
def pin_switch_golden(switch):
    for f in sorted(GOLDEN.glob("switch_*.json")):
        g = json.loads(f.read_text())
        x = np.array(g["x"], dtype=np.float32).reshape(g["shape"])
        y = switch(x, g["from_dim"], g["to_dim"], g["n_chunks"])
        assert list(y.shape) == g["y_shape"], f.name
        assert np.array_equal(y.ravel(), np.array(g["y"], dtype=np.float32)), f.name


def pin_switch_index_loops(switch, index_map):
    rng = np.random.default_rng(7)
    for shape, fd, td, n in [((2, 3, 4, 2), 1, 2, 2), ((1, 4, 6, 3), 1, 2, 3), ((3, 4, 2, 1), 2, 1, 2),
                              ((2, 2, 3, 2), 1, 2, 1)]:
        x = rng.integers(0, 60000, size=shape).astype(np.uint16)
        y = switch(x, fd, td, n)
        for oidx, iidx in index_map(shape, fd, td, n):
            assert y[oidx] == x[iidx]


def pin_switch_round_trip(switch, unswitch):
    rng = np.random.default_rng(8)
    for shape in [(1, 4, 8, 3), (2, 3, 5, 4), (3, 1, 2, 5)]:
        x = rng.standard_normal(shape).astype(np.float32)
        # T->S then S->T, one chunk each: the identity for any B
        y = switch(x, 1, 2, 1)[0]
        assert np.array_equal(switch(y, 1, 2, 1)[0], x)
        # unpacking any chunk count restores x
        for n in [d for d in range(1, shape[2] + 1) if shape[2] % d == 0]:
            assert np.array_equal(unswitch(switch(x, 1, 2, n), 1, 2), x)


def pin_switch_b1_transpose(switch):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((1, 6, 8, 4)).astype(np.float32)
    t = np.ascontiguousarray(x.transpose(0, 2, 1, 3))
    for n in (1, 2, 4, 8):
        y = switch(x, 1, 2, n)
        assert y.tobytes() == t.tobytes()


def pin_switch_bits_and_copy(switch):
    # bit patterns (NaN payloads, signed zeros) survive; from == to is a copy
    x = np.array([0x7FC1, 0x8000, 0x0000, 0xFF81, 0x3F80, 0x0001, 0x7F80, 0xFFFF],
                 dtype=np.uint16).reshape(1, 2, 2, 2)
    y = switch(x, 1, 2, 2)
    assert sorted(y.ravel().tolist()) == sorted(x.ravel().tolist())
    assert np.array_equal(switch(x, 1, 1, 1), x)
    assert np.array_equal(switch(x, 2, 2, 3), x)


def pin_switch_nrank_simulation(switch, exchange_unpack):
    """The paper's exactness claim: resharding only moves data.  N ranks each
    hold a T-shard; after switch + all-to-all + unpack, rank n holds exactly the
    S-shard n of the globally permuted tensor."""
    rng = np.random.default_rng(10)
    for B, T, S, C in [(1, 8, 8, 3), (2, 4, 6, 2), (2, 6, 4, 1), (3, 4, 4, 2)]:
        for N_ in (1, 2, 4):
            if T % N_ or S % N_:
                continue
            X = rng.standard_normal((B, T, S, C)).astype(np.float32)
            shards = np.split(X, N_, axis=1)
            packed = [switch(s, 1, 2, N_) for s in shards]
            got = exchange_unpack(packed)
            G = np.ascontiguousarray(X.transpose(0, 2, 1, 3))
            want = np.split(G, N_, axis=1)
            for n in range(N_):
                assert np.array_equal(got[n], want[n])


def _k3_source(shape, f, t, n_chunks, out_idx):
    """Input index of packed element out_idx = (n, b, o_1, o_2, i, c) for a K = 3
    switch, by the definition: the other two sequence dims in their order (the
    to-dim's index offset by its chunk), the from-dim index i, then c."""
    n, b, o1, o2, i, c = out_idx
    others = [d for d in (1, 2, 3) if d != f]
    src = [b, 0, 0, 0, c]
    for d, o in zip(others, (o1, o2)):
        src[d] = o + (n * (shape[t] // n_chunks) if d == t else 0)
    src[f] = i
    return tuple(src)


def pin_switch_k3_index_loops(switch):
    rng = np.random.default_rng(11)
    for shape in [(2, 2, 3, 4, 2), (1, 4, 2, 2, 3)]:
        x = rng.integers(0, 60000, size=shape).astype(np.uint16)
        for f, t in itertools.permutations((1, 2, 3), 2):
            for n in [d for d in (1, 2, 4) if shape[t] % d == 0]:
                y = switch(x, f, t, n)
                assert y.size == x.size
                for out_idx in itertools.product(*(range(e) for e in y.shape)):
                    assert y[out_idx] == x[_k3_source(shape, f, t, n, out_idx)]


def pin_switch_k3_unit_dim(switch):
    """A K = 3 tensor with a unit sequence dimension switches as the K = 2 tensor."""
    rng = np.random.default_rng(12)
    x = rng.standard_normal((2, 4, 6, 3)).astype(np.float32)
    for n in (1, 2, 3):
        want = switch(x, 1, 2, n)                                   # [n, B, 6/n, 4, C]
        got = switch(x[:, :, :, None, :], 1, 2, n)                  # [n, B, 6/n, 1, 4, C]
        assert np.array_equal(got.reshape(want.shape), want)
        got = switch(x[:, None], 2, 3, n)                           # unit dim in front
        assert np.array_equal(got.reshape(want.shape), want)
        got = switch(x[:, :, None], 1, 3, n)                        # unit dim between
        assert np.array_equal(got.reshape(want.shape), want)
    want = switch(x, 2, 1, 2)
    assert np.array_equal(switch(x[:, :, :, None], 2, 1, 2).reshape(want.shape), want)


def pin_switch_nrank_simulation_k3(switch, exchange_unpack):
    """K = 3: N ranks hold the from-dim shards of X; after switch + all-to-all +
    unpack rank n holds shard n of the to-dim of X with the from-dim next to C
    (the layout of Eq. 7 for the from-dim)."""
    rng = np.random.default_rng(13)
    X = rng.standard_normal((2, 4, 2, 4, 3)).astype(np.float32)
    for f, t in itertools.permutations((1, 2, 3), 2):
        for N_ in (1, 2):
            shards = np.split(X, N_, axis=f)
            got = exchange_unpack([switch(s, f, t, N_) for s in shards])
            G = np.moveaxis(X, f, -2)
            want = np.split(G, N_, axis=t if t < f else t - 1)
            for n in range(N_):
                assert np.array_equal(got[n], want[n])


def pin_split_gather(split, gather):
    rng = np.random.default_rng(14)
    for shape in [(2, 4, 6, 3), (1, 2, 4, 6, 2)]:
        x = rng.integers(0, 60000, size=shape).astype(np.uint16)
        for d in range(1, len(shape) - 1):
            for N_ in [k for k in (1, 2, 3, 4) if shape[d] % k == 0]:
                per = shape[d] // N_
                parts = [split(x, d, N_, r) for r in range(N_)]
                for r, part in enumerate(parts):
                    idx = [slice(None)] * len(shape)
                    idx[d] = slice(r * per, (r + 1) * per)
                    assert np.array_equal(part, x[tuple(idx)])
                assert np.array_equal(gather(parts, d), x)
                # gather by explicit loops: element e of shard m lands at m*per + e on d
                y = gather(parts, d)
                for m in range(N_):
                    for e in range(per):
                        assert np.array_equal(np.take(y, m * per + e, axis=d),
                                              np.take(parts[m], e, axis=d))


def pin_switch_is_gather_then_split(switch, exchange_unpack, split, gather):
    """The Switch's all-to-all moves what a Gather on the from-dim followed by a
    Split on the to-dim would leave on each rank (primitive table), laid out with
    the from-dim next to C."""
    rng = np.random.default_rng(15)
    X = rng.standard_normal((1, 4, 6, 2)).astype(np.float32)
    N_ = 2
    shards = [split(X, 1, N_, r) for r in range(N_)]
    got = exchange_unpack([switch(s, 1, 2, N_) for s in shards])
    for n in range(N_):
        want = split(gather(shards, 1), 2, N_, n)                    # [B, T, S/N, C]
        assert np.array_equal(got[n], np.moveaxis(want, 1, -2))


# ----------------------------------------------------------------------------- attention
def _brute_attention(q, k, v, scale):
    Lq, d = q.shape
    L = k.shape[0]
    out = np.zeros((Lq, v.shape[1]))
    for i in range(Lq):
        z = [math.fsum(float(q[i, a]) * float(k[j, a]) for a in range(d)) * scale for j in range(L)]
        m = max(z)
        e = [math.exp(t - m) for t in z]
        s = math.fsum(e)
        for c in range(v.shape[1]):
            out[i, c] = math.fsum(e[j] * float(v[j, c]) for j in range(L)) / s
    return out


def pin_attention_brute(attention):
    rng = np.random.default_rng(11)
    for Lq, L, d in [(3, 5, 4), (2, 1, 3), (4, 7, 72)]:
        q, k, v = (rng.standard_normal(s) for s in ((Lq, d), (L, d), (L, d)))
        got = attention(q, k, v)
        want = _brute_attention(q, k, v, 1.0 / math.sqrt(d))
        assert np.allclose(got, want, rtol=1e-12, atol=1e-13)


def pin_attention_l1_is_v(attention):
    rng = np.random.default_rng(12)
    q, k, v = rng.standard_normal((5, 72)), rng.standard_normal((1, 72)), rng.standard_normal((1, 72))
    assert np.array_equal(attention(q, k, v), np.repeat(v, 5, axis=0))


def pin_attention_zero_q_mean(attention):
    rng = np.random.default_rng(13)
    k, v = rng.standard_normal((9, 16)), rng.standard_normal((9, 16))
    q = np.zeros((4, 16))
    assert np.allclose(attention(q, k, v), np.tile(v.mean(axis=0), (4, 1)), atol=1e-14)
    # identical keys: any query gives the mean as well
    k1 = np.tile(rng.standard_normal((1, 16)), (9, 1))
    q1 = rng.standard_normal((4, 16))
    assert np.allclose(attention(q1, k1, v), np.tile(v.mean(axis=0), (4, 1)), atol=1e-14)


def pin_attention_two_keys_closed_form(attention):
    # L = 2: the weight of key 0 is the logistic function of the score gap
    rng = np.random.default_rng(14)
    d = 72
    q, k, v = rng.standard_normal((3, d)), rng.standard_normal((2, d)), rng.standard_normal((2, 5))
    got = attention(q, k, v)
    for i in range(3):
        gap = (q[i] @ k[0] - q[i] @ k[1]) / math.sqrt(d)
        w0 = 1.0 / (1.0 + math.exp(-gap))
        assert np.allclose(got[i], w0 * v[0] + (1.0 - w0) * v[1], rtol=1e-12, atol=1e-14)


def pin_attention_rows_stochastic(attention):
    # with V = I the output is the probability matrix: rows nonnegative, sum to 1,
    # and row i ranks keys like the scores of query i
    rng = np.random.default_rng(15)
    q, k = rng.standard_normal((6, 8)), rng.standard_normal((10, 8))
    P = attention(q, k, np.eye(10))
    assert (P >= 0).all() and np.allclose(P.sum(axis=1), 1.0, atol=1e-14)
    z = q @ k.T
    for i in range(6):
        assert np.array_equal(np.argsort(P[i], kind="stable"), np.argsort(z[i], kind="stable"))


def pin_attention_hard_max(attention):
    rng = np.random.default_rng(16)
    q, k, v = rng.standard_normal((4, 8)), rng.standard_normal((6, 8)), rng.standard_normal((6, 3))
    got = attention(q, k, v, scale=1e4)
    idx = np.argmax(q @ k.T, axis=1)
    assert np.allclose(got, v[idx], atol=1e-9)


def pin_attention_permutations(attention):
    rng = np.random.default_rng(17)
    q, k, v = rng.standard_normal((5, 8)), rng.standard_normal((7, 8)), rng.standard_normal((7, 8))
    base = attention(q, k, v)
    pk = rng.permutation(7)
    assert np.allclose(attention(q, k[pk], v[pk]), base, atol=1e-14)
    pq = rng.permutation(5)
    assert np.allclose(attention(q[pq], k, v), base[pq], atol=1e-14)


def pin_attention_scale_default(attention):
    # default scale is 1/sqrt(d) with the true d (never a padded width)
    rng = np.random.default_rng(18)
    q, k, v = rng.standard_normal((3, 72)), rng.standard_normal((4, 72)), rng.standard_normal((4, 2))
    assert np.allclose(attention(q, k, v), attention(q, k, v, scale=1.0 / math.sqrt(72)), atol=0)
    assert not np.allclose(attention(q, k, v), attention(q, k, v, scale=1.0 / math.sqrt(80)))


def pin_spatial_temporal_units(spatial, temporal, temporal_strided, switch):
    """Per-unit independence, head split, and the switch/strided equivalence."""
    rng = np.random.default_rng(19)
    B, T, S, H, d = 2, 3, 5, 2, 4
    C = H * d
    q, k, v = (rng.standard_normal((B, T, S, C)) for _ in range(3))
    o = spatial(q, k, v, H)
    # every (b, t, h) unit is plain attention over S
    for b, t, h in itertools.product(range(B), range(T), range(H)):
        cs = slice(h * d, (h + 1) * d)
        want = _brute_attention(q[b, t, :, cs], k[b, t, :, cs], v[b, t, :, cs], 1 / math.sqrt(d))
        assert np.allclose(o[b, t, :, cs], want, rtol=1e-12, atol=1e-13)
    # perturbing one unit changes only that unit
    k2 = k.copy()
    k2[1, 2, :, d:2 * d] += 1.0
    o2 = spatial(q, k2, v, H)
    diff = np.abs(o2 - o) > 0
    assert diff[1, 2, :, d:2 * d].any()
    diff[1, 2, :, d:2 * d] = False
    assert not diff.any()
    # temporal attention after the switch == temporal attention read strided
    sw = lambda a: switch(a, 1, 2, 1)[0]
    ot = temporal(sw(q), sw(k), sw(v), H)
    ots = temporal_strided(q, k, v, H)
    assert np.allclose(ot, sw(ots), rtol=1e-13, atol=1e-14)
    for b, s, h in itertools.product(range(B), range(S), range(H)):
        cs = slice(h * d, (h + 1) * d)
        want = _brute_attention(q[b, :, s, cs], k[b, :, s, cs], v[b, :, s, cs], 1 / math.sqrt(d))
        assert np.allclose(ot[b, s, :, cs], want, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------- attention backward
def _fd_grad(f, x, h=1e-6):
    """Central finite differences of the scalar f at x (float64)."""
    g = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        xp = x.copy(); xp[idx] += h
        xm = x.copy(); xm[idx] -= h
        g[idx] = (f(xp) - f(xm)) / (2 * h)
    return g


def pin_attention_bwd_fd(attention, attention_bwd):
    """<dO, attention(q, k, v)> differentiated numerically in each input."""
    rng = np.random.default_rng(30)
    for U, Lq, L, d, scale in [(2, 3, 4, 4, None), (1, 5, 5, 3, 0.7)]:
        q, k, v, do = (rng.standard_normal(sh) for sh in [(U, Lq, d), (U, L, d), (U, L, d), (U, Lq, d)])
        dq, dk, dv = attention_bwd(q, k, v, do, scale)
        loss = lambda qq, kk, vv: float((do * attention(qq, kk, vv, scale)).sum())
        assert np.allclose(dq, _fd_grad(lambda a: loss(a, k, v), q), atol=1e-8, rtol=1e-7)
        assert np.allclose(dk, _fd_grad(lambda a: loss(q, a, v), k), atol=1e-8, rtol=1e-7)
        assert np.allclose(dv, _fd_grad(lambda a: loss(q, k, a), v), atol=1e-8, rtol=1e-7)


def pin_attention_bwd_invariants(attention_bwd):
    rng = np.random.default_rng(31)
    q, k, v, do = (rng.standard_normal((3, 6, 5)) for _ in range(4))
    _, dk, _ = attention_bwd(q, k, v, do)
    # softmax is invariant to a common shift of a row's scores, so the key
    # gradients of a unit sum to zero
    assert np.allclose(dk.sum(axis=-2), 0.0, atol=1e-12)
    # one key: the output is v whatever q and k are
    dq, dk, dv = attention_bwd(q[:, :, :], k[:, :1], v[:, :1], do)
    assert np.allclose(dq, 0.0, atol=1e-14) and np.allclose(dk, 0.0, atol=1e-14)
    assert np.allclose(dv[:, 0], do.sum(axis=1))
    # identical keys: P is uniform, so dq = 0 and dv = the column sums of dO / L
    kk = np.repeat(k[:, :1], 6, axis=1)
    dq, _, dv = attention_bwd(q, kk, v, do)
    assert np.allclose(dq, 0.0, atol=1e-12)
    assert np.allclose(dv, np.repeat(do.sum(axis=1, keepdims=True) / 6, 6, axis=1))


def pin_attention_lse(attention_lse):
    from scipy.special import logsumexp
    rng = np.random.default_rng(32)
    q, k = rng.standard_normal((2, 4, 8)) * 3, rng.standard_normal((2, 7, 8)) * 3
    z = np.einsum("uid,ujd->uij", q, k) / math.sqrt(8)
    lse = attention_lse(q, k)
    assert np.allclose(lse, logsumexp(z, axis=-1))
    assert (lse >= z.max(axis=-1)).all()
    assert np.allclose(np.exp(z - lse[..., None]).sum(axis=-1), 1.0)
    assert np.allclose(attention_lse(q, k, 0.25), logsumexp(z * math.sqrt(8) * 0.25, axis=-1))


def pin_attention_bwd_units(attention_bwd, attention_bwd_units, attention_lse_units,
                            attention_lse, attention_delta_units, attention):
    """The (B, X, L, C) wrappers run each (b, x, head) unit on its own columns."""
    rng = np.random.default_rng(33)
    B, X, L, H, d = 2, 3, 5, 2, 4
    q, k, v, do = (rng.standard_normal((B, X, L, H * d)) for _ in range(4))
    dq, dk, dv = attention_bwd_units(q, k, v, do, H)
    lse = attention_lse_units(q, k, H)
    o = np.zeros_like(q)
    for b, x, h in itertools.product(range(B), range(X), range(H)):
        cs = slice(h * d, (h + 1) * d)
        g = attention_bwd(q[b, x, :, cs], k[b, x, :, cs], v[b, x, :, cs], do[b, x, :, cs])
        assert np.allclose(dq[b, x, :, cs], g[0]) and np.allclose(dk[b, x, :, cs], g[1])
        assert np.allclose(dv[b, x, :, cs], g[2])
        u = (b * X + x) * H + h
        assert np.allclose(lse[u], attention_lse(q[b, x, :, cs], k[b, x, :, cs]))
        o[b, x, :, cs] = attention(q[b, x, :, cs], k[b, x, :, cs], v[b, x, :, cs])
    delta = attention_delta_units(o, do, H)
    for b, x, h in itertools.product(range(B), range(X), range(H)):
        cs = slice(h * d, (h + 1) * d)
        assert np.allclose(delta[(b * X + x) * H + h], (o[b, x, :, cs] * do[b, x, :, cs]).sum(-1))


# ----------------------------------------------------------------------------- LN / linear / GELU
def pin_layernorm(layernorm):
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    eps = 1e-6
    want = (x - 2.5) / math.sqrt(1.25 + eps)
    assert np.allclose(layernorm(x, eps), want, rtol=1e-15, atol=1e-15)
    rng = np.random.default_rng(20)
    y = rng.standard_normal((5, 33)) * 3 + 1
    z = layernorm(y, eps)
    var = y.var(axis=1, keepdims=True)
    assert np.allclose(z.mean(axis=1), 0, atol=1e-14)
    assert np.allclose((z ** 2).mean(axis=1, keepdims=True), var / (var + eps), rtol=1e-12)
    # exact invariance to affine maps of the input when eps = 0
    assert np.allclose(layernorm(2.5 * y - 7.0, 0.0), layernorm(y, 0.0), atol=1e-12)


def pin_linear(linear):
    rng = np.random.default_rng(21)
    x, w, b = rng.standard_normal((3, 4)), rng.standard_normal((4, 5)), rng.standard_normal(5)
    got = linear(x, w, b)
    for i in range(3):
        for j in range(5):
            assert math.isclose(got[i, j], math.fsum(x[i, a] * w[a, j] for a in range(4)) + b[j],
                                rel_tol=1e-12, abs_tol=1e-14)
    assert np.array_equal(linear(x, np.eye(4)), x)


def pin_gelu(gelu):
    x = np.linspace(-6, 6, 97)
    assert np.allclose(gelu(x), x * norm.cdf(x), rtol=1e-14, atol=1e-15)
    assert np.allclose(gelu(x) - gelu(-x), x, atol=1e-14)
    assert gelu(np.array([0.0]))[0] == 0.0
    # Phi(1) = 0.841344746068542948585...
    assert math.isclose(gelu(np.array([1.0]))[0], 0.8413447460685429, rel_tol=1e-15)


def pin_relu(relu):
    """Eq. (5): max(0, x).  relu(x) - relu(-x) = x and relu(x) + relu(-x) = |x|."""
    x = np.linspace(-5, 5, 101)
    assert np.array_equal(relu(x) - relu(-x), x)
    assert np.array_equal(relu(x) + relu(-x), np.abs(x))
    assert relu(np.array([0.0]))[0] == 0.0
    assert np.array_equal(relu(np.array([-2.5, 3.25])), np.array([0.0, 3.25]))


# ----------------------------------------------------------------------------- block
def _block_params(rng, C, F, scale=0.3, bias=False):
    p = {"wqkv_s": rng.standard_normal((C, 3 * C)) * scale, "wo_s": rng.standard_normal((C, C)) * scale,
         "wqkv_t": rng.standard_normal((C, 3 * C)) * scale, "wo_t": rng.standard_normal((C, C)) * scale,
         "w1": rng.standard_normal((C, F)) * scale, "w2": rng.standard_normal((F, C)) * scale}
    if bias:
        for n, w in (("bqkv_s", 3 * C), ("bo_s", C), ("bqkv_t", 3 * C), ("bo_t", C), ("b1", F), ("b2", C)):
            p[n] = rng.standard_normal(w) * scale
    return p


def pin_block_identities(st_block, layernorm, linear, gelu, switch):
    rng = np.random.default_rng(22)
    B, T, S, C, H, F = 1, 3, 4, 8, 2, 16
    x = rng.standard_normal((B, T, S, C))
    p = _block_params(rng, C, F)
    # zero output projections: only the switched residual stream is left
    z = dict(p, wo_s=np.zeros((C, C)), wo_t=np.zeros((C, C)), w2=np.zeros((F, C)))
    assert np.array_equal(st_block(x, z, H), switch(x, 1, 2, 1)[0])
    # Q = K = 0: attention is the mean of V over the attended axis (S, then T)
    qk0 = dict(p)
    for n in ("wqkv_s", "wqkv_t"):
        w = p[n].copy()
        w[:, :2 * C] = 0.0
        qk0[n] = w
    qk0["w2"] = np.zeros((F, C))
    got = st_block(x, qk0, H)
    xs = x + linear(linear(layernorm(x), qk0["wqkv_s"][:, 2 * C:]).mean(axis=2, keepdims=True)
                    .repeat(S, axis=2), p["wo_s"])
    y = np.ascontiguousarray(xs.transpose(0, 2, 1, 3))
    y = y + linear(linear(layernorm(y), qk0["wqkv_t"][:, 2 * C:]).mean(axis=2, keepdims=True)
                   .repeat(T, axis=2), p["wo_t"])
    assert np.allclose(got, y, rtol=1e-12, atol=1e-12)
    # MLP path alone (attention projections zero): y = x^T + GELU(LN(x^T) W1) W2
    m = dict(p, wo_s=np.zeros((C, C)), wo_t=np.zeros((C, C)))
    xt = np.ascontiguousarray(x.transpose(0, 2, 1, 3))
    want = xt + linear(gelu(linear(layernorm(xt), p["w1"])), p["w2"])
    assert np.allclose(st_block(x, m, H), want, rtol=1e-12, atol=1e-12)


def pin_block_t1_s1(st_block, layernorm, linear, gelu):
    """A sequence of length 1 makes attention return its V projection.
    T = 1: the temporal sublayer is LN(y) W_v Wo_t.  S = 1: the spatial sublayer
    is LN(x) W_v Wo_s.  Each reduction is checked against the block itself
    with the other half's output projection zeroed."""
    rng = np.random.default_rng(23)
    C, H, F = 8, 2, 12
    p = _block_params(rng, C, F)
    zc, zf = np.zeros((C, C)), np.zeros((F, C))
    # T = 1
    x = rng.standard_normal((2, 1, 5, C))
    y0 = st_block(x, dict(p, wo_t=zc, w2=zf), H)            # spatial half + switch only
    want = y0 + linear(linear(layernorm(y0), p["wqkv_t"][:, 2 * C:]), p["wo_t"])
    want = want + linear(gelu(linear(layernorm(want), p["w1"])), p["w2"])
    assert np.allclose(st_block(x, p, H), want, rtol=1e-12, atol=1e-12)
    # S = 1
    x = rng.standard_normal((2, 4, 1, C))
    xs = x + linear(linear(layernorm(x), p["wqkv_s"][:, 2 * C:]), p["wo_s"])
    want = st_block(xs, dict(p, wo_s=zc), H)
    assert np.allclose(st_block(x, p, H), want, rtol=1e-12, atol=1e-12)


def pin_block_sharded_equals_unsharded(st_block, layernorm, linear, gelu, switch, exchange_unpack,
                                       spatial, temporal):
    """DSP's central claim: with the activation sharded on T for the spatial stage
    and on S for the temporal stage (one switch between them), every rank's
    result equals the matching slice of the unsharded block."""
    rng = np.random.default_rng(24)
    B, T, S, C, H, F, N = 1, 4, 6, 8, 2, 12, 2
    x = rng.standard_normal((B, T, S, C))
    p = _block_params(rng, C, F, bias=True)
    want = st_block(x, p, H)

    def attn_sub(h, wq, bq, wo, bo, attn):
        qkv = linear(h, wq, bq)
        return linear(attn(qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:], H), wo, bo)

    shards = np.split(x, N, axis=1)                       # rank m holds T-shard m
    xs = [s + attn_sub(layernorm(s), p["wqkv_s"], p["bqkv_s"], p["wo_s"], p["bo_s"], spatial)
          for s in shards]
    ys = exchange_unpack([switch(s, 1, 2, N) for s in xs])   # rank n holds S-shard n, all T
    outs = []
    for y in ys:
        y = y + attn_sub(layernorm(y), p["wqkv_t"], p["bqkv_t"], p["wo_t"], p["bo_t"], temporal)
        y = y + linear(gelu(linear(layernorm(y), p["w1"], p["b1"])), p["w2"], p["b2"])
        outs.append(y)
    assert np.allclose(np.concatenate(outs, axis=1), want, rtol=1e-12, atol=1e-12)


def pin_block_post_ln_relu(st_block, layernorm, linear, relu, switch, post_flag, relu_flag):
    """The paper's own block, Eq. (4)-(6): x <- LN(x + sublayer(x)) with a ReLU FFN.
    * Every output row is LN's: mean 0 and (with eps = 0) variance 1.
    * Zero output projections leave LN(LN(LN(switch(x)))) = switch(LN(x)).
    * The MLP path alone is LN(y + ReLU(y W1) W2) with y = LN(switch(x))."""
    rng = np.random.default_rng(26)
    B, T, S, C, H, F = 1, 3, 4, 8, 2, 16
    x = rng.standard_normal((B, T, S, C)) * 2.0 + 0.5
    p = _block_params(rng, C, F)
    flags = post_flag | relu_flag
    out = st_block(x, p, H, 0.0, flags)
    assert np.allclose(out.mean(axis=-1), 0.0, atol=1e-12)
    assert np.allclose(out.var(axis=-1), 1.0, atol=1e-12)
    zc, zf = np.zeros((C, C)), np.zeros((F, C))
    xt = np.ascontiguousarray(switch(x, 1, 2, 1)[0])
    y0 = layernorm(xt, 0.0)
    assert np.allclose(st_block(x, dict(p, wo_s=zc, wo_t=zc, w2=zf), H, 0.0, flags), y0,
                       rtol=1e-12, atol=1e-12)
    want = layernorm(y0 + linear(relu(linear(y0, p["w1"])), p["w2"]), 0.0)
    assert np.allclose(st_block(x, dict(p, wo_s=zc, wo_t=zc), H, 0.0, flags), want,
                       rtol=1e-12, atol=1e-12)
    # post-LN alone keeps the GELU MLP; ReLU alone keeps the pre-LN placement
    g = st_block(x, dict(p, wo_s=zc, wo_t=zc), H, 0.0, post_flag)
    assert not np.allclose(g, want)
    r = st_block(x, dict(p, wo_s=zc, wo_t=zc), H, 0.0, relu_flag)
    assert np.allclose(r, xt + linear(relu(linear(layernorm(xt, 0.0), p["w1"])), p["w2"]),
                       rtol=1e-12, atol=1e-12)


def pin_tiny_chain(tiny_chain, st_block):
    # the chain is the block with LN, residuals and MLP removed: check it against
    # an explicit composition built from per-unit brute-force attention
    rng = np.random.default_rng(25)
    B, T, S, C, H = 1, 2, 3, 4, 2
    d = C // H
    x = rng.standard_normal((B, T, S, C))
    p = {n: rng.standard_normal(s) * 0.5 for n, s in
         (("wqkv_s", (C, 3 * C)), ("wo_s", (C, C)), ("wqkv_t", (C, 3 * C)), ("wo_t", (C, C)))}
    got = tiny_chain(x, p, H)

    def attn_all(qkv, axis_len, spatial):
        out = np.zeros(qkv.shape[:-1] + (C,))
        for idx in itertools.product(range(qkv.shape[0]), range(qkv.shape[1]), range(H)):
            b, o_, h = idx
            cs = slice(h * d, (h + 1) * d)
            q = qkv[b, o_, :, cs]
            k = qkv[b, o_, :, C + h * d:C + (h + 1) * d]
            v = qkv[b, o_, :, 2 * C + h * d:2 * C + (h + 1) * d]
            out[b, o_, :, cs] = _brute_attention(q, k, v, 1 / math.sqrt(d))
        return out

    y = attn_all(x @ p["wqkv_s"], S, True) @ p["wo_s"]
    y = np.ascontiguousarray(y.transpose(0, 2, 1, 3))
    y = attn_all(y @ p["wqkv_t"], T, False) @ p["wo_t"]
    assert np.allclose(got, y, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------- block backward
def pin_linear_bwd(linear, linear_bwd):
    """<dy, x W + b> differentiated numerically in x, W and b."""
    rng = np.random.default_rng(40)
    x, w, b, dy = rng.standard_normal((2, 3, 4)), rng.standard_normal((4, 5)), \
        rng.standard_normal(5), rng.standard_normal((2, 3, 5))
    dx, dw, db = linear_bwd(x, w, dy)
    loss = lambda xx, ww, bb: float((dy * linear(xx, ww, bb)).sum())
    assert np.allclose(dx, _fd_grad(lambda a: loss(a, w, b), x), atol=1e-8)
    assert np.allclose(dw, _fd_grad(lambda a: loss(x, a, b), w), atol=1e-8)
    assert np.allclose(db, _fd_grad(lambda a: loss(x, w, a), b), atol=1e-8)


def pin_layernorm_bwd(layernorm, layernorm_bwd):
    rng = np.random.default_rng(41)
    for eps in (1e-6, 0.3):
        x, dy = rng.standard_normal((3, 7)) * 2 + 1, rng.standard_normal((3, 7))
        dx = layernorm_bwd(x, dy, eps)
        assert np.allclose(dx, _fd_grad(lambda a: float((dy * layernorm(a, eps)).sum()), x), atol=1e-7)
        # the output is invariant to adding a constant to a row (and, for eps = 0,
        # to scaling it), so the gradient has no component along the ones vector
        assert np.allclose(dx.sum(axis=-1), 0.0, atol=1e-12)
    x, dy = rng.standard_normal((4, 9)), rng.standard_normal((4, 9))
    y = layernorm(x, 0.0)
    assert np.allclose((layernorm_bwd(x, dy, 0.0) * (x - x.mean(-1, keepdims=True))).sum(-1), 0.0,
                       atol=1e-11)
    # a gradient along the output itself or along ones gives zero
    assert np.allclose(layernorm_bwd(x, y, 0.0), 0.0, atol=1e-12)
    assert np.allclose(layernorm_bwd(x, np.ones_like(x), 0.0), 0.0, atol=1e-12)


def pin_gelu_bwd(gelu, gelu_bwd, relu, relu_bwd):
    rng = np.random.default_rng(42)
    u, dy = rng.standard_normal(50) * 3, rng.standard_normal(50)
    assert np.allclose(gelu_bwd(u, dy), _fd_grad(lambda a: float((dy * gelu(a)).sum()), u), atol=1e-8)
    # GELU(u) - GELU(-u) = u, so GELU'(u) + GELU'(-u) = 1
    one = np.ones_like(u)
    assert np.allclose(gelu_bwd(u, one) + gelu_bwd(-u, one), 1.0)
    assert gelu_bwd(np.array([0.0]), np.array([1.0]))[0] == 0.5
    v = u[np.abs(u) > 1e-3]
    assert np.allclose(relu_bwd(v, dy[:v.size]), np.where(v > 0, dy[:v.size], 0.0))


def _block_case(seed, B=1, T=3, S=4, C=8, H=2, F=12, bias=False):
    rng = np.random.default_rng(seed)
    p = {"wqkv_s": rng.standard_normal((C, 3 * C)) * 0.3, "wo_s": rng.standard_normal((C, C)) * 0.3,
         "wqkv_t": rng.standard_normal((C, 3 * C)) * 0.3, "wo_t": rng.standard_normal((C, C)) * 0.3,
         "w1": rng.standard_normal((C, F)) * 0.3, "w2": rng.standard_normal((F, C)) * 0.3}
    if bias:
        for n, k in (("bqkv_s", 3 * C), ("bo_s", C), ("bqkv_t", 3 * C), ("bo_t", C), ("b1", F), ("b2", C)):
            p[n] = rng.standard_normal(k) * 0.2
    x = rng.standard_normal((B, T, S, C))
    dy = rng.standard_normal((B, S, T, C))
    return x, p, dy, H


def pin_block_bwd_fd(st_block, st_block_bwd, flag_sets):
    """Finite differences of <dy, st_block(x)> in x and in sampled entries of
    every weight and bias, for each flag combination."""
    for i, flags in enumerate(flag_sets):
        x, p, dy, H = _block_case(50 + i, bias=True)
        dx, g = st_block_bwd(x, p, H, dy, flags=flags)
        f = lambda xx, pp: float((dy * st_block(xx, pp, H, flags=flags)).sum())
        assert np.allclose(dx, _fd_grad(lambda a: f(a, p), x, h=1e-5), atol=1e-6, rtol=1e-5), flags
        rng = np.random.default_rng(60 + i)
        for name, w in p.items():
            assert g[name].shape == w.shape, name
            for _ in range(3):
                idx = tuple(rng.integers(s) for s in w.shape)
                def fw(val):
                    q = dict(p)
                    q[name] = w.copy()
                    q[name][idx] = val
                    return f(x, q)
                num = (fw(w[idx] + 1e-5) - fw(w[idx] - 1e-5)) / 2e-5
                assert abs(g[name][idx] - num) <= 1e-6 + 1e-5 * abs(num), (flags, name, idx)


def pin_block_bwd_autograd(st_block_bwd, flag_sets):
    """The same gradients from torch autograd in float64 on the CPU: an
    independent differentiation of the block written with torch operations."""
    import torch
    for i, flags in enumerate(flag_sets):
        x, p, dy, H = _block_case(70 + i, B=2, T=3, S=5, C=12, H=3, F=20, bias=(i % 2 == 0))
        dx, g = st_block_bwd(x, p, H, dy, flags=flags)
        tx = torch.tensor(x, requires_grad=True)
        tp = {n: torch.tensor(v, requires_grad=True) for n, v in p.items()}
        C = x.shape[-1]

        def ln(v):
            mu = v.mean(-1, keepdim=True)
            return (v - mu) / torch.sqrt(((v - mu) ** 2).mean(-1, keepdim=True) + 1e-6)

        def lin(v, w, b):
            return v @ tp[w] + (tp[b] if b in tp else 0.0)

        def attn(q, k, v, dim):
            # attention over sequence axis `dim` (1 = T, 2 = S) of (B, T, S, C), per head
            qs, ks, vs = (t.movedim(dim, 2) for t in (q, k, v))          # (B, X, L, C)
            Bq, X, L, _ = qs.shape
            sh = lambda t: t.reshape(Bq, X, L, H, C // H).permute(0, 1, 3, 2, 4)
            qh, kh, vh = sh(qs), sh(ks), sh(vs)
            z = qh @ kh.transpose(-1, -2) / math.sqrt(C // H)
            o = torch.softmax(z, dim=-1) @ vh
            return o.permute(0, 1, 3, 2, 4).reshape(Bq, X, L, C).movedim(2, dim)

        post, relu_ = bool(flags & 4), bool(flags & 8)
        act = torch.relu if relu_ else (lambda u: 0.5 * u * (1 + torch.erf(u / math.sqrt(2.0))))

        def sub_attn(v, tag, dim):
            qkv = lin(v, "wqkv_" + tag, "bqkv_" + tag)
            return lin(attn(qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:], dim), "wo_" + tag, "bo_" + tag)
        x1 = ln(tx + sub_attn(tx, "s", 2)) if post else tx + sub_attn(ln(tx), "s", 2)
        y0 = x1                                                   # kept in (B, T, S, C): temporal attends over dim 1
        y1 = ln(y0 + sub_attn(y0, "t", 1)) if post else y0 + sub_attn(ln(y0), "t", 1)
        ffn = lambda v: lin(act(lin(v, "w1", "b1")), "w2", "b2")
        if flags & 1:
            out = y1 + ffn(y1)
        else:
            out = ln(y1 + ffn(y1)) if post else y1 + ffn(ln(y1))
        (out.transpose(1, 2) * torch.tensor(dy)).sum().backward()
        assert np.allclose(dx, tx.grad.numpy(), atol=1e-10, rtol=1e-8), flags
        for n in p:
            assert np.allclose(g[n], tp[n].grad.numpy(), atol=1e-10, rtol=1e-8), (flags, n)


# ----------------------------------------------------------------------------- grouped / cross attention
def pin_attention_grouped(attention_grouped, spatial_attention, attention):
    rng = np.random.default_rng(80)
    B, X, Lq, Lk, H, d = 2, 3, 5, 7, 4, 3
    q = rng.standard_normal((B, X, Lq, H * d))
    # Hkv = H with Lq = Lk: plain multi-head attention per unit
    k, v = rng.standard_normal((B, X, Lq, H * d)), rng.standard_normal((B, X, Lq, H * d))
    assert np.allclose(attention_grouped(q, k, v, H, H), spatial_attention(q, k, v, H))
    # grouped heads equal multi-head attention with each key/value head repeated
    # for the query heads of its group (head h reads group h // (H / Hkv))
    for Hkv in (1, 2):
        k, v = rng.standard_normal((B, X, Lk, Hkv * d)), rng.standard_normal((B, X, Lk, Hkv * d))
        rep = lambda a: np.concatenate([a[..., (h // (H // Hkv)) * d:(h // (H // Hkv) + 1) * d]
                                        for h in range(H)], axis=-1)
        got = attention_grouped(q, k, v, H, Hkv)
        assert got.shape == q.shape
        for b, x, h in itertools.product(range(B), range(X), range(H)):
            cq, ck = slice(h * d, (h + 1) * d), slice((h // (H // Hkv)) * d, (h // (H // Hkv) + 1) * d)
            assert np.allclose(got[b, x, :, cq], attention(q[b, x, :, cq], k[b, x, :, ck], v[b, x, :, ck]))
        # brute force over Python floats for the cross-attention lengths (Lq != Lk)
        for b, x, h, i in [(1, 2, 3, 4), (0, 0, 1, 0)]:
            g = h // (H // Hkv)
            z = [sum(q[b, x, i, h * d + e] * k[b, x, j, g * d + e] for e in range(d)) / math.sqrt(d)
                 for j in range(Lk)]
            m = max(z)
            w = [math.exp(zz - m) for zz in z]
            s = math.fsum(w)
            for e in range(d):
                want = math.fsum(w[j] * v[b, x, j, g * d + e] for j in range(Lk)) / s
                assert abs(got[b, x, i, h * d + e] - want) < 1e-12
        assert np.allclose(got, spatial_attention(q, rep(k), rep(v), H) if Lq == Lk else got)


def pin_attention_grouped_bwd(attention_grouped, attention_grouped_bwd, attention_bwd_units):
    rng = np.random.default_rng(81)
    B, X, Lq, Lk, H, d = 1, 2, 3, 4, 4, 2
    for Hkv in (1, 2, 4):
        q, do = rng.standard_normal((B, X, Lq, H * d)), rng.standard_normal((B, X, Lq, H * d))
        k, v = rng.standard_normal((B, X, Lk, Hkv * d)), rng.standard_normal((B, X, Lk, Hkv * d))
        dq, dk, dv = attention_grouped_bwd(q, k, v, do, H, Hkv)
        loss = lambda qq, kk, vv: float((do * attention_grouped(qq, kk, vv, H, Hkv)).sum())
        assert np.allclose(dq, _fd_grad(lambda a: loss(a, k, v), q), atol=1e-8, rtol=1e-7)
        assert np.allclose(dk, _fd_grad(lambda a: loss(q, a, v), k), atol=1e-8, rtol=1e-7)
        assert np.allclose(dv, _fd_grad(lambda a: loss(q, k, a), v), atol=1e-8, rtol=1e-7)
    # Hkv = H, Lq = Lk: the multi-head gradients
    q, k, v, do = (rng.standard_normal((2, 2, 5, 6)) for _ in range(4))
    for a, b in zip(attention_grouped_bwd(q, k, v, do, 3, 3), attention_bwd_units(q, k, v, do, 3)):
        assert np.allclose(a, b)
