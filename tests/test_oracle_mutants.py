"""Each plausible mistake planted in the oracle (on the CPU) must make at least
one pin fail.  This is what makes the pins worth trusting: a dropped term,
a wrong sign, axis or index, or a transposed operand anywhere in the oracle
is caught."""
import math
import sys
import types

import numpy as np
import pytest
from scipy.special import erf as SCIPY_ERF

import oracle  # noqa: F401  (loads the submodules)
from tests import oracle_pins as P

SW = sys.modules["oracle.switch"]
AT = sys.modules["oracle.attention"]
BL = sys.modules["oracle.block"]
BW = sys.modules["oracle.backward"]
OB = sys.modules["oracle.block_bwd"]
BWD_FLAGS = [0, BL.BLOCK_NO_MLP_LN, BL.BLOCK_POST_LN, BL.BLOCK_POST_LN | BL.BLOCK_RELU,
             BL.BLOCK_RELU | BL.BLOCK_NO_MLP_LN]


def _impl():
    return types.SimpleNamespace(
        switch=SW.switch, unswitch=SW.unswitch, exchange_unpack=SW.exchange_unpack,
        index_map=SW.switch_index_map, split=SW.split, gather=SW.gather, attention=AT.attention, spatial=AT.spatial_attention,
        temporal=AT.temporal_attention, strided=AT.temporal_attention_strided,
        layernorm=BL.layernorm, linear=BL.linear, gelu=BL.gelu, relu=BL.relu, st_block=BL.st_block,
        tiny_chain=BL.tiny_chain, attention_bwd=BW.attention_bwd,
        attention_bwd_units=BW.attention_bwd_units, attention_lse=BW.attention_lse,
        attention_lse_units=BW.attention_lse_units, attention_delta_units=BW.attention_delta_units,
        linear_bwd=OB.linear_bwd, layernorm_bwd=OB.layernorm_bwd, gelu_bwd=OB.gelu_bwd,
        relu_bwd=OB.relu_bwd, st_block_bwd=OB.st_block_bwd, attention_grouped=AT.attention_grouped,
        attention_grouped_bwd=BW.attention_grouped_bwd)


def _pins(i):
    return [
        lambda: P.pin_switch_golden(i.switch),
        lambda: P.pin_switch_index_loops(i.switch, i.index_map),
        lambda: P.pin_switch_round_trip(i.switch, i.unswitch),
        lambda: P.pin_switch_b1_transpose(i.switch),
        lambda: P.pin_switch_bits_and_copy(i.switch),
        lambda: P.pin_switch_nrank_simulation(i.switch, i.exchange_unpack),
        lambda: P.pin_switch_k3_index_loops(i.switch),
        lambda: P.pin_switch_k3_unit_dim(i.switch),
        lambda: P.pin_switch_nrank_simulation_k3(i.switch, i.exchange_unpack),
        lambda: P.pin_split_gather(i.split, i.gather),
        lambda: P.pin_switch_is_gather_then_split(i.switch, i.exchange_unpack, i.split, i.gather),
        lambda: P.pin_attention_brute(i.attention),
        lambda: P.pin_attention_l1_is_v(i.attention),
        lambda: P.pin_attention_zero_q_mean(i.attention),
        lambda: P.pin_attention_two_keys_closed_form(i.attention),
        lambda: P.pin_attention_rows_stochastic(i.attention),
        lambda: P.pin_attention_hard_max(i.attention),
        lambda: P.pin_attention_permutations(i.attention),
        lambda: P.pin_attention_scale_default(i.attention),
        lambda: P.pin_spatial_temporal_units(i.spatial, i.temporal, i.strided, i.switch),
        lambda: P.pin_layernorm(i.layernorm),
        lambda: P.pin_linear(i.linear),
        lambda: P.pin_gelu(i.gelu),
        lambda: P.pin_relu(i.relu),
        lambda: P.pin_block_post_ln_relu(i.st_block, i.layernorm, i.linear, i.relu, i.switch,
                                         BL.BLOCK_POST_LN, BL.BLOCK_RELU),
        lambda: P.pin_block_identities(i.st_block, i.layernorm, i.linear, i.gelu, i.switch),
        lambda: P.pin_block_t1_s1(i.st_block, i.layernorm, i.linear, i.gelu),
        lambda: P.pin_block_sharded_equals_unsharded(i.st_block, i.layernorm, i.linear, i.gelu,
                                                     i.switch, i.exchange_unpack, i.spatial,
                                                     i.temporal),
        lambda: P.pin_tiny_chain(i.tiny_chain, i.st_block),
        lambda: P.pin_attention_bwd_fd(i.attention, i.attention_bwd),
        lambda: P.pin_attention_bwd_invariants(i.attention_bwd),
        lambda: P.pin_attention_lse(i.attention_lse),
        lambda: P.pin_attention_bwd_units(i.attention_bwd, i.attention_bwd_units,
                                          i.attention_lse_units, i.attention_lse,
                                          i.attention_delta_units, i.attention),
        lambda: P.pin_attention_grouped(i.attention_grouped, i.spatial, i.attention),
        lambda: P.pin_attention_grouped_bwd(i.attention_grouped, i.attention_grouped_bwd, i.attention_bwd_units),
        # the block backward pins last: they are the slowest
        lambda: P.pin_linear_bwd(i.linear, i.linear_bwd),
        lambda: P.pin_layernorm_bwd(i.layernorm, i.layernorm_bwd),
        lambda: P.pin_gelu_bwd(i.gelu, i.gelu_bwd, i.relu, i.relu_bwd),
        lambda: P.pin_block_bwd_fd(i.st_block, i.st_block_bwd, BWD_FLAGS),
        lambda: P.pin_block_bwd_autograd(i.st_block_bwd, BWD_FLAGS),
    ]


def _n_failed(stop_at_first: bool = False):
    failed = 0
    for pin in _pins(_impl()):
        try:
            pin()
        except Exception:
            failed += 1
            if stop_at_first:
                break
    return failed


# ---------------------------------------------------------------- mutants
_orig_switch = SW.switch
_orig_attention = AT.attention
_orig_layernorm = BL.layernorm
_orig_linear = BL.linear


def sw_interleaved_chunks(x, f, t, n):
    # chunks take every n-th index of the to-dim instead of contiguous slices
    y = _orig_switch(x, f, t, 1)[0]
    if f == t:
        return y.copy()
    B, D, F, C = y.shape
    return np.ascontiguousarray(y.reshape(B, D // n, n, F, C).transpose(2, 0, 1, 3, 4))


def sw_batch_outside(x, f, t, n):
    # batch outermost: [b][n][...] instead of [n][b][...]
    y = _orig_switch(x, f, t, n)
    if f == t:
        return y
    return np.ascontiguousarray(y.transpose(1, 0, 2, 3, 4)).reshape(y.shape)


def sw_no_transpose(x, f, t, n):
    if f == t:
        return x.copy()
    B, D1, D2, C = x.shape
    # slices the to-dim into chunks but keeps the from-dim outer inside each chunk
    return np.ascontiguousarray(x.reshape(B, D1, n, D2 // n, C).transpose(2, 0, 1, 3, 4)
                                .reshape(n, B, D2 // n, D1, C)) if t == 2 else _orig_switch(x, f, t, n)


def sw_off_by_one(x, f, t, n):
    y = _orig_switch(x, f, t, n)
    return np.roll(y, 1, axis=3) if f != t else y


def sw_k3_others_reversed(x, f, t, n):
    # K = 3: the two other sequence dims swapped inside each chunk
    y = _orig_switch(x, f, t, n)
    if x.ndim != 5 or f == t:
        return y
    return np.ascontiguousarray(np.swapaxes(y, 2, 3))


def sw_k3_from_dim_outer(x, f, t, n):
    # K = 3: the from-dim placed first instead of next to C
    y = _orig_switch(x, f, t, n)
    if x.ndim != 5 or f == t:
        return y
    return np.ascontiguousarray(np.moveaxis(y, -2, 2))


_orig_split = SW.split
_orig_gather = SW.gather


def split_from_end(x, dim, n_chunks, rank):
    return _orig_split(x, dim, n_chunks, n_chunks - 1 - rank)


def gather_reversed(shards, dim):
    return _orig_gather(list(shards)[::-1], dim)


def exchange_outer_axis(packed_per_rank):
    # the received chunks joined on the outermost sequence axis, not the from-dim
    N = len(packed_per_rank)
    return [np.concatenate([p[n] for p in packed_per_rank], axis=1) for n in range(N)]


def att_no_scale(q, k, v, scale=None):
    return _orig_attention(q, k, v, 1.0 if scale is None else scale)


def att_padded_scale(q, k, v, scale=None):
    d = q.shape[-1]
    dp = -(-d // 16) * 16 if d % 16 else d + 8
    return _orig_attention(q, k, v, 1.0 / math.sqrt(dp) if scale is None else scale)


def att_softmax_over_queries(q, k, v, scale=None):
    q = np.asarray(q, float); k = np.asarray(k, float); v = np.asarray(v, float)
    s = (1 / math.sqrt(q.shape[-1])) if scale is None else scale
    z = np.matmul(q, np.swapaxes(k, -1, -2)) * s
    p = np.exp(z - z.max(axis=-2, keepdims=True))
    p = p / p.sum(axis=-2, keepdims=True)
    return np.matmul(p, v)


def att_k_for_v(q, k, v, scale=None):
    if np.shape(k) != np.shape(v):
        return _orig_attention(q, k, v, scale)
    return _orig_attention(q, k, k, scale)


def att_negated_scores(q, k, v, scale=None):
    s = (1 / math.sqrt(np.shape(q)[-1])) if scale is None else scale
    return _orig_attention(q, k, v, -s)


def att_unnormalised(q, k, v, scale=None):
    q = np.asarray(q, float); k = np.asarray(k, float); v = np.asarray(v, float)
    s = (1 / math.sqrt(q.shape[-1])) if scale is None else scale
    z = np.matmul(q, np.swapaxes(k, -1, -2)) * s
    return np.matmul(np.exp(z - z.max(axis=-1, keepdims=True)), v)


def ln_unbiased(x, eps=1e-6):
    x = np.asarray(x, float)
    return (x - x.mean(-1, keepdims=True)) / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps)


def ln_eps_outside(x, eps=1e-6):
    x = np.asarray(x, float)
    return (x - x.mean(-1, keepdims=True)) / (np.sqrt(x.var(-1, keepdims=True)) + eps)


def ln_no_centre(x, eps=1e-6):
    x = np.asarray(x, float)
    return x / np.sqrt(x.var(-1, keepdims=True) + eps)


def gelu_tanh(x):
    x = np.asarray(x, float)
    return 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))


def gelu_no_sqrt2(x):
    from scipy.special import erf
    x = np.asarray(x, float)
    return 0.5 * x * (1 + erf(x))


def lin_no_bias(x, w, b=None):
    return _orig_linear(x, w, None)


def lin_transposed(x, w, b=None):
    w = np.asarray(w)
    if w.shape[0] == w.shape[1]:
        w = w.T
    return _orig_linear(x, w, b)


def block_wrong_axes(x, p, H, eps=1e-6, flags=0):
    # spatial half attends over T instead of S
    saved = BL.spatial_attention
    BL.spatial_attention = lambda q, k, v, H_, scale=None: AT.temporal_attention_strided(q, k, v, H_, scale)
    try:
        return _orig_block(x, p, H, eps, flags)
    finally:
        BL.spatial_attention = saved


def block_no_temporal_residual(x, p, H, eps=1e-6, flags=0):
    saved = BL.temporal_attention
    calls = {}

    def t_attn(q, k, v, H_, scale=None):
        return saved(q, k, v, H_, scale)
    # drop the residual of the temporal half: subtract the switched input back out
    y_in = BL.switch(x + BL._attn_sublayer(BL.layernorm(x, eps), p["wqkv_s"], p.get("bqkv_s"),
                                           p["wo_s"], p.get("bo_s"), H, BL.spatial_attention),
                     1, 2, 1)[0]
    y = _orig_block(x, p, H, eps, flags)
    return y - y_in


def block_post_mlp_ln(x, p, H, eps=1e-6, flags=0):
    y = _orig_block(x, p, H, eps, flags | BL.BLOCK_NO_MLP_LN)
    return y


def relu_leaky(x):
    x = np.asarray(x, float)
    return np.where(x > 0, x, 0.01 * x)


def block_post_ln_inside(x, p, H, eps=1e-6, flags=0):
    # post-LN placed on the sublayer output instead of the sum: x + LN(F(x))
    if not flags & BL.BLOCK_POST_LN:
        return _orig_block(x, p, H, eps, flags)
    saved = BL.layernorm
    f = flags & ~BL.BLOCK_POST_LN

    def attn_sub(h, wq, bq, wo, bo, attn):
        return saved(BL._attn_sublayer(h, wq, bq, wo, bo, H, attn), eps)
    act = BL.relu if flags & BL.BLOCK_RELU else BL.gelu
    x = np.asarray(x, float)
    x = x + attn_sub(x, p["wqkv_s"], p.get("bqkv_s"), p["wo_s"], p.get("bo_s"), BL.spatial_attention)
    y = BL.switch(x, 1, 2, 1)[0]
    y = y + attn_sub(y, p["wqkv_t"], p.get("bqkv_t"), p["wo_t"], p.get("bo_t"), BL.temporal_attention)
    return y + saved(BL.linear(act(BL.linear(y, p["w1"], p.get("b1"))), p["w2"], p.get("b2")), eps)


def block_post_ln_no_final(x, p, H, eps=1e-6, flags=0):
    # post-LN without the LN after the MLP's residual add
    if not flags & BL.BLOCK_POST_LN:
        return _orig_block(x, p, H, eps, flags)
    return _orig_block(x, p, H, eps, flags | BL.BLOCK_NO_MLP_LN)


_orig_abwd = BW.attention_bwd
_orig_lse = BW.attention_lse


def abwd_no_delta(q, k, v, do, scale=None):
    # the softmax Jacobian without the row-sum term: dz = P * dP
    q, k, v, do = (np.asarray(a, float) for a in (q, k, v, do))
    s = 1 / math.sqrt(q.shape[-1]) if scale is None else scale
    z = np.matmul(q, np.swapaxes(k, -1, -2)) * s
    p = np.exp(z - z.max(-1, keepdims=True)); p /= p.sum(-1, keepdims=True)
    dz = p * np.matmul(do, np.swapaxes(v, -1, -2))
    return np.matmul(dz, k) * s, np.matmul(np.swapaxes(dz, -1, -2), q) * s, \
        np.matmul(np.swapaxes(p, -1, -2), do)


def abwd_dk_unscaled(q, k, v, do, scale=None):
    dq, dk, dv = _orig_abwd(q, k, v, do, scale)
    s = 1 / math.sqrt(np.shape(q)[-1]) if scale is None else scale
    return dq, dk / s, dv


def abwd_dq_from_v(q, k, v, do, scale=None):
    # dq built with v in place of k
    dq, dk, dv = _orig_abwd(q, k, v, do, scale)
    dq_v, _, _ = _orig_abwd(q, v, v, do, scale)
    return dq_v if np.shape(k) == np.shape(v) else dq, dk, dv


def abwd_dv_untransposed(q, k, v, do, scale=None):
    dq, dk, dv = _orig_abwd(q, k, v, do, scale)
    if np.shape(q)[-2] != np.shape(k)[-2]:
        return dq, dk, dv
    q_, k_ = np.asarray(q, float), np.asarray(k, float)
    s = 1 / math.sqrt(q_.shape[-1]) if scale is None else scale
    z = np.matmul(q_, np.swapaxes(k_, -1, -2)) * s
    p = np.exp(z - z.max(-1, keepdims=True)); p /= p.sum(-1, keepdims=True)
    return dq, dk, np.matmul(p, np.asarray(do, float))


def lse_log2(q, k, scale=None):
    return _orig_lse(q, k, scale) / math.log(2)


_orig_block = BL.st_block
_orig_grouped = AT.attention_grouped
_orig_grouped_bwd = BW.attention_grouped_bwd


def grouped_modulo_heads(q, k, v, H, Hkv, scale=None):
    # query head h reading key/value head h % Hkv instead of h // (H / Hkv)
    q, k, v = (np.asarray(a, float) for a in (q, k, v))
    d = q.shape[-1] // H
    out = np.empty(q.shape)
    for h in range(H):
        cq, ck = slice(h * d, (h + 1) * d), slice((h % Hkv) * d, (h % Hkv + 1) * d)
        out[..., cq] = _orig_attention(q[..., cq], k[..., ck], v[..., ck], scale)
    return out


def grouped_bwd_last_head_only(q, k, v, do, H, Hkv, scale=None):
    # a key/value head's gradient taken from the last query head of its group, not summed
    q, k, v, do = (np.asarray(a, float) for a in (q, k, v, do))
    d = q.shape[-1] // H
    grp = H // Hkv
    dq, dk, dv = np.empty(q.shape), np.zeros(k.shape), np.zeros(v.shape)
    for h in range(H):
        cq, ck = slice(h * d, (h + 1) * d), slice((h // grp) * d, (h // grp + 1) * d)
        gq, gk, gv = _orig_abwd(q[..., cq], k[..., ck], v[..., ck], do[..., cq], scale)
        dq[..., cq], dk[..., ck], dv[..., ck] = gq, gk, gv
    return dq, dk, dv
_orig_ln_bwd = OB.layernorm_bwd
_orig_lin_bwd = OB.linear_bwd
_orig_sub_bwd = OB._attn_sublayer_bwd


def lnb_no_projection(x, dy, eps=1e-6):
    # drops the term along the normalised row: (dy - mean(dy)) / sigma
    x = np.asarray(x, float)
    mu = x.mean(-1, keepdims=True)
    sigma = np.sqrt(((x - mu) ** 2).mean(-1, keepdims=True) + eps)
    dy = np.asarray(dy, float)
    return (dy - dy.mean(-1, keepdims=True)) / sigma


def gelub_cdf_only(u, dy):
    # d/du (u Phi(u)) taken as Phi(u): the u phi(u) term dropped
    u = np.asarray(u, float)
    return np.asarray(dy, float) * 0.5 * (1 + SCIPY_ERF(u / math.sqrt(2)))


def linb_db_mean(x, w, dy):
    dx, dw, db = _orig_lin_bwd(x, w, dy)
    return dx, dw, db / max(1, np.asarray(dy).reshape(-1, np.shape(dy)[-1]).shape[0])


def subb_wo_transposed(saved, p, tag, H, d_out, grads):
    dh = _orig_sub_bwd(saved, p, tag, H, d_out, grads)
    grads["wo_" + tag] = grads["wo_" + tag].T
    return dh

MUTANTS = {
    "switch: interleaved chunks": [(SW, "switch", sw_interleaved_chunks), (BL, "switch", sw_interleaved_chunks)],
    "switch: batch outside chunks": [(SW, "switch", sw_batch_outside), (BL, "switch", sw_batch_outside)],
    "switch: missing transpose": [(SW, "switch", sw_no_transpose), (BL, "switch", sw_no_transpose)],
    "switch: off-by-one index": [(SW, "switch", sw_off_by_one), (BL, "switch", sw_off_by_one)],
    "switch K=3: other dims swapped": [(SW, "switch", sw_k3_others_reversed)],
    "switch K=3: from-dim outermost": [(SW, "switch", sw_k3_from_dim_outer)],
    "split: slices counted from the end": [(SW, "split", split_from_end)],
    "gather: shards in reverse order": [(SW, "gather", gather_reversed)],
    "exchange: joined on the outer axis": [(SW, "exchange_unpack", exchange_outer_axis)],
    "attention bwd: no row-sum term": [(BW, "attention_bwd", abwd_no_delta)],
    "attention bwd: dk without the scale": [(BW, "attention_bwd", abwd_dk_unscaled)],
    "attention bwd: dq from v": [(BW, "attention_bwd", abwd_dq_from_v)],
    "attention bwd: dv = P dO": [(BW, "attention_bwd", abwd_dv_untransposed)],
    "attention lse: base 2": [(BW, "attention_lse", lse_log2)],
    "grouped attention: head h reads kv head h % Hkv": [(AT, "attention_grouped", grouped_modulo_heads)],
    "grouped attention bwd: kv gradients not summed over the group":
        [(BW, "attention_grouped_bwd", grouped_bwd_last_head_only)],
    "layernorm bwd: no projection on the output": [(OB, "layernorm_bwd", lnb_no_projection)],
    "gelu bwd: Phi only": [(OB, "gelu_bwd", gelub_cdf_only)],
    "linear bwd: bias gradient averaged": [(OB, "linear_bwd", linb_db_mean)],
    "block bwd: switch adjoint without the transpose": [(OB, "switch", sw_no_transpose)],
    "block bwd: out-projection weight gradient transposed": [(OB, "_attn_sublayer_bwd", subb_wo_transposed)],
    "attention: no 1/sqrt(d)": [(AT, "attention", att_no_scale)],
    "attention: padded-width scale": [(AT, "attention", att_padded_scale)],
    "attention: softmax over queries": [(AT, "attention", att_softmax_over_queries)],
    "attention: K used as V": [(AT, "attention", att_k_for_v)],
    "attention: negated scores": [(AT, "attention", att_negated_scores)],
    "attention: missing normalisation": [(AT, "attention", att_unnormalised)],
    "layernorm: unbiased variance": [(BL, "layernorm", ln_unbiased)],
    "layernorm: eps outside sqrt": [(BL, "layernorm", ln_eps_outside)],
    "layernorm: no centring": [(BL, "layernorm", ln_no_centre)],
    "gelu: tanh approximation": [(BL, "gelu", gelu_tanh)],
    "gelu: erf(x) without 1/sqrt(2)": [(BL, "gelu", gelu_no_sqrt2)],
    "linear: bias dropped": [(BL, "linear", lin_no_bias)],
    "linear: square weight transposed": [(BL, "linear", lin_transposed)],
    "block: spatial half over T": [(BL, "st_block", block_wrong_axes)],
    "block: temporal residual dropped": [(BL, "st_block", block_no_temporal_residual)],
    "block: no LN before the MLP": [(BL, "st_block", block_post_mlp_ln)],
    "relu: leaky negative slope": [(BL, "relu", relu_leaky)],
    "block: post-LN on the sublayer, not the sum": [(BL, "st_block", block_post_ln_inside)],
    "block: post-LN without the MLP's LN": [(BL, "st_block", block_post_ln_no_final)],
}


def test_unmutated_oracle_passes_every_pin():
    assert _n_failed() == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    for mod, attr, fn in MUTANTS[name]:
        monkeypatch.setattr(mod, attr, fn)
    assert _n_failed(stop_at_first=True) >= 1, f"no pin catches the planted mistake: {name}"
