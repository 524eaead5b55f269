"""Oracle for the backward pass of the spatial-temporal block (test
infrastructure only).

The paper trains the models it parallelises (its weak-scaling runs are taken
as a training stage, with ZeRO-2 sharding the optimizer state), so every
operation of the block has a gradient.  These are the vector-Jacobian products
of the forward definitions in ``block.py``, written out by the chain rule in
float64, step by step in reverse order of the forward:

* ``linear_bwd``: y = x W + b  ->  dx = dy W^T, dW = x^T dy, db = sum over rows of dy.
* ``layernorm_bwd``: y = (x - mu) / sigma with sigma = sqrt(var + eps) (biased
  variance, no affine part)  ->  dx = (dy - mean(dy) - y * mean(dy * y)) / sigma.
* ``gelu_bwd``: GELU(u) = u Phi(u)  ->  du = dy (Phi(u) + u phi(u)).
* ``relu_bwd``: du = dy where u > 0, else 0.
* the Switch: a permutation of rows, so its adjoint is the inverse permutation
  (the switch back, S -> T).
* ``st_block_bwd``: the whole block, pre-LN (the default) or post-LN
  (``BLOCK_POST_LN``), GELU or ReLU, with or without the MLP's LayerNorm,
  using the attention backward of ``backward.py``.

Pinned by: central finite differences of <dy, f(x)> in float64 for every
function and for the block with respect to its input and to sampled weight
entries; an independent evaluation of the same gradients by torch autograd in
float64; LayerNorm gradients are orthogonal to the ones vector and to the
normalised row; GELU's derivative against the odd-part identity.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

from .attention import spatial_attention, temporal_attention
from .backward import attention_bwd_units
from .block import BLOCK_NO_MLP_LN, BLOCK_POST_LN, BLOCK_RELU, gelu, layernorm, linear, relu
from .switch import switch


def linear_bwd(x, w, dy):
    """y = x W (+ b), x [..., in], W [in, out], dy [..., out] -> (dx, dW, db)."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    x2 = x.reshape(-1, x.shape[-1])
    dy2 = dy.reshape(-1, dy.shape[-1])
    dx = np.matmul(dy, w.T)
    dw = np.matmul(x2.T, dy2)
    db = dy2.sum(axis=0)
    return dx, dw, db


def layernorm_bwd(x, dy, eps: float = 1e-6):
    """Gradient of ``layernorm`` with respect to its input, row by row."""
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    sigma = np.sqrt(var + eps)
    y = (x - mu) / sigma
    return (dy - dy.mean(axis=-1, keepdims=True) - y * (dy * y).mean(axis=-1, keepdims=True)) / sigma


def gelu_bwd(u, dy):
    """d/du of u Phi(u) is Phi(u) + u phi(u), phi the standard normal density."""
    u = np.asarray(u, dtype=np.float64)
    cdf = 0.5 * (1.0 + erf(u / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)
    return np.asarray(dy, dtype=np.float64) * (cdf + u * pdf)


def relu_bwd(u, dy):
    return np.where(np.asarray(u) > 0.0, np.asarray(dy, dtype=np.float64), 0.0)


def _sum_bias(grads, name, db):
    if grads is not None:
        grads[name] = db


def _attn_sublayer_fwd(h, p, tag, H, attn):
    """Forward of one attention sublayer, keeping what its backward needs."""
    C = h.shape[-1]
    qkv = linear(h, p["wqkv_" + tag], p.get("bqkv_" + tag))
    q, k, v = qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:]
    a = attn(q, k, v, H)
    return linear(a, p["wo_" + tag], p.get("bo_" + tag)), (h, q, k, v, a)


def _attn_sublayer_bwd(saved, p, tag, H, d_out, grads):
    """Backward of one attention sublayer: d_out -> d(its input h); weight
    gradients into grads.  The attention runs over axis 2 of (B, X, L, C)."""
    h, q, k, v, a = saved
    da, grads["wo_" + tag], db = linear_bwd(a, p["wo_" + tag], d_out)
    if p.get("bo_" + tag) is not None:
        grads["bo_" + tag] = db
    dq, dk, dv = attention_bwd_units(q, k, v, da, H)
    dqkv = np.concatenate([dq, dk, dv], axis=-1)
    dh, grads["wqkv_" + tag], db = linear_bwd(h, p["wqkv_" + tag], dqkv)
    if p.get("bqkv_" + tag) is not None:
        grads["bqkv_" + tag] = db
    return dh


def st_block_bwd(x, p: dict, H: int, dy, eps: float = 1e-6, flags: int = 0):
    """Gradients of sum(dy * st_block(x, p, H, eps, flags)).

    x: (B, T, S, C); dy: (B, S, T, C), the gradient of the block output.
    Returns (dx in (B, T, S, C), grads) with grads[name] shaped like p[name]
    for every weight and every bias that is not None."""
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    post = bool(flags & BLOCK_POST_LN)
    use_relu = bool(flags & BLOCK_RELU)
    act, act_bwd = (relu, relu_bwd) if use_relu else (gelu, gelu_bwd)
    ln = lambda v: layernorm(v, eps)
    grads: dict = {}

    # ---- forward, keeping the inputs of every step
    # spatial half (attention over S in each frame)
    if post:
        o1, sv1 = _attn_sublayer_fwd(x, p, "s", H, spatial_attention)
        r1 = x + o1
        x1 = ln(r1)
    else:
        o1, sv1 = _attn_sublayer_fwd(ln(x), p, "s", H, spatial_attention)
        x1 = x + o1
    # the Switch T -> S: (B, T, S, C) -> (B, S, T, C)
    y0 = switch(x1, 1, 2, 1)[0]
    # temporal half (attention over T at each location)
    if post:
        o2, sv2 = _attn_sublayer_fwd(y0, p, "t", H, temporal_attention)
        r2 = y0 + o2
        y1 = ln(r2)
    else:
        o2, sv2 = _attn_sublayer_fwd(ln(y0), p, "t", H, temporal_attention)
        y1 = y0 + o2
    # MLP
    no_mlp_ln = bool(flags & BLOCK_NO_MLP_LN)
    h3 = y1 if (post or no_mlp_ln) else ln(y1)
    u = linear(h3, p["w1"], p.get("b1"))
    g = act(u)
    # output: y = ln(y1 + m) (post-LN with the MLP's LN), else y1 + m

    # ---- backward, in reverse order
    if post and not no_mlp_ln:
        r3 = y1 + linear(g, p["w2"], p.get("b2"))
        dr3 = layernorm_bwd(r3, dy, eps)
    else:
        dr3 = dy
    # m = g W2 + b2
    dg, grads["w2"], db = linear_bwd(g, p["w2"], dr3)
    if p.get("b2") is not None:
        grads["b2"] = db
    du = act_bwd(u, dg)
    dh3, grads["w1"], db = linear_bwd(h3, p["w1"], du)
    if p.get("b1") is not None:
        grads["b1"] = db
    dy1 = dr3 + (dh3 if (post or no_mlp_ln) else layernorm_bwd(y1, dh3, eps))
    # temporal half
    if post:
        dr2 = layernorm_bwd(r2, dy1, eps)
        dy0 = dr2 + _attn_sublayer_bwd(sv2, p, "t", H, dr2, grads)
    else:
        dh2 = _attn_sublayer_bwd(sv2, p, "t", H, dy1, grads)
        dy0 = dy1 + layernorm_bwd(y0, dh2, eps)
    # the Switch's adjoint: the inverse permutation, (B, S, T, C) -> (B, T, S, C)
    dx1 = switch(dy0, 1, 2, 1)[0]
    # spatial half
    if post:
        dr1 = layernorm_bwd(r1, dx1, eps)
        dx = dr1 + _attn_sublayer_bwd(sv1, p, "s", H, dr1, grads)
    else:
        dh1 = _attn_sublayer_bwd(sv1, p, "s", H, dx1, grads)
        dx = dx1 + layernorm_bwd(x, dh1, eps)
    return dx, grads
