"""Oracle for the spatial-temporal transformer block (test infrastructure only).

Building blocks, all float64:

* ``layernorm`` -- normalisation over the hidden size, as used around every
  sublayer (Eq. 4 and Eq. 6): (x - mean) / sqrt(var + eps) with the biased
  variance.  The paper gives neither eps nor an affine part; the reading here
  is eps as an argument (1e-6 by default) and no affine part.
* ``linear`` -- y = x W (+ b) with W of shape [in, out], the x W_1 convention
  of Eq. (5).
* ``gelu`` -- x * Phi(x) with the exact error function.  The paper's FFN uses
  ReLU (Eq. 5); the 720M-model block configuration uses GELU.
* ``relu`` -- max(x, 0), the FFN activation of Eq. (5).
* ``st_block`` -- one GPU's share of one layer of the 2D transformer (the two
  per-dimension blocks of the model-details appendix): pre-LN spatial
  attention with residual, the Switch T->S, pre-LN temporal attention with
  residual, then a pre-LN GELU MLP with residual.  Output in (B, S, T, C).
  ``BLOCK_NO_MLP_LN`` drops the LN of the MLP.  ``BLOCK_POST_LN`` places every
  LN after its residual add instead, x <- LN(x + sublayer(x)), the form of
  Eq. (4) and Eq. (6); ``BLOCK_RELU`` uses the ReLU FFN of Eq. (5).  Both
  together are the paper's own block.
* ``tiny_chain`` -- projection, spatial attention, output projection, switch,
  projection, temporal attention, output projection, no LN, residual, MLP or
  biases.

Readings where the paper is silent: QKV columns ordered [Q | K | V], each C
wide, head h at columns [h*d, (h+1)*d) of each (Eq. 1 concatenates heads in
order); the residual stream is kept at full precision.

Pinned by: hand-computed LayerNorm values and its moment identities, explicit
loops for the linear map, GELU against the normal CDF of scipy.stats and its
odd-part identity, and block identities (zero output projections leave only
the switched residual; T=1 / S=1 reduce attention to the V path; the N-rank
sharded evaluation equals the unsharded one).
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

from .attention import spatial_attention, temporal_attention
from .switch import switch

BLOCK_NO_MLP_LN = 1
BLOCK_POST_LN = 4
BLOCK_RELU = 8


def layernorm(x: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def linear(x: np.ndarray, w: np.ndarray, b: np.ndarray | None = None) -> np.ndarray:
    """x [..., in] times W [in, out] plus optional b [out]."""
    y = np.matmul(np.asarray(x, dtype=np.float64), np.asarray(w, dtype=np.float64))
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)
    return y


def gelu(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def relu(x: np.ndarray) -> np.ndarray:
    """The FFN activation of Eq. (5): max(x, 0)."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x, 0.0)


def _attn_sublayer(h, wqkv, bqkv, wo, bo, H, attn):
    C = h.shape[-1]
    qkv = linear(h, wqkv, bqkv)
    q, k, v = qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:]
    return linear(attn(q, k, v, H), wo, bo)


def st_block(x: np.ndarray, p: dict, H: int, eps: float = 1e-6, flags: int = 0) -> np.ndarray:
    """x: (B, T, S, C) residual stream.  p: weights in the paper's [in, out] layout
    (wqkv_s [C, 3C], wo_s [C, C], wqkv_t, wo_t, w1 [C, F], w2 [F, C]) and biases
    (b*, may be None).  Returns the block output in (B, S, T, C)."""
    x = np.asarray(x, dtype=np.float64)
    post = bool(flags & BLOCK_POST_LN)
    act = relu if (flags & BLOCK_RELU) else gelu
    ln = lambda v: layernorm(v, eps)
    # pre-LN: x + F(LN(x));  post-LN (Eq. 4, 6): LN(x + F(x))
    sub = (lambda v, f: ln(v + f(v))) if post else (lambda v, f: v + f(ln(v)))
    # spatial half: attention over S inside each frame, residual
    x = sub(x, lambda h: _attn_sublayer(h, p["wqkv_s"], p.get("bqkv_s"), p["wo_s"], p.get("bo_s"),
                                        H, spatial_attention))
    # the Switch T -> S on one GPU (a single chunk): (B, T, S, C) -> (B, S, T, C)
    y = switch(x, 1, 2, 1)[0]
    # temporal half: attention over T at each location, residual
    y = sub(y, lambda h: _attn_sublayer(h, p["wqkv_t"], p.get("bqkv_t"), p["wo_t"], p.get("bo_t"),
                                        H, temporal_attention))
    # MLP (Eq. 5 with the chosen activation), residual
    ffn = lambda h: linear(act(linear(h, p["w1"], p.get("b1"))), p["w2"], p.get("b2"))
    if flags & BLOCK_NO_MLP_LN:
        return y + ffn(y)
    return sub(y, ffn)


def tiny_chain(x: np.ndarray, p: dict, H: int) -> np.ndarray:
    """x (B, T, S, C) -> (B, S, T, C): Wqkv_s, spatial attention, Wo_s, switch,
    Wqkv_t, temporal attention, Wo_t.  Weights in [in, out] layout."""
    x = np.asarray(x, dtype=np.float64)
    y = _attn_sublayer(x, p["wqkv_s"], None, p["wo_s"], None, H, spatial_attention)
    y = switch(y, 1, 2, 1)[0]
    return _attn_sublayer(y, p["wqkv_t"], None, p["wo_t"], None, H, temporal_attention)
