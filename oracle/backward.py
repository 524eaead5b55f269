"""Oracle for the backward pass (test infrastructure only).

The paper trains its models (the weak-scaling runs are taken as a training
stage, with ZeRO-2), so every operation of the block also has a gradient.
These are the vector-Jacobian products of the forward definitions, written
out by the chain rule in float64:

* attention, Eq. (3) per head: with z = q k^T * scale, P = softmax(z) row-wise
  and O = P v,
      dV = P^T dO,  dP = dO v^T,  dz = P * (dP - rowsum(dP * P)),
      dq = dz k * scale,  dk = dz^T q * scale;
  rowsum(dP * P) equals rowsum(dO * O) (the form the GPU uses).
  ``attention_lse`` is the natural-log row logsumexp of z, the statistic a
  forward pass saves for its backward.

Pinned by: central finite differences of <dO, f(x)> in float64; the key
gradients of a unit sum to zero (softmax is shift invariant); L = 1 gives
dq = dk = 0 and dv = dO; the logsumexp against scipy's and against the row
maximum; unit independence of the per-dimension wrappers.
"""
from __future__ import annotations

import math

import numpy as np

from .attention import _merge_heads, _split_heads


def attention_lse(q: np.ndarray, k: np.ndarray, scale: float | None = None) -> np.ndarray:
    """q: [..., Lq, d], k: [..., L, d] -> [..., Lq]: log sum_j exp(q.k_j * scale)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    z = np.matmul(q, np.swapaxes(k, -1, -2)) * scale
    m = z.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))[..., 0]


def attention_bwd(q, k, v, do, scale: float | None = None):
    """Gradients (dq, dk, dv) of sum(dO * attention(q, k, v)); shapes as ``attention``."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    kt = np.swapaxes(k, -1, -2)
    z = np.matmul(q, kt) * scale
    z = z - z.max(axis=-1, keepdims=True)
    p = np.exp(z)
    p = p / p.sum(axis=-1, keepdims=True)                      # softmax rows
    dv = np.matmul(np.swapaxes(p, -1, -2), do)                 # P^T dO
    dp = np.matmul(do, np.swapaxes(v, -1, -2))                 # dO v^T
    dz = p * (dp - (dp * p).sum(axis=-1, keepdims=True))       # softmax Jacobian, row by row
    dq = np.matmul(dz, k) * scale
    dk = np.matmul(np.swapaxes(dz, -1, -2), q) * scale
    return dq, dk, dv


def _units(x, H):
    h = _split_heads(np.asarray(x, dtype=np.float64), H)
    B, X, _, L, d = h.shape
    return h.reshape(B * X * H, L, d), h.shape


def attention_bwd_units(q, k, v, do, H: int, scale: float | None = None, unit_chunk: int = 64):
    """(B, X, L, C) tensors, attention over L per (b, x, head) unit -> (dq, dk, dv),
    each (B, X, L, C)."""
    (qf, shp), (kf, _), (vf, _), (df, _) = (_units(a, H) for a in (q, k, v, do))
    outs = [np.empty(qf.shape) for _ in range(3)]
    for u0 in range(0, qf.shape[0], unit_chunk):
        u1 = min(u0 + unit_chunk, qf.shape[0])
        for o, g in zip(outs, attention_bwd(qf[u0:u1], kf[u0:u1], vf[u0:u1], df[u0:u1], scale)):
            o[u0:u1] = g
    return tuple(_merge_heads(o.reshape(shp)) for o in outs)


def attention_lse_units(q, k, H: int, scale: float | None = None) -> np.ndarray:
    """(B, X, L, C) -> logsumexp per unit and query, [B * X * H, L] (unit = (b X + x) H + h)."""
    (qf, _), (kf, _) = _units(q, H), _units(k, H)
    return attention_lse(qf, kf, scale)


def attention_delta_units(o, do, H: int) -> np.ndarray:
    """rowsum(dO * O) per unit and query, [B * X * H, L]: the term the softmax
    Jacobian subtracts, rowsum(dP * P), in the form computed from the output."""
    (of, _), (df, _) = _units(o, H), _units(do, H)
    return (of * df).sum(axis=-1)


def attention_grouped_bwd(q, k, v, do, H: int, Hkv: int, scale: float | None = None):
    """Gradients (dq, dk, dv) of sum(dO * attention_grouped(q, k, v, H, Hkv)).
    A key/value head is read by the H // Hkv query heads of its group, so its
    gradients are the sums of theirs."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    B, X, Lq, C = q.shape
    d = C // H
    grp = H // Hkv
    dq = np.empty(q.shape)
    dk = np.zeros(k.shape)
    dv = np.zeros(v.shape)
    for h in range(H):
        cq = slice(h * d, (h + 1) * d)
        ck = slice((h // grp) * d, (h // grp + 1) * d)
        gq, gk, gv = attention_bwd(q[..., cq], k[..., ck], v[..., ck], do[..., cq], scale)
        dq[..., cq] = gq
        dk[..., ck] += gk
        dv[..., ck] += gv
    return dq, dk, dv
