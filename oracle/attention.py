"""Oracle for scaled dot-product attention along one sequence dimension
(test infrastructure only).

Eq. (3): Att(Q, K, V) = softmax(Q K^T / sqrt(d_k)) V, computed independently
for each head (Eq. 1-2; head h owns columns [h*d, (h+1)*d) of the hidden size,
heads are concatenated in order).  In a multi-dimensional transformer the
block runs on Reshape(X, [B * prod_{j != i} S_j, S_i, C]) (Eq. 7-8): every
(batch, other-dimension index, head) triple is an independent attention
problem ("unit") of length L = S_i.

* spatial attention: x in (B, T, S, C), units (b, t, h), L = S;
* temporal attention: x in (B, S, T, C) (after the switch), units (b, s, h),
  L = T.

The softmax is the plain two-pass form: z = q.k / sqrt(d), subtract the row
maximum, exponentiate, divide by the row sum.  d is the true head width (never
a padded width).  No causal mask: the paper's attention has none.  All
arithmetic is float64.

Pinned by: L=1 gives V; zero queries or identical keys give the mean of V; the
closed form at L=2; brute force over Python floats with math.exp and
math.fsum; a huge scale selects V at the arg-max key; permutation
(equi)variance; unit independence; the strided temporal reading equals the
switched one.
"""
from __future__ import annotations

import math

import numpy as np


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float | None = None) -> np.ndarray:
    """q: [..., Lq, d], k: [..., L, d], v: [..., L, dv] -> [..., Lq, dv] in float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    d = q.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    z = np.matmul(q, np.swapaxes(k, -1, -2)) * scale          # [..., Lq, L]
    z = z - z.max(axis=-1, keepdims=True)
    p = np.exp(z)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.matmul(p, v)


def attention_rows(q_rows: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float | None = None):
    """Attention outputs for a chosen set of query rows of one unit (same definition)."""
    return attention(q_rows, k, v, scale)


def _split_heads(x: np.ndarray, H: int) -> np.ndarray:
    """(B, X, L, C) -> (B, X, H, L, d)."""
    B, X, L, C = x.shape
    return x.reshape(B, X, L, H, C // H).transpose(0, 1, 3, 2, 4)


def _merge_heads(o: np.ndarray) -> np.ndarray:
    B, X, H, L, d = o.shape
    return o.transpose(0, 1, 3, 2, 4).reshape(B, X, L, H * d)


def _per_unit(q, k, v, H, scale, unit_chunk=64):
    qh, kh, vh = _split_heads(q, H), _split_heads(k, H), _split_heads(v, H)
    B, X, _, L, d = qh.shape
    out = np.empty(qh.shape, dtype=np.float64)
    qf = qh.reshape(B * X * H, L, d)
    kf = kh.reshape(B * X * H, L, d)
    vf = vh.reshape(B * X * H, L, d)
    of = out.reshape(B * X * H, L, d)
    # units are independent; they are taken a few at a time only to bound memory
    for u0 in range(0, qf.shape[0], unit_chunk):
        u1 = min(u0 + unit_chunk, qf.shape[0])
        of[u0:u1] = attention(qf[u0:u1], kf[u0:u1], vf[u0:u1], scale)
    return _merge_heads(out)


def spatial_attention(q, k, v, H: int, scale: float | None = None) -> np.ndarray:
    """Attention over S within each frame: inputs (B, T, S, C), output (B, T, S, C)."""
    return _per_unit(q, k, v, H, scale)


def temporal_attention(q, k, v, H: int, scale: float | None = None) -> np.ndarray:
    """Attention over T at each spatial location: inputs (B, S, T, C), output (B, S, T, C)."""
    return _per_unit(q, k, v, H, scale)


def temporal_attention_strided(q, k, v, H: int, scale: float | None = None) -> np.ndarray:
    """Temporal attention read straight from (B, T, S, C) tensors (no switch);
    output in (B, T, S, C).  Same units as ``temporal_attention``."""
    sw = lambda a: np.swapaxes(np.asarray(a, dtype=np.float64), 1, 2)
    return np.swapaxes(_per_unit(sw(q), sw(k), sw(v), H, scale), 1, 2)


def attention_grouped(q, k, v, H: int, Hkv: int, scale: float | None = None) -> np.ndarray:
    """Attention with grouped key/value heads and separate query and key lengths
    -- the variants the paper states DSP is compatible with (multi-query and
    grouped-query attention, cross-attention), on the same per-(b, x) units.

    q: (B, X, Lq, H*d); k, v: (B, X, Lk, Hkv*d), Hkv dividing H.  Query head h
    attends with key/value head h // (H // Hkv) (Hkv = H: multi-head; Hkv = 1:
    multi-query).  Lq may differ from Lk (cross-attention: the keys and values
    come from another sequence).  Returns (B, X, Lq, H*d)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if H % Hkv:
        raise ValueError("Hkv must divide H")
    B, X, Lq, C = q.shape
    d = C // H
    grp = H // Hkv
    out = np.empty((B, X, Lq, C))
    for h in range(H):
        cq = slice(h * d, (h + 1) * d)
        ck = slice((h // grp) * d, (h // grp + 1) * d)
        out[..., cq] = attention(q[..., cq], k[..., ck], v[..., ck], scale)
    return out
