"""Oracle for the DSP primitives on one GPU (test infrastructure only).

The paper's Switch (primitive table, row s_i -> s_j; Eq. 10) takes a tensor
sharded on sequence dimension i (local length S_i/N) to one sharded on
dimension j (local length S_j/N) with one all-to-all.  One GPU's share of that
operation, before the exchange, is:

1. the permute that moves dimension i (the one about to become whole) next to
   C and keeps the other sequence dimensions in their order -- the Reshape of
   Eq. (7), [B * prod_{k != i} S_k, S_i, C], that lets the next stage run on
   contiguous sequences along i;
2. the pack of that permuted tensor into ``n_chunks`` contiguous chunks, chunk
   n holding the n-th slice of dimension j, destined for rank n.

For a 4-D tensor [B, D1, D2, C] with from_dim=1, to_dim=2 (for example
(B,T,S,C), T sharded, switching to S) the packed output is

    y[n][b][j'][i][c] = x[b][i][n*D2/N + j'][c],

chunk n of shape [B, D2/N, D1, C].  With from_dim=2, to_dim=1 no transpose is
needed: y[n][b][i'][j][c] = x[b][n*D1/N + i'][j][c].  from_dim == to_dim is
the table's no-op row and returns a copy.  Tensors with K = 3 sequence
dimensions, [B, S1, S2, S3, C], follow the same two steps (Eq. 7 for K = 3).

The table's other two rows need no all-to-all: Split (s^ -> s_i) keeps one
slice of a replicated tensor, Gather (s_i -> s^) is the all-gather that
concatenates every rank's slice.  ``split`` is one rank's slice; ``gather`` is
the receiver's concatenation of the N slices it got.

Readings where the paper is silent: the batch index sits inside each chunk;
D_to must be divisible by n_chunks (the paper assumes S_j/N is an integer);
K is 2 or 3.

Everything is done on unsigned-integer views of the data, so the result is a
pure bit copy.  Pinned by: a hand-worked fixture, explicit index loops (K = 2
and K = 3), the round trip, the B=1 transpose identity, the K = 3 reduction to
K = 2 over a unit dimension, the N-rank exchange simulation (K = 2 and 3) and
split / gather inverses.
"""
from __future__ import annotations

import numpy as np


def _bits(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x)
    return x.view({1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[x.itemsize])


def _check_seq_dim(ndim: int, *dims: int) -> None:
    if ndim not in (4, 5):
        raise ValueError("tensors are [B, S_1, ..., S_K, C] with K = 2 or 3")
    for d in dims:
        if not 1 <= d <= ndim - 2:
            raise ValueError("dimension must be a sequence dimension 1..K")


def switch(x: np.ndarray, from_dim: int, to_dim: int, n_chunks: int) -> np.ndarray:
    """Permute + pack of one GPU's shard.  Returns the packed chunks as an array of
    shape [n_chunks, B, (other dims, D_to/n_chunks in place of D_to), D_from, C]
    (same dtype as ``x``); for K = 2 that is [n_chunks, B, D_to/n_chunks, D_from, C]."""
    _check_seq_dim(x.ndim, from_dim, to_dim)
    if n_chunks < 1:
        raise ValueError("n_chunks must be positive")
    xb = _bits(x)
    if from_dim == to_dim:
        return xb.copy().view(x.dtype)
    if x.shape[to_dim] % n_chunks:
        raise ValueError("the switched-to dimension must divide evenly into n_chunks")
    # step 1 (Eq. 7): the from-dim next to C, the other dims in their order
    perm = np.moveaxis(xb, from_dim, -2)
    t = to_dim if to_dim < from_dim else to_dim - 1          # the to-dim's axis after the move
    # step 2: n_chunks contiguous slices of the to-dim, the chunk index outermost
    packed = np.stack(np.split(perm, n_chunks, axis=t))
    return np.ascontiguousarray(packed).view(x.dtype)


def split(x: np.ndarray, dim: int, n_chunks: int, rank: int) -> np.ndarray:
    """Split (s^ -> s_i): rank ``rank``'s slice of the replicated tensor x along ``dim``."""
    _check_seq_dim(x.ndim, dim)
    if n_chunks < 1 or not 0 <= rank < n_chunks or x.shape[dim] % n_chunks:
        raise ValueError("dim must divide into n_chunks and 0 <= rank < n_chunks")
    return np.ascontiguousarray(np.split(_bits(x), n_chunks, axis=dim)[rank]).view(x.dtype)


def gather(shards, dim: int) -> np.ndarray:
    """Gather (s_i -> s^): the full tensor from the N slices along ``dim``, in rank order."""
    if len(shards) < 1:
        raise ValueError("at least one shard")
    _check_seq_dim(shards[0].ndim, dim)
    if any(s.shape != shards[0].shape or s.dtype != shards[0].dtype for s in shards):
        raise ValueError("shards must share shape and dtype")
    y = np.concatenate([_bits(s) for s in shards], axis=dim)
    return np.ascontiguousarray(y).view(shards[0].dtype)


def switch_index_map(shape, from_dim: int, to_dim: int, n_chunks: int):
    """Yields (output multi-index, input multi-index) pairs of the switch, one element at a time."""
    B, D1, D2, C = shape
    dims = {1: D1, 2: D2}
    d_to, d_from = dims[to_dim], dims[from_dim]
    per = d_to // n_chunks
    for n in range(n_chunks):
        for b in range(B):
            for jj in range(per):
                for i in range(d_from):
                    for c in range(C):
                        j = n * per + jj
                        src = [b, 0, 0, c]
                        src[to_dim] = j
                        src[from_dim] = i
                        yield (n, b, jj, i, c), tuple(src)


def unswitch(packed: np.ndarray, from_dim: int, to_dim: int) -> np.ndarray:
    """Inverse of ``switch`` on one GPU: rebuild x [B, S_1, .., S_K, C] from its packed chunks."""
    nb = _bits(packed)
    ndim = packed.ndim - 1
    _check_seq_dim(ndim, from_dim, to_dim)
    t = to_dim if to_dim < from_dim else to_dim - 1
    perm = np.concatenate(list(nb), axis=t)                   # the chunks joined on the to-dim
    x = np.moveaxis(perm, -2, from_dim)
    return np.ascontiguousarray(x).view(packed.dtype)


def exchange_unpack(packed_per_rank):
    """All-to-all of the packed chunks followed by the receiver's unpack.

    ``packed_per_rank[m]`` is rank m's switch output, [N, B, D_to/N, D_from_local, C]
    (K = 3: [N, B, .., D_from_local, C]).  Rank n receives chunk n of every rank m
    and concatenates them along the from-dimension (next to C) in rank order:
        y_n[b][j'][m*D_from_local + i][c] = packed_per_rank[m][n][b][j'][i][c].
    Returns the list of per-rank results [B, D_to/N, D_from_local*N, C].
    """
    N = len(packed_per_rank)
    out = []
    for n in range(N):
        recv = [_bits(packed_per_rank[m])[n] for m in range(N)]      # each [B, per, d_loc, C]
        y = np.concatenate(recv, axis=-2)
        out.append(np.ascontiguousarray(y).view(packed_per_rank[0].dtype))
    return out
