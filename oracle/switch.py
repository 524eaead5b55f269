"""Oracle for the DSP Switch primitive on one GPU (test infrastructure only).

The paper's Switch (primitive table, row s_i -> s_j; Eq. 10) takes a tensor
sharded on sequence dimension i (local length S_i/N) to one sharded on
dimension j (local length S_j/N) with one all-to-all.  One GPU's share of that
operation, before the exchange, is:

1. the permute that makes dimension j (the dimension about to be sharded) the
   outer sequence dimension and dimension i (the one about to become whole)
   the inner one, next to C -- this is the Reshape of Eq. (7) that lets the
   next stage run on contiguous sequences along i;
2. the pack of that permuted tensor into ``n_chunks`` contiguous chunks, chunk
   n holding the n-th slice of dimension j, destined for rank n.

For a 4-D tensor [B, D1, D2, C] with from_dim=1, to_dim=2 (for example
(B,T,S,C), T sharded, switching to S) the packed output is

    y[n][b][j'][i][c] = x[b][i][n*D2/N + j'][c],

chunk n of shape [B, D2/N, D1, C].  With from_dim=2, to_dim=1 no transpose is
needed: y[n][b][i'][j][c] = x[b][n*D1/N + i'][j][c].  from_dim == to_dim is
the table's no-op row and returns a copy.

Readings where the paper is silent: the batch index sits inside each chunk;
D_to must be divisible by n_chunks (the paper assumes S_j/N is an integer);
only K=2 sequence dimensions are built.

Everything is done on unsigned-integer views of the data, so the result is a
pure bit copy.  Pinned by: a hand-worked fixture, explicit index loops, the
round trip, the B=1 transpose identity and the N-rank exchange simulation.
"""
from __future__ import annotations

import numpy as np


def _bits(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x)
    return x.view({1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[x.itemsize])


def switch(x: np.ndarray, from_dim: int, to_dim: int, n_chunks: int) -> np.ndarray:
    """Permute + pack of one GPU's shard.  Returns the packed chunks as an array of
    shape [n_chunks, B, D_to/n_chunks, D_from, C] (same dtype as ``x``)."""
    if x.ndim != 4:
        raise ValueError("only [B, D1, D2, C] tensors (two sequence dimensions) are defined")
    if from_dim not in (1, 2) or to_dim not in (1, 2):
        raise ValueError("from_dim and to_dim must be sequence dimensions 1 or 2")
    if n_chunks < 1:
        raise ValueError("n_chunks must be positive")
    xb = _bits(x)
    if from_dim == to_dim:
        return xb.copy().view(x.dtype)
    B, C = x.shape[0], x.shape[3]
    d_to, d_from = x.shape[to_dim], x.shape[from_dim]
    if d_to % n_chunks:
        raise ValueError("the switched-to dimension must divide evenly into n_chunks")
    # step 1: bring the to-dim outermost, the from-dim innermost before C
    perm = xb.transpose(0, to_dim, from_dim, 3)              # [B, D_to, D_from, C]
    # step 2: split the to-dim into n_chunks slices and make the chunk index outermost
    per = d_to // n_chunks
    packed = perm.reshape(B, n_chunks, per, d_from, C).transpose(1, 0, 2, 3, 4)
    return np.ascontiguousarray(packed).view(x.dtype)


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
    """Inverse of ``switch`` on one GPU: rebuild x [B, D1, D2, C] from its packed chunks."""
    nb = _bits(packed)
    n, B, per, d_from, C = packed.shape
    perm = nb.transpose(1, 0, 2, 3, 4).reshape(B, n * per, d_from, C)   # [B, D_to, D_from, C]
    if from_dim == 1 and to_dim == 2:
        x = perm.transpose(0, 2, 1, 3)
    else:
        x = perm
    return np.ascontiguousarray(x).view(packed.dtype)


def exchange_unpack(packed_per_rank):
    """All-to-all of the packed chunks followed by the receiver's unpack.

    ``packed_per_rank[m]`` is rank m's switch output, [N, B, D_to/N, D_from_local, C].
    Rank n receives chunk n of every rank m and concatenates them along the
    from-dimension in rank order:
        y_n[b][j'][m*D_from_local + i][c] = packed_per_rank[m][n][b][j'][i][c].
    Returns the list of per-rank results [B, D_to/N, D_from_local*N, C].
    """
    N = len(packed_per_rank)
    out = []
    for n in range(N):
        recv = [_bits(packed_per_rank[m])[n] for m in range(N)]      # each [B, per, d_loc, C]
        y = np.concatenate(recv, axis=2)
        out.append(np.ascontiguousarray(y).view(packed_per_rank[0].dtype))
    return out
