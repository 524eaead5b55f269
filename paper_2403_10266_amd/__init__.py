"""Python binding of libdsp: one GPU's share of a Dynamic Sequence Parallelism
spatial-temporal block on MI355X.

Argument marshalling only.  Every computation runs in the HIP kernels of
``libdsp.so`` (built in-tree by ``paper_2403_10266_amd.build``); this module
turns torch tensors into device pointers, sizes and the current HIP stream,
calls the C entry point of the same name and raises ``DspError`` on a nonzero
status.  There is no fallback: if the library is missing, importing the
binding's functions raises.

Entry points (see ``include/dsp.h`` for the exact contracts):
``dsp_switch``, ``dsp_exchange_unpack``, ``dsp_split``, ``dsp_gather``,
``dsp_spatial_attn``, ``dsp_temporal_attn``, ``dsp_attn_strided``,
``dsp_attn_fwd_lse``, ``dsp_attn_bwd``, ``dsp_attn_general``, ``dsp_attn_general_bwd``, ``dsp_layernorm_bwd``, ``dsp_linear_bwd_data``, ``dsp_linear_bwd_weight``,
``dsp_layernorm``, ``dsp_linear``, ``dsp_st_block_forward``.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from pathlib import Path

_PKG = Path(__file__).resolve().parent
LIB_PATH = _PKG / "libdsp.so"

# status codes and enums of include/dsp.h
DSP_OK, DSP_ERR_NULL, DSP_ERR_DIM, DSP_ERR_SHAPE, DSP_ERR_DTYPE, DSP_ERR_ALIGN, DSP_ERR_HIP, \
    DSP_ERR_WORKSPACE, DSP_ERR_ARG = range(9)
DSP_F32, DSP_BF16 = 0, 1
DSP_EPI_NONE, DSP_EPI_GELU, DSP_EPI_RESID, DSP_EPI_F32, DSP_EPI_RELU = 0, 1, 2, 3, 4
DSP_BLOCK_NO_MLP_LN, DSP_BLOCK_ATTN_ONLY, DSP_BLOCK_POST_LN, DSP_BLOCK_RELU = 1, 2, 4, 8
DSP_GRAD_EPI_F32, DSP_GRAD_EPI_BF16, DSP_GRAD_EPI_GELU_BWD, DSP_GRAD_EPI_RELU_BWD = 0, 1, 2, 3

BLOCK_WEIGHT_FIELDS = ("wqkv_s", "bqkv_s", "wo_s", "bo_s", "wqkv_t", "bqkv_t", "wo_t", "bo_t",
                       "w1", "b1", "w2", "b2")


class DspError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


class BlockWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_WEIGHT_FIELDS]


class BlockGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_WEIGHT_FIELDS]


_lib = None

_c = ctypes
_P, _I, _I64, _F, _SZ = _c.c_void_p, _c.c_int, _c.c_int64, _c.c_float, _c.c_size_t
_SIGNATURES = {
    "dsp_status_str": (_c.c_char_p, [_I]),
    "dsp_version": (_I, []),
    "dsp_switch": (_I, [_P, _P, _c.POINTER(_I64), _I, _I, _I, _I, _I, _P]),
    "dsp_switch_variant": (_I, [_P, _P, _c.POINTER(_I64), _I, _I, _I, _I, _I, _I, _P]),
    "dsp_exchange_unpack": (_I, [_c.POINTER(_P), _c.POINTER(_P), _c.POINTER(_I64), _I, _P]),
    "dsp_split": (_I, [_P, _P, _c.POINTER(_I64), _I, _I, _I, _I, _I, _P]),
    "dsp_gather": (_I, [_c.POINTER(_P), _P, _c.POINTER(_I64), _I, _I, _I, _I, _P]),
    "dsp_spatial_attn": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _I, _I64, _I64, _F, _I, _P]),
    "dsp_temporal_attn": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _I, _I64, _I64, _F, _I, _P]),
    "dsp_attn_strided": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _I, _c.POINTER(_I64),
                              _c.POINTER(_I64), _F, _I, _P]),
    "dsp_attn_fwd_lse": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I, _I, _c.POINTER(_I64),
                              _c.POINTER(_I64), _F, _I, _P]),
    "dsp_attn_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I, _I,
                          _c.POINTER(_I64), _c.POINTER(_I64), _F, _I, _P]),
    "dsp_attn_bwd_noalloc_max_rows": (_I64, []),
    "dsp_attn_bwd_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I, _I,
                                  _c.POINTER(_I64), _c.POINTER(_I64), _F, _I, _P]),
    "dsp_layernorm": (_I, [_P, _I, _P, _I, _I64, _I, _F, _P]),
    "dsp_attn_general": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _I, _I, _I, _c.POINTER(_I64),
                              _c.POINTER(_I64), _c.POINTER(_I64), _F, _I, _P]),
    "dsp_attn_general_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _I, _I, _I,
                                  _c.POINTER(_I64), _c.POINTER(_I64), _c.POINTER(_I64), _F, _I, _P]),
    "dsp_layernorm_bwd": (_I, [_P, _I, _P, _I, _P, _P, _I64, _I, _F, _P]),
    "dsp_linear_bwd_data": (_I, [_P, _P, _P, _P, _I64, _I, _I, _I, _I, _P]),
    "dsp_linear_bwd_weight_workspace_bytes": (_SZ, [_I64, _I, _I, _I]),
    "dsp_linear_bwd_weight": (_I, [_P, _P, _P, _P, _P, _SZ, _I64, _I, _I, _I, _P]),
    "dsp_linear": (_I, [_P, _P, _P, _P, _P, _I64, _I, _I, _I, _I, _P]),
    "dsp_st_block_workspace_bytes": (_SZ, [_I64, _I64, _I64, _I, _I, _I, _I]),
    "dsp_st_block_train_saved_bytes": (_SZ, [_I64, _I64, _I64, _I, _I, _I, _I, _I]),
    "dsp_probe_mfma_workspace_bytes": (_SZ, []),
    "dsp_probe_mfma_flops": (_c.c_double, [_I]),
    "dsp_probe_mfma": (_I, [_P, _SZ, _I, _P]),
    "dsp_st_block_backward_workspace_bytes": (_SZ, [_I64, _I64, _I64, _I, _I, _I, _I]),
    "dsp_st_block_forward_train": (_I, [_P, _P, _c.POINTER(BlockWeights), _P, _SZ, _I64, _I64, _I64, _I, _I,
                                        _I, _F, _I, _I, _P]),
    "dsp_st_block_backward": (_I, [_P, _P, _c.POINTER(BlockWeights), _P, _SZ, _P, _SZ, _P,
                                   _c.POINTER(BlockGrads), _I64, _I64, _I64, _I, _I, _I, _F, _I, _I, _P]),
    "dsp_st_block_forward": (_I, [_P, _P, _c.POINTER(BlockWeights), _P, _SZ, _I64, _I64, _I64, _I,
                                  _I, _I, _F, _I, _I, _P]),
}


def lib() -> ctypes.CDLL:
    """The loaded libdsp.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(f"libdsp.so not found at {LIB_PATH}; build it with "
                               "`python -m paper_2403_10266_amd.build`")
        L = ctypes.CDLL(str(LIB_PATH))
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().dsp_status_str(int(status)).decode()


def _check_status(status: int, where: str) -> None:
    if status != DSP_OK:
        raise DspError(status, where)


# --------------------------------------------------------------------------- torch marshalling
#
# Every wrapper validates the tensors it is given (device, dtype, shape and
# strides) and raises before anything is launched: the library reads and
# writes them in place, so a tensor that does not have the layout the C entry
# point assumes is an error here, never silently copied.  New outputs and
# workspaces are allocated, and the call is enqueued, on `stream` (default:
# the current stream), so the caching allocator orders their reuse after the
# kernels that use them.

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return DSP_F32
    if t.dtype == torch.bfloat16:
        return DSP_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


@contextlib.contextmanager
def _on(stream):
    """Run the body with `stream` current; yields the stream as a ctypes handle."""
    torch = _torch()
    if stream is None:
        yield ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    else:
        with torch.cuda.stream(stream):
            yield ctypes.c_void_p(stream.cuda_stream)


def _require_device(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libdsp operates on device tensors only")


def _check(where, name, t, *, dtype=None, shape=None, numel=None, contiguous=True, like=None, strides=None):
    """Raise ValueError unless tensor `t` is on the device of `like` (if given)
    and has the given dtype, shape / element count, strides or contiguity."""
    if t is None:
        raise ValueError(f"{where}: {name} is required")
    if not t.is_cuda:
        raise ValueError(f"{where}: {name} must be a device tensor")
    if like is not None and t.device != like.device:
        raise ValueError(f"{where}: {name} is on {t.device}, the inputs on {like.device}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{where}: {name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{where}: {name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{where}: {name} must have {numel} elements, got {t.numel()}")
    if strides is not None and tuple(t.stride()) != tuple(strides):
        raise ValueError(f"{where}: {name} must have strides {tuple(strides)}, got {tuple(t.stride())}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{where}: {name} must be contiguous (the library works on it in place; "
                         "pass a contiguous tensor)")
    return t


def _float_dtype(where, t):
    torch = _torch()
    if t.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError(f"{where}: unsupported dtype {t.dtype}; use float32 or bfloat16")
    return t.dtype


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _switch_out_shape(dims, from_dim, to_dim, n_chunks):
    nd = len(dims)
    if from_dim == to_dim or not (1 <= from_dim <= nd - 2 and 1 <= to_dim <= nd - 2):
        return tuple(dims)
    others = [k for k in range(1, nd - 1) if k != from_dim]
    mid = [dims[k] // max(n_chunks, 1) if k == to_dim else dims[k] for k in others]
    return (n_chunks, dims[0], *mid, dims[from_dim], dims[-1])


def dsp_switch(x, from_dim: int, to_dim: int, n_chunks: int, out=None, variant: int = 0,
               stream=None):
    """Permute + pack of a contiguous [B, S_1, .., S_K, C] shard, K = 2 or 3 (see
    dsp.h).  Returns ``out``: a tensor of shape [n_chunks, B, (the other sequence
    dims, the to-dim cut to D_to/n_chunks), D_from, C] (or x's shape when
    from_dim == to_dim); a given ``out`` needs x's dtype and element count."""
    torch = _torch()
    w = "dsp_switch"
    _check(w, "x", x)
    dt = _float_dtype(w, x)
    if x.dim() not in (4, 5):
        raise ValueError(f"{w}: x must be [B, S_1, .., S_K, C] with K = 2 or 3")
    dims = list(x.shape)
    with _on(stream) as s:
        if out is None:
            out = torch.empty(_switch_out_shape(dims, from_dim, to_dim, n_chunks), dtype=dt, device=x.device)
        _check(w, "out", out, dtype=dt, numel=x.numel(), like=x)
        shape = (ctypes.c_int64 * x.dim())(*dims)
        _check_status(lib().dsp_switch_variant(_ptr(x), _ptr(out), shape, x.dim(), from_dim, to_dim, n_chunks,
                                               _dtype_code(x), variant, s), w)
    return out


def dsp_split(x, dim: int, n_chunks: int, rank: int, out=None, stream=None):
    """Split (primitive table, s^ -> s_i): rank ``rank``'s slice of the replicated
    contiguous tensor x [B, S_1, .., S_K, C] along sequence dimension ``dim``."""
    torch = _torch()
    w = "dsp_split"
    _check(w, "x", x)
    dt = _float_dtype(w, x)
    if x.dim() not in (4, 5):
        raise ValueError(f"{w}: x must be [B, S_1, .., S_K, C] with K = 2 or 3")
    dims = list(x.shape)
    oshape = list(dims)
    if 1 <= dim < x.dim() - 1 and n_chunks >= 1:
        oshape[dim] //= n_chunks
    with _on(stream) as s:
        if out is None:
            out = torch.empty(oshape, dtype=dt, device=x.device)
        _check(w, "out", out, dtype=dt, shape=oshape, like=x)
        shape = (ctypes.c_int64 * x.dim())(*dims)
        _check_status(lib().dsp_split(_ptr(x), _ptr(out), shape, x.dim(), dim, n_chunks, rank, _dtype_code(x), s), w)
    return out


def dsp_gather(shards, dim: int, out=None, stream=None):
    """Gather (primitive table, s_i -> s^): the concatenation along sequence
    dimension ``dim`` of N equal contiguous shards [B, S_1, .., S_K, C], in rank
    order; the receiving side of the all-gather, every rank's shard on one GPU."""
    torch = _torch()
    w = "dsp_gather"
    shards = list(shards)
    if not shards:
        raise ValueError(f"{w}: at least one shard")
    x0 = shards[0]
    _check(w, "shards[0]", x0)
    dt = _float_dtype(w, x0)
    for i, t in enumerate(shards):
        _check(w, f"shards[{i}]", t, dtype=dt, shape=x0.shape, like=x0)
    if x0.dim() not in (4, 5):
        raise ValueError(f"{w}: shards must be [B, S_1, .., S_K, C] with K = 2 or 3")
    dims = list(x0.shape)
    oshape = list(dims)
    if 1 <= dim < x0.dim() - 1:
        oshape[dim] *= len(shards)
    with _on(stream) as s:
        if out is None:
            out = torch.empty(oshape, dtype=dt, device=x0.device)
        _check(w, "out", out, dtype=dt, shape=oshape, like=x0)
        ptrs = (ctypes.c_void_p * len(shards))(*[t.data_ptr() for t in shards])
        shape = (ctypes.c_int64 * x0.dim())(*dims)
        _check_status(lib().dsp_gather(ptrs, _ptr(out), shape, x0.dim(), dim, len(shards), _dtype_code(x0), s), w)
    return out


def _row_views(w, q, k, v, C, ld_in):
    """q, k, v: 4-D views [B, X, L, >= C] whose (B, X, L) rows follow each other
    at stride ld_in (a dense tensor, or a column slice of a packed one)."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(w, name, t, contiguous=False, like=q, dtype=q.dtype)
        if t.dim() != 4 or tuple(t.shape[:3]) != tuple(q.shape[:3]) or t.shape[3] < C:
            raise ValueError(f"{w}: {name} must be a 4-D view [B, X, L, >= {C}] like q")
        B, X, L = t.shape[:3]
        want = (X * L * ld_in, L * ld_in, ld_in, 1)
        if any(n > 1 and st != ws for n, st, ws in zip(t.shape, t.stride(), want)):
            raise ValueError(f"{w}: {name} must have row stride {ld_in} with rows packed densely "
                             f"(strides {want}), got {tuple(t.stride())}")
    _float_dtype(w, q)


def _attn(name, q, k, v, B, X, L, H, out, ld_in, ld_out, scale, stream, C):
    torch = _torch()
    if C % H:
        raise ValueError(f"{name}: C = {C} is not a multiple of H = {H}")
    _row_views(name, q, k, v, C, ld_in)
    with _on(stream) as s:
        if out is None:
            if ld_out is not None and ld_out != C:
                raise ValueError(f"{name}: pass `out` for an output row stride other than C")
            out = torch.empty((B, X, L, C), dtype=q.dtype, device=q.device)
        if ld_out is None:
            ld_out = out.stride(2)
        _row_views(name, out, out, out, C, ld_out)
        _check(name, "out", out, dtype=q.dtype, like=q, contiguous=False)
        if tuple(out.shape[:3]) != (B, X, L):
            raise ValueError(f"{name}: out must be [B, X, L, >= C] like q")
        fn = getattr(lib(), name)
        _check_status(fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, X, L, H, C // H, ld_in, ld_out, float(scale),
                         _dtype_code(q), s), name)
    return out


def dsp_exchange_unpack(packed, out=None, stream=None):
    """Exchange + unpack of N ranks' packed switch outputs on one GPU (see
    dsp.h).  ``packed``: N contiguous tensors of shape [N, B, P, F, C] (same
    dtype).  Returns N tensors of shape [B, P, N*F, C]: rank n's result."""
    torch = _torch()
    w = "dsp_exchange_unpack"
    packed = list(packed)
    N = len(packed)
    if N == 0:
        raise ValueError(f"{w}: no ranks")
    p0 = packed[0]
    _check(w, "packed[0]", p0)
    dt = _float_dtype(w, p0)
    shape = tuple(p0.shape)
    if len(shape) != 5 or shape[0] != N:
        raise ValueError(f"{w}: packed[0] has shape {shape}, want [N={N}, B, P, F, C]")
    for i, t in enumerate(packed):
        _check(w, f"packed[{i}]", t, dtype=dt, shape=shape, like=p0)
    _, B, P, F, C = shape
    with _on(stream) as s:
        if out is None:
            out = [torch.empty((B, P, N * F, C), dtype=dt, device=p0.device) for _ in range(N)]
        out = list(out)
        if len(out) != N:
            raise ValueError(f"{w}: out must hold N = {N} tensors")
        for i, o in enumerate(out):
            _check(w, f"out[{i}]", o, dtype=dt, shape=(B, P, N * F, C), like=p0)
        src = (ctypes.c_void_p * N)(*[t.data_ptr() for t in packed])
        dst = (ctypes.c_void_p * N)(*[o.data_ptr() for o in out])
        shp = (ctypes.c_int64 * 5)(N, B, P, F, C)
        _check_status(lib().dsp_exchange_unpack(src, dst, shp, _dtype_code(p0), s), w)
    return out


def dsp_spatial_attn(q, k, v, H: int, out=None, scale: float = 0.0, C: int | None = None,
                     ld_in: int | None = None, ld_out: int | None = None, stream=None):
    """Attention over S within each frame.  q, k, v: (B, T, S, ld_in) views whose
    first C = H*D columns hold the heads (pass C explicitly for packed QKV views)."""
    B, T, S = q.shape[0], q.shape[1], q.shape[2]
    C = C if C is not None else q.shape[3]
    ld_in = ld_in if ld_in is not None else q.stride(2)
    return _attn("dsp_spatial_attn", q, k, v, B, T, S, H, out, ld_in, ld_out, scale, stream, C)


def dsp_temporal_attn(q, k, v, H: int, out=None, scale: float = 0.0, C: int | None = None,
                      ld_in: int | None = None, ld_out: int | None = None, stream=None):
    """Attention over T at each spatial location.  q, k, v: (B, S, T, ld_in) views."""
    B, S, T = q.shape[0], q.shape[1], q.shape[2]
    C = C if C is not None else q.shape[3]
    ld_in = ld_in if ld_in is not None else q.stride(2)
    return _attn("dsp_temporal_attn", q, k, v, B, S, T, H, out, ld_in, ld_out, scale, stream, C)


def _qkv_views(where, q, k, v, H):
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(where, name, t, contiguous=False, like=q, dtype=q.dtype)
    _float_dtype(where, q)
    if q.dim() != 4 or q.shape != k.shape or q.shape != v.shape:
        raise ValueError(f"{where}: q, k, v must be 4-D views of one shape [B, X, L, C]")
    if q.stride() != k.stride() or q.stride() != v.stride() or q.stride(3) != 1:
        raise ValueError(f"{where}: q, k, v must share strides, with a unit last stride")
    B, X, L, C = q.shape
    if C % H:
        raise ValueError(f"{where}: C must be a multiple of H")
    return B, X, L, C


def _like_view(where, t, like, name):
    _check(where, name, t, contiguous=False, like=like, dtype=like.dtype)
    if t.shape != like.shape or t.stride(3) != 1:
        raise ValueError(f"{where}: {name} must be a view of shape {tuple(like.shape)} with a unit last stride")


def dsp_attn_strided(q, k, v, H: int, out=None, scale: float = 0.0, stream=None):
    """Attention over dim 2 of the 4-D views q, k, v [B, X, L, >=H*D] (any
    strides, last one 1, the same for q, k and v), per (b, x, head): e.g.
    temporal attention on a (B, T, S, C) tensor x is ``q = x.permute(0, 2, 1, 3)``.
    The output is a new contiguous [B, X, L, C] tensor, or ``out`` (any 4-D
    view with last stride 1)."""
    torch = _torch()
    w = "dsp_attn_strided"
    B, X, L, C = _qkv_views(w, q, k, v, H)
    with _on(stream) as s:
        if out is None:
            out = torch.empty((B, X, L, C), dtype=q.dtype, device=q.device)
        _like_view(w, out, q, "out")
        ins = (ctypes.c_int64 * 3)(*q.stride()[:3])
        outs = (ctypes.c_int64 * 3)(*out.stride()[:3])
        _check_status(lib().dsp_attn_strided(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, X, L, H, C // H, ins, outs,
                                             float(scale), _dtype_code(q), s), w)
    return out


def dsp_attn_fwd_lse(q, k, v, H: int, out=None, lse=None, scale: float = 0.0, stream=None):
    """dsp_attn_strided that also returns the row log-sum-exp: (out, lse) with
    lse a float32 tensor [B, X, H, L]."""
    torch = _torch()
    w = "dsp_attn_fwd_lse"
    B, X, L, C = _qkv_views(w, q, k, v, H)
    with _on(stream) as s:
        if out is None:
            out = torch.empty((B, X, L, C), dtype=q.dtype, device=q.device)
        _like_view(w, out, q, "out")
        if lse is None:
            lse = torch.empty((B, X, H, L), dtype=torch.float32, device=q.device)
        _check(w, "lse", lse, dtype=torch.float32, numel=B * X * H * L, like=q)
        ins = (ctypes.c_int64 * 3)(*q.stride()[:3])
        outs = (ctypes.c_int64 * 3)(*out.stride()[:3])
        _check_status(lib().dsp_attn_fwd_lse(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, X, L, H, C // H,
                                             ins, outs, float(scale), _dtype_code(q), s), w)
    return out, lse


def dsp_attn_bwd(q, k, v, o, dout, lse, H: int, dq=None, dk=None, dv=None, delta=None,
                 scale: float = 0.0, stream=None):
    """Gradients (dq, dk, dv) of attention over dim 2 of the 4-D views q, k, v
    (as dsp_attn_strided), given its output o, the row log-sum-exp ``lse``
    from dsp_attn_fwd_lse and the output gradient ``dout`` (o and dout share
    one layout).  New contiguous gradients unless dq/dk/dv (views with the
    strides of q) are given.  ``delta``: optional float32 workspace of
    B*X*H*L elements (holds rowsum(dout * o) on return)."""
    torch = _torch()
    w = "dsp_attn_bwd"
    B, X, L, C = _qkv_views(w, q, k, v, H)
    _like_view(w, o, q, "o")
    _like_view(w, dout, q, "dout")
    if dout.stride() != o.stride():
        raise ValueError(f"{w}: dout must have the strides of o")
    _check(w, "lse", lse, dtype=torch.float32, numel=B * X * H * L, like=q)
    with _on(stream) as s:
        if dq is None or dk is None or dv is None:
            if not q.is_contiguous():
                raise ValueError(f"{w}: for a non-contiguous q pass dq, dk, dv views with its strides")
            dq, dk, dv = (torch.empty_like(q) if g is None else g for g in (dq, dk, dv))
        for g, name in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
            _like_view(w, g, q, name)
            if tuple(g.stride()) != tuple(q.stride()):
                raise ValueError(f"{w}: {name} must have the strides of q, k, v")
        if delta is None:
            delta = torch.empty(B * X * H * L, dtype=torch.float32, device=q.device)
        _check(w, "delta", delta, dtype=torch.float32, numel=B * X * H * L, like=q)
        qs = (ctypes.c_int64 * 3)(*q.stride()[:3])
        os_ = (ctypes.c_int64 * 3)(*o.stride()[:3])
        _check_status(lib().dsp_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq),
                                         _ptr(dk), _ptr(dv), _ptr(delta), B, X, L, H, C // H, qs, os_,
                                         float(scale), _dtype_code(q), s), w)
    return dq, dk, dv


def attn_bwd_noalloc_max_rows() -> int:
    """Largest B*X*H*L that dsp_attn_bwd_noalloc accepts."""
    return int(lib().dsp_attn_bwd_noalloc_max_rows())


def dsp_attn_bwd_noalloc(q, k, v, o, dout, lse, H: int, dq, dk, dv, scale: float = 0.0, stream=None):
    """dsp_attn_bwd for callers that cannot allocate: no Delta workspace (the
    library keeps Delta in a static per-device array; calls overlapping on one
    GPU race) and caller-given dq, dk, dv (views with the strides of q)."""
    torch = _torch()
    w = "dsp_attn_bwd_noalloc"
    B, X, L, C = _qkv_views(w, q, k, v, H)
    _like_view(w, o, q, "o")
    _like_view(w, dout, q, "dout")
    if dout.stride() != o.stride():
        raise ValueError(f"{w}: dout must have the strides of o")
    _check(w, "lse", lse, dtype=torch.float32, numel=B * X * H * L, like=q)
    for g, name in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
        _like_view(w, g, q, name)
        if tuple(g.stride()) != tuple(q.stride()):
            raise ValueError(f"{w}: {name} must have the strides of q, k, v")
    with _on(stream) as s:
        qs = (ctypes.c_int64 * 3)(*q.stride()[:3])
        os_ = (ctypes.c_int64 * 3)(*o.stride()[:3])
        _check_status(lib().dsp_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse),
                                                 _ptr(dq), _ptr(dk), _ptr(dv), B, X, L, H, C // H, qs, os_,
                                                 float(scale), _dtype_code(q), s), w)
    return dq, dk, dv


def dsp_layernorm(x, eps: float = 1e-6, out=None, out_dtype=None, stream=None):
    """y = (x - mean) / sqrt(var + eps) over the last dimension of the
    contiguous x; y in out_dtype (default x's), or into ``out``."""
    torch = _torch()
    w = "dsp_layernorm"
    _check(w, "x", x)
    _float_dtype(w, x)
    C = x.shape[-1]
    rows = x.numel() // C if C else 0
    with _on(stream) as s:
        if out is None:
            out = torch.empty(x.shape, dtype=out_dtype or x.dtype, device=x.device)
        _check(w, "out", out, shape=x.shape, like=x)
        _float_dtype(w, out)
        _check_status(lib().dsp_layernorm(_ptr(x), _dtype_code(x), _ptr(out), _dtype_code(out), rows, C,
                                          float(eps), s), w)
    return out


def _st3(t):
    return (ctypes.c_int64 * 3)(*t.stride()[:3])


def _general_views(w, q, k, v, H, Hkv):
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(w, name, t, contiguous=False, like=q, dtype=q.dtype)
    _float_dtype(w, q)
    if q.dim() != 4 or k.dim() != 4 or k.shape != v.shape or k.stride() != v.stride() or q.stride(3) != 1 \
            or k.stride(3) != 1:
        raise ValueError(f"{w}: q [B, X, Lq, C] and k, v [B, X, Lk, Ckv] views of one layout")
    B, X, Lq, C = q.shape
    if H < 1 or Hkv < 1 or C % H or tuple(k.shape[:2]) != (B, X):
        raise ValueError(f"{w}: shapes do not match")
    D = C // H
    if k.shape[3] != Hkv * D:
        raise ValueError(f"{w}: k and v must hold Hkv heads of the query head width")
    return B, X, Lq, k.shape[2], C, D


def dsp_attn_general(q, k, v, H: int, Hkv: int, out=None, lse=None, with_lse: bool = False,
                     scale: float = 0.0, stream=None):
    """Grouped-query / multi-query / cross-attention over dim 2 of 4-D views:
    q [B, X, Lq, H*D], k and v [B, X, Lk, Hkv*D] (same strides; a 0 stride
    broadcasts).  Returns out [B, X, Lq, H*D] (and lse [B, X, H, Lq] fp32 when
    with_lse or lse is given)."""
    torch = _torch()
    w = "dsp_attn_general"
    B, X, Lq, Lk, C, D = _general_views(w, q, k, v, H, Hkv)
    with _on(stream) as s:
        if out is None:
            out = torch.empty((B, X, Lq, C), dtype=q.dtype, device=q.device)
        _like_view(w, out, q, "out")
        if with_lse and lse is None:
            lse = torch.empty((B, X, H, Lq), dtype=torch.float32, device=q.device)
        if lse is not None:
            _check(w, "lse", lse, dtype=torch.float32, numel=B * X * H * Lq, like=q)
        _check_status(lib().dsp_attn_general(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, X, Lq, Lk, H,
                                             Hkv, D, _st3(q), _st3(k), _st3(out), float(scale), _dtype_code(q), s), w)
    return (out, lse) if lse is not None else out


def dsp_attn_general_bwd(q, k, v, o, dout, lse, H: int, Hkv: int, dq=None, dk=None, dv=None, delta=None,
                         scale: float = 0.0, stream=None):
    """Gradients of dsp_attn_general: (dq like q, dk and dv like k and v)."""
    torch = _torch()
    w = "dsp_attn_general_bwd"
    B, X, Lq, Lk, C, D = _general_views(w, q, k, v, H, Hkv)
    _like_view(w, o, q, "o")
    _like_view(w, dout, q, "dout")
    if dout.stride() != o.stride():
        raise ValueError(f"{w}: dout must have the strides of o")
    _check(w, "lse", lse, dtype=torch.float32, numel=B * X * H * Lq, like=q)
    with _on(stream) as s:
        dq = torch.empty_like(q) if dq is None else dq
        dk = torch.empty_like(k) if dk is None else dk
        dv = torch.empty_like(v) if dv is None else dv
        _check(w, "dq", dq, dtype=q.dtype, shape=q.shape, strides=q.stride(), contiguous=False, like=q)
        _check(w, "dk", dk, dtype=q.dtype, shape=k.shape, strides=k.stride(), contiguous=False, like=q)
        _check(w, "dv", dv, dtype=q.dtype, shape=k.shape, strides=k.stride(), contiguous=False, like=q)
        if delta is None:
            delta = torch.empty(B * X * H * Lq, dtype=torch.float32, device=q.device)
        _check(w, "delta", delta, dtype=torch.float32, numel=B * X * H * Lq, like=q)
        _check_status(lib().dsp_attn_general_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse),
                                                 _ptr(dq), _ptr(dk), _ptr(dv), _ptr(delta), B, X, Lq, Lk, H, Hkv, D,
                                                 _st3(q), _st3(k), _st3(o), float(scale), _dtype_code(q), s), w)
    return dq, dk, dv


def dsp_layernorm_bwd(x, dy, eps: float = 1e-6, dres=None, out=None, stream=None):
    """dx (fp32) = dres + the LayerNorm backward of dy at x (contiguous rows of C)."""
    torch = _torch()
    w = "dsp_layernorm_bwd"
    _check(w, "x", x)
    _float_dtype(w, x)
    _check(w, "dy", dy, shape=x.shape, like=x)
    _float_dtype(w, dy)
    if dres is not None:
        _check(w, "dres", dres, dtype=torch.float32, shape=x.shape, like=x)
    C = x.shape[-1]
    rows = x.numel() // C if C else 0
    with _on(stream) as s:
        if out is None:
            out = torch.empty(x.shape, dtype=torch.float32, device=x.device)
        _check(w, "out", out, dtype=torch.float32, shape=x.shape, like=x)
        _check_status(lib().dsp_layernorm_bwd(_ptr(x), _dtype_code(x), _ptr(dy), _dtype_code(dy), _ptr(dres),
                                              _ptr(out), rows, C, float(eps), s), w)
    return out


def dsp_linear(a, w, bias=None, residual=None, epilogue: int = DSP_EPI_NONE, out=None,
               stream=None):
    """out = epilogue(a @ w.T + bias); a [..., K] and w [N, K] contiguous, one dtype."""
    torch = _torch()
    where = "dsp_linear"
    _check(where, "a", a)
    dt = _float_dtype(where, a)
    K = a.shape[-1]
    M = a.numel() // K if K else 0
    _check(where, "w", w, dtype=dt, like=a)
    if w.dim() != 2 or w.shape[1] != K:
        raise ValueError(f"{where}: w must be [N, K = {K}]")
    N = w.shape[0]
    if bias is not None:
        _check(where, "bias", bias, dtype=dt, numel=N, like=a)
    oshape = (*a.shape[:-1], N)
    if residual is not None:
        _check(where, "residual", residual, dtype=torch.float32, numel=M * N, like=a)
    odt = torch.float32 if epilogue in (DSP_EPI_RESID, DSP_EPI_F32) else dt
    with _on(stream) as s:
        if out is None:
            out = torch.empty(oshape, dtype=odt, device=a.device)
        _check(where, "out", out, dtype=odt, numel=M * N, like=a)
        _check_status(lib().dsp_linear(_ptr(a), _ptr(w), _ptr(bias), _ptr(residual), _ptr(out), M, N, K,
                                       epilogue, _dtype_code(a), s), where)
    return out


def dsp_linear_bwd_data(dy, w, u=None, epilogue: int = DSP_GRAD_EPI_F32, out=None, stream=None):
    """dx = epilogue(dy @ w) for y = x @ w.T (w stored [N, K]); u: the saved
    pre-activation [..., K] for the GELU/ReLU backward epilogues."""
    torch = _torch()
    where = "dsp_linear_bwd_data"
    _check(where, "dy", dy)
    dt = _float_dtype(where, dy)
    _check(where, "w", w, dtype=dt, like=dy)
    if w.dim() != 2 or w.shape[0] != dy.shape[-1]:
        raise ValueError(f"{where}: w must be [N = {dy.shape[-1]}, K]")
    N, K = w.shape
    M = dy.numel() // N if N else 0
    if u is not None:
        _check(where, "u", u, dtype=dt, numel=M * K, like=dy)
    odt = torch.float32 if epilogue == DSP_GRAD_EPI_F32 else dt
    with _on(stream) as s:
        if out is None:
            out = torch.empty((*dy.shape[:-1], K), dtype=odt, device=dy.device)
        _check(where, "out", out, dtype=odt, numel=M * K, like=dy)
        _check_status(lib().dsp_linear_bwd_data(_ptr(dy), _ptr(w), _ptr(u), _ptr(out), M, N, K, epilogue,
                                                _dtype_code(dy), s), where)
    return out


def dsp_linear_bwd_weight(dy, x, with_bias: bool = False, dw=None, db=None, workspace=None, stream=None):
    """(dw [N, K] fp32, db [N] fp32 or None) for y = x @ w.T + b: dw = dy^T x."""
    torch = _torch()
    where = "dsp_linear_bwd_weight"
    _check(where, "dy", dy)
    dt = _float_dtype(where, dy)
    _check(where, "x", x, dtype=dt, like=dy)
    N, K = dy.shape[-1], x.shape[-1]
    M = dy.numel() // N if N else 0
    if K == 0 or x.numel() != M * K:
        raise ValueError(f"{where}: x must hold the same {M} rows as dy")
    with _on(stream) as s:
        if dw is None:
            dw = torch.empty((N, K), dtype=torch.float32, device=dy.device)
        _check(where, "dw", dw, dtype=torch.float32, numel=N * K, like=dy)
        if with_bias and db is None:
            db = torch.empty(N, dtype=torch.float32, device=dy.device)
        if db is not None:
            _check(where, "db", db, dtype=torch.float32, numel=N, like=dy)
        need = int(lib().dsp_linear_bwd_weight_workspace_bytes(M, N, K, _dtype_code(dy)))
        if workspace is None and need:
            workspace = torch.empty(need, dtype=torch.uint8, device=dy.device)
        if workspace is not None:
            _check(where, "workspace", workspace, like=dy)
        ws_bytes = _nbytes(workspace) if workspace is not None else 0
        _check_status(lib().dsp_linear_bwd_weight(_ptr(dy), _ptr(x), _ptr(dw), _ptr(db), _ptr(workspace), ws_bytes,
                                                  M, N, K, _dtype_code(dy), s), where)
    return dw, db


def block_workspace_bytes(B, T, S, C, H, F, dtype_code) -> int:
    return int(lib().dsp_st_block_workspace_bytes(B, T, S, C, H, F, dtype_code))


def _block_args(where, x, weights, H, flags, dtype, need_mlp=True):
    """Validate x (B, T, S, C) fp32 and the weights; returns (B, T, S, C, F, code, wt)."""
    torch = _torch()
    _check(where, "x", x, dtype=torch.float32)
    if x.dim() != 4:
        raise ValueError(f"{where}: x must be (B, T, S, C)")
    B, T, S, C = x.shape
    w0 = weights.get("wqkv_s")
    if w0 is None:
        raise ValueError(f"{where}: wqkv_s is required")
    wdt = dtype or w0.dtype
    if wdt not in (torch.float32, torch.bfloat16):
        raise ValueError(f"{where}: unsupported weight dtype {wdt}")
    w1 = weights.get("w1")
    mlp = need_mlp and not (flags & DSP_BLOCK_ATTN_ONLY)
    if mlp and w1 is None:
        raise ValueError(f"{where}: w1 and w2 are required unless DSP_BLOCK_ATTN_ONLY")
    F = w1.shape[0] if w1 is not None else 0
    shapes = {"wqkv_s": (3 * C, C), "bqkv_s": (3 * C,), "wo_s": (C, C), "bo_s": (C,),
              "wqkv_t": (3 * C, C), "bqkv_t": (3 * C,), "wo_t": (C, C), "bo_t": (C,),
              "w1": (F, C), "b1": (F,), "w2": (C, F), "b2": (C,)}
    required = {"wqkv_s", "wo_s", "wqkv_t", "wo_t"} | ({"w1", "w2"} if mlp else set())
    for n in BLOCK_WEIGHT_FIELDS:
        t = weights.get(n)
        if t is None:
            if n in required:
                raise ValueError(f"{where}: {n} is required")
            continue
        _check(where, n, t, dtype=wdt, shape=shapes[n], like=x)
    code = DSP_BF16 if wdt == torch.bfloat16 else DSP_F32
    wt = BlockWeights(**{n: (weights[n].data_ptr() if weights.get(n) is not None else None)
                         for n in BLOCK_WEIGHT_FIELDS})
    return B, T, S, C, F, code, wt


def dsp_st_block_forward(x, weights: dict, H: int, eps: float = 1e-6, flags: int = 0,
                         out=None, workspace=None, dtype=None, stream=None):
    """One spatial-temporal block on x (B, T, S, C) fp32; returns (B, S, T, C) fp32.
    ``weights`` maps the dsp_block_weights_t field names to device tensors (or None)."""
    torch = _torch()
    where = "dsp_st_block_forward"
    B, T, S, C, F, code, wt = _block_args(where, x, weights, H, flags, dtype)
    with _on(stream) as s:
        if out is None:
            out = torch.empty((B, S, T, C), dtype=torch.float32, device=x.device)
        _check(where, "out", out, dtype=torch.float32, shape=(B, S, T, C), like=x)
        need = block_workspace_bytes(B, T, S, C, H, F, code)
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
        _check(where, "workspace", workspace, like=x)
        _check_status(lib().dsp_st_block_forward(_ptr(x), _ptr(out), ctypes.byref(wt), _ptr(workspace),
                                                 _nbytes(workspace), B, T, S, C, H, F, float(eps), flags, code, s),
                      where)
    return out


def dsp_st_block_forward_train(x, weights: dict, H: int, eps: float = 1e-6, flags: int = 0, out=None,
                               saved=None, dtype=None, stream=None):
    """dsp_st_block_forward that also keeps the activations the backward needs:
    returns (y (B, S, T, C) fp32, saved: a uint8 device tensor)."""
    torch = _torch()
    where = "dsp_st_block_forward_train"
    B, T, S, C, F, code, wt = _block_args(where, x, weights, H, flags, dtype)
    with _on(stream) as s:
        if out is None:
            out = torch.empty((B, S, T, C), dtype=torch.float32, device=x.device)
        _check(where, "out", out, dtype=torch.float32, shape=(B, S, T, C), like=x)
        need = int(lib().dsp_st_block_train_saved_bytes(B, T, S, C, H, F, flags, code))
        if saved is None:
            saved = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
        _check(where, "saved", saved, like=x)
        _check_status(lib().dsp_st_block_forward_train(_ptr(x), _ptr(out), ctypes.byref(wt), _ptr(saved),
                                                       _nbytes(saved), B, T, S, C, H, F, float(eps), flags, code, s),
                      where)
    return out, saved


def dsp_st_block_backward(x, dy, weights: dict, saved, H: int, eps: float = 1e-6, flags: int = 0, dx=None,
                          grads=None, with_bias: bool = False, workspace=None, dtype=None, stream=None):
    """Backward of the block: returns (dx (B, T, S, C) fp32, grads: dict of fp32
    tensors shaped like the weights, plus the biases when with_bias)."""
    torch = _torch()
    where = "dsp_st_block_backward"
    B, T, S, C, F, code, wt = _block_args(where, x, weights, H, flags, dtype)
    _check(where, "dy", dy, dtype=torch.float32, shape=(B, S, T, C), like=x)
    _check(where, "saved", saved, like=x)
    shapes = {"wqkv_s": (3 * C, C), "wo_s": (C, C), "wqkv_t": (3 * C, C), "wo_t": (C, C), "w1": (F, C),
              "w2": (C, F), "bqkv_s": (3 * C,), "bo_s": (C,), "bqkv_t": (3 * C,), "bo_t": (C,), "b1": (F,),
              "b2": (C,)}
    with _on(stream) as s:
        if dx is None:
            dx = torch.empty((B, T, S, C), dtype=torch.float32, device=x.device)
        _check(where, "dx", dx, dtype=torch.float32, shape=(B, T, S, C), like=x)
        if grads is None:
            names = [n for n in BLOCK_WEIGHT_FIELDS if n.startswith("w") or with_bias]
            grads = {n: torch.empty(shapes[n], dtype=torch.float32, device=x.device) for n in names}
        for n, g in grads.items():
            if n not in shapes:
                raise ValueError(f"{where}: unknown gradient {n}")
            if g is not None:
                _check(where, f"grads[{n}]", g, dtype=torch.float32, shape=shapes[n], like=x)
        need = int(lib().dsp_st_block_backward_workspace_bytes(B, T, S, C, H, F, code))
        if workspace is None:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
        _check(where, "workspace", workspace, like=x)
        gt = BlockGrads(**{n: (grads[n].data_ptr() if grads.get(n) is not None else None)
                           for n in BLOCK_WEIGHT_FIELDS})
        _check_status(lib().dsp_st_block_backward(_ptr(x), _ptr(dy), ctypes.byref(wt), _ptr(saved), _nbytes(saved),
                                                  _ptr(workspace), _nbytes(workspace), _ptr(dx), ctypes.byref(gt),
                                                  B, T, S, C, H, F, float(eps), flags, code, s), where)
    return dx, grads


def probe_mfma_workspace_bytes() -> int:
    return int(lib().dsp_probe_mfma_workspace_bytes())


def probe_mfma_flops(iters: int) -> float:
    """Flops one dsp_probe_mfma launch of `iters` iterations issues."""
    return float(lib().dsp_probe_mfma_flops(iters))


def dsp_probe_mfma(iters: int, workspace, stream=None):
    """Launch the sustained-MFMA-rate probe (a measurement aid): time it with
    events on `stream` and divide probe_mfma_flops(iters) by the time."""
    _check("dsp_probe_mfma", "workspace", workspace)
    with _on(stream) as s:
        _check_status(lib().dsp_probe_mfma(_ptr(workspace), _nbytes(workspace), iters, s), "dsp_probe_mfma")


__all__ = ["lib", "status_str", "DspError", "BlockWeights", "dsp_switch", "dsp_spatial_attn",
           "dsp_temporal_attn", "dsp_layernorm", "dsp_linear", "dsp_st_block_forward",
           "dsp_st_block_forward_train", "dsp_st_block_backward", "block_workspace_bytes", "LIB_PATH"]
