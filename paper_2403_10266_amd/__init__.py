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


def _check(status: int, where: str) -> None:
    if status != DSP_OK:
        raise DspError(status, where)


# --------------------------------------------------------------------------- torch marshalling

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


def _stream(stream=None):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _require_device(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libdsp operates on device tensors only")


def dsp_switch(x, from_dim: int, to_dim: int, n_chunks: int, out=None, variant: int = 0,
               stream=None):
    """Permute + pack of a [B, S_1, .., S_K, C] shard, K = 2 or 3 (see dsp.h).
    Returns ``out`` as a tensor of shape [n_chunks, B, (the other sequence dims,
    the to-dim cut to D_to/n_chunks), D_from, C] (or x's shape when
    from_dim == to_dim)."""
    torch = _torch()
    _require_device(x)
    if x.dim() not in (4, 5):
        raise ValueError("x must be [B, S_1, .., S_K, C] with K = 2 or 3")
    x = x.contiguous()
    nd = x.dim()
    dims = list(x.shape)
    if from_dim == to_dim or not (1 <= from_dim <= nd - 2 and 1 <= to_dim <= nd - 2):
        oshape = tuple(x.shape)
    else:
        others = [k for k in range(1, nd - 1) if k != from_dim]
        mid = [dims[k] // max(n_chunks, 1) if k == to_dim else dims[k] for k in others]
        oshape = (n_chunks, dims[0], *mid, dims[from_dim], dims[-1])
    if out is None:
        out = torch.empty(oshape, dtype=x.dtype, device=x.device)
    shape = (ctypes.c_int64 * nd)(*dims)
    st = lib().dsp_switch_variant(_ptr(x), _ptr(out), shape, nd, from_dim, to_dim, n_chunks,
                                  _dtype_code(x), variant, _stream(stream))
    _check(st, "dsp_switch")
    return out


def dsp_split(x, dim: int, n_chunks: int, rank: int, out=None, stream=None):
    """Split (primitive table, s^ -> s_i): rank ``rank``'s slice of the replicated
    tensor x [B, S_1, .., S_K, C] along sequence dimension ``dim`` (see dsp.h)."""
    torch = _torch()
    _require_device(x, out)
    if x.dim() not in (4, 5):
        raise ValueError("x must be [B, S_1, .., S_K, C] with K = 2 or 3")
    x = x.contiguous()
    dims = list(x.shape)
    if out is None:
        oshape = list(dims)
        if 1 <= dim < x.dim() - 1 and n_chunks >= 1:
            oshape[dim] //= n_chunks
        out = torch.empty(oshape, dtype=x.dtype, device=x.device)
    shape = (ctypes.c_int64 * x.dim())(*dims)
    st = lib().dsp_split(_ptr(x), _ptr(out), shape, x.dim(), dim, n_chunks, rank, _dtype_code(x),
                         _stream(stream))
    _check(st, "dsp_split")
    return out


def dsp_gather(shards, dim: int, out=None, stream=None):
    """Gather (primitive table, s_i -> s^): the concatenation along sequence
    dimension ``dim`` of N equal shards [B, S_1, .., S_K, C], in rank order; the
    receiving side of the all-gather, with every rank's shard on one GPU."""
    torch = _torch()
    shards = [s.contiguous() for s in shards]
    _require_device(*shards, out)
    if not shards:
        raise ValueError("at least one shard")
    x0 = shards[0]
    if any(s.shape != x0.shape or s.dtype != x0.dtype for s in shards):
        raise ValueError("shards must share shape and dtype")
    if x0.dim() not in (4, 5):
        raise ValueError("shards must be [B, S_1, .., S_K, C] with K = 2 or 3")
    dims = list(x0.shape)
    if out is None:
        oshape = list(dims)
        if 1 <= dim < x0.dim() - 1:
            oshape[dim] *= len(shards)
        out = torch.empty(oshape, dtype=x0.dtype, device=x0.device)
    ptrs = (ctypes.c_void_p * len(shards))(*[_ptr(s) for s in shards])
    shape = (ctypes.c_int64 * x0.dim())(*dims)
    st = lib().dsp_gather(ptrs, _ptr(out), shape, x0.dim(), dim, len(shards), _dtype_code(x0),
                          _stream(stream))
    _check(st, "dsp_gather")
    return out


def _attn(name, q, k, v, B, X, L, H, out, ld_in, ld_out, scale, stream, C):
    torch = _torch()
    _require_device(q, k, v, out)
    D = C // H
    if out is None:
        out = torch.empty((B, X, L, C), dtype=q.dtype, device=q.device)
    fn = getattr(lib(), name)
    st = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, X, L, H, D, ld_in, ld_out, float(scale),
            _dtype_code(q), _stream(stream))
    _check(st, name)
    return out


def dsp_exchange_unpack(packed, out=None, stream=None):
    """Exchange + unpack of N ranks' packed switch outputs on one GPU (see
    dsp.h).  ``packed``: N tensors of shape [N, B, P, F, C] (same dtype).
    Returns N tensors of shape [B, P, N*F, C]: rank n's result."""
    torch = _torch()
    packed = list(packed)
    N = len(packed)
    if N == 0:
        raise ValueError("dsp_exchange_unpack: no ranks")
    shape = tuple(packed[0].shape)
    if len(shape) != 5 or shape[0] != N:
        raise ValueError(f"dsp_exchange_unpack: packed[0] has shape {shape}, want [N={N}, B, P, F, C]")
    _require_device(*packed)
    for t in packed:
        if tuple(t.shape) != shape or t.dtype != packed[0].dtype or not t.is_contiguous():
            raise ValueError("dsp_exchange_unpack: packed tensors must share one contiguous shape and dtype")
    _, B, P, F, C = shape
    if out is None:
        out = [torch.empty((B, P, N * F, C), dtype=packed[0].dtype, device=packed[0].device)
               for _ in range(N)]
    out = list(out)
    _require_device(*out)
    if len(out) != N or any(tuple(o.shape) != (B, P, N * F, C) or not o.is_contiguous() for o in out):
        raise ValueError("dsp_exchange_unpack: out must be N contiguous tensors of shape [B, P, N*F, C]")
    src = (ctypes.c_void_p * N)(*[t.data_ptr() for t in packed])
    dst = (ctypes.c_void_p * N)(*[o.data_ptr() for o in out])
    shp = (ctypes.c_int64 * 5)(N, B, P, F, C)
    _check(lib().dsp_exchange_unpack(src, dst, shp, _dtype_code(packed[0]), _stream(stream)),
           "dsp_exchange_unpack")
    return out


def dsp_spatial_attn(q, k, v, H: int, out=None, scale: float = 0.0, C: int | None = None,
                     ld_in: int | None = None, ld_out: int | None = None, stream=None):
    """Attention over S within each frame.  q, k, v: (B, T, S, ld_in) views whose
    first C = H*D columns hold the heads (pass C explicitly for packed QKV views)."""
    B, T, S = q.shape[0], q.shape[1], q.shape[2]
    C = C if C is not None else q.shape[3]
    ld_in = ld_in if ld_in is not None else q.stride(2)
    ld_out = ld_out if ld_out is not None else (out.stride(2) if out is not None else C)
    return _attn("dsp_spatial_attn", q, k, v, B, T, S, H, out, ld_in, ld_out, scale, stream, C)


def dsp_temporal_attn(q, k, v, H: int, out=None, scale: float = 0.0, C: int | None = None,
                      ld_in: int | None = None, ld_out: int | None = None, stream=None):
    """Attention over T at each spatial location.  q, k, v: (B, S, T, ld_in) views."""
    B, S, T = q.shape[0], q.shape[1], q.shape[2]
    C = C if C is not None else q.shape[3]
    ld_in = ld_in if ld_in is not None else q.stride(2)
    ld_out = ld_out if ld_out is not None else (out.stride(2) if out is not None else C)
    return _attn("dsp_temporal_attn", q, k, v, B, S, T, H, out, ld_in, ld_out, scale, stream, C)


def dsp_attn_strided(q, k, v, H: int, out=None, scale: float = 0.0, stream=None):
    """Attention over dim 2 of the 4-D views q, k, v [B, X, L, >=H*D] (any
    strides, last one 1, the same for q, k and v), per (b, x, head): e.g.
    temporal attention on a (B, T, S, C) tensor x is ``q = x.permute(0, 2, 1, 3)``.
    The output is a new contiguous [B, X, L, C] tensor, or ``out`` (any 4-D
    view with last stride 1)."""
    torch = _torch()
    _require_device(q, k, v, out)
    if q.dim() != 4 or q.shape != k.shape or q.shape != v.shape:
        raise ValueError("q, k, v must be 4-D views of one shape [B, X, L, C]")
    if q.stride() != k.stride() or q.stride() != v.stride() or q.stride(3) != 1:
        raise ValueError("q, k, v must share strides, with a unit last stride")
    B, X, L, C = q.shape
    if C % H:
        raise ValueError("C must be a multiple of H")
    if out is None:
        out = torch.empty((B, X, L, C), dtype=q.dtype, device=q.device)
    if out.shape != q.shape or out.stride(3) != 1:
        raise ValueError("out must be a view of shape [B, X, L, C] with a unit last stride")
    ins = (ctypes.c_int64 * 3)(*q.stride()[:3])
    outs = (ctypes.c_int64 * 3)(*out.stride()[:3])
    _check(lib().dsp_attn_strided(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, X, L, H, C // H, ins, outs,
                                  float(scale), _dtype_code(q), _stream(stream)), "dsp_attn_strided")
    return out


def _qkv_views(where, q, k, v, H):
    _require_device(q, k, v)
    if q.dim() != 4 or q.shape != k.shape or q.shape != v.shape:
        raise ValueError(f"{where}: q, k, v must be 4-D views of one shape [B, X, L, C]")
    if q.stride() != k.stride() or q.stride() != v.stride() or q.stride(3) != 1:
        raise ValueError(f"{where}: q, k, v must share strides, with a unit last stride")
    B, X, L, C = q.shape
    if C % H:
        raise ValueError(f"{where}: C must be a multiple of H")
    return B, X, L, C


def _like_view(where, t, shape, name):
    if t.shape != shape or t.stride(3) != 1:
        raise ValueError(f"{where}: {name} must be a view of shape {tuple(shape)} with a unit last stride")


def dsp_attn_fwd_lse(q, k, v, H: int, out=None, lse=None, scale: float = 0.0, stream=None):
    """dsp_attn_strided that also returns the row log-sum-exp: (out, lse) with
    lse a float32 tensor [B, X, H, L]."""
    torch = _torch()
    B, X, L, C = _qkv_views("dsp_attn_fwd_lse", q, k, v, H)
    _require_device(out, lse)
    if out is None:
        out = torch.empty((B, X, L, C), dtype=q.dtype, device=q.device)
    _like_view("dsp_attn_fwd_lse", out, q.shape, "out")
    if lse is None:
        lse = torch.empty((B, X, H, L), dtype=torch.float32, device=q.device)
    if lse.dtype != torch.float32 or lse.numel() != B * X * H * L or not lse.is_contiguous():
        raise ValueError("dsp_attn_fwd_lse: lse must be a contiguous float32 tensor of B*X*H*L elements")
    ins = (ctypes.c_int64 * 3)(*q.stride()[:3])
    outs = (ctypes.c_int64 * 3)(*out.stride()[:3])
    _check(lib().dsp_attn_fwd_lse(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, X, L, H, C // H,
                                  ins, outs, float(scale), _dtype_code(q), _stream(stream)),
           "dsp_attn_fwd_lse")
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
    B, X, L, C = _qkv_views("dsp_attn_bwd", q, k, v, H)
    _require_device(o, dout, lse, dq, dk, dv, delta)
    _like_view("dsp_attn_bwd", o, q.shape, "o")
    if dout.shape != o.shape or dout.stride() != o.stride():
        raise ValueError("dsp_attn_bwd: dout must have the shape and strides of o")
    if lse.dtype != torch.float32 or lse.numel() != B * X * H * L or not lse.is_contiguous():
        raise ValueError("dsp_attn_bwd: lse must be a contiguous float32 tensor of B*X*H*L elements")
    if dq is None or dk is None or dv is None:
        if not q.is_contiguous():
            raise ValueError("dsp_attn_bwd: for a non-contiguous q pass dq, dk, dv views with its strides")
        dq, dk, dv = (torch.empty_like(q) if g is None else g for g in (dq, dk, dv))
    for g, name in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
        _like_view("dsp_attn_bwd", g, q.shape, name)
        if tuple(g.stride()) != tuple(q.stride()):
            raise ValueError(f"dsp_attn_bwd: {name} must have the strides of q, k, v")
    if delta is None:
        delta = torch.empty(B * X * H * L, dtype=torch.float32, device=q.device)
    if delta.dtype != torch.float32 or delta.numel() != B * X * H * L or not delta.is_contiguous():
        raise ValueError("dsp_attn_bwd: delta must be a contiguous float32 tensor of B*X*H*L elements")
    qs = (ctypes.c_int64 * 3)(*q.stride()[:3])
    os_ = (ctypes.c_int64 * 3)(*o.stride()[:3])
    _check(lib().dsp_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq),
                              _ptr(dk), _ptr(dv), _ptr(delta), B, X, L, H, C // H, qs, os_,
                              float(scale), _dtype_code(q), _stream(stream)), "dsp_attn_bwd")
    return dq, dk, dv


def dsp_layernorm(x, eps: float = 1e-6, out=None, out_dtype=None, stream=None):
    torch = _torch()
    _require_device(x, out)
    x = x.contiguous()
    C = x.shape[-1]
    rows = x.numel() // C
    if out is None:
        out = torch.empty(x.shape, dtype=out_dtype or x.dtype, device=x.device)
    st = lib().dsp_layernorm(_ptr(x), _dtype_code(x), _ptr(out), _dtype_code(out), rows, C,
                             float(eps), _stream(stream))
    _check(st, "dsp_layernorm")
    return out


def _st3(t):
    return (ctypes.c_int64 * 3)(*t.stride()[:3])


def dsp_attn_general(q, k, v, H: int, Hkv: int, out=None, lse=None, with_lse: bool = False,
                     scale: float = 0.0, stream=None):
    """Grouped-query / multi-query / cross-attention over dim 2 of 4-D views:
    q [B, X, Lq, H*D], k and v [B, X, Lk, Hkv*D] (same strides; a 0 stride
    broadcasts).  Returns out [B, X, Lq, H*D] (and lse [B, X, H, Lq] fp32 when
    with_lse or lse is given)."""
    torch = _torch()
    _require_device(q, k, v, out, lse)
    if q.dim() != 4 or k.shape != v.shape or k.stride() != v.stride() or q.stride(3) != 1 or k.stride(3) != 1:
        raise ValueError("dsp_attn_general: q [B, X, Lq, C] and k, v [B, X, Lk, Ckv] views of one layout")
    B, X, Lq, C = q.shape
    if C % H or tuple(k.shape[:2]) != (B, X):
        raise ValueError("dsp_attn_general: shapes do not match")
    D = C // H
    Lk = k.shape[2]
    if k.shape[3] != Hkv * D:
        raise ValueError("dsp_attn_general: k and v must hold Hkv heads of the query head width")
    if out is None:
        out = torch.empty((B, X, Lq, C), dtype=q.dtype, device=q.device)
    if (with_lse or lse is not None) and lse is None:
        lse = torch.empty((B, X, H, Lq), dtype=torch.float32, device=q.device)
    _check(lib().dsp_attn_general(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, X, Lq, Lk, H, Hkv, D,
                                  _st3(q), _st3(k), _st3(out), float(scale), _dtype_code(q), _stream(stream)),
           "dsp_attn_general")
    return (out, lse) if lse is not None else out


def dsp_attn_general_bwd(q, k, v, o, dout, lse, H: int, Hkv: int, dq=None, dk=None, dv=None, delta=None,
                         scale: float = 0.0, stream=None):
    """Gradients of dsp_attn_general: (dq like q, dk and dv like k and v)."""
    torch = _torch()
    _require_device(q, k, v, o, dout, lse, dq, dk, dv, delta)
    B, X, Lq, C = q.shape
    D = C // H
    Lk = k.shape[2]
    if dout.stride() != o.stride() or dout.shape != o.shape:
        raise ValueError("dsp_attn_general_bwd: dout must have the shape and strides of o")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    if dq.stride() != q.stride() or dk.stride() != k.stride() or dv.stride() != k.stride():
        raise ValueError("dsp_attn_general_bwd: dq must have q's strides, dk and dv k's")
    if delta is None:
        delta = torch.empty(B * X * H * Lq, dtype=torch.float32, device=q.device)
    _check(lib().dsp_attn_general_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq),
                                      _ptr(dk), _ptr(dv), _ptr(delta), B, X, Lq, Lk, H, Hkv, D, _st3(q), _st3(k),
                                      _st3(o), float(scale), _dtype_code(q), _stream(stream)),
           "dsp_attn_general_bwd")
    return dq, dk, dv


def dsp_layernorm_bwd(x, dy, eps: float = 1e-6, dres=None, out=None, stream=None):
    """dx (fp32) = dres + the LayerNorm backward of dy at x (rows of C)."""
    torch = _torch()
    _require_device(x, dy, dres, out)
    x, dy = x.contiguous(), dy.contiguous()
    C = x.shape[-1]
    rows = x.numel() // C
    if out is None:
        out = torch.empty(x.shape, dtype=torch.float32, device=x.device)
    _check(lib().dsp_layernorm_bwd(_ptr(x), _dtype_code(x), _ptr(dy), _dtype_code(dy), _ptr(dres), _ptr(out), rows,
                                   C, float(eps), _stream(stream)), "dsp_layernorm_bwd")
    return out


def dsp_linear(a, w, bias=None, residual=None, epilogue: int = DSP_EPI_NONE, out=None,
               stream=None):
    """out = epilogue(a @ w.T + bias); w stored [N, K]."""
    torch = _torch()
    _require_device(a, w, bias, residual, out)
    a = a.contiguous()
    K = a.shape[-1]
    M = a.numel() // K
    N = w.shape[0]
    if out is None:
        odt = torch.float32 if epilogue in (DSP_EPI_RESID, DSP_EPI_F32) else a.dtype
        out = torch.empty((*a.shape[:-1], N), dtype=odt, device=a.device)
    st = lib().dsp_linear(_ptr(a), _ptr(w), _ptr(bias), _ptr(residual), _ptr(out), M, N, K,
                          epilogue, _dtype_code(a), _stream(stream))
    _check(st, "dsp_linear")
    return out


def dsp_linear_bwd_data(dy, w, u=None, epilogue: int = DSP_GRAD_EPI_F32, out=None, stream=None):
    """dx = epilogue(dy @ w) for y = x @ w.T (w stored [N, K]); u: the saved
    pre-activation for the GELU/ReLU backward epilogues."""
    torch = _torch()
    _require_device(dy, w, u, out)
    dy = dy.contiguous()
    N, K = w.shape
    M = dy.numel() // N
    if out is None:
        odt = torch.float32 if epilogue == DSP_GRAD_EPI_F32 else dy.dtype
        out = torch.empty((*dy.shape[:-1], K), dtype=odt, device=dy.device)
    _check(lib().dsp_linear_bwd_data(_ptr(dy), _ptr(w.contiguous()), _ptr(u), _ptr(out), M, N, K, epilogue,
                                     _dtype_code(dy), _stream(stream)), "dsp_linear_bwd_data")
    return out


def dsp_linear_bwd_weight(dy, x, with_bias: bool = False, dw=None, db=None, workspace=None, stream=None):
    """(dw [N, K] fp32, db [N] fp32 or None) for y = x @ w.T + b: dw = dy^T x."""
    torch = _torch()
    _require_device(dy, x, dw, db, workspace)
    dy, x = dy.contiguous(), x.contiguous()
    N, K = dy.shape[-1], x.shape[-1]
    M = dy.numel() // N
    if dw is None:
        dw = torch.empty((N, K), dtype=torch.float32, device=dy.device)
    if with_bias and db is None:
        db = torch.empty(N, dtype=torch.float32, device=dy.device)
    need = int(lib().dsp_linear_bwd_weight_workspace_bytes(M, N, K, _dtype_code(dy)))
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dy.device)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().dsp_linear_bwd_weight(_ptr(dy), _ptr(x), _ptr(dw), _ptr(db), _ptr(workspace), ws_bytes, M, N, K,
                                       _dtype_code(dy), _stream(stream)), "dsp_linear_bwd_weight")
    return dw, db


def block_workspace_bytes(B, T, S, C, H, F, dtype_code) -> int:
    return int(lib().dsp_st_block_workspace_bytes(B, T, S, C, H, F, dtype_code))


def dsp_st_block_forward(x, weights: dict, H: int, eps: float = 1e-6, flags: int = 0,
                         out=None, workspace=None, dtype=None, stream=None):
    """One spatial-temporal block on x (B, T, S, C) fp32; returns (B, S, T, C) fp32.
    ``weights`` maps the dsp_block_weights_t field names to device tensors (or None)."""
    torch = _torch()
    _require_device(x, out, workspace, *weights.values())
    B, T, S, C = x.shape
    wdt = weights["wqkv_s"].dtype
    code = DSP_BF16 if (dtype or wdt) == torch.bfloat16 else DSP_F32
    F = weights["w1"].shape[0] if weights.get("w1") is not None else 0
    if out is None:
        out = torch.empty((B, S, T, C), dtype=torch.float32, device=x.device)
    need = block_workspace_bytes(B, T, S, C, H, F, code)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    wt = BlockWeights(**{n: (weights[n].data_ptr() if weights.get(n) is not None else None)
                         for n in BLOCK_WEIGHT_FIELDS})
    st = lib().dsp_st_block_forward(_ptr(x), _ptr(out), ctypes.byref(wt), _ptr(workspace),
                                    workspace.numel(), B, T, S, C, H, F, float(eps), flags, code,
                                    _stream(stream))
    _check(st, "dsp_st_block_forward")
    return out


def _block_sizes(x, weights, dtype):
    torch = _torch()
    B, T, S, C = x.shape
    code = DSP_BF16 if (dtype or weights["wqkv_s"].dtype) == torch.bfloat16 else DSP_F32
    return B, T, S, C, weights["w1"].shape[0], code


def dsp_st_block_forward_train(x, weights: dict, H: int, eps: float = 1e-6, flags: int = 0, out=None,
                               saved=None, dtype=None, stream=None):
    """dsp_st_block_forward that also keeps the activations the backward needs:
    returns (y (B, S, T, C) fp32, saved: a uint8 device tensor)."""
    torch = _torch()
    _require_device(x, out, saved, *weights.values())
    B, T, S, C, F, code = _block_sizes(x, weights, dtype)
    if out is None:
        out = torch.empty((B, S, T, C), dtype=torch.float32, device=x.device)
    need = int(lib().dsp_st_block_train_saved_bytes(B, T, S, C, H, F, flags, code))
    if saved is None:
        saved = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    wt = BlockWeights(**{n: (weights[n].data_ptr() if weights.get(n) is not None else None)
                         for n in BLOCK_WEIGHT_FIELDS})
    _check(lib().dsp_st_block_forward_train(_ptr(x), _ptr(out), ctypes.byref(wt), _ptr(saved), saved.numel(), B, T,
                                            S, C, H, F, float(eps), flags, code, _stream(stream)),
           "dsp_st_block_forward_train")
    return out, saved


def dsp_st_block_backward(x, dy, weights: dict, saved, H: int, eps: float = 1e-6, flags: int = 0, dx=None,
                          grads=None, with_bias: bool = False, workspace=None, dtype=None, stream=None):
    """Backward of the block: returns (dx (B, T, S, C) fp32, grads: dict of fp32
    tensors shaped like the weights, plus the biases when with_bias)."""
    torch = _torch()
    _require_device(x, dy, saved, dx, workspace, *weights.values())
    B, T, S, C, F, code = _block_sizes(x, weights, dtype)
    if dx is None:
        dx = torch.empty((B, T, S, C), dtype=torch.float32, device=x.device)
    if grads is None:
        shapes = {"wqkv_s": (3 * C, C), "wo_s": (C, C), "wqkv_t": (3 * C, C), "wo_t": (C, C), "w1": (F, C),
                  "w2": (C, F)}
        if with_bias:
            shapes.update({"bqkv_s": (3 * C,), "bo_s": (C,), "bqkv_t": (3 * C,), "bo_t": (C,), "b1": (F,),
                           "b2": (C,)})
        grads = {n: torch.empty(s, dtype=torch.float32, device=x.device) for n, s in shapes.items()}
    need = int(lib().dsp_st_block_backward_workspace_bytes(B, T, S, C, H, F, code))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    wt = BlockWeights(**{n: (weights[n].data_ptr() if weights.get(n) is not None else None)
                         for n in BLOCK_WEIGHT_FIELDS})
    gt = BlockGrads(**{n: (grads[n].data_ptr() if grads.get(n) is not None else None) for n in BLOCK_WEIGHT_FIELDS})
    _check(lib().dsp_st_block_backward(_ptr(x), _ptr(dy.contiguous()), ctypes.byref(wt), _ptr(saved), saved.numel(),
                                       _ptr(workspace), workspace.numel(), _ptr(dx), ctypes.byref(gt), B, T, S, C,
                                       H, F, float(eps), flags, code, _stream(stream)), "dsp_st_block_backward")
    return dx, grads


def probe_mfma_workspace_bytes() -> int:
    return int(lib().dsp_probe_mfma_workspace_bytes())


def probe_mfma_flops(iters: int) -> float:
    """Flops one dsp_probe_mfma launch of `iters` iterations issues."""
    return float(lib().dsp_probe_mfma_flops(iters))


def dsp_probe_mfma(iters: int, workspace, stream=None):
    """Launch the sustained-MFMA-rate probe (a measurement aid): time it with
    events on `stream` and divide probe_mfma_flops(iters) by the time."""
    _require_device(workspace)
    _check(lib().dsp_probe_mfma(_ptr(workspace), workspace.numel() * workspace.element_size(), iters,
                                _stream(stream)), "dsp_probe_mfma")


__all__ = ["lib", "status_str", "DspError", "BlockWeights", "dsp_switch", "dsp_spatial_attn",
           "dsp_temporal_attn", "dsp_layernorm", "dsp_linear", "dsp_st_block_forward",
           "dsp_st_block_forward_train", "dsp_st_block_backward", "block_workspace_bytes", "LIB_PATH"]
