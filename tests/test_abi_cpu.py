"""The C ABI without a GPU: the library loads, exports every symbol that
include/*.h declares, and rejects bad arguments with the documented status
before touching the device (only calls that fail validation are made)."""
import ctypes
import re
from pathlib import Path

import pytest

import paper_2403_10266_amd as dsp

ROOT = Path(__file__).resolve().parent.parent
FAKE = 0x10000          # a 256-byte aligned address that is never dereferenced
FAKE2 = 0x20000000
MIS = FAKE + 2          # misaligned


def _declared():
    names = set()
    for h in (ROOT / "include").glob("*.h"):
        text = re.sub(r"/\*.*?\*/", "", h.read_text(), flags=re.S)
        for m in re.finditer(r"^[A-Za-z_][\w \t\*]*?\b(dsp_\w+)\s*\(", text, flags=re.M):
            names.add(m.group(1))
    return sorted(names)


def test_header_declares_entry_points():
    names = _declared()
    for n in ("dsp_switch", "dsp_spatial_attn", "dsp_temporal_attn", "dsp_layernorm", "dsp_linear",
              "dsp_st_block_forward", "dsp_st_block_workspace_bytes", "dsp_status_str"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(str(dsp.LIB_PATH))
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_signatures_cover_header():
    assert set(_declared()) <= set(dsp._SIGNATURES)


def test_status_strings():
    for code in range(9):
        s = dsp.status_str(code)
        assert s.startswith("DSP_")
    assert "unknown" in dsp.status_str(99)
    assert dsp.lib().dsp_version() >= 10000


def _shape(*v):
    return (ctypes.c_int64 * len(v))(*v)


L = None


@pytest.fixture(scope="module")
def lib():
    return dsp.lib()


def test_switch_validation(lib):
    sw = lambda x, y, shape, ndim, f, t, n, dt, var=0: lib.dsp_switch_variant(
        x, y, shape, ndim, f, t, n, dt, var, None)
    s = _shape(1, 4, 6, 8)
    assert sw(None, FAKE2, s, 4, 1, 2, 2, 1) == dsp.DSP_ERR_NULL
    assert sw(FAKE, None, s, 4, 1, 2, 2, 1) == dsp.DSP_ERR_NULL
    assert sw(FAKE, FAKE2, None, 4, 1, 2, 2, 1) == dsp.DSP_ERR_NULL
    assert sw(FAKE, FAKE2, s, 3, 1, 2, 2, 1) == dsp.DSP_ERR_DIM
    assert sw(FAKE, FAKE2, s, 4, 0, 2, 2, 1) == dsp.DSP_ERR_DIM
    assert sw(FAKE, FAKE2, s, 4, 1, 3, 2, 1) == dsp.DSP_ERR_DIM
    assert sw(FAKE, FAKE2, s, 4, 1, 2, 4, 1) == dsp.DSP_ERR_SHAPE      # 6 % 4
    assert sw(FAKE, FAKE2, s, 4, 1, 2, 0, 1) == dsp.DSP_ERR_SHAPE
    assert sw(FAKE, FAKE2, _shape(1, -1, 6, 8), 4, 1, 2, 1, 1) == dsp.DSP_ERR_SHAPE
    assert sw(FAKE, FAKE2, s, 4, 1, 2, 2, 7) == dsp.DSP_ERR_DTYPE
    assert sw(FAKE, FAKE + 16, s, 4, 1, 2, 2, 1) == dsp.DSP_ERR_ARG      # overlapping buffers
    assert sw(FAKE, FAKE2, s, 4, 1, 2, 2, 1, 3) == dsp.DSP_ERR_ARG     # unknown variant
    assert sw(MIS, FAKE2, s, 4, 1, 2, 2, 1, 1) == dsp.DSP_ERR_ALIGN    # rows variant needs 16 B
    # empty tensors are accepted and launch nothing
    assert sw(FAKE, FAKE2, _shape(0, 4, 6, 8), 4, 1, 2, 2, 1) == dsp.DSP_OK
    assert sw(FAKE, FAKE2, _shape(1, 4, 6, 0), 4, 1, 2, 2, 1) == dsp.DSP_OK


def test_switch_k3_split_gather_validation(lib):
    sw = lambda x, y, shape, ndim, f, t, n, dt, var=0: lib.dsp_switch_variant(
        x, y, shape, ndim, f, t, n, dt, var, None)
    s5 = _shape(1, 4, 2, 6, 8)
    assert sw(FAKE, FAKE2, s5, 5, 1, 4, 2, 1) == dsp.DSP_ERR_DIM        # 4 is C when K = 3
    assert sw(FAKE, FAKE2, _shape(1, 2, 2, 2, 2, 2), 6, 1, 2, 1, 1) == dsp.DSP_ERR_DIM
    assert sw(FAKE, FAKE2, s5, 5, 1, 3, 4, 1) == dsp.DSP_ERR_SHAPE      # 6 % 4
    assert sw(FAKE, FAKE2, s5, 5, 1, 3, 2, 1, 1) == dsp.DSP_ERR_ARG     # one kernel for K = 3
    assert sw(FAKE, FAKE + 16, s5, 5, 1, 3, 2, 1) == dsp.DSP_ERR_ARG    # overlapping buffers
    assert sw(None, FAKE2, s5, 5, 1, 3, 2, 1) == dsp.DSP_ERR_NULL
    assert sw(FAKE, FAKE2, _shape(1, 4, 0, 6, 8), 5, 1, 3, 2, 1) == dsp.DSP_OK
    split = lambda x=FAKE, y=FAKE2, s=s5, nd=5, dim=3, n=2, r=0, dt=1: lib.dsp_split(
        x, y, s, nd, dim, n, r, dt, None)
    assert split(x=None) == dsp.DSP_ERR_NULL
    assert split(s=None) == dsp.DSP_ERR_NULL
    assert split(nd=3) == dsp.DSP_ERR_DIM
    assert split(dim=4) == dsp.DSP_ERR_DIM
    assert split(dim=0) == dsp.DSP_ERR_DIM
    assert split(n=4) == dsp.DSP_ERR_SHAPE                 # 6 % 4
    assert split(n=0) == dsp.DSP_ERR_SHAPE
    assert split(r=2) == dsp.DSP_ERR_ARG
    assert split(r=-1) == dsp.DSP_ERR_ARG
    assert split(dt=5) == dsp.DSP_ERR_DTYPE
    assert split(y=FAKE + 16) == dsp.DSP_ERR_ARG           # overlaps x
    assert split(s=_shape(0, 4, 2, 6, 8)) == dsp.DSP_OK
    P = ctypes.c_void_p
    def gather(ptrs=(FAKE, FAKE + 0x1000), y=FAKE2, s=s5, nd=5, dim=1, n=None, dt=1):
        arr = (P * len(ptrs))(*ptrs) if ptrs is not None else None
        return lib.dsp_gather(arr, y, s, nd, dim, len(ptrs or ()) if n is None else n, dt, None)
    assert gather(ptrs=None, n=2) == dsp.DSP_ERR_NULL
    assert gather(ptrs=(FAKE, None)) == dsp.DSP_ERR_NULL
    assert gather(y=None) == dsp.DSP_ERR_NULL
    assert gather(s=None) == dsp.DSP_ERR_NULL
    assert gather(dim=4) == dsp.DSP_ERR_DIM
    assert gather(nd=6) == dsp.DSP_ERR_DIM
    assert gather(n=0) == dsp.DSP_ERR_SHAPE
    assert gather(ptrs=(FAKE,) * 65) == dsp.DSP_ERR_SHAPE
    assert gather(dt=3) == dsp.DSP_ERR_DTYPE
    assert gather(y=FAKE + 0x1000 + 64) == dsp.DSP_ERR_ARG  # y overlaps a shard
    assert gather(s=_shape(1, 4, 2, 0, 8)) == dsp.DSP_OK


def test_exchange_validation(lib):
    P = ctypes.c_void_p
    def call(srcs, dsts, shape, dt=1):
        s = (P * len(srcs))(*srcs) if srcs is not None else None
        d = (P * len(dsts))(*dsts) if dsts is not None else None
        return lib.dsp_exchange_unpack(s, d, shape, dt, None)
    ok = _shape(2, 1, 4, 3, 8)                  # N=2 ranks, 2*1*4*3*8 = 192 elements each
    a, b, c, d = 0x100000, 0x200000, 0x300000, 0x400000
    assert call([a, b], [c, d], None) == dsp.DSP_ERR_NULL
    assert call(None, [c, d], ok) == dsp.DSP_ERR_NULL
    assert call([a, b], None, ok) == dsp.DSP_ERR_NULL
    assert call([a, None], [c, d], ok) == dsp.DSP_ERR_NULL
    assert call([a, b], [c, d], _shape(0, 1, 4, 3, 8)) == dsp.DSP_ERR_SHAPE
    assert call([a] * 65, [c] * 65, _shape(65, 1, 1, 1, 1)) == dsp.DSP_ERR_SHAPE
    assert call([a, b], [c, d], _shape(2, 1, -4, 3, 8)) == dsp.DSP_ERR_SHAPE
    assert call([a, b], [c, d], _shape(2, 1, 2 ** 40, 2 ** 20, 8)) == dsp.DSP_ERR_SHAPE
    assert call([a, b], [c, d], ok, dt=7) == dsp.DSP_ERR_DTYPE
    assert call([a, b], [b + 64, d], ok) == dsp.DSP_ERR_ARG     # an output overlaps a source
    assert call([a, b], [c, c + 256], ok) == dsp.DSP_ERR_ARG    # two outputs overlap
    # an empty exchange launches nothing (pointers are not looked at)
    assert call([a, b], [c, d], _shape(2, 0, 4, 3, 8)) == dsp.DSP_OK


@pytest.mark.parametrize("fn", ["dsp_spatial_attn", "dsp_temporal_attn"])
def test_attention_validation(lib, fn):
    f = getattr(lib, fn)
    call = lambda q=FAKE, k=FAKE, v=FAKE, o=FAKE2, B=2, X=3, L=5, H=16, D=72, ldi=1152, ldo=1152, \
        sc=0.0, dt=1: f(q, k, v, o, B, X, L, H, D, ldi, ldo, sc, dt, None)
    assert call(q=None) == dsp.DSP_ERR_NULL
    assert call(o=None) == dsp.DSP_ERR_NULL
    assert call(dt=5) == dsp.DSP_ERR_DTYPE
    assert call(H=0) == dsp.DSP_ERR_SHAPE
    assert call(B=-1) == dsp.DSP_ERR_SHAPE
    assert call(ldi=1000) == dsp.DSP_ERR_SHAPE            # H*D > ld
    assert call(D=70, ldi=1120, ldo=1120) == dsp.DSP_ERR_SHAPE   # unsupported bf16 head width
    assert call(q=MIS) == dsp.DSP_ERR_ALIGN
    assert call(ldi=1156) == dsp.DSP_ERR_ALIGN
    assert call(sc=float("nan")) == dsp.DSP_ERR_ARG
    assert call(dt=0, D=300, H=1, ldi=300, ldo=300) == dsp.DSP_ERR_SHAPE
    assert call(B=0) == dsp.DSP_OK                         # empty: nothing launched
    assert call(L=0) == dsp.DSP_OK


def test_attn_strided_validation(lib):
    ok_in, ok_out = _shape(8 * 1152 * 5, 1152, 8 * 1152), _shape(3 * 5 * 1152, 5 * 1152, 1152)
    call = lambda q=FAKE, o=FAKE2, B=2, X=3, L=5, H=16, D=72, si=ok_in, so=ok_out, sc=0.0, dt=1: \
        lib.dsp_attn_strided(q, q, q, o, B, X, L, H, D, si, so, sc, dt, None)
    assert call(si=None) == dsp.DSP_ERR_NULL
    assert call(q=None) == dsp.DSP_ERR_NULL
    assert call(si=_shape(-8, 1152, 9216)) == dsp.DSP_ERR_SHAPE
    assert call(so=_shape(0, 0, 1152), B=2) == dsp.DSP_ERR_ARG          # rows of different b coincide
    assert call(so=_shape(3 * 5 * 1152, 5 * 1152, 576)) == dsp.DSP_ERR_ARG   # rows narrower than H*D
    assert call(si=_shape(8 * 1152 * 5, 1152, 8 * 1152 + 4)) == dsp.DSP_ERR_ALIGN
    assert call(dt=9) == dsp.DSP_ERR_DTYPE
    assert call(D=70) == dsp.DSP_ERR_SHAPE
    assert call(si=_shape(0, 0, 2 ** 28)) == dsp.DSP_ERR_SHAPE          # 64 rows exceed a 2^31-byte range
    assert call(B=0) == dsp.DSP_OK


def test_attn_fwd_lse_validation(lib):
    ok_in, ok_out = _shape(8 * 1152 * 5, 1152, 8 * 1152), _shape(3 * 5 * 1152, 5 * 1152, 1152)
    call = lambda q=FAKE, o=FAKE2, lse=FAKE2 + 2 ** 24, B=2, X=3, L=5, H=16, D=72, dt=1: \
        lib.dsp_attn_fwd_lse(q, q, q, o, lse, B, X, L, H, D, ok_in, ok_out, 0.0, dt, None)
    assert call(lse=None) == dsp.DSP_ERR_NULL
    assert call(lse=FAKE2 + 2 ** 24 + 2) == dsp.DSP_ERR_ALIGN
    assert call(q=None) == dsp.DSP_ERR_NULL
    assert call(dt=4) == dsp.DSP_ERR_DTYPE
    assert call(D=70) == dsp.DSP_ERR_SHAPE
    assert call(B=0, lse=None) == dsp.DSP_OK


def test_attn_bwd_validation(lib):
    st_qkv = _shape(3 * 5 * 3456, 5 * 3456, 3456)     # a packed [Q|K|V] layout
    st_o = _shape(3 * 5 * 1152, 5 * 1152, 1152)
    A, BUF = 2 ** 24, 2 ** 26

    def call(q=FAKE, o=FAKE + BUF, lse=FAKE + 2 * BUF, dq=FAKE + 3 * BUF, delta=FAKE + 4 * BUF, B=2, X=3,
             L=5, H=16, D=72, sq=st_qkv, so=st_o, sc=0.0, dt=1):
        return lib.dsp_attn_bwd(q, q, q, o, o, lse, dq, dq, dq, delta, B, X, L, H, D, sq, so, sc, dt, None)
    assert call(sq=None) == dsp.DSP_ERR_NULL
    assert call(so=None) == dsp.DSP_ERR_NULL
    assert call(lse=None) == dsp.DSP_ERR_NULL
    assert call(delta=None) == dsp.DSP_ERR_NULL
    assert call(dq=None) == dsp.DSP_ERR_NULL
    assert call(dt=3) == dsp.DSP_ERR_DTYPE
    assert call(H=0) == dsp.DSP_ERR_SHAPE
    assert call(L=-1) == dsp.DSP_ERR_SHAPE
    assert call(D=70) == dsp.DSP_ERR_SHAPE                   # unsupported bf16 head width
    assert call(D=48, H=24) == dsp.DSP_ERR_SHAPE             # 48 % 32 > 16: no 16-row slab
    assert call(dt=0, D=300, H=1) == dsp.DSP_ERR_SHAPE
    assert call(q=MIS) == dsp.DSP_ERR_ALIGN
    assert call(dq=FAKE + 3 * BUF + 8) == dsp.DSP_ERR_ALIGN
    assert call(sq=_shape(3 * 5 * 3456, 5 * 3456, 3460)) == dsp.DSP_ERR_ALIGN
    assert call(lse=FAKE + 2 * BUF + 2) == dsp.DSP_ERR_ALIGN
    assert call(sc=float("inf")) == dsp.DSP_ERR_ARG
    assert call(sq=_shape(0, 0, 3456)) == dsp.DSP_ERR_ARG   # gradient rows of different units coincide
    assert call(sq=_shape(3 * 5 * 3456, 5 * 3456, 576)) == dsp.DSP_ERR_ARG   # rows narrower than H*D
    assert call(delta=FAKE + 2 * BUF + 4) == dsp.DSP_ERR_ARG   # delta overlaps lse
    assert call(B=1, sq=_shape(0, 2 ** 33, 2 ** 26)) == dsp.DSP_ERR_SHAPE   # 64 rows exceed a 2^31-byte range
    assert call(B=0, q=None, o=None, lse=None, dq=None, delta=None) == dsp.DSP_OK
    assert call(L=0) == dsp.DSP_OK


def test_linear_bwd_validation(lib):
    A = 2 ** 24
    data = lambda dy=FAKE, w=FAKE + A, u=None, dx=FAKE + 2 * A, M=64, N=72, K=136, epi=0, dt=1: \
        lib.dsp_linear_bwd_data(dy, w, u, dx, M, N, K, epi, dt, None)
    assert data(w=None) == dsp.DSP_ERR_NULL
    assert data(dy=None) == dsp.DSP_ERR_NULL
    assert data(epi=2) == dsp.DSP_ERR_NULL                      # GELU backward needs u
    assert data(epi=7) == dsp.DSP_ERR_ARG
    assert data(dt=0, epi=1) == dsp.DSP_ERR_ARG                  # fp32 path: fp32 output only
    assert data(dt=5) == dsp.DSP_ERR_DTYPE
    assert data(N=0) == dsp.DSP_ERR_SHAPE
    assert data(M=-1) == dsp.DSP_ERR_SHAPE
    assert data(N=70) == dsp.DSP_ERR_ALIGN
    assert data(K=130) == dsp.DSP_ERR_ALIGN
    assert data(dy=MIS) == dsp.DSP_ERR_ALIGN
    assert data(dx=FAKE + 64) == dsp.DSP_ERR_ARG                 # dx overlaps dy
    assert data(M=0, dy=None, dx=None) == dsp.DSP_OK
    ws_need = lib.dsp_linear_bwd_weight_workspace_bytes(32768, 3456, 1152, 1)
    assert ws_need > 0 and lib.dsp_linear_bwd_weight_workspace_bytes(32768, 3456, 1152, 0) == 0
    wgt = lambda dy=FAKE, x=FAKE + A, dw=FAKE + 2 * A, db=None, ws=None, wsb=0, M=64, N=72, K=136, dt=1: \
        lib.dsp_linear_bwd_weight(dy, x, dw, db, ws, wsb, M, N, K, dt, None)
    assert wgt(dw=None) == dsp.DSP_ERR_NULL
    assert wgt(x=None) == dsp.DSP_ERR_NULL
    assert wgt(dt=4) == dsp.DSP_ERR_DTYPE
    assert wgt(K=0) == dsp.DSP_ERR_SHAPE
    assert wgt(N=12) == dsp.DSP_ERR_ALIGN
    assert wgt(dw=FAKE + 2 * A + 4) == dsp.DSP_ERR_ALIGN
    assert wgt(db=FAKE + 2 * A) == dsp.DSP_ERR_ARG                # db overlaps dw
    big = dict(M=32768, N=3456, K=1152, dy=2 ** 36, x=2 ** 37, dw=2 ** 38)
    assert wgt(**big) == dsp.DSP_ERR_WORKSPACE
    assert wgt(ws=2 ** 39, wsb=ws_need - 16, **big) == dsp.DSP_ERR_WORKSPACE


def test_layernorm_bwd_validation(lib):
    f = lambda x=FAKE, xd=0, dy=FAKE2, dyd=1, dres=None, dx=FAKE2 + 2 ** 24, rows=4, C=8, eps=1e-6: \
        lib.dsp_layernorm_bwd(x, xd, dy, dyd, dres, dx, rows, C, eps, None)
    assert f(x=None) == dsp.DSP_ERR_NULL
    assert f(dx=None) == dsp.DSP_ERR_NULL
    assert f(dyd=2) == dsp.DSP_ERR_DTYPE
    assert f(C=0) == dsp.DSP_ERR_SHAPE
    assert f(eps=float("nan")) == dsp.DSP_ERR_ARG
    assert f(dx=FAKE + 4) == dsp.DSP_ERR_ARG                      # dx overlaps x
    assert f(dres=FAKE2 + 2 ** 24 + 4) == dsp.DSP_ERR_ARG          # dres partly overlaps dx
    assert f(rows=0, x=None) == dsp.DSP_OK


def test_block_train_validation(lib):
    import ctypes as c
    W = dsp.BlockWeights(**{n: (FAKE + 2 ** 26 * i if n.startswith("w") else None)
                            for i, n in enumerate(dsp.BLOCK_WEIGHT_FIELDS)})
    G = dsp.BlockGrads(**{n: (2 ** 40 + 2 ** 26 * i if n.startswith("w") else None)
                          for i, n in enumerate(dsp.BLOCK_WEIGHT_FIELDS)})
    dims = (1, 4, 8, 144, 2, 576)
    need = lib.dsp_st_block_train_saved_bytes(*dims, 0, 1)
    ws_need = lib.dsp_st_block_backward_workspace_bytes(*dims, 1)
    assert need > 0 and ws_need > 0
    assert lib.dsp_st_block_train_saved_bytes(1, 4, 8, 144, 5, 576, 0, 1) == 0     # C % H
    # post-LN with the MLP's LayerNorm keeps one more fp32 stream (tokens x C), else the same
    post = dsp.DSP_BLOCK_POST_LN
    assert lib.dsp_st_block_train_saved_bytes(*dims, post, 1) == need + 32 * 144 * 4
    assert lib.dsp_st_block_train_saved_bytes(*dims, post | dsp.DSP_BLOCK_NO_MLP_LN, 1) == need
    assert lib.dsp_st_block_train_saved_bytes(*dims, dsp.DSP_BLOCK_RELU, 1) == need
    X, Y, SV, WS, DX = 2 ** 34, 2 ** 35, 2 ** 36, 2 ** 37, 2 ** 38
    fwd = lambda flags=0, sv=SV, svb=need, dt=1, F=576: lib.dsp_st_block_forward_train(
        X, Y, c.byref(W), sv, svb, 1, 4, 8, 144, 2, F, 1e-6, flags, dt, None)
    assert fwd(flags=dsp.DSP_BLOCK_ATTN_ONLY) == dsp.DSP_ERR_ARG               # no training path
    assert fwd(flags=16) == dsp.DSP_ERR_ARG                                     # unknown flag
    assert fwd(flags=post) == dsp.DSP_ERR_WORKSPACE                             # post-LN needs the r3 slot
    assert fwd(sv=None) == dsp.DSP_ERR_WORKSPACE
    assert fwd(svb=need - 1) == dsp.DSP_ERR_WORKSPACE
    assert fwd(sv=SV + 16) == dsp.DSP_ERR_ALIGN
    assert fwd(dt=2) == dsp.DSP_ERR_DTYPE
    assert fwd(F=0) == dsp.DSP_ERR_SHAPE
    bwd = lambda grads=c.byref(G), ws=WS, wsb=ws_need, dx=DX, flags=0: lib.dsp_st_block_backward(
        X, Y, c.byref(W), SV, need, ws, wsb, dx, grads, 1, 4, 8, 144, 2, 576, 1e-6, flags, 1, None)
    assert bwd(grads=None) == dsp.DSP_ERR_NULL
    assert bwd(dx=None) == dsp.DSP_ERR_NULL
    assert bwd(wsb=ws_need - 1) == dsp.DSP_ERR_WORKSPACE
    assert bwd(dx=X + 16) == dsp.DSP_ERR_ARG                                     # dx overlaps x
    assert bwd(flags=dsp.DSP_BLOCK_POST_LN | dsp.DSP_BLOCK_RELU) == dsp.DSP_ERR_WORKSPACE
    assert bwd(flags=dsp.DSP_BLOCK_ATTN_ONLY) == dsp.DSP_ERR_ARG


def test_attn_general_validation(lib):
    qs, kvs, os_ = _shape(3 * 5 * 1152, 5 * 1152, 1152), _shape(3 * 7 * 288, 7 * 288, 288), \
        _shape(3 * 5 * 1152, 5 * 1152, 1152)
    A = 2 ** 26
    fwd = lambda Lq=5, Lk=7, H=16, Hkv=4, D=72, k=FAKE + A, kst=kvs, dt=1, lse=None: lib.dsp_attn_general(
        FAKE, k, k, FAKE + 2 * A, lse, 2, 3, Lq, Lk, H, Hkv, D, qs, kst, os_, 0.0, dt, None)
    assert fwd(Hkv=5) == dsp.DSP_ERR_SHAPE          # Hkv must divide H
    assert fwd(Hkv=0) == dsp.DSP_ERR_SHAPE
    assert fwd(Lk=0) == dsp.DSP_ERR_SHAPE           # queries without keys
    assert fwd(Lk=-1) == dsp.DSP_ERR_SHAPE
    assert fwd(k=None) == dsp.DSP_ERR_NULL
    assert fwd(kst=None) == dsp.DSP_ERR_NULL
    assert fwd(kst=_shape(3 * 7 * 288, 7 * 288, 290)) == dsp.DSP_ERR_ALIGN
    assert fwd(lse=FAKE + 3 * A + 2) == dsp.DSP_ERR_ALIGN
    assert fwd(dt=7) == dsp.DSP_ERR_DTYPE
    assert fwd(Lq=0, Lk=0) == dsp.DSP_OK
    bwd = lambda kst=kvs, Lk=7, Hkv=4: lib.dsp_attn_general_bwd(
        FAKE, FAKE + A, FAKE + A, FAKE + 2 * A, FAKE + 2 * A, FAKE + 3 * A, FAKE + 4 * A, FAKE + 5 * A,
        FAKE + 6 * A, FAKE + 7 * A, 2, 3, 5, Lk, 16, Hkv, 72, qs, kst, os_, 0.0, 1, None)
    assert bwd(kst=_shape(0, 0, 288)) == dsp.DSP_ERR_ARG      # broadcast k/v: no single owner of dk rows
    assert bwd(Hkv=3) == dsp.DSP_ERR_SHAPE
    assert bwd(Lk=0) == dsp.DSP_ERR_SHAPE


def test_layernorm_validation(lib):
    f = lambda x=FAKE, xd=1, y=FAKE2, yd=1, rows=4, C=8, eps=1e-6: lib.dsp_layernorm(
        x, xd, y, yd, rows, C, eps, None)
    assert f(x=None) == dsp.DSP_ERR_NULL
    assert f(xd=3) == dsp.DSP_ERR_DTYPE
    assert f(C=0) == dsp.DSP_ERR_SHAPE
    assert f(rows=-2) == dsp.DSP_ERR_SHAPE
    assert f(eps=-1.0) == dsp.DSP_ERR_ARG
    assert f(eps=float("inf")) == dsp.DSP_ERR_ARG
    assert f(y=FAKE + 4) == dsp.DSP_ERR_ARG
    assert f(rows=0) == dsp.DSP_OK


def test_linear_validation(lib):
    f = lambda a=FAKE, w=FAKE2, b=None, r=None, o=0x40000000, M=4, N=8, K=16, epi=0, dt=1: \
        lib.dsp_linear(a, w, b, r, o, M, N, K, epi, dt, None)
    assert f(a=None) == dsp.DSP_ERR_NULL
    assert f(epi=2) == dsp.DSP_ERR_NULL                    # residual required
    assert f(epi=9) == dsp.DSP_ERR_ARG
    assert f(epi=5) == dsp.DSP_ERR_ARG                      # one past DSP_EPI_RELU
    assert f(dt=9) == dsp.DSP_ERR_DTYPE
    assert f(N=0) == dsp.DSP_ERR_SHAPE
    assert f(K=12) == dsp.DSP_ERR_ALIGN                    # bf16 needs K % 8 == 0
    assert f(a=MIS) == dsp.DSP_ERR_ALIGN
    assert f(o=FAKE + 8) == dsp.DSP_ERR_ARG                # out overlaps a
    assert f(M=0) == dsp.DSP_OK


def test_block_validation_and_workspace(lib):
    B, T, S, C, H, F = 1, 4, 16, 64, 4, 256
    need = lib.dsp_st_block_workspace_bytes(B, T, S, C, H, F, 1)
    tokens = B * T * S
    up = lambda v: (v + 255) // 256 * 256
    assert need == up(tokens * C * 2) + up(tokens * 3 * C * 2) + up(tokens * C * 2) + \
        up(tokens * F * 2) + up(tokens * C * 4)
    assert lib.dsp_st_block_workspace_bytes(B, T, S, C, 5, F, 1) == 0     # C % H != 0
    w = dsp.BlockWeights(wqkv_s=FAKE, wo_s=FAKE, wqkv_t=FAKE, wo_t=FAKE, w1=FAKE, w2=FAKE)
    f = lambda x=0x100000, y=0x200000, wp=ctypes.byref(w), ws=0x40000000, wsb=need, flags=0, \
        dt=1, eps=1e-6, F_=F: lib.dsp_st_block_forward(x, y, wp, ws, wsb, B, T, S, C, H, F_, eps,
                                                     flags, dt, None)
    assert f(x=None) == dsp.DSP_ERR_NULL
    assert f(wp=None) == dsp.DSP_ERR_NULL
    assert f(ws=None) == dsp.DSP_ERR_WORKSPACE
    assert f(wsb=need - 1) == dsp.DSP_ERR_WORKSPACE
    assert f(ws=0x40000010) == dsp.DSP_ERR_ALIGN
    assert f(flags=16) == dsp.DSP_ERR_ARG                   # unknown flag bit
    assert f(dt=4) == dsp.DSP_ERR_DTYPE
    assert f(eps=-1.0) == dsp.DSP_ERR_ARG
    assert f(F_=0) == dsp.DSP_ERR_SHAPE                     # the MLP needs F >= 1
    assert f(y=0x100000 + 64) == dsp.DSP_ERR_ARG            # x and y overlap
    w2 = dsp.BlockWeights(wqkv_s=FAKE, wo_s=FAKE, wqkv_t=FAKE, wo_t=None)
    assert f(wp=ctypes.byref(w2)) == dsp.DSP_ERR_NULL


def test_binding_rejects_host_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 2, 2, 8), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        dsp.dsp_switch(x, 1, 2, 1)


def test_probe_mfma_validation(lib):
    need = lib.dsp_probe_mfma_workspace_bytes()
    assert need == 2048 * 256 * 4
    assert lib.dsp_probe_mfma_flops(10) == 2048 * 4 * 10 * 8 * 2.0 * 32 * 32 * 16
    assert lib.dsp_probe_mfma_flops(0) == 0.0
    assert lib.dsp_probe_mfma(FAKE, need, 0, None) == dsp.DSP_ERR_ARG
    assert lib.dsp_probe_mfma(None, need, 10, None) == dsp.DSP_ERR_NULL
    assert lib.dsp_probe_mfma(FAKE, need - 1, 10, None) == dsp.DSP_ERR_WORKSPACE
    assert lib.dsp_probe_mfma(FAKE + 4, need, 10, None) == dsp.DSP_ERR_ALIGN
