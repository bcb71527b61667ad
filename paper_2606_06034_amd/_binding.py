"""ctypes marshalling for libgdninv.so (see include/gdninv.h for the contract)."""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgdninv.so")

GDN_F32, GDN_BF16, GDN_I8 = 0, 1, 2
GDN_INT_PLAIN = 1  # integer inverses: the unit diagonal inside the codes

_c_int, _c_i64, _vp = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p

# name -> argtypes (all return int unless noted)
_SIGS = {
    "gdn_abi_version": [],
    "gdn_status_string": [_c_int],
    "gdn_default_order": [_c_int, ctypes.POINTER(_c_int), ctypes.POINTER(_c_int)],
    "gdn_build_A": [_vp, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_chunk_inverse_neumann": [_vp, _vp, _c_i64, _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_chunk_inverse_fwdsub": [_vp, _vp, _c_i64, _c_int, _c_int, _vp],
    "gdn_chunk_inverse_blockwise": [_vp, _vp, _c_i64, _c_int, _c_int, _vp],
    "gdn_wy_apply": [_vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                     _c_int, _vp],
    "gdn_chunk_wy_fused": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int, _c_int,
                           _c_int, _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_chunk_wy_fused_blockwise": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int,
                                     _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_quantize_tiles_i8": [_vp, _vp, _vp, _c_i64, _c_int, _vp],
    "gdn_chunk_inverse_neumann_i8": [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _c_int, _c_int,
                                     _c_int, _vp],
    "gdn_chunk_inverse_neumann_i8_fused": [_vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int,
                                           _c_int, _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_quantize_tiles_i16": [_vp, _vp, _vp, _c_i64, _c_int, _vp],
    "gdn_chunk_inverse_neumann_i16": [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _c_int, _c_int,
                                      _c_int, _vp],
    "gdn_chunk_inverse_fwdsub_i16": [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _vp],
    "gdn_chunk_inverse_fwdsub_i8": [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _vp],
    "gdn_chunk_inverse_neumann_i16_fused": [_vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int,
                                            _c_int, _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_chunk_forward": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _c_int,
                          _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, ctypes.c_float,
                          _c_int, _vp],
    "gdn_chunk_forward_noalloc": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _c_int,
                                  _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                  ctypes.c_float, _c_int, _vp],
    "gdn_chunk_forward_varlen": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _vp, _vp,
                                 _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                 _c_int, _c_int, ctypes.c_float, _c_int, _vp],
    "gdn_chunk_forward_workspace": [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                    ctypes.POINTER(_c_i64)],
    "gdn_chunk_wy_fused_varlen": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int,
                                  _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                  _c_int, _vp],
    "gdn_chunk_forward_prepare": [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _c_int, _c_int,
                                  _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _vp],
    "gdn_chunk_forward_state": [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_int, _c_int, _c_int,
                                _c_int, _c_int, _c_int, ctypes.c_float, _c_int, _vp],
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python paper_2606_06034_amd/csrc/build.py`")
    L = ctypes.CDLL(LIB_PATH)
    for name, args in _SIGS.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name == "gdn_status_string" else _c_int
    return L


lib = _load()


def abi_symbols():
    return list(_SIGS)


class GdnError(RuntimeError):
    def __init__(self, fn: str, code: int):
        self.code = code
        super().__init__(f"{fn}: {code} ({lib.gdn_status_string(code).decode()})")


def _check(fn: str, code: int):
    if code != 0:
        raise GdnError(fn, code)


def gdn_abi_version() -> int:
    return lib.gdn_abi_version()


def gdn_status_string(code: int) -> str:
    return lib.gdn_status_string(code).decode()


def gdn_default_order(C: int) -> Tuple[int, int]:
    n, s = _c_int(), _c_int()
    _check("gdn_default_order", lib.gdn_default_order(C, ctypes.byref(n), ctypes.byref(s)))
    return n.value, s.value


# ---------------------------------------------------------------------------

_FDT = {torch.float32: GDN_F32, torch.bfloat16: GDN_BF16}
_TDT = {GDN_F32: torch.float32, GDN_BF16: torch.bfloat16}


def _dev(t: torch.Tensor, name: str, dtype=None, numel: Optional[int] = None) -> int:
    """Device pointer of a contiguous tensor, after checking its dtype and
    element count (the C ABI takes sizes from the shape arguments alone)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements (got {t.numel()})")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    return t.data_ptr()


def _fdtype(t: torch.Tensor, name: str) -> int:
    if t.dtype not in _FDT:
        raise TypeError(f"{name}: dtype {t.dtype} not supported (float32 or bfloat16)")
    return _FDT[t.dtype]


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _tiles(A: torch.Tensor) -> Tuple[int, int]:
    if A.dim() < 2 or A.shape[-1] != A.shape[-2]:
        raise ValueError("tile tensor must end in (C, C)")
    C = A.shape[-1]
    return A.numel() // (C * C), C


def gdn_build_A(K: torch.Tensor, beta: torch.Tensor, g: torch.Tensor, C: int,
                a_dtype: Optional[torch.dtype] = None, A: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """A [B, H, L/C, C, C] from K [B, L, H, dk], beta, g [B, L, H] (fp32)."""
    B, L, H, dk = K.shape
    kdt = _fdtype(K, "K")
    adt = _FDT[a_dtype] if a_dtype is not None else (_fdtype(A, "A") if A is not None else kdt)
    if A is None:
        A = torch.empty((B, H, L // C if C else 0, C, C), dtype=_TDT[adt], device=K.device)
    tok = B * L * H
    _check("gdn_build_A", lib.gdn_build_A(
        _dev(K, "K"), _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok),
        _dev(A, "A", _TDT[adt], B * H * (L // C if C else 0) * C * C), B, L, H, dk, C, kdt, adt,
        _stream(stream)))
    return A


def gdn_chunk_inverse_neumann(A: torch.Tensor, N: int, S: int, Tinv: Optional[torch.Tensor] = None,
                              stream=None) -> torch.Tensor:
    """T_hat(N, S) of every C x C tile of A (same shape and dtype)."""
    n, C = _tiles(A)
    dt = _fdtype(A, "A")
    if Tinv is None:
        Tinv = torch.empty_like(A)
    _check("gdn_chunk_inverse_neumann", lib.gdn_chunk_inverse_neumann(
        _dev(A, "A"), _dev(Tinv, "Tinv", A.dtype, A.numel()), n, C, N, S, dt, _stream(stream)))
    return Tinv


def gdn_chunk_inverse_fwdsub(A: torch.Tensor, Tinv: Optional[torch.Tensor] = None,
                             stream=None) -> torch.Tensor:
    """Exact (I + A)^-1 of every tile by forward substitution."""
    n, C = _tiles(A)
    dt = _fdtype(A, "A")
    if Tinv is None:
        Tinv = torch.empty_like(A)
    _check("gdn_chunk_inverse_fwdsub", lib.gdn_chunk_inverse_fwdsub(
        _dev(A, "A"), _dev(Tinv, "Tinv", A.dtype, A.numel()), n, C, dt, _stream(stream)))
    return Tinv


def gdn_chunk_inverse_blockwise(A: torch.Tensor, Tinv: Optional[torch.Tensor] = None,
                                stream=None) -> torch.Tensor:
    """Exact (I + A)^-1 of every tile by 16 x 16 block recursion (products only)."""
    n, C = _tiles(A)
    dt = _fdtype(A, "A")
    if Tinv is None:
        Tinv = torch.empty_like(A)
    _check("gdn_chunk_inverse_blockwise", lib.gdn_chunk_inverse_blockwise(
        _dev(A, "A"), _dev(Tinv, "Tinv", A.dtype, A.numel()), n, C, dt, _stream(stream)))
    return Tinv


def gdn_wy_apply(Tinv: torch.Tensor, K: torch.Tensor, V: torch.Tensor, beta: torch.Tensor, C: int,
                 W: Optional[torch.Tensor] = None, U: Optional[torch.Tensor] = None,
                 stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """W = T diag(beta) K, U = T diag(beta) V per chunk."""
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    W = torch.empty_like(K) if W is None else W
    U = torch.empty_like(V) if U is None else U
    tok = B * L * H
    _check("gdn_wy_apply", lib.gdn_wy_apply(
        _dev(Tinv, "Tinv", K.dtype, B * H * (L // C if C else 0) * C * C), _dev(K, "K"),
        _dev(V, "V", K.dtype, tok * dv), _dev(beta, "beta", torch.float32, tok),
        _dev(W, "W", K.dtype, tok * dk), _dev(U, "U", K.dtype, tok * dv),
        B, L, H, dk, dv, C, dt, _stream(stream)))
    return W, U


def gdn_chunk_wy_fused(K: torch.Tensor, V: torch.Tensor, beta: torch.Tensor, g: torch.Tensor,
                       C: int, N: int, S: int, want_T: bool = False,
                       W: Optional[torch.Tensor] = None, U: Optional[torch.Tensor] = None,
                       Tinv: Optional[torch.Tensor] = None, stream=None):
    """Fused build A -> T_hat(N, S) -> (W, U[, Tinv])."""
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    W = torch.empty_like(K) if W is None else W
    U = torch.empty_like(V) if U is None else U
    if want_T and Tinv is None:
        Tinv = torch.empty((B, H, L // C, C, C), dtype=K.dtype, device=K.device)
    tok = B * L * H
    tp = (_dev(Tinv, "Tinv", K.dtype, B * H * (L // C if C else 0) * C * C)
          if Tinv is not None else None)
    _check("gdn_chunk_wy_fused", lib.gdn_chunk_wy_fused(
        _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv), _dev(beta, "beta", torch.float32, tok),
        _dev(g, "g", torch.float32, tok), _dev(W, "W", K.dtype, tok * dk),
        _dev(U, "U", K.dtype, tok * dv), tp, B, L, H, dk, dv, C, N, S, dt, _stream(stream)))
    return (W, U, Tinv) if Tinv is not None else (W, U)


def gdn_chunk_wy_fused_blockwise(K: torch.Tensor, V: torch.Tensor, beta: torch.Tensor,
                                 g: torch.Tensor, C: int, want_T: bool = False,
                                 W: Optional[torch.Tensor] = None, U: Optional[torch.Tensor] = None,
                                 Tinv: Optional[torch.Tensor] = None, stream=None):
    """Fused build A -> exact inverse (block-wise) -> (W, U[, Tinv])."""
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    W = torch.empty_like(K) if W is None else W
    U = torch.empty_like(V) if U is None else U
    if want_T and Tinv is None:
        Tinv = torch.empty((B, H, L // C, C, C), dtype=K.dtype, device=K.device)
    tok = B * L * H
    tp = (_dev(Tinv, "Tinv", K.dtype, B * H * (L // C if C else 0) * C * C)
          if Tinv is not None else None)
    _check("gdn_chunk_wy_fused_blockwise", lib.gdn_chunk_wy_fused_blockwise(
        _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv), _dev(beta, "beta", torch.float32, tok),
        _dev(g, "g", torch.float32, tok), _dev(W, "W", K.dtype, tok * dk),
        _dev(U, "U", K.dtype, tok * dv), tp, B, L, H, dk, dv, C, dt, _stream(stream)))
    return (W, U, Tinv) if Tinv is not None else (W, U)


def _nexp(C: int) -> int:
    """Exponents per tile of the integer paths (C = 128: blocks 11, 21, 22)."""
    return 3 if C == 128 else 1


def gdn_quantize_tiles_i8(A: torch.Tensor, Aq: Optional[torch.Tensor] = None,
                          eA: Optional[torch.Tensor] = None, stream=None):
    """(Aq int8 tiles, eA int32 per tile) with A ~ Aq * 2^eA; C = 128:
    eA [n, 3], one exponent per block (11, 21, 22)."""
    n, C = _tiles(A)
    ne = _nexp(C)
    Aq = torch.empty(A.shape, dtype=torch.int8, device=A.device) if Aq is None else Aq
    if eA is None:
        eA = torch.empty((n, 3) if ne == 3 else n, dtype=torch.int32, device=A.device)
    _check("gdn_quantize_tiles_i8", lib.gdn_quantize_tiles_i8(
        _dev(A, "A", torch.float32), _dev(Aq, "Aq", torch.int8, A.numel()),
        _dev(eA, "eA", torch.int32, n * ne), n, C, _stream(stream)))
    return Aq, eA


def gdn_chunk_inverse_neumann_i8(Aq: torch.Tensor, eA: torch.Tensor, N: int, S: int,
                                 want_deq: bool = False, plain: bool = False,
                                 Tq: Optional[torch.Tensor] = None,
                                 eT: Optional[torch.Tensor] = None,
                                 Tdeq: Optional[torch.Tensor] = None, stream=None):
    """(Tq int8, eT int32[, Tdeq fp32]) with T_hat = I + Tq * 2^eT (plain:
    T_hat = Tq * 2^eT, the diagonal in the codes; GDN_INT_PLAIN); C = 128:
    block-wise, eA and eT [n, 3] (blocks 11, 21, 22)."""
    n, C = _tiles(Aq)
    Tq = torch.empty_like(Aq) if Tq is None else Tq
    eT = torch.empty_like(eA) if eT is None else eT
    Td = Tdeq
    if want_deq and Td is None:
        Td = torch.empty(Aq.shape, dtype=torch.float32, device=Aq.device)
    ne = _nexp(C)
    _check("gdn_chunk_inverse_neumann_i8", lib.gdn_chunk_inverse_neumann_i8(
        _dev(Aq, "Aq", torch.int8), _dev(eA, "eA", torch.int32, n * ne),
        _dev(Tq, "Tq", torch.int8, Aq.numel()), _dev(eT, "eT", torch.int32, n * ne),
        _dev(Td, "Tdeq", torch.float32, Aq.numel()) if Td is not None else None, n, C, N, S,
        GDN_INT_PLAIN if plain else 0, _stream(stream)))
    return (Tq, eT, Td) if Td is not None else (Tq, eT)


def gdn_chunk_inverse_neumann_i8_fused(K: torch.Tensor, beta: torch.Tensor, g: torch.Tensor,
                                       C: int, N: int, S: int, want_deq: bool = False,
                                       Tq: Optional[torch.Tensor] = None,
                                       eT: Optional[torch.Tensor] = None,
                                       Tdeq: Optional[torch.Tensor] = None, stream=None):
    """K [B, L, H, dk] -> (Tq int8 [B, H, L/C, C, C], eT int32[, Tdeq fp32]):
    build A, quantise and invert in one launch."""
    B, L, H, dk = K.shape
    nc = L // C if C else 0
    shape = (B, H, nc, C, C)
    n = B * H * nc
    Tq = torch.empty(shape, dtype=torch.int8, device=K.device) if Tq is None else Tq
    ne = _nexp(C)
    if eT is None:
        eT = torch.empty((n, 3) if ne == 3 else n, dtype=torch.int32, device=K.device)
    Td = Tdeq
    if want_deq and Td is None:
        Td = torch.empty(shape, dtype=torch.float32, device=K.device)
    tok = B * L * H
    _check("gdn_chunk_inverse_neumann_i8_fused", lib.gdn_chunk_inverse_neumann_i8_fused(
        _dev(K, "K"), _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok),
        _dev(Tq, "Tq", torch.int8, n * C * C), _dev(eT, "eT", torch.int32, n * ne),
        _dev(Td, "Tdeq", torch.float32, n * C * C) if Td is not None else None,
        B, L, H, dk, C, N, S, _fdtype(K, "K"), _stream(stream)))
    return (Tq, eT, Td) if Td is not None else (Tq, eT)


def gdn_quantize_tiles_i16(A: torch.Tensor, Aq: Optional[torch.Tensor] = None,
                           eA: Optional[torch.Tensor] = None, stream=None):
    """(Aq int16 tiles, eA int32 per tile) with A ~ Aq * 2^eA; C = 128:
    eA [n, 3], one exponent per block (11, 21, 22)."""
    n, C = _tiles(A)
    ne = _nexp(C)
    Aq = torch.empty(A.shape, dtype=torch.int16, device=A.device) if Aq is None else Aq
    if eA is None:
        eA = torch.empty((n, 3) if ne == 3 else n, dtype=torch.int32, device=A.device)
    _check("gdn_quantize_tiles_i16", lib.gdn_quantize_tiles_i16(
        _dev(A, "A", torch.float32), _dev(Aq, "Aq", torch.int16, A.numel()),
        _dev(eA, "eA", torch.int32, n * ne), n, C, _stream(stream)))
    return Aq, eA


def gdn_chunk_inverse_neumann_i16(Aq: torch.Tensor, eA: torch.Tensor, N: int, S: int,
                                  want_deq: bool = False, plain: bool = False,
                                  Tq: Optional[torch.Tensor] = None,
                                  eT: Optional[torch.Tensor] = None,
                                  Tdeq: Optional[torch.Tensor] = None, stream=None):
    """(Tq int16, eT int32[, Tdeq fp32]) with T_hat = I + Tq * 2^eT (plain:
    T_hat = Tq * 2^eT, the diagonal in the codes; GDN_INT_PLAIN); C = 128:
    block-wise, eA and eT [n, 3] (blocks 11, 21, 22)."""
    n, C = _tiles(Aq)
    Tq = torch.empty_like(Aq) if Tq is None else Tq
    eT = torch.empty_like(eA) if eT is None else eT
    Td = Tdeq
    if want_deq and Td is None:
        Td = torch.empty(Aq.shape, dtype=torch.float32, device=Aq.device)
    ne = _nexp(C)
    _check("gdn_chunk_inverse_neumann_i16", lib.gdn_chunk_inverse_neumann_i16(
        _dev(Aq, "Aq", torch.int16), _dev(eA, "eA", torch.int32, n * ne),
        _dev(Tq, "Tq", torch.int16, Aq.numel()), _dev(eT, "eT", torch.int32, n * ne),
        _dev(Td, "Tdeq", torch.float32, Aq.numel()) if Td is not None else None, n, C, N, S,
        GDN_INT_PLAIN if plain else 0, _stream(stream)))
    return (Tq, eT, Td) if Td is not None else (Tq, eT)


def gdn_chunk_inverse_fwdsub_i16(Aq: torch.Tensor, eA: torch.Tensor, want_deq: bool = False,
                                 Tq: Optional[torch.Tensor] = None,
                                 eT: Optional[torch.Tensor] = None,
                                 Tdeq: Optional[torch.Tensor] = None, stream=None):
    """(Tq int16, eT int32[, Tdeq fp32]): integer forward substitution,
    T = I + Tq * 2^eT."""
    n, C = _tiles(Aq)
    Tq = torch.empty_like(Aq) if Tq is None else Tq
    eT = torch.empty_like(eA) if eT is None else eT
    Td = Tdeq
    if want_deq and Td is None:
        Td = torch.empty(Aq.shape, dtype=torch.float32, device=Aq.device)
    _check("gdn_chunk_inverse_fwdsub_i16", lib.gdn_chunk_inverse_fwdsub_i16(
        _dev(Aq, "Aq", torch.int16), _dev(eA, "eA", torch.int32, n),
        _dev(Tq, "Tq", torch.int16, Aq.numel()), _dev(eT, "eT", torch.int32, n),
        _dev(Td, "Tdeq", torch.float32, Aq.numel()) if Td is not None else None, n, C,
        _stream(stream)))
    return (Tq, eT, Td) if Td is not None else (Tq, eT)


def gdn_chunk_inverse_fwdsub_i8(Aq: torch.Tensor, eA: torch.Tensor, want_deq: bool = False,
                                Tq: Optional[torch.Tensor] = None,
                                eT: Optional[torch.Tensor] = None,
                                Tdeq: Optional[torch.Tensor] = None, stream=None):
    """(Tq int8, eT int32[, Tdeq fp32]): integer forward substitution,
    T = I + Tq * 2^eT."""
    n, C = _tiles(Aq)
    Tq = torch.empty_like(Aq) if Tq is None else Tq
    eT = torch.empty_like(eA) if eT is None else eT
    Td = Tdeq
    if want_deq and Td is None:
        Td = torch.empty(Aq.shape, dtype=torch.float32, device=Aq.device)
    _check("gdn_chunk_inverse_fwdsub_i8", lib.gdn_chunk_inverse_fwdsub_i8(
        _dev(Aq, "Aq", torch.int8), _dev(eA, "eA", torch.int32, n),
        _dev(Tq, "Tq", torch.int8, Aq.numel()), _dev(eT, "eT", torch.int32, n),
        _dev(Td, "Tdeq", torch.float32, Aq.numel()) if Td is not None else None, n, C,
        _stream(stream)))
    return (Tq, eT, Td) if Td is not None else (Tq, eT)


def gdn_chunk_inverse_neumann_i16_fused(K: torch.Tensor, beta: torch.Tensor, g: torch.Tensor,
                                        C: int, N: int, S: int, want_deq: bool = False,
                                        Tq: Optional[torch.Tensor] = None,
                                        eT: Optional[torch.Tensor] = None,
                                        Tdeq: Optional[torch.Tensor] = None, stream=None):
    """K [B, L, H, dk] -> (Tq int16 [B, H, L/C, C, C], eT int32[, Tdeq fp32]):
    build A, quantise and invert in one launch."""
    B, L, H, dk = K.shape
    nc = L // C if C else 0
    shape = (B, H, nc, C, C)
    n = B * H * nc
    Tq = torch.empty(shape, dtype=torch.int16, device=K.device) if Tq is None else Tq
    ne = _nexp(C)
    if eT is None:
        eT = torch.empty((n, 3) if ne == 3 else n, dtype=torch.int32, device=K.device)
    Td = Tdeq
    if want_deq and Td is None:
        Td = torch.empty(shape, dtype=torch.float32, device=K.device)
    tok = B * L * H
    _check("gdn_chunk_inverse_neumann_i16_fused", lib.gdn_chunk_inverse_neumann_i16_fused(
        _dev(K, "K"), _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok),
        _dev(Tq, "Tq", torch.int16, n * C * C), _dev(eT, "eT", torch.int32, n * ne),
        _dev(Td, "Tdeq", torch.float32, n * C * C) if Td is not None else None,
        B, L, H, dk, C, N, S, _fdtype(K, "K"), _stream(stream)))
    return (Tq, eT, Td) if Td is not None else (Tq, eT)


def gdn_chunk_forward_workspace(B: int, L: int, H: int, dk: int, dv: int, C: int,
                                dtype: torch.dtype) -> int:
    """Bytes of workspace gdn_chunk_forward needs for these sizes."""
    n = _c_i64()
    _check("gdn_chunk_forward_workspace", lib.gdn_chunk_forward_workspace(
        B, L, H, dk, dv, C, _FDT[dtype], ctypes.byref(n)))
    return n.value


_FWD_MODES = {"neumann": 0, "exact": 1, "int16": 2, "int8": 3}


def _fwd_mode(exact: bool, inverse: Optional[str]) -> int:
    """The inverse mode of the layer forward: T_hat(N, S) ("neumann"), the
    exact inverse ("exact", or exact=True), or T_hat(N, S) on 16- or 8-bit
    codes ("int16", "int8")."""
    if inverse is None:
        return 1 if exact else 0
    if inverse not in _FWD_MODES:
        raise ValueError(f"inverse must be one of {sorted(_FWD_MODES)}")
    return _FWD_MODES[inverse]


def gdn_chunk_forward(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, beta: torch.Tensor,
                      g: torch.Tensor, C: int, S0: Optional[torch.Tensor] = None,
                      N: Optional[int] = None, S: Optional[int] = None, exact: bool = False,
                      scale: Optional[float] = None, want_state: bool = True,
                      O: Optional[torch.Tensor] = None, S_final: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, stream=None,
                      inverse: Optional[str] = None):
    """Chunk-wise Gated DeltaNet forward: (O [B, L, H, dv], S_final [B, H, dk, dv] fp32 or
    None).  N, S default to gdn_default_order(C); scale defaults to dk ** -0.5.  The
    workspace (a byte tensor of gdn_chunk_forward_workspace() bytes) is allocated when
    not given.  inverse: "neumann" (default), "exact" (as exact=True), "int16" or "int8"
    (the integer T_hat(N, S) inside the layer)."""
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    if N is None or S is None:
        dn, ds = gdn_default_order(C) if C in (16, 32, 64, 128) else (0, 0)
        N = dn if N is None else N
        S = ds if S is None else S
    scale = dk ** -0.5 if scale is None else float(scale)
    tok = B * L * H
    O = torch.empty_like(V) if O is None else O
    if want_state and S_final is None:
        S_final = torch.empty((B, H, dk, dv), dtype=torch.float32, device=K.device)
    need = gdn_chunk_forward_workspace(B, L, H, dk, dv, C, K.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=K.device)
    sp = _dev(S0, "S0", torch.float32, B * H * dk * dv) if S0 is not None else None
    fp = _dev(S_final, "S_final", torch.float32, B * H * dk * dv) if S_final is not None else None
    _check("gdn_chunk_forward", lib.gdn_chunk_forward(
        _dev(Q, "Q", K.dtype, tok * dk), _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv),
        _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok), sp,
        _dev(O, "O", K.dtype, tok * dv), fp, _dev(workspace, "workspace"), workspace.numel() *
        workspace.element_size(), B, L, H, dk, dv, C, N, S, _fwd_mode(exact, inverse), scale,
        dt, _stream(stream)))
    return O, S_final


GDN_FORWARD_SCRATCH_BYTES = 128 << 20  # the allocation-free forward's scratch


def gdn_chunk_forward_noalloc(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                              beta: torch.Tensor, g: torch.Tensor, C: int, O: torch.Tensor,
                              S0: Optional[torch.Tensor] = None,
                              S_final: Optional[torch.Tensor] = None, N: Optional[int] = None,
                              S: Optional[int] = None, exact: bool = False,
                              scale: Optional[float] = None, stream=None,
                              inverse: Optional[str] = None):
    """gdn_chunk_forward with the library's device scratch as its workspace:
    the call allocates nothing (O and, when wanted, S_final are the caller's).
    Returns (O, S_final)."""
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    if N is None or S is None:
        dn, ds = gdn_default_order(C) if C in (16, 32, 64, 128) else (0, 0)
        N = dn if N is None else N
        S = ds if S is None else S
    scale = dk ** -0.5 if scale is None else float(scale)
    tok = B * L * H
    sp = _dev(S0, "S0", torch.float32, B * H * dk * dv) if S0 is not None else None
    fp = _dev(S_final, "S_final", torch.float32, B * H * dk * dv) if S_final is not None else None
    _check("gdn_chunk_forward_noalloc", lib.gdn_chunk_forward_noalloc(
        _dev(Q, "Q", K.dtype, tok * dk), _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv),
        _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok), sp,
        _dev(O, "O", K.dtype, tok * dv), fp, B, L, H, dk, dv, C, N, S,
        _fwd_mode(exact, inverse), scale, dt, _stream(stream)))
    return O, S_final


def gdn_chunk_forward_prepare(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                              beta: torch.Tensor, g: torch.Tensor, C: int,
                              workspace: torch.Tensor, N: Optional[int] = None,
                              S: Optional[int] = None, exact: bool = False, stream=None,
                              inverse: Optional[str] = None):
    """First phase of gdn_chunk_forward: the per-chunk factors into `workspace`."""
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    if N is None or S is None:
        dn, ds = gdn_default_order(C) if C in (16, 32, 64, 128) else (0, 0)
        N = dn if N is None else N
        S = ds if S is None else S
    tok = B * L * H
    _check("gdn_chunk_forward_prepare", lib.gdn_chunk_forward_prepare(
        _dev(Q, "Q", K.dtype, tok * dk), _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv),
        _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        B, L, H, dk, dv, C, N, S, _fwd_mode(exact, inverse), dt, _stream(stream)))
    return workspace


def gdn_chunk_forward_state(Q: torch.Tensor, g: torch.Tensor, C: int, workspace: torch.Tensor,
                            dv: int, S0: Optional[torch.Tensor] = None,
                            scale: Optional[float] = None, want_state: bool = True,
                            O: Optional[torch.Tensor] = None,
                            S_final: Optional[torch.Tensor] = None, stream=None):
    """Second phase of gdn_chunk_forward: the state pass over a prepared workspace."""
    B, L, H, dk = Q.shape
    dt = _fdtype(Q, "Q")
    scale = dk ** -0.5 if scale is None else float(scale)
    tok = B * L * H
    O = torch.empty((B, L, H, dv), dtype=Q.dtype, device=Q.device) if O is None else O
    if want_state and S_final is None:
        S_final = torch.empty((B, H, dk, dv), dtype=torch.float32, device=Q.device)
    sp = _dev(S0, "S0", torch.float32, B * H * dk * dv) if S0 is not None else None
    fp = _dev(S_final, "S_final", torch.float32, B * H * dk * dv) if S_final is not None else None
    _check("gdn_chunk_forward_state", lib.gdn_chunk_forward_state(
        _dev(Q, "Q"), _dev(g, "g", torch.float32, tok), sp, _dev(O, "O", Q.dtype, tok * dv), fp,
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        B, L, H, dk, dv, C, scale, dt, _stream(stream)))
    return O, S_final


def gdn_varlen_tables(cu_seqlens, C: int, device="cuda"):
    """Device tables for packed sequences from host-side sequence offsets
    cu_seqlens (list, numpy array or CPU tensor of nseq + 1 ints): returns
    (cu int32 device tensor, chunk offsets int32 device tensor, n_chunks).
    This is host bookkeeping (a prefix sum of ceil(l / C)); nothing of the
    method runs here."""
    cu = [int(x) for x in (cu_seqlens.tolist() if hasattr(cu_seqlens, "tolist") else cu_seqlens)]
    off = [0]
    for s in range(len(cu) - 1):
        off.append(off[-1] + max(0, cu[s + 1] - cu[s] + C - 1) // C)
    dcu = torch.tensor(cu, dtype=torch.int32, device=device)
    doff = torch.tensor(off, dtype=torch.int32, device=device)
    return dcu, doff, off[-1]


def gdn_chunk_wy_fused_varlen(K: torch.Tensor, V: torch.Tensor, beta: torch.Tensor,
                              g: torch.Tensor, tables, C: int, N: Optional[int] = None,
                              S: Optional[int] = None, exact: bool = False, want_T: bool = False,
                              W: Optional[torch.Tensor] = None, U: Optional[torch.Tensor] = None,
                              Tinv: Optional[torch.Tensor] = None, stream=None):
    """Fused build A -> inverse -> (W, U[, Tinv]) over packed sequences;
    tables = gdn_varlen_tables(cu_seqlens, C)."""
    dcu, doff, n_chunks = tables
    B, T, H, dk = K.shape
    if B != 1:
        raise ValueError("packed sequences use B = 1")
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    if N is None or S is None:
        dn, ds = gdn_default_order(C) if C in (16, 32, 64, 128) else (0, 0)
        N = dn if N is None else N
        S = ds if S is None else S
    W = torch.empty_like(K) if W is None else W
    U = torch.empty_like(V) if U is None else U
    if want_T and Tinv is None:
        Tinv = torch.empty((H, n_chunks, C, C), dtype=K.dtype, device=K.device)
    tok = T * H
    nseq = dcu.numel() - 1
    tp = _dev(Tinv, "Tinv", K.dtype, H * n_chunks * C * C) if Tinv is not None else None
    _check("gdn_chunk_wy_fused_varlen", lib.gdn_chunk_wy_fused_varlen(
        _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv), _dev(beta, "beta", torch.float32, tok),
        _dev(g, "g", torch.float32, tok), _dev(W, "W", K.dtype, tok * dk),
        _dev(U, "U", K.dtype, tok * dv), tp, _dev(dcu, "cu_seqlens", torch.int32),
        _dev(doff, "chunk_offsets", torch.int32, nseq + 1), nseq, n_chunks, T, H, dk, dv, C, N, S,
        int(bool(exact)), dt, _stream(stream)))
    return (W, U, Tinv) if Tinv is not None else (W, U)


def gdn_chunk_forward_varlen(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                             beta: torch.Tensor, g: torch.Tensor, tables, C: int,
                             S0: Optional[torch.Tensor] = None, N: Optional[int] = None,
                             S: Optional[int] = None, exact: bool = False,
                             scale: Optional[float] = None, want_state: bool = True,
                             O: Optional[torch.Tensor] = None,
                             S_final: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None, stream=None,
                             inverse: Optional[str] = None):
    """Layer forward over packed sequences: (O [1, T, H, dv], S_final
    [nseq, H, dk, dv] fp32 or None); tables = gdn_varlen_tables(cu_seqlens, C).
    Defaults and inverse modes as gdn_chunk_forward."""
    dcu, doff, n_chunks = tables
    B, T, H, dk = K.shape
    if B != 1:
        raise ValueError("packed sequences use B = 1")
    dv = V.shape[-1]
    dt = _fdtype(K, "K")
    nseq = dcu.numel() - 1
    if N is None or S is None:
        dn, ds = gdn_default_order(C) if C in (16, 32, 64, 128) else (0, 0)
        N = dn if N is None else N
        S = ds if S is None else S
    scale = dk ** -0.5 if scale is None else float(scale)
    tok = T * H
    O = torch.empty_like(V) if O is None else O
    if want_state and S_final is None:
        S_final = torch.empty((nseq, H, dk, dv), dtype=torch.float32, device=K.device)
    need = gdn_chunk_forward_workspace(1, n_chunks * C, H, dk, dv, C, K.dtype) if n_chunks else 0
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=K.device)
    sp = _dev(S0, "S0", torch.float32, nseq * H * dk * dv) if S0 is not None else None
    fp = _dev(S_final, "S_final", torch.float32, nseq * H * dk * dv) if S_final is not None \
        else None
    _check("gdn_chunk_forward_varlen", lib.gdn_chunk_forward_varlen(
        _dev(Q, "Q", K.dtype, tok * dk), _dev(K, "K"), _dev(V, "V", K.dtype, tok * dv),
        _dev(beta, "beta", torch.float32, tok), _dev(g, "g", torch.float32, tok), sp,
        _dev(O, "O", K.dtype, tok * dv), fp, _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _dev(dcu, "cu_seqlens", torch.int32),
        _dev(doff, "chunk_offsets", torch.int32, nseq + 1), nseq, n_chunks, T, H, dk, dv, C, N, S,
        _fwd_mode(exact, inverse), scale, dt, _stream(stream)))
    return O, S_final
