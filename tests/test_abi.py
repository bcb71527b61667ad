"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects bad arguments before anything reaches the GPU.

No call here passes validation with a non-zero amount of work, so no kernel
is launched (there is no GPU in the build container)."""

import os
import re

import pytest

import paper_2606_06034_amd as g

HDR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "gdninv.h")

OK, NULL, SHAPE, PARAM, DTYPE, ALIGN, ALIAS, HIP, UNSUP, WS = 0, -1, -2, -3, -4, -5, -6, -7, -8, -9
P1, P2, P3, P4, P5, P6, P7 = (0x10000 * k for k in range(1, 8))  # aligned fake addresses
BIG = 1 << 40  # far apart so nothing overlaps unless intended


def _declared():
    src = open(HDR).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(gdn_\w+)\s*\(", src, re.M)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) == 25
    for n in names:
        assert hasattr(g.lib, n), n
    assert sorted(g.abi_symbols()) == names


def test_version_and_status_strings():
    assert g.gdn_abi_version() == 3
    for code in (OK, NULL, SHAPE, PARAM, DTYPE, ALIGN, ALIAS, HIP, UNSUP, WS, 12345):
        assert isinstance(g.gdn_status_string(code), str) and g.gdn_status_string(code)


def test_default_order():
    assert g.gdn_default_order(16) == (3, 2)
    assert g.gdn_default_order(32) == (3, 4)
    assert g.gdn_default_order(64) == (3, 8)
    assert g.gdn_default_order(128) == (3, 8)
    with pytest.raises(g.GdnError):
        g.gdn_default_order(48)
    assert g.lib.gdn_default_order(64, None, None) == NULL


L = g.lib


def test_neumann_validation():
    f = L.gdn_chunk_inverse_neumann
    assert f(P1, BIG, 4, 48, 3, 8, 0, None) == SHAPE
    assert f(P1, BIG, -1, 64, 3, 8, 0, None) == SHAPE
    assert f(P1, BIG, 1 << 31, 64, 3, 8, 0, None) == SHAPE
    assert f(P1, BIG, 4, 64, 64, 8, 0, None) == PARAM
    assert f(P1, BIG, 4, 64, 3, -1, 0, None) == PARAM
    assert f(P1, BIG, 4, 128, 3, 64, 0, None) == PARAM  # 64-blocks at C = 128
    assert f(P1, BIG, 4, 64, 3, 8, 2, None) == DTYPE
    assert f(P1, BIG, 4, 64, 3, 8, 7, None) == DTYPE
    assert f(None, BIG, 4, 64, 3, 8, 0, None) == NULL
    assert f(P1, None, 4, 64, 3, 8, 0, None) == NULL
    assert f(P1 + 4, BIG, 4, 64, 3, 8, 0, None) == ALIGN
    assert f(P1, P1 + 64, 4, 64, 3, 8, 0, None) == ALIAS
    assert f(P1, P1, 4, 64, 3, 8, 1, None) == ALIAS
    # zero tiles: a no-op, even with NULL pointers
    assert f(None, None, 0, 64, 3, 8, 0, None) == OK


def test_fwdsub_validation():
    f = L.gdn_chunk_inverse_fwdsub
    assert f(P1, BIG, 4, 8, 0, None) == SHAPE
    assert f(P1, BIG, 4, 64, 3, None) == DTYPE
    assert f(None, BIG, 4, 64, 0, None) == NULL
    assert f(P1, BIG + 8, 4, 64, 0, None) == ALIGN
    assert f(P1, P1 + 16, 4, 64, 0, None) == ALIAS
    assert f(None, None, 0, 32, 1, None) == OK


def test_build_A_validation():
    f = L.gdn_build_A
    # K, beta, g, A, B, L, H, dk, C, kdt, adt, stream
    assert f(P1, P2, P3, BIG, 1, 100, 4, 128, 64, 1, 1, None) == SHAPE  # L % C
    assert f(P1, P2, P3, BIG, 1, 128, 4, 96, 64, 1, 1, None) == SHAPE  # dk
    assert f(P1, P2, P3, BIG, -1, 128, 4, 128, 64, 1, 1, None) == SHAPE
    assert f(P1, P2, P3, BIG, 1, 128, 4, 128, 64, 2, 1, None) == DTYPE
    assert f(P1, None, P3, BIG, 1, 128, 4, 128, 64, 1, 1, None) == NULL
    assert f(P1, P2 + 8, P3, BIG, 1, 128, 4, 128, 64, 1, 1, None) == ALIGN
    # A overlapping K
    assert f(BIG, P2, P3, BIG + 4096, 1, 128, 4, 128, 64, 1, 1, None) == ALIAS
    assert f(None, None, None, None, 0, 128, 4, 128, 64, 1, 1, None) == OK
    assert f(None, None, None, None, 1, 0, 4, 128, 64, 1, 1, None) == OK


def test_wy_validation():
    f = L.gdn_wy_apply
    # T, K, V, beta, W, U, B, L, H, dk, dv, C, dtype, stream
    args = [P1, P2, P3, P4, BIG, 2 * BIG, 1, 128, 4, 128, 128, 64, 1, None]
    bad = list(args); bad[10] = 32
    assert f(*bad) == SHAPE
    bad = list(args); bad[12] = 5
    assert f(*bad) == DTYPE
    bad = list(args); bad[4] = None
    assert f(*bad) == NULL
    bad = list(args); bad[5] = BIG  # W == U
    assert f(*bad) == ALIAS
    bad = list(args); bad[4] = P2  # W == K
    assert f(*bad) == ALIAS


def test_fused_validation():
    f = L.gdn_chunk_wy_fused
    # K, V, beta, g, W, U, T, B, L, H, dk, dv, C, N, S, dtype, stream
    base = [P1, P2, P3, P4, BIG, 2 * BIG, None, 1, 128, 4, 128, 128, 64, 3, 8, 1, None]
    bad = list(base); bad[13] = 64
    assert f(*bad) == PARAM
    bad = list(base); bad[8] = 96
    assert f(*bad) == SHAPE
    bad = list(base); bad[3] = None
    assert f(*bad) == NULL
    bad = list(base); bad[6] = P1  # Tinv over K
    assert f(*bad) == ALIAS
    bad = list(base); bad[6] = 3 * BIG + 4
    assert f(*bad) == ALIGN
    zero = list(base); zero[7] = 0
    zero[0] = zero[1] = None
    assert f(*zero) == OK


def test_fused_blockwise_validation():
    f = L.gdn_chunk_wy_fused_blockwise
    # K, V, beta, g, W, U, Tinv, B, L, H, dk, dv, C, dtype, stream
    base = [P1, BIG, 2 * BIG, 3 * BIG, 4 * BIG, 5 * BIG, None, 1, 256, 2, 128, 128, 64, 1, None]
    bad = list(base); bad[12] = 48
    assert f(*bad) == SHAPE
    bad = list(base); bad[13] = 2
    assert f(*bad) == DTYPE
    bad = list(base); bad[4] = None
    assert f(*bad) == NULL
    bad = list(base); bad[4] = P1 + 512
    assert f(*bad) == ALIAS
    zero = list(base); zero[7] = 0
    assert f(*zero) == OK


@pytest.mark.parametrize("w", ["i8", "i16"])
def test_int_validation(w):
    q = getattr(L, "gdn_quantize_tiles_" + w)
    assert q(P1, BIG, 2 * BIG, 4, 48, None) == SHAPE
    # C = 128: three exponents per tile (48 bytes for 4 tiles)
    assert q(BIG, 2 * BIG, BIG + 4 * 128 * 128 * 4 - 16, 4, 128, None) == ALIAS
    assert q(P1, None, 2 * BIG, 4, 64, None) == NULL
    assert q(P1, P1, 2 * BIG, 4, 64, None) == ALIAS
    assert q(None, None, None, 0, 64, None) == OK
    n = getattr(L, "gdn_chunk_inverse_neumann_" + w)
    # Aq, eA, Tq, eT, Tdeq, n_tiles, C, N, S, flags, stream
    assert n(P1, P2, BIG, 2 * BIG, None, 4, 64, 64, 8, 0, None) == PARAM
    assert n(P1, P2, BIG, None, None, 4, 64, 3, 8, 0, None) == NULL
    assert n(P1, P2, P1, 2 * BIG, None, 4, 64, 3, 8, 0, None) == ALIAS
    assert n(None, None, None, None, None, 0, 64, 3, 8, 0, None) == OK
    # flags: GDN_INT_PLAIN (1) only, and not at C = 128
    assert n(P1, P2, BIG, 2 * BIG, None, 4, 64, 3, 8, 2, None) == PARAM
    assert n(P1, P2, BIG, 2 * BIG, None, 4, 128, 3, 8, 1, None) == UNSUP
    assert n(None, None, None, None, None, 0, 64, 3, 8, 1, None) == OK
    assert g.GDN_INT_PLAIN == 1
    # C = 128: orders up to 63 (64-blocks); eA, eT hold 3 exponents per tile
    assert n(P1, 2 * BIG, 3 * BIG, 4 * BIG, None, 4, 128, 64, 8, 0, None) == PARAM
    assert n(P1, 2 * BIG, 3 * BIG, 2 * BIG + 16, None, 4, 128, 63, 8, 0, None) == ALIAS
    assert n(None, None, None, None, None, 0, 128, 3, 8, 0, None) == OK
    if w == "i16":
        # Tq starting one int8 extent (4 tiles of 64 x 64 bytes) past Aq lies
        # inside the int16 codes
        assert n(P1, P2, P1 + 4 * 64 * 64, 2 * BIG, None, 4, 64, 3, 8, 0, None) == ALIAS


def test_blockwise_validation():
    f = L.gdn_chunk_inverse_blockwise
    assert f(P1, P2, 4, 48, 1, None) == SHAPE
    assert f(P1, P2, -1, 64, 1, None) == SHAPE
    assert f(P1, P2, 4, 64, 2, None) == DTYPE
    assert f(None, P2, 4, 64, 1, None) == NULL
    assert f(P1, P1 + 256, 4, 64, 1, None) == ALIAS
    assert f(P1 + 8, P2, 4, 64, 1, None) == ALIGN
    assert f(None, None, 0, 64, 1, None) == OK


@pytest.mark.parametrize("w", ["i8", "i16"])
def test_fwdsub_int_validation(w):
    f = getattr(L, "gdn_chunk_inverse_fwdsub_" + w)
    assert f(P1, P2, BIG, 2 * BIG, None, 4, 128, None) == SHAPE
    assert f(P1, P2, BIG, 2 * BIG, None, -1, 64, None) == SHAPE
    assert f(P1, P2, BIG, None, None, 4, 64, None) == NULL
    assert f(P1, P2, P1 + 4 * 64 * 64 - 16, 2 * BIG, None, 4, 64, None) == ALIAS
    assert f(P1, P2, BIG, 2 * BIG, BIG + 1024, 4, 64, None) == ALIAS
    assert f(P1, P2, BIG + 2, 2 * BIG, None, 4, 64, None) == ALIGN
    assert f(None, None, None, None, None, 0, 64, None) == OK


@pytest.mark.parametrize("w", ["i8", "i16"])
def test_int_fused_validation(w):
    f = getattr(L, "gdn_chunk_inverse_neumann_%s_fused" % w)
    # K, beta, g, Tq, eT, Tdeq, B, L, H, dk, C, N, S, k_dtype, stream
    base = [P1, BIG, 2 * BIG, 3 * BIG, 4 * BIG, None, 1, 256, 2, 128, 64, 3, 8, 1, None]

    def call(**kw):
        a = list(base)
        for k, v in kw.items():
            a[["K", "beta", "g", "Tq", "eT", "Tdeq", "B", "L", "H", "dk", "C", "N", "S",
               "kdt"].index(k)] = v
        return f(*a)

    # C = 128 (block-wise): orders up to 63, L % 128 == 0, three exponents per tile
    assert call(C=128, N=64) == PARAM
    assert call(C=128, L=192) == SHAPE
    assert call(C=128, Tdeq=4 * BIG + 32) == ALIAS  # inside eT's 4 tiles x 3 exponents
    assert call(dk=96) == SHAPE
    assert call(L=250) == SHAPE       # L % C != 0
    assert call(N=64) == PARAM
    assert call(kdt=2) == DTYPE
    assert call(Tq=None) == NULL
    assert call(eT=None) == NULL
    assert call(Tq=P1 + 1024) == ALIAS
    assert call(Tdeq=4 * BIG + 16) == ALIAS
    assert call(eT=P1 + 8) == ALIGN
    assert call(B=0, K=None, beta=None, g=None, Tq=None, eT=None) == OK


def test_forward_workspace_size():
    import ctypes
    n = ctypes.c_int64()
    f = L.gdn_chunk_forward_workspace
    assert f(1, 8192, 16, 128, 128, 64, 1, ctypes.byref(n)) == OK
    # per 64-token chunk: W 64x128, U 64x128, K^T 128 x 64, P 6 pair slots of 512
    assert n.value == 2048 * (8192 + 8192 + 8192 + 6 * 512) * 2
    assert f(1, 64, 1, 64, 64, 16, 0, ctypes.byref(n)) == OK
    # C = 16: K^T pairs carry a zero half
    assert n.value == 4 * (1 * 2 * 512 + 4 * 256 + 4 * 512 + 512) * 4
    assert f(1, 64, 1, 64, 64, 16, 0, None) == NULL
    assert f(1, 100, 1, 64, 64, 16, 0, ctypes.byref(n)) == SHAPE
    assert f(1, 128, 1, 96, 64, 16, 0, ctypes.byref(n)) == SHAPE
    assert f(1, 128, 1, 64, 64, 16, 2, ctypes.byref(n)) == DTYPE
    assert f(1, 128, 1, 64, 64, 128, 1, ctypes.byref(n)) == UNSUP
    assert f(0, 128, 1, 64, 64, 64, 1, ctypes.byref(n)) == OK and n.value == 0


def test_forward_validation():
    f = L.gdn_chunk_forward
    names = ["Q", "K", "V", "beta", "g", "S0", "O", "Sf", "ws", "wsb", "B", "L", "H", "dk", "dv",
             "C", "N", "S", "exact", "scale", "dt"]
    need = 2 * (8192 + 8192 + 8192 + 6 * 512) * 2  # B = 1, L = 128, H = 1, C = 64, bf16
    base = dict(Q=P1, K=BIG, V=2 * BIG, beta=3 * BIG, g=4 * BIG, S0=None, O=5 * BIG, Sf=None,
                ws=6 * BIG, wsb=need, B=1, L=128, H=1, dk=128, dv=128, C=64, N=3, S=8, exact=0,
                scale=1.0, dt=1)

    def call(**kw):
        a = dict(base, **kw)
        return f(*[a[n] for n in names], None)

    assert call(C=48) == SHAPE
    assert call(L=100) == SHAPE
    assert call(dv=32) == SHAPE
    assert call(N=64) == PARAM
    assert call(exact=4) == PARAM
    assert call(dt=2) == DTYPE
    assert call(C=128) == UNSUP
    assert call(Q=None) == NULL
    assert call(ws=None) == NULL
    assert call(wsb=need - 1) == WS
    assert call(O=5 * BIG + 4) == ALIGN
    assert call(S0=7 * BIG + 8) == ALIGN
    assert call(O=P1 + 256) == ALIAS            # O over Q
    assert call(ws=BIG + 1024) == ALIAS         # workspace over K
    assert call(ws=5 * BIG + 4096) == ALIAS     # workspace over O
    assert call(S0=7 * BIG, Sf=7 * BIG + 1024) == ALIAS  # partial overlap of the states
    assert call(Sf=4 * BIG) == ALIAS            # S_final over g
    assert call(B=0) == OK
    assert call(H=0, Q=None, K=None) == OK


def test_forward_phase_validation():
    need = 2 * (8192 + 8192 + 8192 + 6 * 512) * 2  # B = 1, L = 128, H = 1, C = 64, bf16
    p = L.gdn_chunk_forward_prepare
    # Q, K, V, beta, g, ws, wsb, B, L, H, dk, dv, C, N, S, exact, dt
    pb = [P1, BIG, 2 * BIG, 3 * BIG, 4 * BIG, 6 * BIG, need, 1, 128, 1, 128, 128, 64, 3, 8, 0, 1]
    bad = list(pb); bad[13] = 70
    assert p(*bad, None) == PARAM
    bad = list(pb); bad[2] = None
    assert p(*bad, None) == NULL
    bad = list(pb); bad[6] = need - 2
    assert p(*bad, None) == WS
    bad = list(pb); bad[5] = 2 * BIG + 64  # workspace over V
    assert p(*bad, None) == ALIAS
    bad = list(pb); bad[8] = 0  # no chunk: nothing to prepare
    assert p(*bad, None) == OK
    # inverse modes: 0 T_hat, 1 exact, 2 / 3 integer T_hat (default order, dk = dv = 128)
    bad = list(pb); bad[15] = 4
    assert p(*bad, None) == PARAM
    bad = list(pb); bad[15] = 2; bad[10] = 64
    assert p(*bad, None) == UNSUP
    bad = list(pb); bad[15] = 3; bad[13] = 2
    assert p(*bad, None) == UNSUP
    bad = list(pb); bad[15] = 2; bad[13] = 70
    assert p(*bad, None) == PARAM
    s = L.gdn_chunk_forward_state
    # Q, g, S0, O, S_final, ws, wsb, B, L, H, dk, dv, C, scale, dt
    sb = [P1, 4 * BIG, None, 5 * BIG, None, 6 * BIG, need, 1, 128, 1, 128, 128, 64, 1.0, 1]
    bad = list(sb); bad[3] = None
    assert s(*bad, None) == NULL
    bad = list(sb); bad[3] = 6 * BIG + 4096  # O over the workspace
    assert s(*bad, None) == ALIAS
    bad = list(sb); bad[6] = 16
    assert s(*bad, None) == WS
    bad = list(sb); bad[12] = 128
    assert s(*bad, None) == UNSUP
    bad = list(sb); bad[7] = 0
    assert s(*bad, None) == OK


def test_fused_varlen_validation():
    f = L.gdn_chunk_wy_fused_varlen
    names = ["K", "V", "beta", "g", "W", "U", "Tinv", "cu", "off", "nseq", "nch", "T", "H", "dk",
             "dv", "C", "N", "S", "exact", "dt"]
    base = dict(K=P1, V=BIG, beta=2 * BIG, g=3 * BIG, W=4 * BIG, U=5 * BIG, Tinv=None,
                cu=6 * BIG, off=6 * BIG + 4096, nseq=3, nch=5, T=200, H=2, dk=128, dv=128, C=64,
                N=3, S=8, exact=0, dt=1)

    def call(**kw):
        a = dict(base, **kw)
        return f(*[a[n] for n in names], None)

    assert call(C=48) == SHAPE
    assert call(nseq=-1) == SHAPE
    assert call(nseq=0) == SHAPE        # chunks without sequences
    assert call(nch=300) == SHAPE       # more chunks than tokens
    assert call(dk=96) == SHAPE
    assert call(N=64) == PARAM
    assert call(exact=3) == PARAM
    assert call(dt=2) == DTYPE
    assert call(C=128, N=64) == PARAM   # C = 128 accepted up to the launch
    assert call(C=128, cu=None) == NULL
    assert call(C=128, nch=0, K=None) == OK
    assert call(cu=None) == NULL
    assert call(W=None) == NULL
    assert call(off=6 * BIG + 2) == ALIGN
    assert call(U=4 * BIG + 256) == ALIAS   # U over W
    assert call(W=6 * BIG) == ALIAS         # W over the tables
    assert call(nch=0, K=None) == OK
    assert call(H=0) == OK


def test_binding_rejects_host_tensors():
    import torch
    A = torch.zeros(2, 64, 64)
    with pytest.raises(ValueError):
        g.gdn_chunk_inverse_neumann(A, 3, 8)
    with pytest.raises(TypeError):
        g.gdn_chunk_inverse_neumann(A.to(torch.float16), 3, 8)


def test_forward_varlen_validation():
    import ctypes
    f = L.gdn_chunk_forward_varlen
    need = ctypes.c_int64()
    assert L.gdn_chunk_forward_workspace(1, 4 * 64, 2, 128, 128, 64, 1, ctypes.byref(need)) == OK
    # Q, K, V, beta, g, S0, O, S_final, ws, ws_bytes, cu, off, nseq, n_chunks, T, H, dk, dv, C,
    # N, S, exact, scale, dtype, stream
    b = [k * BIG for k in range(9)]  # far apart: nothing overlaps unless a case moves it
    base = [b[1], b[2], b[3], b[4], b[5], None, b[6], None, b[7], need.value, b[8], b[8] + 64, 2,
            4, 200, 2, 128, 128, 64, 3, 8, 0, 1.0, 1, None]
    names = ["Q", "K", "V", "beta", "g", "S0", "O", "Sf", "ws", "wsb", "cu", "off", "nseq", "nch",
             "T", "H", "dk", "dv", "C", "N", "S", "exact", "scale", "dt"]

    def call(**kw):
        a = list(base)
        for k, v in kw.items():
            a[names.index(k)] = v
        return f(*a)

    assert call(nseq=0) == SHAPE                 # chunks without sequences
    assert call(nch=300) == SHAPE                # more chunks than tokens
    assert call(C=48) == SHAPE
    assert call(C=128) == UNSUP
    assert call(exact=4) == PARAM
    assert call(N=64) == PARAM
    assert call(dt=2) == DTYPE
    assert call(O=None) == NULL
    assert call(cu=None) == NULL
    assert call(wsb=need.value - 1) == WS
    assert call(cu=b[8] + 2) == ALIGN
    assert call(O=b[1] + 4096) == ALIAS          # O over Q
    assert call(ws=b[8] - 16) == ALIAS           # workspace over the tables
    assert call(Sf=b[6] + 64) == ALIAS           # S_final over O
    assert call(nseq=0, nch=0) == OK
    assert call(H=0) == OK


def test_binding_inverse_modes_and_exponent_layout():
    """Host logic of the binding: the layer forward's inverse modes map onto
    the ABI's `exact` values (0 T_hat, 1 exact, 2 INT16, 3 INT8), and the
    integer paths carry three exponents per tile at C = 128 only."""
    from paper_2606_06034_amd import _binding as b
    assert b._fwd_mode(False, None) == 0 and b._fwd_mode(True, None) == 1
    assert [b._fwd_mode(False, m) for m in ("neumann", "exact", "int16", "int8")] == [0, 1, 2, 3]
    assert b._fwd_mode(True, "int8") == 3  # an explicit mode wins over exact
    with pytest.raises(ValueError):
        b._fwd_mode(False, "int4")
    assert [b._nexp(C) for C in (16, 32, 64, 128)] == [1, 1, 1, 3]


# ---------------------------------------------------------------------------
# HIP's grid bounds a launch to 2^32 - 1 work items: every entry point turns
# a tile count past (2^32 - 1) / (its workgroup size) into GDN_ERR_SHAPE
# before anything is enqueued (pointers are never touched: the sizes fail
# first, so made-up addresses are safe here)

LIM64 = (2 ** 32 - 1) // 64     # 67,108,863 tiles of one wave
LIM128 = (2 ** 32 - 1) // 128   # the two-wave C = 128 kernels
LIM256 = (2 ** 32 - 1) // 256   # the C = 128 quantiser and the state pass


def test_grid_limit_inverse_entry_points():
    for f in (lambda n: L.gdn_chunk_inverse_neumann(P1, BIG, n, 16, 3, 2, 1, None),
              lambda n: L.gdn_chunk_inverse_fwdsub(P1, BIG, n, 16, 1, None),
              lambda n: L.gdn_chunk_inverse_blockwise(P1, BIG, n, 16, 1, None),
              lambda n: L.gdn_chunk_inverse_fwdsub_i8(P1, P2, BIG, 2 * BIG, None, n, 16, None),
              lambda n: L.gdn_chunk_inverse_fwdsub_i16(P1, P2, BIG, 2 * BIG, None, n, 16, None)):
        assert f(LIM64 + 1) == SHAPE
        assert f(1 << 31) == SHAPE
    for w in ("i8", "i16"):
        n = getattr(L, "gdn_chunk_inverse_neumann_" + w)
        assert n(P1, P2, BIG, 2 * BIG, None, LIM64 + 1, 16, 3, 2, 0, None) == SHAPE
        assert n(P1, P2, BIG, 2 * BIG, None, LIM128 + 1, 128, 3, 8, 0, None) == SHAPE
        q = getattr(L, "gdn_quantize_tiles_" + w)
        assert q(P1, BIG, 2 * BIG, LIM64 + 1, 16, None) == SHAPE
        assert q(P1, BIG, 2 * BIG, LIM256 + 1, 128, None) == SHAPE


def test_grid_limit_chunked_entry_points():
    # [B, L, H, d] entry points: B * H * L / C tiles; C = 16 with H = 1 and
    # B * L / 16 = LIM64 + 1 tiles (one over the one-wave limit)
    Lc = 16 * (LIM64 + 1)          # one sequence of that many tokens, B = 1
    assert Lc < 2 ** 31
    assert L.gdn_build_A(P1, P2, P3, BIG, 1, Lc, 1, 128, 16, 1, 1, None) == SHAPE
    f = L.gdn_chunk_wy_fused
    # K, V, beta, g, W, U, Tinv, B, L, H, dk, dv, C, N, S, dtype, stream
    assert f(P1, P2, P3, BIG, 2 * BIG, 3 * BIG, None, 1, Lc, 1, 128, 128, 16, 3, 2, 1,
             None) == SHAPE
    # C = 128 (128 work items per tile): H * L / 128 = 2^10 * 2^15 = LIM128 + 1
    assert LIM128 + 1 == 2 ** 25
    assert f(P1, P2, P3, BIG, 2 * BIG, 3 * BIG, None, 1, 128 * 2 ** 15, 2 ** 10, 128, 128, 128,
             3, 8, 1, None) == SHAPE


def test_noalloc_forward_size_limit():
    # sizes whose workspace exceeds the static scratch fail before any HIP
    # call: 2428 bf16 tiles of C = 64, dk = dv = 128 need 134,258,688 bytes
    assert g.GDN_FORWARD_SCRATCH_BYTES == 128 << 20
    f = L.gdn_chunk_forward_noalloc
    # Q, K, V, beta, g, S0, O, S_final, B, L, H, dk, dv, C, N, S, exact, scale, dtype, stream
    assert f(P1, P2, P3, P4, P5, None, P6, None, 1, 64 * 2428, 1, 128, 128, 64, 3, 8, 0, 0.1, 1,
             None) == WS
    assert f(P1, P2, P3, P4, P5, None, P6, None, 1, 100, 1, 128, 128, 64, 3, 8, 0, 0.1, 1,
             None) == SHAPE
    assert f(None, None, None, None, None, None, None, None, 0, 64, 1, 128, 128, 64, 3, 8, 0, 0.1,
             1, None) == OK
