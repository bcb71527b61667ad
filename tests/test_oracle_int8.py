"""Pins of the exact-integer (INT8) oracle.

The paper fixes the quantiser q(x) = clip(round(x / Delta), qmin, qmax)
(Appendix G) and the method (Algorithm 1); the integer mechanics are this
library's reading, stated in oracle/int8.py.  The pins check the rounding
primitives against exact rational arithmetic, the recipe against a second,
independent pure-Python coding of it on small tiles, exactness where the
paper's setting makes every intermediate representable, and closeness of the
dequantised result to the float64 T_hat(N, S).
"""

from fractions import Fraction

import numpy as np
import pytest

import workloads as wl
from oracle import gdn
from oracle import int8 as qo


def test_rne_shift_matches_exact_rounding():
    rng = np.random.default_rng(0)
    ys = rng.integers(-(1 << 24), 1 << 24, 4000)
    ss = rng.integers(0, 26, 4000)
    got = qo.rne_shift(ys, ss)
    for y, s, g in zip(ys.tolist(), ss.tolist(), got.tolist()):
        assert g == round(Fraction(y, 1 << s))  # Python rounds halves to even
    # exact halves both ways
    assert qo.rne_shift(np.array([1, 3, -1, -3, 5, -5]), 1).tolist() == [0, 2, 0, -2, 2, -2]


def test_quantize_minimal_exponent_and_roundtrip():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((50, 16, 16)) * np.exp(rng.uniform(-20, 5, (50, 1, 1)))).astype(np.float32)
    q, e = qo.quantize(x)
    amax = np.max(np.abs(x.astype(np.float64)), axis=(-1, -2))
    # amax / 2^e <= 127 < amax / 2^(e-1)
    assert np.all(amax <= 127 * np.ldexp(1.0, e))
    assert np.all(amax > 127 * np.ldexp(1.0, e - 1))
    assert np.all(np.abs(q) <= 127)
    err = np.abs(qo.dequant(q, e) - x)
    assert np.all(err <= np.ldexp(0.5, e)[..., None, None])
    # exactly representable values come back exactly
    q0 = rng.integers(-127, 128, (10, 8, 8))
    q0[:, 0, 0] = 127
    e0 = rng.integers(-30, 5, 10)
    x0 = qo.dequant(q0, e0).astype(np.float32)
    q1, e1 = qo.quantize(x0)
    assert np.array_equal(q1, q0) and np.array_equal(e1, e0)
    # all-zero tile
    qz, ez = qo.quantize(np.zeros((1, 4, 4), np.float32))
    assert np.all(qz == 0) and ez[0] == 0


def test_requant_smallest_shift():
    rng = np.random.default_rng(2)
    acc = rng.integers(-(1 << 20), 1 << 20, (200, 8, 8))
    acc[:20] //= 1 << 15  # some already small
    q, e = qo.requant(acc, np.zeros(200, np.int64))
    assert np.all(np.abs(q) <= 127)
    for t in range(200):
        s = int(e[t])
        amax = int(np.max(np.abs(acc[t])))
        assert round(Fraction(amax, 1 << s)) <= 127
        if s > 0:
            assert round(Fraction(amax, 1 << (s - 1))) > 127
        for v, w in zip(acc[t].ravel().tolist(), q[t].ravel().tolist()):
            assert w == round(Fraction(v, 1 << s))


def test_aligned_sum_is_exact_within_guard_bits():
    """Terms no finer than 16 bits below the first term's quantum add
    exactly; the sum carries q * 2^e of every term."""
    rng = np.random.default_rng(3)
    qa = rng.integers(-127, 128, (5, 4, 4))
    qb = rng.integers(-127, 128, (5, 4, 4))
    ea = rng.integers(-12, -4, 5)
    eb = ea - rng.integers(0, 17, 5)
    p = np.ones(5, bool)
    s, es, _ = qo.aligned_sum([(qa, ea, p, 7), (qb, eb, p, 7)])
    assert np.all(es == ea - 16)
    for t in range(5):
        for i in range(4):
            for j in range(4):
                want = Fraction(int(qa[t, i, j])) * Fraction(2) ** int(ea[t]) + \
                    Fraction(int(qb[t, i, j])) * Fraction(2) ** int(eb[t])
                assert Fraction(int(s[t, i, j])) * Fraction(2) ** int(es[t]) == want


def test_aligned_sum_rebases_on_larger_term():
    """A later term above the running range rebases (rounding the sum) and
    the result stays within int32 and within one rounding of the exact sum."""
    qa = np.array([[[100, -3], [7, 1]]])
    qb = np.array([[[127, 64], [-127, 0]]])
    ea = np.array([-10]); eb = np.array([0])
    p = np.ones(1, bool)
    s, es, _ = qo.aligned_sum([(qa, ea, p, 7), (qb, eb, p, 7)])
    assert es[0] == 0 + 7 - 23
    exact = qa[0] * 2.0 ** -10 + qb[0] * 1.0
    assert np.max(np.abs(s[0] * 2.0 ** float(es[0]) - exact)) <= 2.0 ** float(es[0])


# ---------------------------------------------------------------------------
# a second, independent coding of the recipe (pure Python integers, loops)


def _py_rne(y, s):
    return y if s <= 0 else round(Fraction(y, 1 << s))


def _py_requant(M, e):
    amax = max(abs(v) for row in M for v in row)
    s = 0
    while _py_rne(amax, s) > 127:
        s += 1
    return [[_py_rne(v, s) for v in row] for row in M], (e + s if amax > 0 else 0)


def _py_mm(X, Y):
    n = len(X)
    return [[sum(X[i][k] * Y[k][j] for k in range(n)) for j in range(n)] for i in range(n)]


def _py_nz(M):
    return any(v != 0 for row in M for v in row)


def _py_sum(terms, C):
    """terms: (M, e, present, bits), summed in order with the running-exponent
    rule (first term sets e = e0 + bits - 23; rebase when a term's top would
    pass e + 23; finer terms rounded half-even)."""
    out = [[0] * C for _ in range(C)]
    es = None
    for M, e, p, b in terms:
        if not p:
            continue
        top = e + b - 23
        if es is None:
            es = top
        elif top > es:
            out = [[_py_rne(v, top - es) for v in row] for row in out]
            es = top
        for i in range(C):
            for j in range(C):
                v = M[i][j]
                out[i][j] += v << (e - es) if e >= es else _py_rne(v, es - e)
    return out, (0 if es is None else es)


def _py_pipeline(qA, eA, N, S):
    C = len(qA)
    bits = 14 + (C - 1).bit_length()
    L = [[-qA[i][j] if i > j else 0 for j in range(C)] for i in range(C)]
    band = lambda M: [[M[i][j] if 0 < i - j <= N else 0 for j in range(C)] for i in range(C)]
    pw = []
    if N >= 1:
        B, eB = _py_requant(band(L), eA)
        pw.append((B, eB))
        for _ in range(2, N + 1):
            B, eB = _py_requant(band(_py_mm(pw[-1][0], L)), pw[-1][1] + eA)
            pw.append((B, eB))
    if pw:
        N0, eN = _py_requant(*_py_sum([(M, e, _py_nz(M), 7) for M, e in pw], C))
    else:
        N0, eN = [[0] * C for _ in range(C)], 0
    nzL, nzN = _py_nz(L), _py_nz(N0)
    Es, ee = _py_sum([(L, eA, nzL, 7), (_py_mm(L, N0), eA + eN, nzL and nzN, bits),
                      ([[-v for v in r] for r in N0], eN, nzN, 7)], C)
    Es = [[Es[i][j] if i - j > N else 0 for j in range(C)] for i in range(C)]
    E, eE = _py_requant(Es, ee)
    ch = []
    if S >= 1:
        ch.append((E, eE))
        for _ in range(2, S + 1):
            ch.append(_py_requant(_py_mm(E, ch[-1][0]), eE + ch[-1][1]))
    if ch:
        G, eG = _py_requant(*_py_sum([(M, e, _py_nz(M), 7) for M, e in ch], C))
    else:
        G, eG = [[0] * C for _ in range(C)], 0
    nzG = _py_nz(G)
    Ts, et = _py_sum([(N0, eN, nzN, 7), (G, eG, nzG, 7), (_py_mm(N0, G), eN + eG, nzN and nzG, bits)], C)
    Ts = [[Ts[i][j] if i > j else 0 for j in range(C)] for i in range(C)]
    return _py_requant(Ts, et)


@pytest.mark.parametrize("C,N,S", [(8, 3, 2), (8, 1, 3), (16, 3, 2), (16, 2, 5), (8, 0, 3), (8, 3, 0)])
def test_int8_pipeline_matches_independent_coding(C, N, S):
    k, b, g, _ = wl.gen_stress_head(L=2 * C, dk=32, C=C, seed=C + N + S)
    A = gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], C))
    qA, eA = qo.quantize(A.astype(np.float32))
    qT, eT, _ = qo.neumann_inverse_int8(qA, eA, N, S)
    for t in range(A.shape[0]):
        Tp, ep = _py_pipeline(qA[t].tolist(), int(eA[t]), N, S)
        assert qT[t].tolist() == Tp
        assert int(eT[t]) == ep


# ---------------------------------------------------------------------------
# exactness and accuracy in the paper's setting


def test_int8_all_ones_gdn_is_exact():
    """All-ones A (GDN sign): every intermediate is a small integer, so the
    integer pipeline reproduces the exact bidiagonal inverse I - Z."""
    C = 64
    A = np.tril(np.ones((1, C, C), np.float32), -1)
    qA, eA = qo.quantize(A)
    qT, eT, parts = qo.neumann_inverse_int8(qA, eA, 3, 8)
    assert np.array_equal(qo.dequant_unit(qT, eT)[0], np.eye(C) - np.eye(C, k=-1))
    assert np.all(parts["E"][0] == 0)


@pytest.mark.parametrize("gate", ["default", "wide"])
def test_int8_close_to_float_approximation(gate):
    """Dequantised INT8 T_hat(3, 8) against the float64 T_hat(3, 8) on the
    workload distributions: each requantisation keeps 7 bits relative to its
    matrix's largest entry, so the error stays a small multiple of
    2^-8 max|T_hat - I|."""
    w = wl.workload("int8" if gate == "wide" else "tiny")
    k, b, g, _ = wl.gen_head(w, 0, 0, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(k[None, :256, None], b[None, :256, None], g[None, :256, None], 64))
    qA, eA = qo.quantize(A.astype(np.float32))
    qT, eT, _ = qo.neumann_inverse_int8(qA, eA, 3, 8)
    T = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qT, eT) - T), axis=(-1, -2))
    assert np.all(err <= 4 * 2.0 ** -8 * scale)


def test_int8_stress_close_to_float():
    k, b, g, _ = wl.gen_stress_head(L=256, dk=128, C=64, seed=9)
    A = gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], 64))
    qA, eA = qo.quantize(A.astype(np.float32))
    qT, eT, _ = qo.neumann_inverse_int8(qA, eA, 3, 8)
    T = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qT, eT) - T), axis=(-1, -2))
    # stress tiles have |A| up to ~0.5 and larger residual powers: the
    # quantisation noise compounds over the chain (observed ~9 x 2^-8)
    assert np.all(err <= 16 * 2.0 ** -8 * scale)


def test_int8_structure():
    """Strict part only; codes in range; E zero on its band; residual powers
    zero below s (N + 1) (exact in integers)."""
    w = wl.workload("tiny")
    k, b, g, _ = wl.gen_head(w, 0, 1, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(k[None, :128, None], b[None, :128, None], g[None, :128, None], 64))
    qA, eA = qo.quantize(A.astype(np.float32))
    N, S = 3, 8
    qT, eT, parts = qo.neumann_inverse_int8(qA, eA, N, S)
    d = gdn.subdiag_index(64)
    assert np.all(qT[:, d <= 0] == 0)
    assert np.all(np.abs(qT) <= 127)
    assert np.all(parts["E"][0][:, d <= N] == 0)
    for s, (q, e, nz) in enumerate(parts["chain"], start=1):
        assert np.all(q[:, d < s * (N + 1)] == 0)
