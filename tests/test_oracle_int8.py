"""Pins of the exact-integer (INT8 and INT16) oracle.

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


# (qmax, bits of a code, alignment bits) of the two integer settings
PY8 = (127, 7, 23)
PY16 = (32639, 15, 31)


def _py_requant(M, e, P=PY8):
    amax = max(abs(v) for row in M for v in row)
    s = 0
    while _py_rne(amax, s) > P[0]:
        s += 1
    return [[_py_rne(v, s) for v in row] for row in M], (e + s if amax > 0 else 0)


def _py_mm(X, Y):
    n = len(X)
    return [[sum(X[i][k] * Y[k][j] for k in range(n)) for j in range(n)] for i in range(n)]


def _py_nz(M):
    return any(v != 0 for row in M for v in row)


def _py_sum(terms, C, P=PY8):
    """terms: (M, e, present, bits), summed in order with the running-exponent
    rule (first term sets e = e0 + bits - a with a = 23 for INT8, 31 for
    INT16; rebase when a term's top would pass e + a; finer terms rounded
    half-even)."""
    out = [[0] * C for _ in range(C)]
    es = None
    for M, e, p, b in terms:
        if not p:
            continue
        top = e + b - P[2]
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


def _py_pipeline(qA, eA, N, S, P=PY8):
    C = len(qA)
    q = P[1]
    bits = 2 * q + (C - 1).bit_length()
    rq = lambda M, e: _py_requant(M, e, P)
    sm = lambda terms: _py_sum(terms, C, P)
    L = [[-qA[i][j] if i > j else 0 for j in range(C)] for i in range(C)]
    band = lambda M: [[M[i][j] if 0 < i - j <= N else 0 for j in range(C)] for i in range(C)]
    pw = []
    if N >= 1:
        B, eB = rq(band(L), eA)
        pw.append((B, eB))
        for _ in range(2, N + 1):
            B, eB = rq(band(_py_mm(pw[-1][0], L)), pw[-1][1] + eA)
            pw.append((B, eB))
    if pw:
        N0, eN = rq(*sm([(M, e, _py_nz(M), q) for M, e in pw]))
    else:
        N0, eN = [[0] * C for _ in range(C)], 0
    nzL, nzN = _py_nz(L), _py_nz(N0)
    Es, ee = sm([(L, eA, nzL, q), (_py_mm(L, N0), eA + eN, nzL and nzN, bits),
                 ([[-v for v in r] for r in N0], eN, nzN, q)])
    Es = [[Es[i][j] if i - j > N else 0 for j in range(C)] for i in range(C)]
    E, eE = rq(Es, ee)
    ch = []
    if S >= 1:
        ch.append((E, eE))
        for _ in range(2, S + 1):
            ch.append(rq(_py_mm(E, ch[-1][0]), eE + ch[-1][1]))
    if ch:
        G, eG = rq(*sm([(M, e, _py_nz(M), q) for M, e in ch]))
    else:
        G, eG = [[0] * C for _ in range(C)], 0
    nzG = _py_nz(G)
    Ts, et = sm([(N0, eN, nzN, q), (G, eG, nzG, q), (_py_mm(N0, G), eN + eG, nzN and nzG, bits)])
    Ts = [[Ts[i][j] if i > j else 0 for j in range(C)] for i in range(C)]
    return rq(Ts, et)


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


# ---------------------------------------------------------------------------
# INT16: the same recipe with 16-bit codes (|q| <= 32639), 31-bit aligned
# terms; the pins above repeated at that width


def test_int16_quantize_minimal_exponent_and_roundtrip():
    rng = np.random.default_rng(11)
    x = (rng.standard_normal((50, 16, 16)) * np.exp(rng.uniform(-20, 5, (50, 1, 1)))).astype(np.float32)
    q, e = qo.quantize(x, qo.SPEC16)
    amax = np.max(np.abs(x.astype(np.float64)), axis=(-1, -2))
    assert np.all(amax <= 32639 * np.ldexp(1.0, e))
    assert np.all(amax > 32639 * np.ldexp(1.0, e - 1))
    assert np.all(np.abs(q) <= 32639) and np.max(np.abs(q)) > 16319
    for t in range(50):
        for v, w in zip(x[t].ravel().tolist(), q[t].ravel().tolist()):
            assert w == round(Fraction(v) / Fraction(2) ** int(e[t]))
    # codes at the range ends come back exactly
    q0 = rng.integers(-32639, 32640, (10, 8, 8))
    q0[:, 0, 0] = -32639
    e0 = rng.integers(-40, 5, 10)
    q1, e1 = qo.quantize(qo.dequant(q0, e0).astype(np.float32), qo.SPEC16)
    # float32 holds 24 bits: every 15-bit code times a power of two is exact
    assert np.array_equal(q1, q0) and np.array_equal(e1, e0)


def test_int16_requant_smallest_shift():
    rng = np.random.default_rng(12)
    acc = rng.integers(-(1 << 36), 1 << 36, (100, 8, 8))
    acc[:10] //= 1 << 25
    acc[10] = rng.integers(-1000, 1000, (8, 8))
    acc[10, 0, 0] = 32639 * 4 + 2  # 32639.5 * 4 rounds up to 32640: one more bit
    q, e = qo.requant(acc, np.zeros(100, np.int64), qo.SPEC16)
    assert np.all(np.abs(q) <= 32639)
    assert e[10] == 3
    for t in range(100):
        s = int(e[t])
        amax = int(np.max(np.abs(acc[t])))
        assert round(Fraction(amax, 1 << s)) <= 32639
        if s > 0:
            assert round(Fraction(amax, 1 << (s - 1))) > 32639
        for v, w in zip(acc[t].ravel().tolist(), q[t].ravel().tolist()):
            assert w == round(Fraction(v, 1 << s))


def test_int16_aligned_sum_is_exact_within_guard_bits():
    rng = np.random.default_rng(13)
    qa = rng.integers(-32639, 32640, (5, 4, 4))
    qb = rng.integers(-32639, 32640, (5, 4, 4))
    ea = rng.integers(-30, -4, 5)
    eb = ea - rng.integers(0, 17, 5)
    p = np.ones(5, bool)
    s, es, _ = qo.aligned_sum([(qa, ea, p, 15), (qb, eb, p, 15)], qo.SPEC16)
    assert np.all(es == ea - 16)
    for t in range(5):
        for i in range(4):
            for j in range(4):
                want = Fraction(int(qa[t, i, j])) * Fraction(2) ** int(ea[t]) + \
                    Fraction(int(qb[t, i, j])) * Fraction(2) ** int(eb[t])
                assert Fraction(int(s[t, i, j])) * Fraction(2) ** int(es[t]) == want


@pytest.mark.parametrize("C,N,S", [(8, 3, 2), (16, 3, 2), (16, 2, 5), (8, 0, 3), (8, 3, 0)])
def test_int16_pipeline_matches_independent_coding(C, N, S):
    k, b, g, _ = wl.gen_stress_head(L=2 * C, dk=32, C=C, seed=C + N + S + 50)
    A = gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], C))
    qA, eA = qo.quantize(A.astype(np.float32), qo.SPEC16)
    qT, eT, _ = qo.neumann_inverse_int16(qA, eA, N, S)
    for t in range(A.shape[0]):
        Tp, ep = _py_pipeline(qA[t].tolist(), int(eA[t]), N, S, PY16)
        assert qT[t].tolist() == Tp
        assert int(eT[t]) == ep


def test_int16_all_ones_gdn_is_exact():
    C = 64
    A = np.tril(np.ones((1, C, C), np.float32), -1)
    qA, eA = qo.quantize(A, qo.SPEC16)
    qT, eT, parts = qo.neumann_inverse_int16(qA, eA, 3, 8)
    assert np.array_equal(qo.dequant_unit(qT, eT)[0], np.eye(C) - np.eye(C, k=-1))
    assert np.all(parts["E"][0] == 0)


@pytest.mark.parametrize("gate", ["default", "wide"])
def test_int16_close_to_float_approximation(gate):
    """Each requantisation keeps 15 bits relative to its matrix's largest
    entry: the dequantised INT16 T_hat(3, 8) stays within a small multiple of
    2^-16 max|T_hat - I| of the float64 T_hat(3, 8), about 2^8 times closer
    than INT8."""
    w = wl.workload("int8" if gate == "wide" else "tiny")
    k, b, g, _ = wl.gen_head(w, 0, 0, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(k[None, :256, None], b[None, :256, None], g[None, :256, None], 64))
    T = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(64)), axis=(-1, -2))
    q16, e16 = qo.quantize(A.astype(np.float32), qo.SPEC16)
    qT, eT, _ = qo.neumann_inverse_int16(q16, e16, 3, 8)
    err16 = np.max(np.abs(qo.dequant_unit(qT, eT) - T), axis=(-1, -2))
    assert np.all(err16 <= 4 * 2.0 ** -16 * scale)
    q8, e8 = qo.quantize(A.astype(np.float32))
    qT8, eT8, _ = qo.neumann_inverse_int8(q8, e8, 3, 8)
    err8 = np.max(np.abs(qo.dequant_unit(qT8, eT8) - T), axis=(-1, -2))
    assert np.max(err16) * 32 < np.max(err8)


def test_int16_stress_close_to_float():
    k, b, g, _ = wl.gen_stress_head(L=256, dk=128, C=64, seed=9)
    A = gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], 64))
    qA, eA = qo.quantize(A.astype(np.float32), qo.SPEC16)
    qT, eT, _ = qo.neumann_inverse_int16(qA, eA, 3, 8)
    T = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qT, eT) - T), axis=(-1, -2))
    assert np.all(err <= 16 * 2.0 ** -16 * scale)


def test_int16_structure():
    w = wl.workload("tiny")
    k, b, g, _ = wl.gen_head(w, 0, 1, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(k[None, :128, None], b[None, :128, None], g[None, :128, None], 64))
    qA, eA = qo.quantize(A.astype(np.float32), qo.SPEC16)
    N, S = 3, 8
    qT, eT, parts = qo.neumann_inverse_int16(qA, eA, N, S)
    d = gdn.subdiag_index(64)
    assert np.all(qT[:, d <= 0] == 0)
    assert np.all(np.abs(qT) <= 32639) and np.max(np.abs(qT)) > 16319
    assert np.all(parts["E"][0][:, d <= N] == 0)
    for s, (q, e, nz) in enumerate(parts["chain"], start=1):
        assert np.all(q[:, d < s * (N + 1)] == 0)


def test_int16_limbs_split_every_code():
    """32639 = 127 * 256 + 127: every INT16 code is hi * 256 + lo with both
    limbs int8 codes, so a product of 16-bit codes is four int8 products."""
    q = np.arange(-32639, 32640)
    lo = ((q + 128) & 255) - 128
    hi = (q - lo) >> 8
    assert np.all(hi * 256 + lo == q)
    assert lo.min() >= -128 and lo.max() <= 127 and hi.min() >= -127 and hi.max() <= 127


# ---------------------------------------------------------------------------
# the integer forward-substitution baseline (INT16)


def _py_fwdsub(qA, eA, P=PY16):
    """Second coding of the integer forward substitution: Python integers,
    loops, the running-sum rule of _py_sum, the growth of the tile exponent
    searched from 0 upwards."""
    C = len(qA)
    q = P[1]
    bits = 2 * q + (C - 1).bit_length()
    L = [[-qA[i][j] if i > j else 0 for j in range(C)] for i in range(C)]
    X = [[0] * C for _ in range(C)]
    eX = eA

    def scale(y, d):  # rne(y / 2^d), any integer d
        return _py_rne(y, d) if d >= 0 else y << -d

    for i in range(1, C):
        t = [L[i][:]]
        Pm = [[sum(L[i][k] * X[k][j] for k in range(C)) for j in range(C)]]
        nzt, nzX = _py_nz(t), _py_nz(X)
        row, es = _py_sum_rows([(t, eA, nzt, q), (Pm, eA + eX, nzt and nzX, bits)], C, P)
        amax = max(abs(v) for v in row)
        s = 0
        while amax > 0 and scale(amax, eX + s - es) > P[0]:
            s += 1
        if s:
            X = [[_py_rne(v, s) for v in r] for r in X]
            eX += s
        X[i] = [scale(v, eX - es) for v in row] if nzt else [0] * C
    return X, eX


def _py_sum_rows(terms, C, P):
    """_py_sum on 1 x C rows."""
    out = [0] * C
    es = None
    for M, e, p, b in terms:
        if not p:
            continue
        top = e + b - P[2]
        if es is None:
            es = top
        elif top > es:
            out = [_py_rne(v, top - es) for v in out]
            es = top
        for j in range(C):
            v = M[0][j]
            out[j] += v << (e - es) if e >= es else _py_rne(v, es - e)
    return out, (0 if es is None else es)


@pytest.mark.parametrize("C,src", [(8, "stress"), (16, "stress"), (16, "workload"),
                                   (16, "minus_ones")])
def test_int16_fwdsub_matches_independent_coding(C, src):
    if src == "minus_ones":
        A = -np.tril(np.ones((2, C, C)), -1)
        A[1] *= 0.75
    elif src == "stress":
        k, b, g, _ = wl.gen_stress_head(L=2 * C, dk=32, C=C, seed=C + 70)
        A = gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], C))
    else:
        k, b, g, _ = wl.gen_head(wl.workload("int8"), 0, 0, C=C, want_v=False)
        A = gdn.tiles_flat(gdn.build_A(k[None, :3 * C, None], b[None, :3 * C, None],
                                       g[None, :3 * C, None], C))
    qA, eA = qo.quantize(A.astype(np.float32), qo.SPEC16)
    qX, eX = qo.fwdsub_inverse_int(qA, eA)
    for t in range(A.shape[0]):
        Xp, ep = _py_fwdsub(qA[t].tolist(), int(eA[t]))
        assert qX[t].tolist() == Xp
        assert int(eX[t]) == ep


def test_int16_fwdsub_exact_cases():
    """All-ones A: the inverse I - Z, no exponent growth.  Minus-ones A at
    C = 16: the inverse has x_ij = 2^(i-j-1) (up to 2^14), so the tile
    exponent must grow from -14 to 0, rounding earlier rows each time, and
    every step stays exact (power-of-two values on the grid)."""
    C = 64
    qA, eA = qo.quantize(np.tril(np.ones((1, C, C), np.float32), -1), qo.SPEC16)
    qX, eX = qo.fwdsub_inverse_int(qA, eA)
    assert eX[0] == eA[0]
    assert np.array_equal(qo.dequant_unit(qX, eX)[0], np.eye(C) - np.eye(C, k=-1))
    C = 16
    qA, eA = qo.quantize(-np.tril(np.ones((1, C, C), np.float32), -1), qo.SPEC16)
    qX, eX = qo.fwdsub_inverse_int(qA, eA)
    d = gdn.subdiag_index(C)
    want = np.where(d > 0, 2.0 ** np.maximum(d - 1, 0), 0.0) + np.eye(C)
    assert eA[0] == -14 and eX[0] == 0
    assert np.array_equal(qo.dequant_unit(qX, eX)[0], want)


@pytest.mark.parametrize("src", ["workload", "wide", "stress"])
def test_int16_fwdsub_close_to_exact_inverse(src):
    """Against the exact inverse of the float64 A: the error stays a small
    multiple of the 16-bit quantum of max|X - I| (the input quantisation
    alone contributes about 2^-16 of it)."""
    if src == "stress":
        k, b, g, _ = wl.gen_stress_head(L=256, dk=128, C=64, seed=9)
    else:
        k, b, g, _ = wl.gen_head(wl.workload("int8" if src == "wide" else "tiny"), 0, 0,
                                 want_v=False)
    A = gdn.tiles_flat(gdn.build_A(k[None, :256, None], b[None, :256, None], g[None, :256, None], 64))
    X = gdn.forward_substitution_inverse(A)
    qA, eA = qo.quantize(A.astype(np.float32), qo.SPEC16)
    qX, eX = qo.fwdsub_inverse_int(qA, eA)
    scale = np.max(np.abs(X - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qX, eX) - X), axis=(-1, -2))
    assert np.all(err <= 8 * 2.0 ** -15 * scale)
    d = gdn.subdiag_index(64)
    assert np.all(qX[:, d <= 0] == 0) and np.all(np.abs(qX) <= 32639) and np.all(eX >= eA)


@pytest.mark.parametrize("C,src", [(8, "stress"), (16, "stress"), (16, "workload"),
                                   (8, "minus_ones")])
def test_int8_fwdsub_matches_independent_coding(C, src):
    """The integer forward substitution at 8-bit codes (SPEC8) against the
    second coding with INT8's parameters."""
    if src == "minus_ones":
        A = -np.tril(np.ones((2, C, C)), -1)
        A[1] *= 0.75
    elif src == "stress":
        k, b, g, _ = wl.gen_stress_head(L=2 * C, dk=32, C=C, seed=C + 90)
        A = gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], C))
    else:
        k, b, g, _ = wl.gen_head(wl.workload("int8"), 0, 1, C=C, want_v=False)
        A = gdn.tiles_flat(gdn.build_A(k[None, :3 * C, None], b[None, :3 * C, None],
                                       g[None, :3 * C, None], C))
    qA, eA = qo.quantize(A.astype(np.float32))
    qX, eX = qo.fwdsub_inverse_int(qA, eA, qo.SPEC8)
    for t in range(A.shape[0]):
        Xp, ep = _py_fwdsub(qA[t].tolist(), int(eA[t]), PY8)
        assert qX[t].tolist() == Xp
        assert int(eX[t]) == ep


def test_int8_fwdsub_exact_cases_and_accuracy():
    """Minus-ones A at C = 8 (x_ij = 2^(i-j-1) up to 64, the exponent growing
    from -6 to 0, exact); workload tiles within a few 8-bit quanta of
    max|X - I|."""
    C = 8
    qA, eA = qo.quantize(-np.tril(np.ones((1, C, C), np.float32), -1))
    qX, eX = qo.fwdsub_inverse_int(qA, eA, qo.SPEC8)
    d = gdn.subdiag_index(C)
    assert eA[0] == -6 and eX[0] == 0
    assert np.array_equal(qo.dequant_unit(qX, eX)[0],
                          np.where(d > 0, 2.0 ** np.maximum(d - 1, 0), 0.0) + np.eye(C))
    k, b, g, _ = wl.gen_head(wl.workload("int8"), 0, 0, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(k[None, :256, None], b[None, :256, None], g[None, :256, None], 64))
    X = gdn.forward_substitution_inverse(A)
    qA, eA = qo.quantize(A.astype(np.float32))
    qX, eX = qo.fwdsub_inverse_int(qA, eA, qo.SPEC8)
    scale = np.max(np.abs(X - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qX, eX) - X), axis=(-1, -2))
    assert np.all(err <= 8 * 2.0 ** -7 * scale)
    assert np.all(np.abs(qX) <= 127)


# ---------------------------------------------------------------------------
# C = 128, block-wise (Appendix E with 64 x 64 blocks, Appendix H): three
# exponents per tile, X21 = -X22 A21 X11 as two requantised products


def _blocked_A(C, seed, stress=False):
    if stress:
        k, b, g, _ = wl.gen_stress_head(L=2 * C, dk=64, C=C, seed=seed)
    else:
        w = wl.workload("tiny").with_(seed=seed)
        k, b, g, _ = wl.gen_head(w, 0, 0, C=C, want_v=False)
        k, b, g = k[:2 * C], b[:2 * C], g[:2 * C]
    return gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], C))


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_blocked_quantize_per_block_minimal_exponent(spec):
    A = _blocked_A(128, 1).astype(np.float32)
    A[1, 64:, :64] = 0.0  # an all-zero off-diagonal block gets e = 0
    q, e = qo.quantize_blocked(A, spec)
    assert e.shape == (2, 3) and e[1, 1] == 0
    d = gdn.subdiag_index(128)
    assert np.all(q[:, d <= 0] == 0)
    for k, (r, c) in enumerate([(0, 0), (1, 0), (1, 1)]):
        rs, cs = slice(64 * r, 64 * r + 64), slice(64 * c, 64 * c + 64)
        x = np.where(d[rs, cs] > 0, A[:, rs, cs], 0).astype(np.float64)
        for t in range(2):
            et = int(e[t, k])
            if not np.any(x[t]):
                assert et == 0 and not np.any(q[t, rs, cs])
                continue
            qb = q[t, rs, cs]
            assert np.max(np.abs(qb)) <= spec.qmax
            # smallest exponent: one lower would need a code above qmax
            assert np.max(np.abs(x[t])) / 2.0 ** (et - 1) > spec.qmax
            assert np.max(np.abs(qb * 2.0 ** et - x[t])) <= 2.0 ** (et - 1)


def _py_blocked(qA, eA, N, S, P):
    """Independent coding of the block-wise inverse on small tiles: the
    diagonal blocks by _py_pipeline, then P = A21 + A21 N11 and
    X21 = -(P + N22 P), each summed and requantised."""
    C = len(qA)
    h = C // 2
    bits = 2 * P[1] + (h - 1).bit_length()
    blk = lambda r, c: [row[c:c + h] for row in qA[r:r + h]]
    N11, e11 = _py_pipeline(blk(0, 0), eA[0], N, S, P)
    N22, e22 = _py_pipeline(blk(h, h), eA[2], N, S, P)
    A21 = blk(h, 0)
    nzA = _py_nz(A21)
    Ps, ep = _py_sum([(A21, eA[1], nzA, P[1]),
                      (_py_mm(A21, N11), eA[1] + e11, nzA and _py_nz(N11), bits)], h, P)
    Pq, eP = _py_requant(Ps, ep, P)
    Xs, ex = _py_sum([(Pq, eP, _py_nz(Pq), P[1]),
                      (_py_mm(N22, Pq), e22 + eP, _py_nz(N22) and _py_nz(Pq), bits)], h, P)
    X21, e21 = _py_requant(Xs, ex, P)
    out = [[0] * C for _ in range(C)]
    for i in range(h):
        for j in range(h):
            out[i][j] = N11[i][j]
            out[h + i][h + j] = N22[i][j]
            out[h + i][j] = -X21[i][j]
    return out, [e11, e21, e22]


@pytest.mark.parametrize("spec,P", [(qo.SPEC8, PY8), (qo.SPEC16, PY16)])
@pytest.mark.parametrize("C,N,S", [(16, 3, 2), (16, 1, 3), (32, 2, 2)])
def test_blocked_matches_independent_coding(spec, P, C, N, S):
    A = _blocked_A(C, C + N, stress=True).astype(np.float32)
    qA, eA = qo.quantize_blocked(A, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, N, S, spec)
    for t in range(A.shape[0]):
        Tp, ep = _py_blocked(qA[t].tolist(), [int(v) for v in eA[t]], N, S, P)
        assert qT[t].tolist() == Tp
        assert [int(v) for v in eT[t]] == ep


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_blocked_closed_forms(spec):
    """A21 = 0: X21 = 0 and the diagonal blocks are the 64 x 64 integer
    inverses; A11 = A22 = 0: A^2 = 0, so (I + A)^-1 = I - A and the codes of
    X21 are those of -A21 at A21's exponent; all-ones A: the pipeline
    reproduces the exact inverse I - Z (Z the unit sub-diagonal) across the
    block boundary."""
    A = _blocked_A(128, 2).astype(np.float32)
    Ad = A.copy()
    Ad[:, 64:, :64] = 0.0
    qA, eA = qo.quantize_blocked(Ad, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    assert not np.any(qT[:, 64:, :64]) and np.all(eT[:, 1] == 0)
    for k, s in ((0, slice(0, 64)), (2, slice(64, 128))):
        q1, e1 = qo.quantize(np.tril(A[:, s, s], -1), spec)
        t1, f1, _ = qo.neumann_inverse_int8(q1, e1, 3, 8, spec)
        assert np.array_equal(qT[:, s, s], t1) and np.array_equal(eT[:, k], f1)
    Ao = np.zeros_like(A)
    Ao[:, 64:, :64] = A[:, 64:, :64]
    qA, eA = qo.quantize_blocked(Ao, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    assert np.array_equal(qT[:, 64:, :64], -qA[:, 64:, :64]) and np.array_equal(eT[:, 1], eA[:, 1])
    assert not np.any(qT[:, :64, :64]) and not np.any(qT[:, 64:, 64:])
    ones = np.tril(np.ones((1, 128, 128), np.float32), -1)
    qA, eA = qo.quantize_blocked(ones, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    assert np.array_equal(qo.dequant_unit_blocked(qT, eT)[0], np.eye(128) - np.eye(128, k=-1))


@pytest.mark.parametrize("spec,bits", [(qo.SPEC8, 8), (qo.SPEC16, 16)])
@pytest.mark.parametrize("src", ["workload", "stress"])
def test_blocked_close_to_float_approximation(spec, bits, src):
    """Dequantised block-wise inverse against the float64 block-wise
    T_hat(3, 8) (Appendix E formula on float64 diagonal inverses): the merge
    adds two requantisations and X22's gain to the diagonal blocks' error."""
    A = _blocked_A(128, 3, stress=src == "stress")
    qA, eA = qo.quantize_blocked(A.astype(np.float32), spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    T = gdn.neumann_inverse_blocked(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(128)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit_blocked(qT, eT) - T), axis=(-1, -2))
    assert np.all(err <= 16 * 2.0 ** -bits * scale)
    # the 64 x 64 inverses alone: same bound as the unblocked pins
    err11 = np.max(np.abs(qo.dequant_unit_blocked(qT, eT)[:, :64, :64] - T[:, :64, :64]))
    assert err11 <= 16 * 2.0 ** -bits * np.max(scale)


# ---------------------------------------------------------------------------
# the integer inverse inside the layer forward (dequantized_inverse)


@pytest.mark.parametrize("spec,bits", [(qo.SPEC8, 8), (qo.SPEC16, 16)])
def test_dequantized_inverse_padding_and_closeness(spec, bits):
    """Padding a partial tile with tokens that write nothing (zero rows and
    columns) leaves an identity block (the integer recipe keeps every power
    block diagonal), and the dequantised inverse stays within the pinned
    integer error of the float64 T_hat(N, S); all-ones A stays exact."""
    A = _blocked_A(64, 4)
    T = qo.dequantized_inverse(A, 3, 8, spec)
    Tf = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(Tf - np.eye(64)), axis=(-1, -2))
    assert np.all(np.max(np.abs(T - Tf), axis=(-1, -2)) <= 4 * 2.0 ** -bits * scale)
    m = 40
    Ap = np.zeros_like(A)
    Ap[:, :m, :m] = A[:, :m, :m]
    Tp = qo.dequantized_inverse(Ap, 3, 8, spec)
    n = A.shape[0]
    assert np.array_equal(Tp[:, m:, m:], np.broadcast_to(np.eye(64 - m), (n, 64 - m, 64 - m)))
    assert not np.any(Tp[:, m:, :m]) and not np.any(Tp[:, :m, m:])
    assert np.array_equal(qo.dequantized_inverse(A[:, :m, :m], 3, 8, spec, C=64), Tp[:, :m, :m])
    ones = np.tril(np.ones((1, 64, 64)), -1)
    assert np.array_equal(qo.dequantized_inverse(ones, 3, 8, spec)[0], np.eye(64) - np.eye(64, k=-1))


@pytest.mark.parametrize("spec,bits", [(qo.SPEC8, 8), (qo.SPEC16, 16)])
def test_forward_with_integer_inverse_close_to_float(spec, bits):
    """The layer forward (chunk-wise oracle) with the integer inverse differs
    from the one with the float64 T_hat(3, 8) only through the inverse's
    quantisation error: INT16 about 2^8 times closer than INT8."""
    from oracle import gdn_forward
    C = 64
    w = wl.workload("tiny").with_(B=1, L=2 * C, H=2, dk=32, dv=16, C=C)
    Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w, C=C)
    Of, Sf = gdn_forward.gdn_chunked(Q, K, V, beta, g, C, S0, 0.5,
                                     inverse=lambda A: gdn.neumann_inverse(A, 3, 8))
    Oi, Si = gdn_forward.gdn_chunked(Q, K, V, beta, g, C, S0, 0.5,
                                     inverse=lambda A: qo.dequantized_inverse(A, 3, 8, spec))
    err = max(np.max(np.abs(Oi - Of)) / np.max(np.abs(Of)), np.max(np.abs(Si - Sf)) / np.max(np.abs(Sf)))
    assert 0 < err <= 2.0 ** (6 - bits)
