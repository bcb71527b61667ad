"""Pins of the exact-integer (INT8 and INT16) oracle.

The paper fixes the quantiser q(x) = clip(round(x / Delta), qmin, qmax)
(Appendix G) and the method (Algorithm 1); where the integer tensors are
quantised is this library's reading, stated in oracle/int8.py: every
operator of Algorithm 1 is evaluated exactly and its result quantised once.
The pins check the rounding primitives against exact rational arithmetic,
the pipeline against a second coding in exact rational arithmetic
(fractions) on small tiles, hand-derived closed forms on structured inputs
(where every intermediate is a power of two, or where the quantised sum
loses its band to the outliers of the unmasked powers), and closeness of
the dequantised result to the float64 T_hat(N, S).
"""

from fractions import Fraction

import numpy as np
import pytest

import workloads as wl
from oracle import gdn
from oracle import int8 as qo


def _py_rne(y, s):
    return y if s <= 0 else round(Fraction(y, 1 << s))


def _py_nz(M):
    return any(v != 0 for row in M for v in row)


# (qmax, bits of a code, alignment bits) of the two integer settings
PY8 = (127, 7, 23)
PY16 = (32639, 15, 31)


def _stress_A(C, seed, L=None):
    k, b, g, _ = wl.gen_stress_head(L=L or 2 * C, dk=32, C=C, seed=seed)
    return gdn.tiles_flat(gdn.build_A(k[None, :, None], b[None, :, None], g[None, :, None], C))


def _workload_A(C, name="int8", h=0, tiles=2):
    k, b, g, _ = wl.gen_head(wl.workload(name), 0, h, C=C, want_v=False)
    n = tiles * C
    return gdn.tiles_flat(gdn.build_A(k[None, :n, None], b[None, :n, None], g[None, :n, None], C))


# ---------------------------------------------------------------------------
# rounding primitives


def test_rne_shift_matches_exact_rounding():
    rng = np.random.default_rng(0)
    ys = rng.integers(-(1 << 24), 1 << 24, 4000)
    ss = rng.integers(0, 26, 4000)
    got = qo.rne_shift(ys, ss)
    for y, s, g in zip(ys.tolist(), ss.tolist(), got.tolist()):
        assert g == round(Fraction(y, 1 << s))  # Python rounds halves to even
    # exact halves both ways
    assert qo.rne_shift(np.array([1, 3, -1, -3, 5, -5]), 1).tolist() == [0, 2, 0, -2, 2, -2]


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_quantize_minimal_exponent_and_roundtrip(spec):
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((50, 16, 16)) * np.exp(rng.uniform(-20, 5, (50, 1, 1)))).astype(np.float32)
    q, e = qo.quantize(x, spec)
    amax = np.max(np.abs(x.astype(np.float64)), axis=(-1, -2))
    # amax / 2^e < qmax + 1/2 <= amax / 2^(e-1): the finest scale at which
    # rounding keeps every code in range
    assert np.all(amax < (spec.qmax + 0.5) * np.ldexp(1.0, e))
    assert np.all(amax >= (spec.qmax + 0.5) * np.ldexp(1.0, e - 1))
    assert np.all(np.abs(q) <= spec.qmax)
    err = np.abs(qo.dequant(q, e) - x)
    assert np.all(err <= np.ldexp(0.5, e)[..., None, None])
    # exactly representable values come back exactly
    q0 = rng.integers(-spec.qmax, spec.qmax + 1, (10, 8, 8))
    q0[:, 0, 0] = spec.qmax
    e0 = rng.integers(-30, 5, 10)
    x0 = qo.dequant(q0, e0).astype(np.float32)
    if spec.qbits <= 23:
        q1, e1 = qo.quantize(x0, spec)
        assert np.array_equal(q1, q0) and np.array_equal(e1, e0)
    # all-zero tile
    qz, ez = qo.quantize(np.zeros((1, 4, 4), np.float32), spec)
    assert np.all(qz == 0) and ez[0] == 0


def _fr_exp(amax, qmax):
    """The smallest e with round(amax / 2^e) <= qmax (Python's round: half
    to even), searched over the rationals."""
    e = 0
    while round(amax / Fraction(2) ** e) > qmax:
        e += 1
    while round(amax / Fraction(2) ** (e - 1)) <= qmax:
        e -= 1
    return e


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_requant_is_the_quantiser_on_exact_values(spec):
    """requant(Y, e) = the quantiser's rule applied to the rational values
    Y 2^e: the smallest exponent at which the rounded codes fit (shifting
    left when the values are small), codes rounded half to even; int64 and
    Python-integer inputs (values past 2^62) alike."""
    rng = np.random.default_rng(2)
    for t in range(300):
        hi = 1 << int(rng.integers(1, 45))
        Y = rng.integers(-hi, hi, (3, 3))
        if t % 7 == 0:
            Y = Y.astype(object) * (1 << 70) + 1  # beyond int64
        e = int(rng.integers(-40, 40))
        q, eo = qo.requant(np.asarray(Y)[None], np.array([e]), spec)
        vals = [Fraction(int(v)) * Fraction(2) ** e for v in np.ravel(Y)]
        amax = max(abs(v) for v in vals)
        if amax == 0:
            assert eo[0] == 0 and not np.any(q)
            continue
        E = _fr_exp(amax, spec.qmax)
        assert int(eo[0]) == E
        assert [int(v) for v in np.ravel(q)] == [round(v / Fraction(2) ** E) for v in vals]
    # the INT16 bound: codes above 32639 move the exponent up even below 2^15
    q, eo = qo.requant(np.array([[[16350]]]), np.array([0]), qo.SPEC16)
    assert int(eo[0]) == 0 and int(q[0, 0, 0]) == 16350
    q, eo = qo.requant(np.array([[[32700]]]), np.array([0]), qo.SPEC16)
    assert int(eo[0]) == 1 and int(q[0, 0, 0]) == 16350
    # a value whose rounding lands on qmax keeps the finer scale; one whose
    # rounding would reach qmax + 1 does not (255 / 2 = 127.5 rounds to 128)
    q, eo = qo.requant(np.array([[[254, 3]]]), np.array([0]))
    assert int(eo[0]) == 1 and q[0].tolist() == [[127, 2]]
    q, eo = qo.requant(np.array([[[255, 3]]]), np.array([0]))
    assert int(eo[0]) == 2 and q[0].tolist() == [[64, 1]]


def test_exact_sum_is_exact():
    """exact_sum carries every term exactly (aligned at the finest exponent
    of the non-zero terms), also across exponent gaps beyond int64."""
    rng = np.random.default_rng(3)
    for t in range(100):
        n = int(rng.integers(1, 4))
        gap = int(rng.integers(0, 90))
        terms = []
        for k in range(n):
            q = rng.integers(-(1 << 20), 1 << 20, (2, 3, 3))
            if rng.random() < 0.2:
                q[0] = 0  # an all-zero term in one tile
            e = rng.integers(-gap - 10, 10, 2)
            terms.append((q, e))
        Y, em = qo.exact_sum(terms)
        for b in range(2):
            for i in range(3):
                for j in range(3):
                    want = sum(Fraction(int(q[b, i, j])) * Fraction(2) ** int(e[b])
                               for q, e in terms)
                    got = Fraction(int(Y[b, i, j])) * Fraction(2) ** int(em[b])
                    assert got == want


# ---------------------------------------------------------------------------
# a second coding of the pipeline in exact rational arithmetic: every
# statement of Algorithm 1 evaluated on fractions, its result passed through
# the quantiser q(); the unit diagonal of T0, T and T_hat kept out of the
# quantised tensor (split form) or inside it (plain form)


def _fr_q(M, qmax):
    """q() of a matrix of fractions: (codes, e) with the quantiser's rule."""
    amax = max(abs(v) for row in M for v in row)
    if amax == 0:
        return [[0] * len(M[0]) for _ in M], 0
    e = _fr_exp(amax, qmax)
    sc = Fraction(2) ** e
    return [[round(v / sc) for v in row] for row in M], e


def _fr_val(codes, e):
    sc = Fraction(2) ** e
    return [[c * sc for c in row] for row in codes]


def _fr_mm(X, Y):
    n = len(X)
    return [[sum(X[i][k] * Y[k][j] for k in range(n)) for j in range(n)] for i in range(n)]


def _fr_add(X, Y):
    return [[a + b for a, b in zip(r, s)] for r, s in zip(X, Y)]


def _fr_pipeline(qA, eA, N, S, qmax, plain=False):
    C = len(qA)
    I = [[Fraction(int(i == j)) for j in range(C)] for i in range(C)]
    Z = [[Fraction(0)] * C for _ in range(C)]
    A = [[Fraction(qA[i][j]) * Fraction(2) ** eA if i > j else Fraction(0) for j in range(C)]
         for i in range(C)]
    L = [[-v for v in row] for row in A]
    q = lambda M: _fr_val(*_fr_q(M, qmax))
    unit = (lambda M: _fr_add(I, M)) if not plain else (lambda M: M)   # tensor -> value
    strip = (lambda M: _fr_add(M, [[-v for v in r] for r in I])) if not plain else (lambda M: M)
    # T0 = I + sum P_n, P_n = P_{n-1} L
    T0 = Z if not plain else I  # the quantised tensor (strict part in split form)
    P = None
    for n in range(1, N + 1):
        P = L if n == 1 else q(_fr_mm(P, L))
        T0 = q(strip(_fr_add(unit(T0), P)))
    T0 = [[T0[i][j] if i - j <= N else Fraction(0) for j in range(C)] for i in range(C)]
    # E = I - q((I + A) T0)
    M = q(strip(_fr_mm(_fr_add(I, A), unit(T0))))
    E = q(_fr_add(I, [[-v for v in r] for r in unit(M)]))
    T = Z if not plain else I
    for s in range(1, S + 1):
        P = E if s == 1 else q(_fr_mm(P, E))
        T = q(strip(_fr_add(unit(T), P)))
    return _fr_q(strip(_fr_mm(unit(T0), unit(T))), qmax)


def _random_codes(C, qmax, seed, n=2):
    rng = np.random.default_rng(seed)
    q = rng.integers(-qmax, qmax + 1, (n, C, C))
    q = np.where(gdn.subdiag_index(C) > 0, q, 0)
    # sparse tiles and tiles with one large code make uneven scales
    q[0][rng.random((C, C)) < 0.7] = 0
    e = rng.integers(-12, 2, n)
    return q, e


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
@pytest.mark.parametrize("plain", [False, True])
@pytest.mark.parametrize("src,C,N,S", [("stress", 8, 3, 2), ("stress", 8, 1, 3),
                                       ("stress", 16, 3, 2), ("stress", 16, 2, 5),
                                       ("stress", 8, 0, 3), ("stress", 8, 3, 0),
                                       ("workload", 16, 3, 2), ("random", 8, 3, 4),
                                       ("random", 16, 2, 3)])
def test_pipeline_matches_rational_coding(spec, plain, src, C, N, S):
    if src == "random":
        qA, eA = _random_codes(C, spec.qmax, C * 10 + N + S + spec.qbits)
    else:
        A = _stress_A(C, C + N + S) if src == "stress" else _workload_A(C)
        qA, eA = qo.quantize(A.astype(np.float32), spec)
    qT, eT, _ = qo.neumann_inverse_int(qA, eA, N, S, spec, plain=plain)
    for t in range(qA.shape[0]):
        Tp, ep = _fr_pipeline(qA[t].tolist(), int(eA[t]), N, S, spec.qmax, plain)
        assert qT[t].tolist() == Tp
        assert int(eT[t]) == ep


# ---------------------------------------------------------------------------
# closed forms on structured inputs


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_zero_and_single_entry(spec):
    """A = 0 gives T_hat = I (split: no codes; plain: the identity at the
    smallest exponent that holds 1).  A with one non-zero entry has A^2 = 0,
    so every power past the first vanishes: on the band (i - j <= N) T0 =
    I - A and E = 0, off the band T0 = I and E = -A with E^2 = 0; either way
    T_hat = I - A exactly."""
    C = 16
    z = np.zeros((1, C, C), np.int64)
    for N, S in ((3, 2), (0, 0), (5, 7)):
        qT, eT, _ = qo.neumann_inverse_int(z, np.zeros(1, np.int64), N, S, spec)
        assert not np.any(qT) and eT[0] == 0
        qT, eT, _ = qo.neumann_inverse_int(z, np.zeros(1, np.int64), N, S, spec, plain=True)
        e1 = -(spec.qbits - 1)  # 1 = 2^(qbits-1) 2^e1 and 2^qbits > qmax
        assert eT[0] == e1 and np.array_equal(qT[0], np.eye(C, dtype=np.int64) << (spec.qbits - 1))
    rng = np.random.default_rng(5)
    for t in range(20):
        i = int(rng.integers(1, C))
        j = int(rng.integers(0, i))
        qA = np.zeros((1, C, C), np.int64)
        qA[0, i, j] = int(rng.integers(1, spec.qmax + 1)) * (1 if t % 2 else -1)
        eA = np.array([int(rng.integers(-20, 3))])
        qT, eT, parts = qo.neumann_inverse_int(qA, eA, 3, 4, spec)
        want = qo.dequant(-qA, eA)[0]
        assert np.array_equal(qo.dequant(qT, eT)[0], want)
        if i - j <= 3:
            assert not np.any(parts["E"][0])
        else:
            assert np.array_equal(qo.dequant(*parts["E"])[0], want)


@pytest.mark.parametrize("spec,S", [(qo.SPEC8, 2), (qo.SPEC8, 8), (qo.SPEC16, 3), (qo.SPEC16, 8)])
@pytest.mark.parametrize("C", [16, 64])
def test_half_subdiagonal_gives_the_quantised_inverse(spec, S, C):
    """A = Z/2 (Z the unit sub-diagonal): X = sum_d (-1/2)^d Z^d.  Every
    power, T0 = I - Z/2 + Z^2/4 - Z^3/8 and E = Z^4/16 are exact, and so are
    the residual powers 2^(-4s) Z^(4s) as long as they fit the 8 (16) bits
    of the running sum T, i.e. up to s = 2 (s = 4); T_hat's strict part then
    holds (-1/2)^d up to d = 11 (19), which its exponent -7 (-15) rounds to
    the codes of X's strict part: T_hat = q(X) exactly.  In plain form the
    identity sets the scale (1 = 2^(qbits-1) 2^e): T = I + Z^4/16 (+ Z^8/256
    and Z^12/4096 at 16 bits) and T_hat = q(X) again, at the exponent of 1."""
    A = np.full((1, C, C), 0.0)
    A[0][gdn.subdiag_index(C) == 1] = 0.5
    X = gdn.forward_substitution_inverse(A)
    qA, eA = qo.quantize(A.astype(np.float32), spec)
    qT, eT, parts = qo.neumann_inverse_int(qA, eA, 3, S, spec)
    qX, eX = qo.quantize((X - np.eye(C)).astype(np.float32), spec)
    assert eT[0] == eX[0] == -spec.qbits
    assert np.array_equal(qT, qX)
    d = gdn.subdiag_index(C)
    assert np.array_equal(qo.dequant(*parts["E"])[0], np.where(d == 4, 1 / 16, 0.0))
    assert np.array_equal(qo.dequant(*parts["T0"])[0],
                          np.where((d >= 1) & (d <= 3), (-0.5) ** np.maximum(d, 0), 0.0))
    qP, eP, _ = qo.neumann_inverse_int(qA, eA, 3, S, spec, plain=True)
    qXp, eXp = qo.quantize(X.astype(np.float32), spec)
    assert eP[0] == eXp[0] == 1 - spec.qbits
    assert np.array_equal(qP, qXp)


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_off_band_powers_of_two_are_exact(spec):
    """A = Z^4 / 2 at C = 16, N = 3: A has nothing on the band d <= 3, so the
    masked T0 = I and E = -A; the residual powers (-1/2)^s Z^(4s) are exact,
    and with (S + 1)(N + 1) >= C the result is the exact inverse,
    X = I - Z^4/2 + Z^8/4 - Z^12/8."""
    C, N, S = 16, 3, 3
    d = gdn.subdiag_index(C)
    A = np.where(d == 4, 0.5, 0.0)[None]
    qA, eA = qo.quantize(A.astype(np.float32), spec)
    qT, eT, parts = qo.neumann_inverse_int(qA, eA, N, S, spec)
    X = np.eye(C) + np.where((d > 0) & (d % 4 == 0), (-0.5) ** (d // 4), 0.0)
    assert np.array_equal(qo.dequant_unit(qT, eT)[0], X)
    assert not np.any(parts["T0"][0])
    assert np.array_equal(parts["E"][0], -qA) and np.array_equal(parts["E"][1], eA)


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_mask_after_the_quantised_sum(spec):
    """Algorithm 1 masks T0 once, after its sum.  For the all-ones A (GDN
    sign) the unmasked powers reach |L^3|_ij = binom(d - 1, 2), up to
    binom(62, 2) = 1891 at C = 64, and T0 = I + L + L^2 + L^3 about 1830:
    at 8 bits its exponent is 4, whose quantum 16 rounds the band entries
    (-1, 0, 0 for d = 1, 2, 3) to 0, so the masked T0 is I and E = -A.  At
    16 bits (exponent -4) the band survives exactly: T0 = I - Z, E = 0 and
    T_hat = I - Z, the exact inverse."""
    C = 64
    A = np.tril(np.ones((1, C, C), np.float32), -1)
    qA, eA = qo.quantize(A, spec)
    qT, eT, parts = qo.neumann_inverse_int(qA, eA, 3, 8, spec)
    d = gdn.subdiag_index(C)
    if spec.qbits == 7:
        T0 = parts["T0"]
        assert not np.any(T0[0])
        assert np.array_equal(qo.dequant(*parts["E"]), -A.astype(np.float64))
    else:
        assert np.array_equal(qo.dequant(*parts["T0"])[0], np.where(d == 1, -1.0, 0.0))
        assert not np.any(parts["E"][0])
        assert np.array_equal(qo.dequant_unit(qT, eT)[0], np.eye(C) - np.eye(C, k=-1))


def test_residual_keeps_the_rounding_of_T0():
    """E = I - (I + A) T0 is formed from the quantised T0, so on the band
    d <= N, where T0 would equal the inverse in real arithmetic, E holds
    T0's rounding error instead of zero (A = a Z with a = 90/128: the power
    a^2 = 8100/16384 is rounded in P_2 and again in the sum T0, so E's
    second sub-diagonal is -(t2 + a t1), t1 = -a and t2 the entries of T0's
    first two sub-diagonals, up to E's own rounding); the residual
    correction then removes that error too."""
    C, N = 16, 3
    d = gdn.subdiag_index(C)
    a = 90 / 128
    A = np.where(d == 1, a, 0.0)[None]
    qA, eA = qo.quantize(A.astype(np.float32))
    assert qA[0, 1, 0] == 90 and eA[0] == -7
    _, _, parts = qo.neumann_inverse_int(qA, eA, N, 8)
    E = qo.dequant(*parts["E"])[0]
    T0 = qo.dequant(*parts["T0"])[0]
    assert T0[1, 0] == -a and T0[2, 0] != a * a
    want = -(T0[2, 0] + a * T0[1, 0])
    assert E[2, 0] != 0 and abs(E[2, 0] - want) <= 2.0 ** (int(parts["E"][1][0]) - 1)
    # with S = 8 the error against the exact inverse of the quantised A is
    # below the quantum of T_hat; without correction (S = 0) it is T0's
    X = gdn.forward_substitution_inverse(A)
    err = lambda S: np.max(np.abs(qo.dequant_unit(*qo.neumann_inverse_int(qA, eA, N, S)[:2]) - X))
    assert err(8) < err(0)


# ---------------------------------------------------------------------------
# accuracy in the paper's setting


@pytest.mark.parametrize("spec,bits", [(qo.SPEC8, 8), (qo.SPEC16, 16)])
@pytest.mark.parametrize("gate", ["default", "wide"])
def test_close_to_float_approximation(spec, bits, gate):
    """Dequantised integer T_hat(3, 8) against the float64 T_hat(3, 8) on the
    workload distributions (fast decay, |A| <= ~0.2): each quantisation keeps
    qbits bits relative to its tensor's largest entry, so the error stays a
    small multiple of 2^-bits max|T_hat - I|; 16-bit codes land well over
    32 times closer than 8-bit ones."""
    A = _workload_A(64, "int8" if gate == "wide" else "tiny", tiles=4)
    qA, eA = qo.quantize(A.astype(np.float32), spec)
    qT, eT, _ = qo.neumann_inverse_int(qA, eA, 3, 8, spec)
    T = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qT, eT) - T), axis=(-1, -2))
    assert np.all(err <= 4 * 2.0 ** -bits * scale)
    if bits == 16:
        q8, e8 = qo.quantize(A.astype(np.float32))
        t8, f8, _ = qo.neumann_inverse_int(q8, e8, 3, 8)
        err8 = np.max(np.abs(qo.dequant_unit(t8, f8) - T))
        assert err8 > 32 * np.max(err)


def test_int16_stress_close_to_float():
    """Stress tiles (shared key direction, slow decay, |A| up to ~0.5): the
    unmasked powers grow, but 16 bits keep the band of T0 and the INT16
    result stays close to the float64 T_hat(3, 8)."""
    A = _stress_A(64, 9, L=256)
    qA, eA = qo.quantize(A.astype(np.float32), qo.SPEC16)
    qT, eT, _ = qo.neumann_inverse_int(qA, eA, 3, 8, qo.SPEC16)
    T = gdn.neumann_inverse(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit(qT, eT) - T), axis=(-1, -2))
    assert np.all(err <= 64 * 2.0 ** -16 * scale)


def test_split_form_beats_plain_form_at_8_bits():
    """Keeping the unit diagonal out of the codes (split form) leaves the
    small off-diagonal entries of T0, T and T_hat their own scale; with the
    identity inside (plain form) the scale is at least 1.  On the workload
    tiles the split form is several times closer to the exact inverse."""
    A = _workload_A(64, "int8", tiles=4)
    X = gdn.forward_substitution_inverse(A)
    qA, eA = qo.quantize(A.astype(np.float32))
    qs, es, _ = qo.neumann_inverse_int(qA, eA, 3, 8)
    qp, ep, _ = qo.neumann_inverse_int(qA, eA, 3, 8, plain=True)
    err_split = np.max(np.abs(qo.dequant_unit(qs, es) - X))
    err_plain = np.max(np.abs(qo.dequant(qp, ep) - X))
    assert err_plain > 3 * err_split


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_structure(spec):
    """Split form: strict part only, codes in range, the exponent of the
    smallest scale that fits (the largest code above qmax / 2); the
    residual powers vanish below the s-th sub-diagonal; plain form: lower
    triangular with the diagonal."""
    A = _workload_A(64, "tiny", h=1, tiles=2)
    qA, eA = qo.quantize(A.astype(np.float32), spec)
    N, S = 3, 8
    qT, eT, parts = qo.neumann_inverse_int(qA, eA, N, S, spec)
    d = gdn.subdiag_index(64)
    assert np.all(qT[:, d <= 0] == 0)
    assert np.all(np.abs(qT) <= spec.qmax)
    assert np.all(np.max(np.abs(qT), axis=(-1, -2)) > spec.qmax // 2)
    for s, (q, e) in enumerate(parts["chain"], start=1):
        assert np.all(q[:, d < s] == 0)
    qp, ep, _ = qo.neumann_inverse_int(qA, eA, N, S, spec, plain=True)
    assert np.all(qp[:, d < 0] == 0) and np.all(np.diagonal(qp, axis1=-2, axis2=-1) != 0)


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




# ---------------------------------------------------------------------------
# C = 128, block-wise (Appendix E with 64 x 64 blocks, Appendix H): three
# exponents per tile, X21 = -X22 A21 X11 as two MatMuls, each one rounding


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


def _fr_blocked(qA, eA, N, S, qmax):
    """Second coding of the block-wise inverse on small tiles, in exact
    rational arithmetic: the diagonal blocks by _fr_pipeline, then
    P = q(A21 (I + N11)) and X21 = -q((I + N22) P)."""
    C = len(qA)
    h = C // 2
    blk = lambda r, c: [row[c:c + h] for row in qA[r:r + h]]
    N11, e11 = _fr_pipeline(blk(0, 0), eA[0], N, S, qmax)
    N22, e22 = _fr_pipeline(blk(h, h), eA[2], N, S, qmax)
    I = [[Fraction(int(i == j)) for j in range(h)] for i in range(h)]
    A21 = _fr_val(blk(h, 0), eA[1])
    Pq, eP = _fr_q(_fr_mm(A21, _fr_add(I, _fr_val(N11, e11))), qmax)
    X21, e21 = _fr_q(_fr_mm(_fr_add(I, _fr_val(N22, e22)), _fr_val(Pq, eP)), qmax)
    out = [[0] * C for _ in range(C)]
    for i in range(h):
        for j in range(h):
            out[i][j] = N11[i][j]
            out[h + i][h + j] = N22[i][j]
            out[h + i][j] = -X21[i][j]
    return out, [e11, e21, e22]


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
@pytest.mark.parametrize("C,N,S", [(16, 3, 2), (16, 1, 3), (32, 2, 2)])
def test_blocked_matches_rational_coding(spec, C, N, S):
    A = _blocked_A(C, C + N, stress=True).astype(np.float32)
    qA, eA = qo.quantize_blocked(A, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, N, S, spec)
    for t in range(A.shape[0]):
        Tp, ep = _fr_blocked(qA[t].tolist(), [int(v) for v in eA[t]], N, S, spec.qmax)
        assert qT[t].tolist() == Tp
        assert [int(v) for v in eT[t]] == ep


@pytest.mark.parametrize("spec", [qo.SPEC8, qo.SPEC16])
def test_blocked_closed_forms(spec):
    """A21 = 0: X21 = 0 and the diagonal blocks are the 64 x 64 integer
    inverses; A11 = A22 = 0: A^2 = 0, so (I + A)^-1 = I - A and the codes of
    X21 are those of -A21 at A21's exponent; A = Z/2 across the block
    boundary: both merge products are exact and X21 carries the quantised
    (-1/2)^d of X (its codes round to 0 past the block's exponent)."""
    A = _blocked_A(128, 2).astype(np.float32)
    Ad = A.copy()
    Ad[:, 64:, :64] = 0.0
    qA, eA = qo.quantize_blocked(Ad, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    assert not np.any(qT[:, 64:, :64]) and np.all(eT[:, 1] == 0)
    for k, s in ((0, slice(0, 64)), (2, slice(64, 128))):
        q1, e1 = qo.quantize(np.tril(A[:, s, s], -1), spec)
        t1, f1, _ = qo.neumann_inverse_int(q1, e1, 3, 8, spec)
        assert np.array_equal(qT[:, s, s], t1) and np.array_equal(eT[:, k], f1)
    Ao = np.zeros_like(A)
    Ao[:, 64:, :64] = A[:, 64:, :64]
    qA, eA = qo.quantize_blocked(Ao, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    assert np.array_equal(qT[:, 64:, :64], -qA[:, 64:, :64]) and np.array_equal(eT[:, 1], eA[:, 1])
    assert not np.any(qT[:, :64, :64]) and not np.any(qT[:, 64:, 64:])
    # A = Z / 2: A21 has the single entry 1/2 at (64, 63); P = A21 X11 is
    # row 0 of 1/2 X11's last row, X21 = -X22 P; with X11, X22 the
    # quantised inverses (exact on the sub-diagonals their codes hold) both
    # products are exact and X21 = q(-(1/2) x22[:, 0] x11[63, :])
    C = 128
    d = gdn.subdiag_index(C)
    Ah = np.where(d == 1, 0.5, 0.0)[None].astype(np.float32)
    qA, eA = qo.quantize_blocked(Ah, spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    D = qo.dequant_unit_blocked(qT, eT)[0]
    x11 = D[:64, :64]
    x22 = D[64:, 64:]
    want = -0.5 * np.outer(x22[:, 0], x11[63, :])
    q21, e21 = qo.quantize(want[None].astype(np.float32), spec)
    assert np.array_equal(qT[0, 64:, :64], q21[0]) and eT[0, 1] == e21[0]


@pytest.mark.parametrize("spec,bits", [(qo.SPEC8, 8), (qo.SPEC16, 16)])
def test_blocked_close_to_float_approximation(spec, bits):
    """Dequantised block-wise inverse against the float64 block-wise
    T_hat(3, 8) (Appendix E formula on float64 diagonal inverses) on the
    workload distributions: the merge adds two quantisations and X22's gain
    to the diagonal blocks' error."""
    A = _blocked_A(128, 3)
    qA, eA = qo.quantize_blocked(A.astype(np.float32), spec)
    qT, eT = qo.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    T = gdn.neumann_inverse_blocked(A, 3, 8)
    scale = np.max(np.abs(T - np.eye(128)), axis=(-1, -2))
    err = np.max(np.abs(qo.dequant_unit_blocked(qT, eT) - T), axis=(-1, -2))
    assert np.all(err <= 16 * 2.0 ** -bits * scale)


# ---------------------------------------------------------------------------
# the integer inverse inside the layer forward (dequantized_inverse)


@pytest.mark.parametrize("spec,bits", [(qo.SPEC8, 8), (qo.SPEC16, 16)])
def test_dequantized_inverse_padding_and_closeness(spec, bits):
    """Padding a partial tile with tokens that write nothing (zero rows and
    columns) leaves an identity block (every power and product keeps the
    block-diagonal structure), and the dequantised inverse stays within the
    pinned integer error of the float64 T_hat(N, S)."""
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
