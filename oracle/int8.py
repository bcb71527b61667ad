"""Exact-integer oracle of the low-bit (INT8 / INT16) inverse path.

Test infrastructure only: tests/, the smoke check and the bench's CPU
baseline call it; the library never does.

The paper runs the masked truncated Neumann expansion and the residual
correction (Algorithm 1, Sections 3.1-3.4) with integer activations
(Section 3.5; Appendix G: the uniform symmetric quantiser
q(x) = clip(round(x / Delta), qmin, qmax), one scale per tensor, INT16 or
INT8 for the matrix inversion).  It does not spell out where the tensors are
quantised.  This module reads Algorithm 1 as a sequence of integer
operators, each of whose outputs is an activation tensor quantised per
tensor:

  * A tensor is codes q with |q| <= qmax and one power-of-two scale
    Delta = 2^e per tile (value q 2^e).  qmax = 127 (INT8; the symmetric
    range, so that negation is exact) or 32639 (INT16; 127 * 256 + 127, so
    that a code splits into two int8 limbs).
  * quantisation of an exactly known tensor v (requant): q =
    round-half-even(v / 2^e) with e the smallest integer at which no code
    leaves [-qmax, qmax], i.e. the finest power-of-two scale at which the
    clip of q(x) does nothing (max|v| < (qmax + 1/2) 2^e).  The same rule
    quantises the float input A (quantize).  An all-zero tensor gets q = 0,
    e = 0.
  * Every operator is evaluated exactly from the codes of its operands and
    its result is quantised once: a MatMul (P <- P A, P <- P E, the final
    T0 T), an Add (T0 <- T0 + P, T <- T + P), and the residual
    E <- I - (I + A) T0, which is the one MatMul (I + A) T0 = T0 + A T0
    followed by the subtraction from I (exact: it cancels the identity).
    The mask M^(N) zeroes codes and keeps the scale (exact).
  * The order is Algorithm 1's: the powers P_n = P_{n-1} L (L = -A, the
    GDN sign) summed into T0, T0 masked once after the sum, E, the residual
    powers P_s = P_{s-1} E summed into T = sum_{s<=S} E^s, and the result
    T0 T (the order of the equation of Section 3.4 and of Appendix D; the
    printed last line T T0 does not converge to the inverse).
  * Split form (the default): the unit diagonal of T0, T and T_hat is kept
    outside the codes, exact, so only their strict lower parts are
    quantised: (I + X)(I + Y) has strict part X + Y + X Y, one rounding.
    Plain form (plain=True): every tensor, identity included, is one tensor
    of codes.  Keeping the unit diagonal exact is a dynamic-range
    mitigation of this library on top of the paper's low order and masking
    (Sections 3.2, 3.3): with the diagonal inside the codes the scale of
    T0, T and T_hat is at least 1, which leaves INT8 about 6 bits for the
    small off-diagonal entries.

All arithmetic after quantize() is on integers: exact sums align their terms
at the finest exponent (numpy int64 when the bounds allow, Python integers
otherwise).

C = 128 runs block-wise (Appendix E, with the 64 x 64 blocks Appendix H
names as the smallest for the integer settings): quantize_blocked gives each
of the blocks A11, A21, A22 its own exponent, neumann_inverse_int_blocked
inverts the diagonal blocks by neumann_inverse_int and forms
X21 = -X22 A21 X11 as two MatMuls from the right, P = A21 X11 and X22 P,
each one rounding of its exact result (the identity parts of X11 and X22
exact).

The integer forward substitution (fwdsub_inverse_int) is the baseline of
the comparison in Appendix I (a "naive" INT16 inverse); it keeps its own
reading, documented there.
"""

from __future__ import annotations

import dataclasses
from typing import List, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class Spec:
    qmax: int        # codes q in [-qmax, qmax]
    qbits: int       # 2^(qbits - 1) <= qmax < 2^qbits
    align_bits: int  # (forward substitution) aligned terms stay below 2^align_bits
    sum_bits: int    # (forward substitution) sums stay below 2^sum_bits


SPEC8 = Spec(qmax=127, qbits=7, align_bits=23, sum_bits=31)
SPEC16 = Spec(qmax=32639, qbits=15, align_bits=31, sum_bits=37)

QMAX = SPEC8.qmax

_I64_BITS = 60  # int64 values are kept below 2^60


# ----------------------------------------------------------------------------
# rounding primitives


def rne_shift(y: np.ndarray, s) -> np.ndarray:
    """round-half-even(y / 2^s) for integer y (int64, |y| < 2^60) and integer
    s >= 0 (per element or broadcast)."""
    y = np.asarray(y, dtype=np.int64)
    assert np.all(np.abs(y) < (1 << 60))
    s = np.asarray(s, dtype=np.int64)
    # |y| < 2^60 gives |y| / 2^s < 1/2 for s >= 62: the result is 0, which
    # shifting by 62 also yields (floor 0 or -1, remainder below one half).
    s_b = np.minimum(np.broadcast_to(s, y.shape), 62)
    out = y.copy()
    pos = s_b > 0
    if np.any(pos):
        ss = np.where(pos, s_b, 0)
        q = y >> ss  # floor
        r = y - (q << ss)
        half = np.where(pos, np.int64(1) << np.maximum(ss - 1, 0), 0)
        up = (r > half) | ((r == half) & ((q & 1) == 1))
        out = np.where(pos, q + up.astype(np.int64), y)
    return out


def _py_rne(y: int, s: int) -> int:
    """round-half-even(y / 2^s) for Python integers, any s (s <= 0 exact)."""
    if s <= 0:
        return y << -s
    q = y >> s
    r = y - (q << s)
    h = 1 << (s - 1)
    return q + (1 if (r > h or (r == h and (q & 1))) else 0)


def _tile_amax(q: np.ndarray) -> np.ndarray:
    return np.max(np.abs(q), axis=(-1, -2))


def _bitlen(a: np.ndarray) -> np.ndarray:
    """bit length of non-negative integers (int64 or Python ints)."""
    a = np.asarray(a)
    if a.dtype != object:
        a = a.astype(np.int64)
        out = np.zeros(a.shape, np.int64)
        nz = a > 0
        out[nz] = np.floor(np.log2(a[nz].astype(np.float64))).astype(np.int64) + 1
        # correct the float estimate near powers of two
        out = np.where(nz & ((np.int64(1) << np.maximum(out - 1, 0)) > a), out - 1, out)
        out = np.where(nz & ((np.int64(1) << np.minimum(out, 62)) <= a) & (out < 63), out + 1, out)
        return out
    return np.vectorize(lambda v: int(v).bit_length(), otypes=[np.int64])(a)


def requant(Y: np.ndarray, e: np.ndarray, spec: Spec = SPEC8) -> Tuple[np.ndarray, np.ndarray]:
    """Quantise the exact values Y 2^e per tile (Y integers [..., R, C],
    int64 or Python ints; e [...]) by the quantiser's rule: codes
    round-half-even(Y 2^(e - e_out)) with e_out the smallest integer at
    which every code lies in [-qmax, qmax] (max|Y 2^e| < (qmax + 1/2)
    2^e_out).  Returns (codes int64, e_out); an all-zero tile gets codes 0,
    e_out 0."""
    Y = np.asarray(Y)
    e = np.asarray(e, dtype=np.int64)
    amax = _tile_amax(Y)
    b = _bitlen(amax)
    # max|Y| lies in [2^(b-1), 2^b), so max|Y| / 2^(b - qbits) is in
    # [2^(qbits-1), 2^qbits): the shift is b - qbits, or one more when that
    # quotient reaches qmax + 1/2 (whose rounding would leave the range)
    s = b - spec.qbits
    over = np.array([(2 * int(a) << max(-int(k), 0)) >= ((2 * spec.qmax + 1) << max(int(k), 0))
                     if int(a) > 0 else False
                     for a, k in zip(np.ravel(amax), np.ravel(s))], dtype=bool).reshape(np.shape(s))
    s = s + over.astype(np.int64)
    nz = np.asarray(amax) != 0
    s = np.where(nz, s, 0)
    if Y.dtype != object and np.all(b - np.minimum(s, 0) <= _I64_BITS):
        sb = s[..., None, None]
        q = np.where(sb > 0, rne_shift(Y.astype(np.int64), np.maximum(sb, 0)),
                     Y.astype(np.int64) << np.maximum(-sb, 0))
    else:
        flat_Y = Y.reshape((-1,) + Y.shape[-2:])
        flat_s = np.ravel(s)
        q = np.zeros(flat_Y.shape, np.int64)
        for t in range(flat_Y.shape[0]):
            st = int(flat_s[t])
            q[t] = np.array([[_py_rne(int(v), st) for v in row] for row in flat_Y[t]],
                            dtype=np.int64)
        q = q.reshape(Y.shape)
    assert np.all(np.abs(q) <= spec.qmax)
    return q, np.where(nz, e + s, 0)


def exact_sum(terms: List[Tuple[np.ndarray, np.ndarray]]) -> Tuple[np.ndarray, np.ndarray]:
    """Exact sum of q_k 2^(e_k) per tile: every term aligned at the finest
    exponent among the tile's non-zero terms.  terms: (q [..., R, C]
    integers, e [...]).  Returns (Y, e_min) with sum = Y 2^e_min (int64 when
    the bounds allow, Python integers otherwise); a tile with no non-zero
    term gets Y = 0, e_min = 0."""
    shape = np.asarray(terms[0][0]).shape
    bshape = shape[:-2]
    BIG = np.int64(1) << 62
    emin = np.full(bshape, BIG, np.int64)
    nzs = []
    for q, e in terms:
        q = np.asarray(q)
        e = np.broadcast_to(np.asarray(e, np.int64), bshape)
        nz = _tile_amax(q) != 0
        nzs.append(nz)
        emin = np.where(nz, np.minimum(emin, e), emin)
    emin = np.where(emin == BIG, 0, emin)
    need = np.zeros(bshape, np.int64)
    for (q, e), nz in zip(terms, nzs):
        e = np.broadcast_to(np.asarray(e, np.int64), bshape)
        need = np.maximum(need, np.where(nz, _bitlen(_tile_amax(np.asarray(q))) + (e - emin), 0))
    need = need + (len(terms) - 1).bit_length()
    if np.all(need <= _I64_BITS) and all(np.asarray(q).dtype != object for q, _ in terms):
        Y = np.zeros(shape, np.int64)
        for (q, e), nz in zip(terms, nzs):
            e = np.broadcast_to(np.asarray(e, np.int64), bshape)
            sh = np.where(nz, e - emin, 0)[..., None, None]
            Y = Y + np.where(nz[..., None, None], np.asarray(q, np.int64) << sh, 0)
        return Y, emin
    Y = np.zeros(shape, dtype=object)
    Y[...] = 0
    for (q, e), nz in zip(terms, nzs):
        e = np.broadcast_to(np.asarray(e, np.int64), bshape)
        qo = np.asarray(q).astype(object)
        for idx in np.ndindex(*bshape):
            if nz[idx]:
                sh = int(e[idx] - emin[idx])
                Y[idx] = Y[idx] + np.vectorize(lambda v: int(v) << sh, otypes=[object])(qo[idx])
    return Y, emin


def _mm(X: np.ndarray, Y: np.ndarray) -> np.ndarray:
    """Exact product of code matrices (|codes| <= 32639, at most 128 terms:
    below 2^37, exact in int64)."""
    return np.asarray(X, np.int64) @ np.asarray(Y, np.int64)


# ----------------------------------------------------------------------------
# quantisation of the float input


def quantize(x: np.ndarray, spec: Spec = SPEC8) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric per-tile quantiser with a power-of-two scale (Appendix G's
    q(x) with Delta = 2^e).

    x float32 tiles [..., C, C].  q = rne(x / 2^e) with e the smallest
    integer at which no code leaves [-qmax, qmax] (the clip never acts):
    amax / 2^e < qmax + 1/2.  From frexp, amax = m 2^p with m in [0.5, 1)
    gives amax / 2^(p - qbits) = 2^qbits m, which stays below qmax + 1/2
    unless m >= (qmax + 1/2) / 2^qbits (INT8: 128 m < 127.5).  All-zero tiles
    get q = 0, e = 0."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    amax = np.max(np.abs(x), axis=(-1, -2))
    m, p = np.frexp(amax)
    e = (p.astype(np.int64) - spec.qbits) + (m * float(1 << spec.qbits) >= spec.qmax + 0.5).astype(np.int64)
    e = np.where(amax > 0, e, 0)
    q = np.rint(np.ldexp(x, -e[..., None, None])).astype(np.int64)
    assert np.all(np.abs(q) <= spec.qmax)
    return q, e


# ----------------------------------------------------------------------------
# the integer inverse (Algorithm 1)


def _subdiag(C: int) -> np.ndarray:
    i = np.arange(C)[:, None]
    j = np.arange(C)[None, :]
    return i - j


def neumann_inverse_int(qA: np.ndarray, eA: np.ndarray, N: int, S: int, spec: Spec = SPEC8,
                        plain: bool = False):
    """Integer T_hat(N, S) (Algorithm 1 as integer operators) from the
    quantised GDN matrix (qA, eA).

    qA int [..., C, C] (only i > j is read), eA int [...].
    Split form (default): returns (qT, eT, parts) with T_hat = I + qT 2^eT,
    qT the codes of the strict lower part (zero on and above the diagonal).
    Plain form: T_hat = qT 2^eT, qT lower triangular with the diagonal.
    parts holds the intermediate tensors (codes, exponent): "T0" (masked;
    strict part in split form), "E", "T" (the residual sum; strict part in
    split form), "powers" (P_1 .. P_N) and "chain" (E^1 .. E^S)."""
    qA = np.asarray(qA, np.int64)
    eA = np.asarray(eA, np.int64)
    C = qA.shape[-1]
    bshape = qA.shape[:-2]
    d = _subdiag(C)
    qA = np.where(d > 0, qA, 0)
    rq = lambda Y, e: requant(Y, e, spec)
    zero = (np.zeros_like(qA), np.zeros(bshape, np.int64))
    eye = (np.broadcast_to(np.eye(C, dtype=np.int64), qA.shape).copy(), np.zeros(bshape, np.int64))
    L = (-qA, eA)  # L = -A (the paper's (I - L)^-1 with the GDN sign)

    # ---- T0 = sum_{n=0}^{N} L^n: P_n = P_{n-1} L, T0 <- T0 + P_n
    T0 = zero if not plain else eye
    powers = []
    P = None
    for n in range(1, N + 1):
        P = L if n == 1 else rq(_mm(P[0], L[0]), P[1] + L[1])
        powers.append(P)
        T0 = rq(*exact_sum([T0, P]))
    # ---- T0 <- M^(N) (.) T0 (codes masked, scale kept)
    T0 = (np.where(d <= N, T0[0], 0), T0[1])

    # ---- E = I - (I + A) T0: the MatMul (I + A) T0 = T0 + A T0, quantised,
    # then subtracted from I
    if not plain:
        # (I + A)(I + N0) = I + (A + N0 + A N0)
        M = rq(*exact_sum([(qA, eA), T0, (_mm(qA, T0[0]), eA + T0[1])]))
        E = (-M[0], M[1])
    else:
        M = rq(*exact_sum([T0, (_mm(qA, T0[0]), eA + T0[1])]))
        E = rq(*exact_sum([eye, (-M[0], M[1])]))

    # ---- T = sum_{s=0}^{S} E^s: P_s = P_{s-1} E, T <- T + P_s
    T = zero if not plain else eye
    chain = []
    for s in range(1, S + 1):
        P = E if s == 1 else rq(_mm(P[0], E[0]), P[1] + E[1])
        chain.append(P)
        T = rq(*exact_sum([T, P]))

    # ---- T_hat = T0 T
    if not plain:
        # (I + N0)(I + R) = I + (N0 + R + N0 R)
        Th = rq(*exact_sum([T0, T, (_mm(T0[0], T[0]), T0[1] + T[1])]))
    else:
        Th = rq(_mm(T0[0], T[0]), T0[1] + T[1])
    parts = {"T0": T0, "E": E, "T": T, "powers": powers, "chain": chain}
    return Th[0], Th[1], parts


def neumann_inverse_int8(qA, eA, N, S, spec: Spec = SPEC8, plain: bool = False):
    """neumann_inverse_int with 8-bit codes (SPEC8 unless another spec is given)."""
    return neumann_inverse_int(qA, eA, N, S, spec, plain)


def neumann_inverse_int16(qA, eA, N, S, plain: bool = False):
    """neumann_inverse_int with 16-bit codes (SPEC16)."""
    return neumann_inverse_int(qA, eA, N, S, SPEC16, plain)


# ----------------------------------------------------------------------------
# the forward-substitution baseline in integers


def _acc_bits(C: int, spec: Spec = SPEC8) -> int:
    # |acc| <= C * qmax^2 < C * 2^(2 qbits)
    return 2 * spec.qbits + int(np.ceil(np.log2(C)))


def aligned_sum(terms: List[Tuple[np.ndarray, np.ndarray, np.ndarray, int]],
                spec: Spec = SPEC8):
    """Running sum of q_k * 2^(e_k), terms taken in the given order (the
    integer forward substitution's row sums).

    terms: list of (q, e, present, bits) with q [..., R, C] int, e [...] int,
    present [...] bool, bits = log2 bound of |q| (7 for int8 codes, 14+log2 C
    for raw products).  Per tile, the sum keeps an exponent e_acc:
      * the first present term sets e_acc = e + bits - align_bits (its
        largest value sits just below 2^align_bits, leaving 16 guard bits
        under a code's quantum);
      * a later present term whose top e + bits would pass e_acc +
        align_bits first rebases the sum to e_acc' = e + bits - align_bits
        (acc = rne(acc / 2^d));
      * the term is then added exactly at e_acc (shifted left) or, when finer,
        rounded to it (round-half-even right shift).
    Absent terms are skipped.  Returns (sum, e_acc, any_present)."""
    shape = terms[0][0].shape[:-2]
    total = np.zeros(terms[0][0].shape, dtype=np.int64)
    e_acc = np.zeros(shape, dtype=np.int64)
    anyp = np.zeros(shape, dtype=bool)
    for q, e, p, bits in terms:
        q = np.asarray(q, np.int64)
        e = np.asarray(e, np.int64)
        p = np.asarray(p, bool)
        top = e + bits - spec.align_bits
        first = p & ~anyp
        rebase = p & anyp & (top > e_acc)
        dd = np.where(rebase, top - e_acc, 0)
        total = np.where(rebase[..., None, None], rne_shift(total, dd[..., None, None]), total)
        e_acc = np.where(first | rebase, top, e_acc)
        sh = (e - e_acc)[..., None, None]
        t = np.where(sh >= 0, q << np.maximum(sh, 0), rne_shift(q, np.maximum(-sh, 0)))
        total = total + np.where(p[..., None, None], t, 0)
        anyp |= p
    e_acc = np.where(anyp, e_acc, 0)
    assert np.all(np.abs(total) < (1 << spec.sum_bits))
    return total, e_acc, anyp


def _scale_rne(y: np.ndarray, d: np.ndarray) -> np.ndarray:
    """round-half-even(y * 2^-d) for integers y and any integer d (d < 0 is
    an exact left shift)."""
    y = np.asarray(y, np.int64)
    d = np.broadcast_to(np.asarray(d, np.int64), y.shape)
    return np.where(d >= 0, rne_shift(y, np.maximum(d, 0)), y << np.maximum(-d, 0))


def fwdsub_inverse_int(qA: np.ndarray, eA: np.ndarray, spec: Spec = SPEC16):
    """The forward-substitution baseline in integer arithmetic (this
    library's reading of an INT16 forward substitution: the recurrence of
    Section 2.2 on codes with one power-of-two exponent per tile, the
    per-tensor scheme of Appendix G).

    With Lm = -A (codes qL = -qA at eA), row i (i = 1 .. C-1) of the strict
    part X of (I + A)^-1 is t + t X_{0:i, 0:i} with t = row i of Lm and X's
    rows 0 .. i-1 already final, i.e. x_ij = -a_ij - sum_{j<k<i} a_ik x_kj.
    X holds codes qX with one exponent eX per tile, starting at eA.  Per row:
      * the two terms t (codes at eA, |t| < 2^qbits) and t X (exact products
        at eA + eX, below C 2^(2 qbits)) are summed by aligned_sum (present:
        t non-zero; t non-zero and X non-zero);
      * eX grows by the smallest s >= 0 with rne(max|row| / 2^(eX + s)) <=
        qmax; when s > 0 every earlier row is rounded to the new exponent
        (qX = rne(qX / 2^s));
      * the row's codes are rne(row / 2^eX), one rounding from the sum.
    Returns (qX codes, strict lower, and eX per tile); T = I + qX 2^eX."""
    qA = np.asarray(qA, np.int64)
    eA = np.asarray(eA, np.int64)
    C = qA.shape[-1]
    L = -np.tril(qA, -1)
    X = np.zeros_like(L)
    eX = eA.copy()
    accb = _acc_bits(C, spec)
    for i in range(1, C):
        t = L[..., i:i + 1, :]
        P = t @ X
        nzt = np.any(t != 0, axis=(-1, -2))
        nzX = np.any(X != 0, axis=(-1, -2))
        row, es, anyp = aligned_sum([(t, eA, nzt, spec.qbits), (P, eA + eX, nzt & nzX, accb)],
                                    spec)
        amax = np.max(np.abs(row), axis=(-1, -2))
        u = es - eX
        # start at a shift where amax 2^(u - s) < 2^16, then the smallest that fits
        bl = np.array([int(v).bit_length() for v in amax.ravel()], np.int64).reshape(amax.shape)
        s = np.where(amax > 0, np.maximum(0, bl + u - 16), 0)
        s = np.maximum(0, s - 1)
        while True:
            big = (amax > 0) & (_scale_rne(amax, s - u) > spec.qmax)
            if not np.any(big):
                break
            s = s + big.astype(np.int64)
        X = np.where((s > 0)[..., None, None], _scale_rne(X, s[..., None, None]), X)
        eX = eX + s
        codes = _scale_rne(row, (eX - es)[..., None, None])
        X[..., i, :] = np.where(anyp[..., None], codes[..., 0, :], 0)
        assert np.all(np.abs(X) <= spec.qmax)
    return X, eX


# ----------------------------------------------------------------------------
# C = 128: block-wise (Appendix E; Appendix H fixes 64 x 64 as the smallest
# block for the integer settings)


def _blocks(C: int):
    """(rows, cols) slices of the blocks 11, 21, 22 of a C x C tile split at
    C / 2 (block 12 is zero in a lower-triangular matrix)."""
    h = C // 2
    return ((slice(0, h), slice(0, h)), (slice(h, C), slice(0, h)), (slice(h, C), slice(h, C)))


def quantize_blocked(x: np.ndarray, spec: Spec = SPEC8) -> Tuple[np.ndarray, np.ndarray]:
    """The quantiser of quantize() applied block by block: the strict lower
    parts of the diagonal blocks A11, A22 and the whole block A21 each get
    their own power-of-two exponent.  x float32 tiles [..., C, C] (only
    i > j read).  Returns q [..., C, C] (zero on and above the diagonal)
    and e [..., 3] for the blocks (11, 21, 22)."""
    x = np.asarray(x, dtype=np.float32)
    C = x.shape[-1]
    x = np.where(_subdiag(C) > 0, x, np.float32(0))
    q = np.zeros(x.shape, np.int64)
    es = []
    for rs, cs in _blocks(C):
        qb, eb = quantize(x[..., rs, cs], spec)
        q[..., rs, cs] = qb
        es.append(eb)
    return q, np.stack(es, axis=-1)


def neumann_inverse_int_blocked(qA: np.ndarray, eA: np.ndarray, N: int, S: int,
                                spec: Spec = SPEC8):
    """Integer inverse of a tile split into two diagonal blocks (Appendix E:
    X11 = T11^-1, X22 = T22^-1, X21 = -X22 A21 X11).

    qA [..., C, C] codes with exponents eA [..., 3] for the blocks
    (11, 21, 22) as quantize_blocked writes them.  The diagonal blocks are
    inverted by neumann_inverse_int (split form, X = I + N).  The
    off-diagonal block is two MatMuls taken from the right, each evaluated
    exactly and quantised once, the identity parts of X11 and X22 exact:
      P   = A21 X11 = A21 + A21 N11,
      X21 = -(X22 P) = -(P + N22 P)
    (the sign is applied to the codes: round-half-even is symmetric).
    Returns qT [..., C, C] (N11, X21 and N22 in their blocks, zero on and
    above the diagonal) and eT [..., 3] for (N11, X21, N22): the inverse is
    I + each block's codes * 2^(its exponent)."""
    qA = np.asarray(qA, np.int64)
    eA = np.asarray(eA, np.int64)
    C = qA.shape[-1]
    b11, b21, b22 = _blocks(C)
    q11, e11, _ = neumann_inverse_int(qA[(Ellipsis,) + b11], eA[..., 0], N, S, spec)
    q22, e22, _ = neumann_inverse_int(qA[(Ellipsis,) + b22], eA[..., 2], N, S, spec)
    a21, ea = qA[(Ellipsis,) + b21], eA[..., 1]
    qP, eP = requant(*exact_sum([(a21, ea), (_mm(a21, q11), ea + e11)]), spec)
    q21, e21 = requant(*exact_sum([(qP, eP), (_mm(q22, qP), e22 + eP)]), spec)
    qT = np.zeros_like(qA)
    qT[(Ellipsis,) + b11] = q11
    qT[(Ellipsis,) + b21] = -q21
    qT[(Ellipsis,) + b22] = q22
    return qT, np.stack([e11, e21, e22], axis=-1)


def dequant_unit_blocked(qT: np.ndarray, eT: np.ndarray) -> np.ndarray:
    """I + (each block's codes) * 2^(its exponent), float64; eT [..., 3]."""
    qT = np.asarray(qT, np.float64)
    eT = np.asarray(eT)
    C = qT.shape[-1]
    out = np.zeros(qT.shape)
    for k, (rs, cs) in enumerate(_blocks(C)):
        out[(Ellipsis, rs, cs)] = np.ldexp(qT[(Ellipsis, rs, cs)], eT[..., k][..., None, None])
    return out + np.eye(C)


def dequantized_inverse(A: np.ndarray, N: int, S: int, spec: Spec = SPEC8,
                        C: int = 0) -> np.ndarray:
    """The integer T_hat(N, S) as a float64 inverse, for the layer forward's
    integer mode: the strictly lower A tiles [..., m, m] rounded to float32
    (the values the quantiser reads), quantised per tile, inverted by
    neumann_inverse_int and dequantised, I + qT 2^eT.  With C > m the tile
    is first padded to C x C with zero rows and columns (tokens that write
    nothing) and the top-left m x m block returned: the kernels run every
    chunk on C x C tiles."""
    A = np.asarray(A, np.float64)
    m = A.shape[-1]
    if C > m:
        P = np.zeros(A.shape[:-2] + (C, C))
        P[..., :m, :m] = A
        return dequantized_inverse(P, N, S, spec)[..., :m, :m]
    qA, eA = quantize(np.tril(A, -1).astype(np.float32), spec)
    qT, eT, _ = neumann_inverse_int(qA, eA, N, S, spec)
    return dequant_unit(qT, eT)


def dequant_unit(qT: np.ndarray, eT: np.ndarray) -> np.ndarray:
    """I + qT * 2^eT as float64."""
    C = qT.shape[-1]
    return np.eye(C) + np.ldexp(np.asarray(qT, np.float64), np.asarray(eT)[..., None, None])


def dequant(q: np.ndarray, e: np.ndarray) -> np.ndarray:
    return np.ldexp(np.asarray(q, np.float64), np.asarray(e)[..., None, None])
