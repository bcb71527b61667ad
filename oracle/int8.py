"""Exact-integer oracle of the low-bit (INT8) inverse path (test infrastructure only).

The paper (Section 3.5 and Appendix G) runs the masked truncated Neumann
expansion and the residual correction on integer hardware with a uniform
symmetric quantiser q(x) = clip(round(x / Delta), qmin, qmax) and a
per-tensor scale, and keeps the order low (N <= 3) so that the dynamic range
of the powers stays small.  It does not spell out the integer mechanics.
This module fixes them (one reading, applied identically by the GPU path):

  * A matrix is stored as int8 codes q in [-127, 127] and one exponent e per
    tile (value = q * 2^e, Delta = 2^e: a power-of-two per-tile scale).
    Unit lower-triangular matrices (T^(0), sum E^s, T_hat) are stored as
    I + (int8 strict part) * 2^e: the unit diagonal is kept exact.
  * quantize(x): e = smallest integer with max|x| / 2^e <= 127,
    q = round-half-even(x / 2^e).
  * Every int8 x int8 product is accumulated exactly in int32
    (|acc| <= C * 127^2 < 2^21 for C <= 64), then requantised ("per-power
    rescaling"): s = smallest s >= 0 with rne(max|acc| / 2^s) <= 127,
    q = rne(acc / 2^s), e = e1 + e2 + s.
  * Sums run in int32 in the order the terms are produced, at an exponent
    set by the first term (16 guard bits below an int8 quantum) and raised
    only when a later term would pass 2^23; terms finer than the running
    exponent are added with round-half-even (aligned_sum).  A term is present
    when the matrix it comes from is not identically zero (a product is
    present when both factors are).
  * The diagonal mask M^(N) is applied to every power before it is
    quantised (in exact arithmetic M (sum L^n) = sum M L^n, and masking first
    keeps the deep sub-diagonal outliers out of every scale).
  * E is formed exactly as Lm + Lm N0 - N0 (= I - (I - Lm)(I + N0)) in int32
    and its band i - j <= N, exactly zero in real arithmetic, is set to 0.
  * The residual powers run as P_s = E P_{s-1} (equal to P_{s-1} E in exact
    arithmetic; fixing the side fixes which quantised factor is used).

All arithmetic here is on Python/numpy integers; no floating point enters
after quantize().

INT16 (the paper's main integer setting, Section 3.5 and Appendix G) is the
same recipe with 16-bit codes: |q| <= 32639 (= 127 * 256 + 127, so a code
splits into two int8 limbs), the running sums 16 guard bits below a code's
quantum (terms kept below 2^31, sums below 2^36), and products exact in
int64.  SPEC8 and SPEC16 hold the two parameter sets; every function takes
the spec (INT8 by default).

C = 128 runs block-wise (Appendix E, with Appendix H's 64 x 64 blocks):
quantize_blocked gives each of the blocks A11, A21, A22 its own exponent,
and neumann_inverse_int_blocked inverts the diagonal blocks with the recipe
above and forms X21 = -X22 A21 X11 as two requantised products (P = A21 X11,
then X22 P), the identity parts of X11 and X22 kept exact.
"""

from __future__ import annotations

from typing import List, Tuple

import numpy as np

import dataclasses


@dataclasses.dataclass(frozen=True)
class Spec:
    qmax: int        # codes q in [-qmax, qmax]
    qbits: int       # 2^(qbits - 1) <= qmax < 2^qbits
    align_bits: int  # aligned sum terms stay below 2^align_bits
    sum_bits: int    # running sums stay below 2^sum_bits


SPEC8 = Spec(qmax=127, qbits=7, align_bits=23, sum_bits=31)
SPEC16 = Spec(qmax=32639, qbits=15, align_bits=31, sum_bits=37)

QMAX = SPEC8.qmax
ALIGN_BITS = SPEC8.align_bits  # aligned terms stay below 2^23 in magnitude


# ----------------------------------------------------------------------------
# rounding primitives


def rne_shift(y: np.ndarray, s) -> np.ndarray:
    """round-half-even(y / 2^s) for integer y and integer s >= 0 (per element
    or broadcast)."""
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


def _tile_amax(q: np.ndarray) -> np.ndarray:
    return np.max(np.abs(q), axis=(-1, -2))


def requant(acc: np.ndarray, e: np.ndarray, spec: Spec = SPEC8) -> Tuple[np.ndarray, np.ndarray]:
    """Per tile: smallest shift s >= 0 with rne(max|acc| / 2^s) <= qmax
    (127 for INT8); returns (q int64 codes, e + s).  An all-zero tile gets
    e = 0."""
    acc = np.asarray(acc, dtype=np.int64)
    e = np.asarray(e, dtype=np.int64)
    amax = _tile_amax(acc)
    s = np.zeros_like(amax)
    while True:
        big = rne_shift(amax, s) > spec.qmax
        if not np.any(big):
            break
        s = s + big.astype(np.int64)
    q = rne_shift(acc, s[..., None, None])
    e_out = np.where(amax > 0, e + s, 0)
    return q, e_out


# ----------------------------------------------------------------------------
# quantisation of the float input


def quantize(x: np.ndarray, spec: Spec = SPEC8) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric per-tile quantiser with a power-of-two scale.

    x float32 tiles [..., C, C].  e = ceil(log2(amax / qmax)) computed
    exactly from frexp: amax = m 2^p, m in [0.5, 1) gives
    amax / 2^(p - qbits) = 2^qbits m, which is <= qmax unless
    m > qmax / 2^qbits (INT8: 128 m <= 127 unless m > 127/128).
    q = rne(x / 2^e).  All-zero tiles get q = 0, e = 0."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    amax = np.max(np.abs(x), axis=(-1, -2))
    m, p = np.frexp(amax)
    e = (p.astype(np.int64) - spec.qbits) + (m * float(1 << spec.qbits) > spec.qmax).astype(np.int64)
    e = np.where(amax > 0, e, 0)
    q = np.rint(np.ldexp(x, -e[..., None, None])).astype(np.int64)
    assert np.all(np.abs(q) <= spec.qmax)
    return q, e


# ----------------------------------------------------------------------------
# exact running sums


def _acc_bits(C: int, spec: Spec = SPEC8) -> int:
    # |acc| <= C * qmax^2 < C * 2^(2 qbits)
    return 2 * spec.qbits + int(np.ceil(np.log2(C)))


def aligned_sum(terms: List[Tuple[np.ndarray, np.ndarray, np.ndarray, int]],
                spec: Spec = SPEC8):
    """Running int32 sum of q_k * 2^(e_k), terms taken in the given order.

    terms: list of (q, e, present, bits) with q [..., C, C] int, e [...] int,
    present [...] bool, bits = log2 bound of |q| (7 for int8 codes, 14+log2 C
    for raw products).  Per tile, the sum keeps an exponent e_acc:
      * the first present term sets e_acc = e + bits - 23 (its largest value
        sits just below 2^23, leaving 16 guard bits under an int8 quantum);
      * a later present term whose top e + bits would pass e_acc + 23 first
        rebases the sum to e_acc' = e + bits - 23 (acc = rne(acc / 2^d));
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
        d = np.where(rebase, top - e_acc, 0)
        total = np.where(rebase[..., None, None], rne_shift(total, d[..., None, None]), total)
        e_acc = np.where(first | rebase, top, e_acc)
        sh = (e - e_acc)[..., None, None]
        t = np.where(sh >= 0, q << np.maximum(sh, 0), rne_shift(q, np.maximum(-sh, 0)))
        total = total + np.where(p[..., None, None], t, 0)
        anyp |= p
    e_acc = np.where(anyp, e_acc, 0)
    assert np.all(np.abs(total) < (1 << spec.sum_bits))
    return total, e_acc, anyp


# ----------------------------------------------------------------------------
# the INT8 pipeline


def _subdiag(C: int) -> np.ndarray:
    i = np.arange(C)[:, None]
    j = np.arange(C)[None, :]
    return i - j


def neumann_inverse_int8(qA: np.ndarray, eA: np.ndarray, N: int, S: int, spec: Spec = SPEC8):
    """Integer T_hat(N, S) from the quantised GDN matrix (qA, eA).

    qA int [..., C, C] (only i > j is read), eA int [...].
    Returns (qT, eT): T_hat = I + qT * 2^eT, qT codes (int8 range, or
    int16 range with SPEC16) of the strict lower part (zero on and above the
    diagonal), and the parts dictionary for inspection."""
    qA = np.asarray(qA, np.int64)
    eA = np.asarray(eA, np.int64)
    C = qA.shape[-1]
    d = _subdiag(C)
    strict = d > 0
    band = (d > 0) & (d <= N)
    accb = _acc_bits(C, spec)
    qb = spec.qbits
    rq = lambda acc, e: requant(acc, e, spec)
    asum = lambda terms: aligned_sum(terms, spec)

    qL = np.where(strict, -qA, 0)
    eL = eA
    nzL = _tile_amax(qL) > 0

    # Section 3.1 / 3.3: masked powers B_n = M (Lm^n), B_n = M (B_{n-1} Lm)
    powers = []
    if N >= 1:
        qB = np.where(band, qL, 0)
        qB, eB = rq(qB, eL)
        powers.append((qB, eB, _tile_amax(qB) > 0))
        for _n in range(2, N + 1):
            qP, eP, nzP = powers[-1]
            acc = np.where(band, qP @ qL, 0)
            q, e = rq(acc, eP + eL)
            powers.append((q, e, (_tile_amax(q) > 0)))

    # N0 = strict part of T^(0) = sum_n B_n
    if powers:
        s_, e_, p_ = asum([(q, e, p, qb) for (q, e, p) in powers])
        qN0, eN0 = rq(s_, e_)
    else:
        qN0 = np.zeros_like(qL)
        eN0 = np.zeros_like(eL)
    nzN0 = _tile_amax(qN0) > 0

    # E = I - (I + A) T0 = Lm + Lm N0 - N0, band zeroed (Section 3.4)
    s_, e_, _ = asum([
        (qL, eL, nzL, qb),
        (qL @ qN0, eL + eN0, nzL & nzN0, accb),
        (-qN0, eN0, nzN0, qb),
    ])
    s_ = np.where(d > N, s_, 0)
    qE, eE = rq(s_, e_)
    nzE = _tile_amax(qE) > 0

    # residual powers P_s = E P_{s-1}, G strict part = sum_{s=1}^{S} P_s
    chain = []
    if S >= 1:
        chain.append((qE, eE, nzE))
        for _s in range(2, S + 1):
            qP, eP, nzP = chain[-1]
            q, e = rq(qE @ qP, eE + eP)
            chain.append((q, e, (_tile_amax(q) > 0)))
    if chain:
        s_, e_, _ = asum([(q, e, p, qb) for (q, e, p) in chain])
        qG, eG = rq(s_, e_)
    else:
        qG = np.zeros_like(qL)
        eG = np.zeros_like(eL)
    nzG = _tile_amax(qG) > 0

    # T_hat = (I + N0)(I + Gs) = I + N0 + Gs + N0 Gs
    s_, e_, _ = asum([
        (qN0, eN0, nzN0, qb),
        (qG, eG, nzG, qb),
        (qN0 @ qG, eN0 + eG, nzN0 & nzG, accb),
    ])
    s_ = np.where(strict, s_, 0)
    qT, eT = rq(s_, e_)
    parts = {"N0": (qN0, eN0), "E": (qE, eE), "G": (qG, eG), "powers": powers, "chain": chain}
    return qT, eT, parts


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


def neumann_inverse_int16(qA: np.ndarray, eA: np.ndarray, N: int, S: int):
    """neumann_inverse_int8 with 16-bit codes (SPEC16)."""
    return neumann_inverse_int8(qA, eA, N, S, SPEC16)


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
    X11 = T11^-1, X22 = T22^-1, X21 = -X22 T21 X11 with T21 = A21).

    qA [..., C, C] codes with exponents eA [..., 3] for the blocks
    (11, 21, 22) as quantize_blocked writes them.  The diagonal blocks are
    inverted by neumann_inverse_int8 (X = I + N, codes N at one exponent).
    The off-diagonal block is two requantised products whose identity parts
    stay exact, taken from the right:
      P   = A21 X11 = A21 + A21 N11,
      X21 = -(X22 P) = -(P + N22 P),
    each an aligned_sum of the code term and the exact product term (in
    that order; a product is present when both factors are non-zero),
    requantised; the sign is applied to the codes (round-half-even is
    symmetric, so negating before or after rounding agrees).
    Returns qT [..., C, C] (N11, X21 and N22 in their blocks, zero on and
    above the diagonal) and eT [..., 3] for (N11, X21, N22): the inverse is
    I + each block's codes * 2^(its exponent)."""
    qA = np.asarray(qA, np.int64)
    eA = np.asarray(eA, np.int64)
    C = qA.shape[-1]
    b11, b21, b22 = _blocks(C)
    q11, e11, _ = neumann_inverse_int8(qA[(Ellipsis,) + b11], eA[..., 0], N, S, spec)
    q22, e22, _ = neumann_inverse_int8(qA[(Ellipsis,) + b22], eA[..., 2], N, S, spec)
    a21, ea = qA[(Ellipsis,) + b21], eA[..., 1]
    accb = _acc_bits(C // 2, spec)
    nzA = _tile_amax(a21) > 0
    nz11 = _tile_amax(q11) > 0
    nz22 = _tile_amax(q22) > 0
    s_, e_, _ = aligned_sum([(a21, ea, nzA, spec.qbits),
                             (a21 @ q11, ea + e11, nzA & nz11, accb)], spec)
    qP, eP = requant(s_, e_, spec)
    nzP = _tile_amax(qP) > 0
    s_, e_, _ = aligned_sum([(qP, eP, nzP, spec.qbits),
                             (q22 @ qP, e22 + eP, nz22 & nzP, accb)], spec)
    q21, e21 = requant(s_, e_, spec)
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
    neumann_inverse_int8 and dequantised, I + qT 2^eT.  With C > m the tile is
    first padded to C x C with zero rows and columns (tokens that write
    nothing) and the top-left m x m block returned: the integer recipe runs on
    C x C tiles, whose product bound sets the alignment of its sums."""
    A = np.asarray(A, np.float64)
    m = A.shape[-1]
    if C > m:
        P = np.zeros(A.shape[:-2] + (C, C))
        P[..., :m, :m] = A
        return dequantized_inverse(P, N, S, spec)[..., :m, :m]
    qA, eA = quantize(np.tril(A, -1).astype(np.float32), spec)
    qT, eT, _ = neumann_inverse_int8(qA, eA, N, S, spec)
    return dequant_unit(qT, eT)


def dequant_unit(qT: np.ndarray, eT: np.ndarray) -> np.ndarray:
    """I + qT * 2^eT as float64."""
    C = qT.shape[-1]
    return np.eye(C) + np.ldexp(np.asarray(qT, np.float64), np.asarray(eT)[..., None, None])


def dequant(q: np.ndarray, e: np.ndarray) -> np.ndarray:
    return np.ldexp(np.asarray(q, np.float64), np.asarray(e)[..., None, None])
