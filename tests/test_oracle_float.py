"""Pins of the float64 oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every check is a closed form,
an exact rational brute force, a library routine, a bound or invariant the
paper proves, or a value the paper prints (tests/golden).
"""

import os
from fractions import Fraction
from math import comb

import numpy as np
import pytest
import scipy.linalg

import workloads as wl
from oracle import gdn

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _tiles_from_workload(name, n_heads=1, C=None, stress=False):
    w = wl.workload(name)
    C = w.C if C is None else C
    if stress:
        k, b, g, _ = wl.gen_stress_head(L=4 * C, dk=w.dk, C=C, seed=5)
        K, beta, gg = k[None, :, None], b[None, :, None], g[None, :, None]
    else:
        heads = [wl.gen_head(w, 0, h, C=C, want_v=False) for h in range(n_heads)]
        K = wl.as_blhd(*[x[0] for x in heads])
        beta = wl.as_blhd(*[x[1] for x in heads])
        gg = wl.as_blhd(*[x[2] for x in heads])
    return gdn.tiles_flat(gdn.build_A(K, beta, gg, C))


@pytest.fixture(scope="module")
def gdn_tiles():
    return _tiles_from_workload("tiny")  # 16 tiles of C = 64


@pytest.fixture(scope="module")
def stress_tiles():
    return _tiles_from_workload("tiny", stress=True)  # 4 tiles of C = 64


# ---------------------------------------------------------------------------
# exact inverse (forward substitution, Section 2.2)


def test_fwdsub_solves_system(gdn_tiles, stress_tiles):
    for A in (gdn_tiles, stress_tiles):
        X = gdn.forward_substitution_inverse(A)
        I = np.eye(A.shape[-1])
        R = (I + A) @ X - I
        assert np.max(np.abs(R)) < 1e-13
        # unit lower triangular
        assert np.all(np.triu(X, 1) == 0)
        assert np.all(np.diagonal(X, axis1=-2, axis2=-1) == 1)


def test_fwdsub_matches_library_inverse(stress_tiles):
    X = gdn.forward_substitution_inverse(stress_tiles)
    Xl = np.linalg.inv(np.eye(64) + stress_tiles)
    assert np.max(np.abs(X - Xl)) < 1e-11 * max(1.0, np.max(np.abs(Xl)))


def _fraction_inverse(M):
    """Gauss-Jordan elimination over the rationals (exact)."""
    n = len(M)
    a = [[Fraction(M[i][j]) for j in range(n)] + [Fraction(int(i == j)) for j in range(n)]
         for i in range(n)]
    for c in range(n):
        p = next(r for r in range(c, n) if a[r][c] != 0)
        a[c], a[p] = a[p], a[c]
        pv = a[c][c]
        a[c] = [x / pv for x in a[c]]
        for r in range(n):
            if r != c and a[r][c] != 0:
                f = a[r][c]
                a[r] = [x - f * y for x, y in zip(a[r], a[c])]
    return [[a[i][n + j] for j in range(n)] for i in range(n)]


@pytest.mark.parametrize("C", [2, 3, 5, 8])
def test_fwdsub_exact_rational_bruteforce(C):
    rng = np.random.default_rng(C)
    A = np.tril(rng.uniform(-1, 1, (C, C)), -1)
    X = gdn.forward_substitution_inverse(A)
    Xr = _fraction_inverse((np.eye(C) + A).tolist())
    for i in range(C):
        for j in range(C):
            assert abs(X[i, j] - float(Xr[i][j])) <= 1e-14 * max(1.0, abs(float(Xr[i][j])))


def test_nilpotent_finite_neumann_is_exact(stress_tiles):
    """Section 2.3: Lm^C = 0 and sum_{n<C} Lm^n = (I - Lm)^-1."""
    Lm = -stress_tiles
    P = np.broadcast_to(np.eye(64), Lm.shape).copy()
    biggest = 1.0
    for _ in range(64):
        P = P @ Lm
        biggest = max(biggest, np.max(np.abs(P)))
    assert np.all(P == 0)
    X = gdn.forward_substitution_inverse(stress_tiles)
    # the sum cancels powers far larger than X (Section 3.2): rounding is
    # relative to the largest power, not to X
    assert biggest > 1e3
    assert np.max(np.abs(gdn.neumann_full(stress_tiles) - X)) < 1e-14 * biggest


# ---------------------------------------------------------------------------
# closed forms


def _toeplitz_inputs(C, b, a, dk=8, n_chunks=2):
    """Identical unit keys, constant beta = b, constant per-token log-decay a."""
    L = C * n_chunks
    k = np.zeros((L, dk))
    k[:, 0] = 1.0
    beta = np.full(L, b)
    g = wl.chunk_cumsum(np.full(L, a), C)
    return k[None, :, None], beta[None, :, None], g[None, :, None]


@pytest.mark.parametrize("C,b,a", [(16, 0.3, -0.1), (64, 0.7, -0.02), (32, 0.5, -1.0)])
def test_gdn_toeplitz_closed_form(C, b, a):
    """Identical keys, constant beta and decay: A_ij = b gamma^(i-j) and
    (I + A)^-1 has X_ij = -b gamma^d (1 - b)^(d-1) for d = i - j >= 1
    (generating-function identity (1 + b gamma z / (1 - gamma z))^-1)."""
    K, beta, g = _toeplitz_inputs(C, b, a)
    A = gdn.tiles_flat(gdn.build_A(K, beta, g, C))
    gam = np.exp(a)
    col = np.r_[0.0, b * gam ** np.arange(1, C)]
    At = scipy.linalg.toeplitz(col, np.zeros(C))
    assert np.allclose(A, At, rtol=1e-13, atol=0)
    X = gdn.forward_substitution_inverse(A)
    d = gdn.subdiag_index(C)
    Xc = np.where(d > 0, -b * gam ** np.maximum(d, 0) * (1 - b) ** np.maximum(d - 1, 0), 0.0) + np.eye(C)
    assert np.max(np.abs(X - Xc)) < 1e-14


def test_build_A_row_scale_is_beta_i():
    """Identical keys, per-token beta, constant decay: A = diag(beta) Toep."""
    C = 16
    K, _, g = _toeplitz_inputs(C, 0.5, -0.2, n_chunks=1)
    beta = np.linspace(0.1, 0.9, C)[None, :, None]
    A = gdn.tiles_flat(gdn.build_A(K, beta, g, C))[0]
    col = np.r_[0.0, np.exp(-0.2) ** np.arange(1, C)]
    Tp = scipy.linalg.toeplitz(col, np.zeros(C))
    assert np.allclose(A, np.diag(beta[0, :, 0]) @ Tp, rtol=1e-13, atol=0)


def test_build_A_orthogonal_keys_gives_identity_inverse():
    C, dk = 16, 16
    K = np.eye(dk)[None, :, None, :]
    beta = np.full((1, C, 1), 0.5)
    g = wl.chunk_cumsum(np.full((1, C, 1), -0.3), C, axis=1)
    A = gdn.tiles_flat(gdn.build_A(K, beta, g, C))
    assert np.all(A == 0)
    assert np.all(gdn.neumann_inverse(A, 3, 2) == np.eye(C))


def test_build_A_properties(gdn_tiles):
    """Strictly lower; |A_ij| <= 1 (unit keys, beta < 1, non-increasing g);
    with beta = 1, g = 0 the symmetric completion A + A^T + I is the Gram
    matrix of dk-dimensional keys, so its rank is at most dk."""
    A = gdn_tiles
    assert np.all(np.triu(A) == 0)
    assert np.max(np.abs(A)) <= 1.0
    w = wl.workload("tiny")
    k, _, _, _ = wl.gen_head(w, 0, 0, want_v=False)
    dk = 16
    kk = k[:64, :dk].astype(np.float64)
    kk = kk / np.linalg.norm(kk, axis=1, keepdims=True)
    A1 = gdn.build_A(kk[None, :, None], np.ones((1, 64, 1)), np.zeros((1, 64, 1)), 64)[0, 0, 0]
    ev = np.linalg.eigvalsh(A1 + A1.T + np.eye(64))
    assert np.sum(np.abs(ev) > 1e-10) <= dk
    assert np.min(ev) > -1e-12  # positive semidefinite


def test_build_A_tile_layout():
    """Tile (b, h, chunk) sits at (b H + h) L/C + chunk and uses tokens
    chunk*C .. chunk*C + C - 1 of head h."""
    w = wl.workload("tiny").with_(L=256, H=3, B=2)
    K, beta, g, _ = wl.gen_inputs(w, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(K, beta, g, w.C))
    for (b, h, c) in [(0, 0, 0), (1, 2, 3), (0, 1, 2)]:
        t = wl.tile_index(w, b, h, c)
        sl = slice(c * w.C, (c + 1) * w.C)
        A1 = gdn.build_A(K[b:b + 1, sl, h:h + 1], beta[b:b + 1, sl, h:h + 1],
                         g[b:b + 1, sl, h:h + 1], w.C)[0, 0, 0]
        assert np.array_equal(A[t], A1)


def test_paper_sign_all_ones_closed_form():
    """Lemma 3 tightness case (Appendix C): the paper's A = all-ones strictly
    lower (our A = -ones).  (A^n)_ij = binom(d-1, n-1) and (I - A)^-1 has
    entries 2^(d-1)."""
    C = 24
    ones = np.tril(np.ones((C, C)), -1)
    X = gdn.forward_substitution_inverse(-ones)
    d = gdn.subdiag_index(C)
    Xc = np.where(d > 0, 2.0 ** np.maximum(d - 1, 0), 0.0) + np.eye(C)
    assert np.array_equal(X, Xc)
    P = np.eye(C)
    for n in range(1, 6):
        P = P @ ones
        ref = np.array([[comb(i - j - 1, n - 1) if i > j else 0 for j in range(C)] for i in range(C)],
                       dtype=np.float64)
        assert np.array_equal(P, ref)


def test_gdn_sign_all_ones_bidiagonal():
    """GDN sign with all-ones A: (I + A)^-1 = I - Z (Z the down-shift);
    then T^(0) = X already on its band, E = 0 and T_hat(N >= 1, S) = X."""
    C = 64
    A = np.tril(np.ones((C, C)), -1)
    X = gdn.forward_substitution_inverse(A)
    assert np.array_equal(X, np.eye(C) - np.eye(C, k=-1))
    for N, S in [(1, 0), (3, 8), (2, 1)]:
        T, parts = gdn.neumann_inverse(A, N, S, return_parts=True)
        assert np.max(np.abs(parts["E"])) == 0
        assert np.array_equal(T, X)


# ---------------------------------------------------------------------------
# masked Neumann + residual structure (Sections 3.1, 3.3, 3.4)


@pytest.mark.parametrize("N", [1, 2, 3, 5])
def test_T0_is_inverse_on_band(stress_tiles, N):
    """Lemma 1: Lm^n vanishes for i - j < n, so on i - j <= N the truncated
    sum already holds every term of the exact inverse; the mask zeroes the
    rest.  Hence E = (I + A)(X - T0) vanishes on the band too."""
    A = stress_tiles
    X = gdn.forward_substitution_inverse(A)
    T0, _ = gdn.masked_truncated_neumann(A, N)
    d = gdn.subdiag_index(64)
    band = d <= N
    assert np.max(np.abs(np.where(band, T0 - X, 0))) < 1e-13
    assert np.all(np.where(band, 0, T0) == 0)
    E = gdn.residual(A, T0)
    assert np.max(np.abs(np.where(band, E, 0))) < 1e-13
    assert np.max(np.abs(np.where(band, 0, E))) > 1e-6  # and not beyond it


@pytest.mark.parametrize("C,N,S", [(64, 3, 8), (64, 3, 15), (64, 2, 3), (32, 3, 4), (32, 3, 7),
                                   (16, 3, 2), (16, 3, 3), (64, 1, 20)])
def test_approx_exact_below_band_limit(C, N, S):
    """E^s vanishes for i - j < s (N + 1), so T_hat(N, S) = X on
    i - j < (S + 1)(N + 1), and exactly everywhere once (S+1)(N+1) >= C."""
    A = _tiles_from_workload("tiny", C=C, stress=True)
    X = gdn.forward_substitution_inverse(A)
    T = gdn.neumann_inverse(A, N, S)
    d = gdn.subdiag_index(C)
    lim = (S + 1) * (N + 1)
    err_in = np.max(np.abs(np.where(d < lim, T - X, 0)))
    assert err_in < 1e-12
    if lim >= C:
        assert np.max(np.abs(T - X)) < 1e-12
    else:
        assert np.max(np.abs(np.where(d >= lim, T - X, 0))) > 1e-12


def test_mask_width_is_N_not_N_minus_1():
    """At C = 16, (N, S) = (3, 3) is exact; a mask one diagonal narrower
    (K = N - 1) would leave E non-zero on d = N and break exactness."""
    A = _tiles_from_workload("tiny", C=16, stress=True)
    X = gdn.forward_substitution_inverse(A)
    assert np.max(np.abs(gdn.neumann_inverse(A, 3, 3) - X)) < 1e-12
    T0w, _ = gdn.masked_truncated_neumann(A, 3)
    T0w = T0w * gdn.band_mask(16, 2)
    E = gdn.residual(A, T0w)
    G, _ = gdn.power_sum(E, 3)
    assert np.max(np.abs(T0w @ G - X)) > 1e-6


def test_printed_return_order_does_not_converge(stress_tiles):
    """Algorithm 1 prints the return as T <- T T^(0), i.e. (sum E^s) T^(0).
    With E = I - (I + A) T^(0) only T^(0) (sum E^s) tends to X (Section 3.4
    equation, Appendix D); the printed order tends to T0^-1 X T0."""
    A = stress_tiles
    X = gdn.forward_substitution_inverse(A)
    good = gdn.neumann_inverse(A, 3, 16)
    bad = gdn.neumann_inverse_printed_order(A, 3, 16)
    assert np.max(np.abs(good - X)) < 1e-12
    assert np.max(np.abs(bad - X)) > 1e-3
    T0, _ = gdn.masked_truncated_neumann(A, 3)
    assert np.max(np.abs(bad - np.linalg.solve(T0, X @ T0))) < 1e-10


def test_newton_iteration_equals_power_sum(stress_tiles):
    """Section 3.4: M Newton steps T <- T + T R equal T^(0) sum_{s<2^M} E^s."""
    A = stress_tiles
    T0, _ = gdn.masked_truncated_neumann(A, 3)
    E = gdn.residual(A, T0)
    for M in (1, 2, 3):
        G, _ = gdn.power_sum(E, 2 ** M - 1)
        assert np.max(np.abs(gdn.newton_residual(A, 3, M) - T0 @ G)) < 1e-12


def test_factorised_product_equals_power_sum(stress_tiles):
    """Appendix F: prod_m (I + E^(2^m)) = sum_{s < 2^M} E^s."""
    T0, _ = gdn.masked_truncated_neumann(stress_tiles, 3)
    E = gdn.residual(stress_tiles, T0)
    for M in (1, 2, 3):
        G, _ = gdn.power_sum(E, 2 ** M - 1)
        assert np.max(np.abs(gdn.factorised_power_sum(E, M) - G)) < 1e-12


def test_two_block_inverse_is_exact(stress_tiles):
    """Appendix E with exact diagonal-block inverses reproduces X."""
    X = gdn.forward_substitution_inverse(stress_tiles)
    Xb = gdn.two_block_inverse(stress_tiles, gdn.forward_substitution_inverse)
    assert np.max(np.abs(Xb - X)) < 1e-12 * np.max(np.abs(X))


def test_blocked_neumann_128_error_within_blocks():
    """C = 128 path: with (S+1)(N+1) >= 64 each 64-block inverse is exact and
    so is the joined 128 inverse."""
    A = _tiles_from_workload("tiny", C=128, stress=True)
    X = gdn.forward_substitution_inverse(A)
    assert np.max(np.abs(gdn.neumann_inverse_blocked(A, 3, 15) - X)) < 1e-11 * np.max(np.abs(X))
    assert np.max(np.abs(gdn.neumann_inverse_blocked(A, 3, 8) - X)) > 0


# ---------------------------------------------------------------------------
# bounds


def test_lemma2_truncation_bound():
    """||E_N|| <= ||A||^(N+1) / (1 - ||A||) for the unmasked truncation,
    in the spectral and infinity norms (both sub-multiplicative)."""
    rng = np.random.default_rng(3)
    C = 64
    for trial in range(5):
        A = np.tril(rng.uniform(-1, 1, (C, C)), -1)
        for ordn in (2, np.inf):
            A = A * (0.6 / np.linalg.norm(A, ordn))
            X = gdn.forward_substitution_inverse(A)
            Lm = -A
            T = np.eye(C)
            P = np.eye(C)
            for N in range(0, 10):
                if N > 0:
                    P = P @ Lm
                    T = T + P
                EN = X - T
                a = np.linalg.norm(A, ordn)
                assert np.linalg.norm(EN, ordn) <= a ** (N + 1) / (1 - a) * (1 + 1e-12)


def test_appendix_d_residual_bound(stress_tiles):
    """||X - T_hat|| <= ||T0|| ||E||^(S+1) / (1 - ||E||) when ||E|| < 1."""
    checked = 0
    for A in stress_tiles:
        X = gdn.forward_substitution_inverse(A)
        for N in (2, 3, 4):
            T0, _ = gdn.masked_truncated_neumann(A, N)
            E = gdn.residual(A, T0)
            e = np.linalg.norm(E, 2)
            if e >= 1:
                continue
            for S in (0, 1, 2, 4, 8):
                T = gdn.neumann_inverse(A, N, S)
                bound = np.linalg.norm(T0, 2) * e ** (S + 1) / (1 - e)
                assert np.linalg.norm(X - T, 2) <= bound * (1 + 1e-9) + 1e-14
                checked += 1
    assert checked > 0


def test_lemma3_entrywise_bound_abs():
    """Lemma 3 in absolute value: |(Lm^n)_ij| <= binom(d-1, n-1) whenever
    |A_ij| <= 1 (triangle inequality on the path expansion of Appendix C)."""
    rng = np.random.default_rng(11)
    C = 32
    d = gdn.subdiag_index(C)
    for trial in range(4):
        Lm = np.tril(rng.uniform(-1, 1, (C, C)), -1)
        P = np.eye(C)
        for n in range(1, 7):
            P = P @ Lm
            bound = np.array([[comb(i - j - 1, n - 1) if i > j else 0 for j in range(C)]
                              for i in range(C)], dtype=np.float64)
            assert np.all(np.abs(P) <= bound * (1 + 1e-12))


# ---------------------------------------------------------------------------
# printed numbers


def test_matmul_counts_match_paper():
    for C, N, S, count in _golden("matmul_counts.txt"):
        A = _tiles_from_workload("tiny", C=int(C))
        _, parts = gdn.neumann_inverse(A, int(N), int(S), return_parts=True)
        assert parts["products"] == int(count)


def test_fig5_captured_structure_proxy():
    """Appendix B / Fig. 5: entries decaying geometrically with the
    sub-diagonal index, rescaled to ||A||_2 = 0.55.  The decay rate is not
    given; fitting it so that r_3 equals the printed 95.5 % reproduces the
    other two printed values, r_5 and r_8, to their printed precision."""
    rows = _golden("fig5_captured_structure.txt")
    C = int(rows[0][0])
    norm = float(rows[0][1])
    want = {int(r[2]): float(r[3]) for r in rows}
    d = gdn.subdiag_index(C)

    def rs(rho):
        A = np.where(d > 0, rho ** (d - 1.0), 0.0)
        A *= norm / np.linalg.norm(A, 2)
        X = gdn.neumann_full(-A)  # paper sign: (I - A)^-1 = sum A^n
        out = {}
        for m in want:
            Tm = np.eye(C)
            P = np.eye(C)
            for _ in range(m):
                P = P @ A
                Tm = Tm + P
            out[m] = gdn.captured_structure(X, Tm)
        return out

    lo, hi = 0.05, 0.95
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        if rs(mid)[3] < want[3]:
            lo = mid
        else:
            hi = mid
    got = rs(mid)
    for m, r in want.items():
        assert abs(got[m] - r) <= 0.0005 + 1e-9, (m, got[m], r)


def test_default_orders():
    assert gdn.default_order(32) == (3, 4)
    assert gdn.default_order(64) == (3, 8)


# ---------------------------------------------------------------------------
# WY application


def test_wy_solves_triangular_system():
    """With the exact inverse, W = X diag(beta) K is the solution of
    (I + A) W = diag(beta) K (checked with a library triangular solve)."""
    w = wl.workload("tiny").with_(L=128, H=2)
    K, beta, g, V = wl.gen_inputs(w)
    A = gdn.build_A(K, beta, g, w.C)
    X = gdn.forward_substitution_inverse(A)
    W, U = gdn.wy_apply(X, K, V, beta, w.C)
    for b in range(w.B):
        for h in range(w.H):
            for c in range(w.L // w.C):
                sl = slice(c * w.C, (c + 1) * w.C)
                M = np.eye(w.C) + A[b, h, c]
                rhsk = beta[b, sl, h, None].astype(np.float64) * K[b, sl, h]
                rhsv = beta[b, sl, h, None].astype(np.float64) * V[b, sl, h]
                Wr = scipy.linalg.solve_triangular(M, rhsk, lower=True, unit_diagonal=True)
                Ur = scipy.linalg.solve_triangular(M, rhsv, lower=True, unit_diagonal=True)
                assert np.max(np.abs(W[b, sl, h] - Wr)) < 1e-12
                assert np.max(np.abs(U[b, sl, h] - Ur)) < 1e-12


def test_metrics_definitions():
    X = np.eye(4)[None]
    T = X.copy()
    T[0, 3, 0] = 0.1
    assert np.isclose(gdn.snr_db(X, T)[0], 10 * np.log10(4 / 0.01))
    assert np.isclose(gdn.diag_power_ratio(X, 0)[0], 1.0)


def test_diag_power_ratio_closed_forms():
    """The accumulated diagonal power ratio on inverses with a closed form.
    A = -S (S the unit sub-diagonal): (I + A)^-1 = sum_k S^k, the all-ones
    lower triangle, whose sub-diagonal d holds C - d ones, so the ratio up to
    n is sum_{d<=n} (C - d) / (C (C + 1) / 2) = (n + 1)(2C - n) / (C (C + 1)).
    A = -r S: the inverse has r^(i-j) below the diagonal, diagonal d has
    power (C - d) r^(2d)."""
    for C in (5, 8, 16):
        A = np.zeros((1, C, C))
        A[0, np.arange(1, C), np.arange(C - 1)] = -1.0
        X = gdn.forward_substitution_inverse(A)
        for n in range(C):
            want = (n + 1) * (2 * C - n) / (C * (C + 1))
            assert np.isclose(gdn.diag_power_ratio(X, n)[0], want, rtol=1e-13, atol=0)
        r = 0.7
        Xg = gdn.forward_substitution_inverse(r * A)
        tot = sum((C - d) * r ** (2 * d) for d in range(C))
        for n in range(C):
            want = sum((C - d) * r ** (2 * d) for d in range(n + 1)) / tot
            assert np.isclose(gdn.diag_power_ratio(Xg, n)[0], want, rtol=1e-12, atol=0)
