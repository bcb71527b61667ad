"""Float64 oracle of the chunk-inverse path (test infrastructure only).

All matrices are stacks of C x C tiles, shape [..., C, C], float64.
Row i is the later token; "strictly lower" means entries with i > j.

Paper references (arXiv 2606.06034):
  Section 2.1  problem statement T = (I - A)^-1, A strictly lower triangular
  Section 2.2  forward substitution, Eq. (forward_sub) + identity augmentation
  Section 2.3  Neumann series, nilpotency, exact finite expansion
  Section 3.1  Lemma 1 (diagonal localisation), low-order truncation T^(0),
               Lemma 2 (truncation error bound)
  Section 3.2  Lemma 3 (entrywise growth, binomial bound)
  Section 3.3  diagonal mask M^(K), K = N
  Section 3.4  residual correction: iterative (Newton) form and the
               parallel power-sum form T ~ T^(0) sum_{s=0}^{S} E^s;
               Algorithm 1
  Appendix B   truncation-error proof, captured-structure proxy r_m
  Appendix D   proof of the residual reformulation and its error bound
  Appendix E   block-wise (two-block) inversion
  Appendix F   factorised Neumann products
"""

from __future__ import annotations

from typing import Optional, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# small helpers


def eye_like(A: np.ndarray) -> np.ndarray:
    C = A.shape[-1]
    return np.broadcast_to(np.eye(C), A.shape).copy()


def strict_lower(A: np.ndarray) -> np.ndarray:
    """Keep entries with i > j; the problem statement (Section 2.1) takes A
    strictly lower triangular, so anything on or above the diagonal is
    treated as zero."""
    return np.tril(np.asarray(A, dtype=np.float64), k=-1)


def subdiag_index(C: int) -> np.ndarray:
    """d[i, j] = i - j, the sub-diagonal index used by Lemma 1 and the mask."""
    i = np.arange(C)[:, None]
    j = np.arange(C)[None, :]
    return i - j


# ----------------------------------------------------------------------------
# Step: build the chunk matrix A


def build_A(K: np.ndarray, beta: np.ndarray, g: np.ndarray, C: int) -> np.ndarray:
    """Gated DeltaNet chunk matrix, one C x C tile per (b, h, chunk).

    A_ij = beta_i * (k_i . k_j) * exp(g_i - g_j) for i > j within a chunk,
    else 0.  (Section 2.1 states A = K K^T with l2-normalised keys; the
    write strength beta and the gate exp(g_i - g_j) complete the Gated
    DeltaNet form.)  The gate is evaluated as exp of the difference, never as
    a product of two exponentials.

    K [B, L, H, dk], beta [B, L, H], g [B, L, H] (g already the within-chunk
    cumulative log-decay).  Returns A [B, H, L/C, C, C] float64.
    """
    K = np.asarray(K, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    B, L, H, dk = K.shape
    assert L % C == 0
    nc = L // C
    # [B, L, H, dk] -> [B, H, nc, C, dk]
    Kc = K.transpose(0, 2, 1, 3).reshape(B, H, nc, C, dk)
    bc = beta.transpose(0, 2, 1).reshape(B, H, nc, C)
    gc = g.transpose(0, 2, 1).reshape(B, H, nc, C)
    gram = Kc @ np.swapaxes(Kc, -1, -2)  # k_i . k_j
    gate = np.exp(gc[..., :, None] - gc[..., None, :])  # exp(g_i - g_j)
    A = bc[..., :, None] * gram * gate
    return strict_lower(A)


def tiles_flat(A: np.ndarray) -> np.ndarray:
    C = A.shape[-1]
    return A.reshape(-1, C, C)


# ----------------------------------------------------------------------------
# Exact inverse: forward substitution (Section 2.2)


def forward_substitution_inverse(A: np.ndarray) -> np.ndarray:
    """X = (I + A)^-1 by the paper's forward substitution with Lm = -A.

    Eq. (forward_sub): starting from T = Lm, for i = 1 .. k-1,
        T[i, 0:i] <- T[i, 0:i] + T[i, 0:i] @ T[0:i, 0:i],
    then the identity augmentation T <- T + I.  Row i still holds Lm[i] when
    it is updated, and rows 0..i-1 already hold the finished strict part of
    the inverse, so each row solves one step of (I - Lm) X = I.
    """
    Lm = -strict_lower(A)
    T = Lm.copy()
    C = T.shape[-1]
    for i in range(1, C):
        row = T[..., i, 0:i]
        T[..., i, 0:i] = row + np.einsum("...t,...tj->...j", row, T[..., 0:i, 0:i])
    return T + eye_like(T)


def neumann_full(A: np.ndarray) -> np.ndarray:
    """Exact finite Neumann expansion sum_{n=0}^{C-1} Lm^n (Section 2.3:
    a strictly lower-triangular matrix is nilpotent, Lm^C = 0)."""
    Lm = -strict_lower(A)
    C = Lm.shape[-1]
    acc = eye_like(Lm)
    P = eye_like(Lm)
    for _ in range(1, C):
        P = P @ Lm
        acc = acc + P
    return acc


# ----------------------------------------------------------------------------
# MatMul-only approximation (Section 3, Algorithm 1)


def band_mask(C: int, K: int) -> np.ndarray:
    """Diagonal mask M^(K) of Section 3.3: 1 where i - j <= K, else 0."""
    return (subdiag_index(C) <= K).astype(np.float64)


def masked_truncated_neumann(A: np.ndarray, N: int) -> Tuple[np.ndarray, int]:
    """T^(0) = M^(N) (Hadamard) sum_{n=0}^{N} Lm^n  (Sections 3.1 and 3.3).

    Returns (T0, number of non-trivial matrix products).  Multiplying by the
    identity is not a product: Lm^1 is taken as is."""
    Lm = -strict_lower(A)
    C = Lm.shape[-1]
    T0 = eye_like(Lm)
    P = None
    products = 0
    for _n in range(1, N + 1):
        if P is None:
            P = Lm.copy()
        else:
            P = P @ Lm
            products += 1
        T0 = T0 + P
    T0 = band_mask(C, N) * T0
    return T0, products


def residual(A: np.ndarray, T0: np.ndarray) -> np.ndarray:
    """E = I - (I - Lm) T^(0) = I - (I + A) T^(0)  (Section 3.4)."""
    IA = eye_like(T0) + strict_lower(A)
    return eye_like(T0) - IA @ T0


def power_sum(E: np.ndarray, S: int) -> Tuple[np.ndarray, int]:
    """G = sum_{s=0}^{S} E^s, accumulated along one power chain P <- P E
    (Algorithm 1's second loop).  Returns (G, non-trivial products)."""
    G = eye_like(E)
    P = None
    products = 0
    for _s in range(1, S + 1):
        if P is None:
            P = E.copy()
        else:
            P = P @ E
            products += 1
        G = G + P
    return G, products


def neumann_inverse(A: np.ndarray, N: int, S: int, return_parts: bool = False):
    """Masked low-order Neumann initialisation + parallel residual correction.

    T_hat(N, S) = T^(0) sum_{s=0}^{S} E^s,
      T^(0) = M^(N) (Hadamard) sum_{n=0}^{N} Lm^n,   E = I - (I + A) T^(0).

    The residual sum multiplies T^(0) from the right of T^(0), as in the
    reformulation of Section 3.4 and its proof in Appendix D (the ordering
    for which T_hat tends to (I + A)^-1 as S grows).

    Returns T_hat, or (T_hat, dict of parts) with T0, E, G and the count of
    non-trivial matrix products (N - 1 for the powers, 1 for E, S - 1 for the
    power chain, 1 for the final product when N, S >= 1).
    """
    T0, p1 = masked_truncated_neumann(A, N)
    E = residual(A, T0)
    p_res = 1 if N >= 1 else 0  # with N = 0, T0 = I and E = -A needs no product
    G, p2 = power_sum(E, S)
    T = T0 @ G
    p_fin = 1 if (S >= 1 and N >= 1) else 0  # T0 = I or G = I make it trivial
    if not return_parts:
        return T
    return T, {"T0": T0, "E": E, "G": G, "products": p1 + p_res + p2 + p_fin}


def neumann_inverse_printed_order(A: np.ndarray, N: int, S: int) -> np.ndarray:
    """Algorithm 1 with its return step read literally, (sum E^s) T^(0).

    Kept only so a test can show this ordering does not converge to the
    inverse when E = I - (I + A) T^(0); the library uses neumann_inverse."""
    T0, _ = masked_truncated_neumann(A, N)
    E = residual(A, T0)
    G, _ = power_sum(E, S)
    return G @ T0


def newton_residual(A: np.ndarray, N: int, M: int) -> np.ndarray:
    """Iterative residual correction of Section 3.4:
    R^(m) = I - (I + A) T^(m),  T^(m+1) = T^(m) + T^(m) R^(m),
    starting from T^(0) (masked truncated Neumann), M iterations."""
    T, _ = masked_truncated_neumann(A, N)
    IA = eye_like(T) + strict_lower(A)
    for _ in range(M):
        R = eye_like(T) - IA @ T
        T = T + T @ R
    return T


def factorised_power_sum(E: np.ndarray, M: int) -> np.ndarray:
    """Appendix F product form: G_M = prod_{m=0}^{M-1} (I + E^(2^m)),
    which equals sum_{s=0}^{2^M - 1} E^s."""
    G = eye_like(E)
    Pm = E.copy()
    for _ in range(M):
        G = G @ (eye_like(E) + Pm)
        Pm = Pm @ Pm
    return G


# ----------------------------------------------------------------------------
# Block-wise inversion (Appendix E), two blocks


def two_block_inverse(A: np.ndarray, inv_diag) -> np.ndarray:
    """Inverse of the block lower-triangular T = I + A split into 2 x 2
    blocks of size C/2 (Appendix E):
      S_11 = T_11^-1,  S_22 = T_22^-1,  S_21 = -T_22^-1 T_21 T_11^-1,
    with T_21 = A_21.  ``inv_diag(A_block)`` inverts I + A_block, e.g. the
    exact forward substitution or the Neumann approximation."""
    A = strict_lower(A)
    C = A.shape[-1]
    h = C // 2
    S11 = inv_diag(A[..., :h, :h])
    S22 = inv_diag(A[..., h:, h:])
    S21 = -(S22 @ A[..., h:, :h] @ S11)
    out = np.zeros_like(A)
    out[..., :h, :h] = S11
    out[..., h:, h:] = S22
    out[..., h:, :h] = S21
    return out


def neumann_inverse_blocked(A: np.ndarray, N: int, S: int) -> np.ndarray:
    """C = 128 path: two C/2 diagonal blocks each by neumann_inverse(N, S),
    joined by the Appendix E off-diagonal formula."""
    return two_block_inverse(A, lambda Ab: neumann_inverse(Ab, N, S))


# ----------------------------------------------------------------------------
# WY application


def wy_apply(T: np.ndarray, K: np.ndarray, V: np.ndarray, beta: np.ndarray, C: int):
    """W = T diag(beta) K,  U = T diag(beta) V per chunk.

    T [B, H, L/C, C, C]; K [B, L, H, dk]; V [B, L, H, dv]; beta [B, L, H].
    Returns W [B, L, H, dk], U [B, L, H, dv] in float64."""
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    beta = np.asarray(beta, np.float64)
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    nc = L // C
    Kc = K.transpose(0, 2, 1, 3).reshape(B, H, nc, C, dk)
    Vc = V.transpose(0, 2, 1, 3).reshape(B, H, nc, C, dv)
    bc = beta.transpose(0, 2, 1).reshape(B, H, nc, C, 1)
    W = np.asarray(T, np.float64) @ (bc * Kc)
    U = np.asarray(T, np.float64) @ (bc * Vc)
    W = W.reshape(B, H, L, dk).transpose(0, 2, 1, 3)
    U = U.reshape(B, H, L, dv).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(W), np.ascontiguousarray(U)


# ----------------------------------------------------------------------------
# default orders per chunk size


def default_order(C: int) -> Tuple[int, int]:
    """(N, S) per chunk size: 32 -> (3, 4) (Section 4.3), 64 -> (3, 8)
    (Section 4.1 defaults), 128 -> two 64-blocks at (3, 8) (Appendix H).
    C = 16 is not covered by the paper: (3, 2) continues the S = C / 8
    pattern of the two sizes it does cover."""
    return {16: (3, 2), 32: (3, 4), 64: (3, 8), 128: (3, 8)}[C]


# ----------------------------------------------------------------------------
# accuracy metrics


def snr_db(X: np.ndarray, T: np.ndarray) -> np.ndarray:
    """Per-tile SNR = 10 log10(||X||_F^2 / ||X - T||_F^2) (the tables of
    Section 4 report an SNR without defining it; this is the reading)."""
    num = np.sum(np.asarray(X, np.float64) ** 2, axis=(-1, -2))
    den = np.sum((np.asarray(X, np.float64) - np.asarray(T, np.float64)) ** 2, axis=(-1, -2))
    with np.errstate(divide="ignore"):
        return 10.0 * np.log10(num / den)


def captured_structure(X: np.ndarray, Tm: np.ndarray) -> np.ndarray:
    """r_m = 1 - ||E_m||_F / ||T||_F with E_m = T - T_m (Appendix B)."""
    return 1.0 - np.linalg.norm(X - Tm, axis=(-1, -2)) / np.linalg.norm(X, axis=(-1, -2))


def diag_power_ratio(X: np.ndarray, n: int) -> np.ndarray:
    """Accumulated diagonal power ratio sum_{d<=n} ||diag_d(X)||^2 / ||X||_F^2
    (Appendix B, real-value experiments; undefined there, this is the
    reading)."""
    C = X.shape[-1]
    keep = (subdiag_index(C) <= n) & (subdiag_index(C) >= 0)
    num = np.sum((X * keep) ** 2, axis=(-1, -2))
    return num / np.sum(X ** 2, axis=(-1, -2))
