"""Float64 oracle of the chunk-wise Gated DeltaNet forward (test infrastructure only).

The chunk inverse is one step of the chunk-wise Gated DeltaNet forward: the
paper motivates it by the chunk-level recurrence of Yang et al. (Section 1)
and writes the chunk output as Y = T^-1 X (Appendix E).  The recurrence
itself is Gated DeltaNet's (the paper's reference for the model, Section 1,
Section 2.1).  This module holds two independent codings of that forward,
per head, with the state S in R^{dk x dv}:

  gdn_recurrent  the token recurrence, the plain definition:
                   S_t = a_t (I - b_t k_t k_t^T) S_{t-1} + b_t k_t v_t^T,
                   o_t = scale * S_t^T q_t,   a_t = exp(inc_t),
                 inc_t the per-token log-decay, b_t = beta_t.

  gdn_chunked    the chunk-wise (WY) form.  For a chunk with local positions
                 i = 0 .. C-1, gamma_i the within-chunk cumulative log-decay
                 (the g input), A the chunk matrix of build_A and
                 T = (I + A)^-1:
                   W     = T diag(beta * exp(gamma)) K,   U = T diag(beta) V,
                   V_new = U - W S,
                   O     = scale (diag(exp(gamma)) Q S + (Q K^T (.) D) V_new),
                           D_ij = exp(gamma_i - gamma_j) for i >= j, else 0,
                   S'    = exp(gamma_{C-1}) S + (diag(exp(gamma_{C-1} - gamma)) K)^T V_new.
                 The inverse is a parameter: the exact one (forward
                 substitution) or T_hat(N, S), to measure what the
                 approximation does to the layer output.

Layouts as in oracle/gdn.py: Q, K [B, L, H, dk], V, O [B, L, H, dv],
beta, g [B, L, H] (g the within-chunk inclusive cumulative log-decay),
states [B, H, dk, dv].
"""

from __future__ import annotations

from typing import Callable, Optional, Tuple

import numpy as np

from . import gdn


def token_log_decay(g: np.ndarray, C: int) -> np.ndarray:
    """Per-token log-decay inc from the within-chunk cumulative sum g
    (inc_t = g_t - g_{t-1} inside a chunk, g_t at a chunk's first token)."""
    g = np.asarray(g, np.float64)
    B, L, H = g.shape
    gc = g.reshape(B, L // C, C, H)
    inc = np.concatenate([gc[:, :, :1], np.diff(gc, axis=2)], axis=2)
    return inc.reshape(B, L, H)


def gdn_recurrent(Q, K, V, beta, g, C: int, S0: Optional[np.ndarray] = None,
                  scale: float = 1.0) -> Tuple[np.ndarray, np.ndarray]:
    """Token-by-token gated delta rule; returns (O, S_final)."""
    Q, K, V = (np.asarray(x, np.float64) for x in (Q, K, V))
    beta = np.asarray(beta, np.float64)
    a = np.exp(token_log_decay(g, C))
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    S = np.zeros((B, H, dk, dv)) if S0 is None else np.array(S0, np.float64)
    O = np.zeros((B, L, H, dv))
    for t in range(L):
        k = K[:, t]                        # [B, H, dk]
        v = V[:, t]
        kS = np.einsum("bhk,bhkv->bhv", k, S)  # k^T S
        # S = a (S - b k (k^T S)) + b k v^T
        S = a[:, t, :, None, None] * (S - beta[:, t, :, None, None] * k[..., :, None] * kS[..., None, :]) \
            + beta[:, t, :, None, None] * k[..., :, None] * v[..., None, :]
        O[:, t] = scale * np.einsum("bhkv,bhk->bhv", S, Q[:, t])
    return O, S


def gdn_chunked(Q, K, V, beta, g, C: int, S0: Optional[np.ndarray] = None,
                scale: float = 1.0,
                inverse: Callable[[np.ndarray], np.ndarray] = gdn.forward_substitution_inverse
                ) -> Tuple[np.ndarray, np.ndarray]:
    """Chunk-wise form (see the module docstring); returns (O, S_final)."""
    Q, K, V = (np.asarray(x, np.float64) for x in (Q, K, V))
    beta = np.asarray(beta, np.float64)
    g = np.asarray(g, np.float64)
    B, L, H, dk = K.shape
    dv = V.shape[-1]
    nc = L // C
    T = inverse(gdn.build_A(K, beta, g, C))            # [B, H, nc, C, C]
    # per chunk, head-major: [B, H, nc, C, d]
    def chunks(x):
        return np.moveaxis(x, 2, 1).reshape(B, H, nc, C, *x.shape[3:])
    Qc, Kc, Vc = chunks(Q), chunks(K), chunks(V)
    bc, gc = chunks(beta), chunks(g)
    W = T @ ((bc * np.exp(gc))[..., None] * Kc)
    U = T @ (bc[..., None] * Vc)
    D = np.tril(np.exp(gc[..., :, None] - gc[..., None, :]))
    P = (Qc @ np.swapaxes(Kc, -1, -2)) * D
    S = np.zeros((B, H, dk, dv)) if S0 is None else np.array(S0, np.float64)
    Oc = np.zeros((B, H, nc, C, dv))
    for c in range(nc):
        Vn = U[:, :, c] - W[:, :, c] @ S
        Oc[:, :, c] = scale * (np.exp(gc[:, :, c])[..., None] * (Qc[:, :, c] @ S) + P[:, :, c] @ Vn)
        last = gc[:, :, c, -1]
        Kd = np.exp(last[..., None] - gc[:, :, c])[..., None] * Kc[:, :, c]
        S = np.exp(last)[..., None, None] * S + np.swapaxes(Kd, -1, -2) @ Vn
    O = np.moveaxis(Oc.reshape(B, H, L, dv), 1, 2)
    return O, S
