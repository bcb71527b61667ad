"""Float64 oracle of the chunk path over packed variable-length sequences
(test infrastructure only).

Serving packs sequences of different lengths along the token axis,
K [1, T, H, dk] with cu_seqlens = [0, l_0, l_0 + l_1, ..., T].  Chunks start
at every sequence start, so a sequence of length l has ceil(l / C) chunks
and its last chunk holds m = l - C (ceil(l / C) - 1) <= C tokens.  For a
chunk of m tokens the method is the one of Section 2.1 on the m x m system:
A_ij = beta_i (k_i . k_j) exp(g_i - g_j) for i > j (i, j < m),
T = (I + A)^-1, W = T diag(beta) K, U = T diag(beta) V, with g the
within-chunk cumulative log-decay (restarted at every chunk).

Tiles are reported C x C per (head, chunk) in the order [H, n_chunks], the
chunk index running over the sequences in order: the m x m inverse in the top
left and the identity on the rows and columns past m (the inverse of the
system padded with tokens that write nothing).

Each chunk is computed on its own m x m matrices with the functions of
oracle/gdn.py; nothing is padded in the arithmetic.

The layer forward over packed sequences (forward_varlen_recurrent,
forward_varlen_chunked) runs the gated delta rule of oracle/gdn_forward.py
on every sequence from its own initial state: the token recurrence, and the
chunk-wise form on every chunk's m x m system.
"""

from __future__ import annotations

from typing import Callable, List, Tuple

import numpy as np

from . import gdn


def chunk_table(cu_seqlens, C: int) -> List[Tuple[int, int, int]]:
    """(sequence, first token, length m) of every chunk, in order."""
    cu = [int(x) for x in cu_seqlens]
    out = []
    for s in range(len(cu) - 1):
        t = cu[s]
        while t < cu[s + 1]:
            m = min(C, cu[s + 1] - t)
            out.append((s, t, m))
            t += m
    return out


def chunk_offsets(cu_seqlens, C: int) -> np.ndarray:
    """First chunk index of every sequence, and the chunk count last."""
    cu = np.asarray(cu_seqlens, np.int64)
    per = (cu[1:] - cu[:-1] + C - 1) // C
    return np.concatenate([[0], np.cumsum(per)]).astype(np.int64)


def varlen_cumsum(inc: np.ndarray, cu_seqlens, C: int) -> np.ndarray:
    """Within-chunk inclusive cumulative sum over packed sequences, chunks
    restarting at every sequence start.  inc [T, ...] along axis 0."""
    out = np.empty_like(np.asarray(inc, np.float64))
    for _, t, m in chunk_table(cu_seqlens, C):
        out[t:t + m] = np.cumsum(inc[t:t + m], axis=0)
    return out


def wy_varlen(K, V, beta, g, cu_seqlens, C: int,
              inverse: Callable[[np.ndarray], np.ndarray] = gdn.forward_substitution_inverse):
    """W [1, T, H, dk], U [1, T, H, dv] and the tiles [H, n_chunks, C, C].

    `inverse` maps a stack of strictly lower m x m tiles A to (I + A)^-1."""
    K = np.asarray(K, np.float64)[0]
    V = np.asarray(V, np.float64)[0]
    beta = np.asarray(beta, np.float64)[0]
    g = np.asarray(g, np.float64)[0]
    T_, H, dk = K.shape
    dv = V.shape[-1]
    table = chunk_table(cu_seqlens, C)
    W = np.zeros((T_, H, dk))
    U = np.zeros((T_, H, dv))
    tiles = np.zeros((H, len(table), C, C))
    for n, (_, t, m) in enumerate(table):
        for h in range(H):
            k = K[t:t + m, h]
            b = beta[t:t + m, h]
            gg = g[t:t + m, h]
            A = gdn.strict_lower(b[:, None] * (k @ k.T) * np.exp(gg[:, None] - gg[None, :]))
            X = inverse(A[None])[0]
            W[t:t + m, h] = X @ (b[:, None] * k)
            U[t:t + m, h] = X @ (b[:, None] * V[t:t + m, h])
            tiles[h, n] = np.eye(C)
            tiles[h, n, :m, :m] = X
    return W[None], U[None], tiles


# ---------------------------------------------------------------------------
# the layer forward over packed sequences


def varlen_log_decay(g, cu_seqlens, C: int) -> np.ndarray:
    """Per-token log-decay inc from the within-chunk cumulative sum g over
    packed sequences (inc_t = g_t - g_{t-1} inside a chunk, g_t at a chunk's
    first token; chunks start at every sequence start).  g [T, ...]."""
    g = np.asarray(g, np.float64)
    inc = np.empty_like(g)
    for _, t, m in chunk_table(cu_seqlens, C):
        inc[t] = g[t]
        inc[t + 1:t + m] = np.diff(g[t:t + m], axis=0)
    return inc


def forward_varlen_recurrent(Q, K, V, beta, g, cu_seqlens, C: int, S0=None, scale: float = 1.0):
    """Token recurrence of the gated delta rule (oracle/gdn_forward.py's
    gdn_recurrent) run on every packed sequence on its own, from its own
    initial state.  Q, K [1, T, H, dk]; V [1, T, H, dv]; beta, g [1, T, H];
    S0 [nseq, H, dk, dv] or None.  Returns O [1, T, H, dv], S_final
    [nseq, H, dk, dv]."""
    Q, K, V = (np.asarray(x, np.float64)[0] for x in (Q, K, V))
    beta = np.asarray(beta, np.float64)[0]
    a = np.exp(varlen_log_decay(np.asarray(g, np.float64)[0], cu_seqlens, C))
    cu = [int(x) for x in cu_seqlens]
    T_, H, dk = K.shape
    dv = V.shape[-1]
    ns = len(cu) - 1
    Sf = np.zeros((ns, H, dk, dv)) if S0 is None else np.array(S0, np.float64)
    O = np.zeros((T_, H, dv))
    for s in range(ns):
        S = Sf[s].copy()
        for t in range(cu[s], cu[s + 1]):
            k, v = K[t], V[t]                      # [H, dk], [H, dv]
            kS = np.einsum("hk,hkv->hv", k, S)
            S = a[t, :, None, None] * (S - beta[t, :, None, None] * k[:, :, None] * kS[:, None, :]) \
                + beta[t, :, None, None] * k[:, :, None] * v[:, None, :]
            O[t] = scale * np.einsum("hkv,hk->hv", S, Q[t])
        Sf[s] = S
    return O[None], Sf


def forward_varlen_chunked(Q, K, V, beta, g, cu_seqlens, C: int, S0=None, scale: float = 1.0,
                           inverse: Callable[[np.ndarray], np.ndarray] =
                           gdn.forward_substitution_inverse):
    """Chunk-wise form over packed sequences: every chunk of m <= C tokens
    on its own m x m system (oracle/gdn_forward.py's gdn_chunked on the
    chunk's tokens), the state carried through a sequence's chunks in order.
    `inverse` maps a stack of strictly lower m x m tiles A to (I + A)^-1."""
    Q, K, V = (np.asarray(x, np.float64)[0] for x in (Q, K, V))
    beta = np.asarray(beta, np.float64)[0]
    g = np.asarray(g, np.float64)[0]
    T_, H, dk = K.shape
    dv = V.shape[-1]
    ns = len(cu_seqlens) - 1
    Sf = np.zeros((ns, H, dk, dv)) if S0 is None else np.array(S0, np.float64)
    O = np.zeros((T_, H, dv))
    for s, t, m in chunk_table(cu_seqlens, C):
        for h in range(H):
            q, k, v = Q[t:t + m, h], K[t:t + m, h], V[t:t + m, h]
            b, gg = beta[t:t + m, h], g[t:t + m, h]
            A = gdn.strict_lower(b[:, None] * (k @ k.T) * np.exp(gg[:, None] - gg[None, :]))
            X = inverse(A[None])[0]
            W = X @ ((b * np.exp(gg))[:, None] * k)
            U = X @ (b[:, None] * v)
            S = Sf[s, h]
            Vn = U - W @ S
            D = np.tril(np.exp(gg[:, None] - gg[None, :]))
            O[t:t + m, h] = scale * (np.exp(gg)[:, None] * (q @ S) + ((q @ k.T) * D) @ Vn)
            last = gg[-1]
            Sf[s, h] = np.exp(last) * S + (np.exp(last - gg)[:, None] * k).T @ Vn
    return O[None], Sf
