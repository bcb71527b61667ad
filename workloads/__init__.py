"""Seeded synthetic inputs for the chunk-wise Gated DeltaNet inverse path.

This module is shared by the HIP path's tests/benchmarks and by the CPU
oracle.  It holds no arithmetic of the method itself: it only draws keys,
values, write strengths (beta) and log-decays (g) with the distributions
of the workloads below, and rounds them to the storage dtype.

Layouts (row-major, contiguous):
  K [B, L, H, dk], V [B, L, H, dv], beta [B, L, H], g [B, L, H]
  g is the within-chunk inclusive cumulative sum of the per-token log-decay.

Each (b, h) head draws from its own counter-addressed numpy stream
(``default_rng([seed, b, h])``), so one head's inputs can be regenerated
without generating the whole batch; within a head the draws come in the
order K, beta, decay increments, V, Q.  Queries are unit rows like the
keys.  An initial state S0 [dk, dv] ~ N(0, 1) comes from a stream of its
own (``default_rng([seed, b, h, 1])``).
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Iterable, Optional, Tuple

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "workload",
    "round_to_bf16",
    "bf16_bits",
    "gen_head",
    "gen_head_qkv",
    "gen_state",
    "gen_forward_inputs",
    "varlen_lengths",
    "gen_varlen",
    "gen_inputs",
    "gen_inputs_heads",
    "chunk_cumsum",
    "n_tiles",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: sizes, storage dtype and decay distribution.

    gate = "default": per-token log-decay -softplus(x + 3), x ~ N(0, 1)
    gate = "wide":    per-token log-decay -softplus(2 x + 1), x ~ N(0, 1)
                      (the larger-spread gates used for the low-bit path)
    """

    name: str
    B: int
    L: int
    H: int
    dk: int
    dv: int
    C: int
    dtype: str  # "f32" | "bf16"
    gate: str = "default"
    seed: int = 1000

    @property
    def tiles(self) -> int:
        return self.B * self.H * (self.L // self.C)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The workloads the library is measured and tested on.  The seeds are
# 1000 + position in this list.
WORKLOADS: Dict[str, Workload] = {
    # 64 tiles, fp32: small enough for the oracle to check every tile.
    "tiny": Workload("tiny", B=1, L=1024, H=4, dk=128, dv=128, C=64, dtype="f32", seed=1000),
    # Qwen3.5-shaped prefill: 16 key heads, 8K tokens, bf16 storage.
    "qwen35_prefill": Workload("qwen35_prefill", B=1, L=8192, H=16, dk=128, dv=128, C=64,
                               dtype="bf16", seed=1001),
    # Chunk-size sweep (C is replaced per run by 16, 32, 64 or 128).
    "sweep": Workload("sweep", B=4, L=16384, H=32, dk=128, dv=128, C=64, dtype="bf16", seed=1002),
    # Low-bit path: wider gate spread.
    "int8": Workload("int8", B=4, L=16384, H=32, dk=128, dv=128, C=64, dtype="bf16",
                     gate="wide", seed=1003),
    # Long context: 128K tokens x 32 heads.
    "long_context": Workload("long_context", B=1, L=131072, H=32, dk=128, dv=128, C=64,
                             dtype="bf16", seed=1004),
}


def workload(name: str, **overrides) -> Workload:
    w = WORKLOADS[name]
    return w.with_(**overrides) if overrides else w


def n_tiles(B: int, L: int, H: int, C: int) -> int:
    return B * H * (L // C)


# ----------------------------------------------------------------------------
# dtype rounding (storage only)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns as uint16.  NaN stays NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    nan = np.isnan(x)
    r = np.where(nan, (u >> np.uint64(16)) | np.uint64(0x40), r)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float64/float32 -> float32 holding the nearest bfloat16 value
    (first rounded to float32, then to bfloat16, both ties-to-even)."""
    return bf16_to_f32(bf16_bits(np.asarray(x, dtype=np.float32)))


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 draws to the storage dtype; returned as float32 arrays
    holding exactly the stored values."""
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype == "bf16":
        return round_to_bf16(x)
    raise ValueError(f"unknown dtype {dtype!r}")


# ----------------------------------------------------------------------------
# generators


def _softplus(x: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, x)


def chunk_cumsum(inc: np.ndarray, C: int, axis: int = 0) -> np.ndarray:
    """Inclusive cumulative sum restarted at every chunk of C positions
    along ``axis`` (the token axis)."""
    inc = np.moveaxis(inc, axis, 0)
    L = inc.shape[0]
    assert L % C == 0
    r = inc.reshape((L // C, C) + inc.shape[1:]).cumsum(axis=1)
    return np.moveaxis(r.reshape(inc.shape), 0, axis)


def _draw_head(w: Workload, b: int, h: int, C: int, want_v: bool, want_q: bool):
    rng = np.random.default_rng([w.seed, b, h])
    z = rng.standard_normal((w.L, w.dk))
    k = z / np.linalg.norm(z, axis=1, keepdims=True)
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal(w.L)))
    x = rng.standard_normal(w.L)
    if w.gate == "default":
        inc = -_softplus(x + 3.0)
    elif w.gate == "wide":
        inc = -_softplus(2.0 * x + 1.0)
    else:
        raise ValueError(w.gate)
    g = chunk_cumsum(inc, C)
    v = rng.standard_normal((w.L, w.dv)) if (want_v or want_q) else None
    q = None
    if want_q:
        z = rng.standard_normal((w.L, w.dk))
        q = z / np.linalg.norm(z, axis=1, keepdims=True)
    return k, beta, g, v, q


def gen_head(w: Workload, b: int, h: int, C: Optional[int] = None,
             want_v: bool = True) -> Tuple[np.ndarray, np.ndarray, np.ndarray, Optional[np.ndarray]]:
    """Inputs of one (b, h) head: K [L, dk], beta [L], g [L], V [L, dv].

    K, V are rounded to the workload's storage dtype (returned as float32
    arrays holding the stored values); beta and g are float32.
    """
    C = w.C if C is None else C
    k, beta, g, v, _ = _draw_head(w, b, h, C, want_v, False)
    return (_store(k, w.dtype), beta.astype(np.float32), g.astype(np.float32),
            None if v is None else _store(v, w.dtype))


def gen_head_qkv(w: Workload, b: int, h: int, C: Optional[int] = None):
    """Inputs of one (b, h) head for the whole layer: Q [L, dk], K [L, dk],
    V [L, dv] (storage dtype values as float32), beta [L], g [L] (float32).
    K, beta, g, V are the values gen_head returns."""
    C = w.C if C is None else C
    k, beta, g, v, q = _draw_head(w, b, h, C, True, True)
    return (_store(q, w.dtype), _store(k, w.dtype), _store(v, w.dtype),
            beta.astype(np.float32), g.astype(np.float32))


def gen_state(w: Workload, b: int, h: int) -> np.ndarray:
    """Initial state S0 [dk, dv] of one head, float32 ~ N(0, 1)."""
    rng = np.random.default_rng([w.seed, b, h, 1])
    return rng.standard_normal((w.dk, w.dv)).astype(np.float32)


def gen_forward_inputs(w: Workload, C: Optional[int] = None, want_state: bool = True):
    """Full-size layer inputs: Q, K [B, L, H, dk], V [B, L, H, dv],
    beta, g [B, L, H], S0 [B, H, dk, dv] (or None); float32 arrays holding
    the stored values."""
    C = w.C if C is None else C
    Q = np.empty((w.B, w.L, w.H, w.dk), np.float32)
    K = np.empty_like(Q)
    V = np.empty((w.B, w.L, w.H, w.dv), np.float32)
    beta = np.empty((w.B, w.L, w.H), np.float32)
    g = np.empty_like(beta)
    S0 = np.empty((w.B, w.H, w.dk, w.dv), np.float32) if want_state else None
    for b in range(w.B):
        for h in range(w.H):
            Q[b, :, h], K[b, :, h], V[b, :, h], beta[b, :, h], g[b, :, h] = gen_head_qkv(w, b, h, C=C)
            if want_state:
                S0[b, h] = gen_state(w, b, h)
    return Q, K, V, beta, g, S0


def gen_inputs_heads(w: Workload, heads: Iterable[Tuple[int, int]], C: Optional[int] = None,
                     want_v: bool = True):
    """Dict (b, h) -> (K, beta, g, V) for the listed heads only."""
    return {bh: gen_head(w, bh[0], bh[1], C=C, want_v=want_v) for bh in heads}


def gen_inputs(w: Workload, C: Optional[int] = None, want_v: bool = True):
    """Full-size inputs in the [B, L, H, *] layouts (float32 arrays holding
    the stored values)."""
    C = w.C if C is None else C
    K = np.empty((w.B, w.L, w.H, w.dk), np.float32)
    beta = np.empty((w.B, w.L, w.H), np.float32)
    g = np.empty((w.B, w.L, w.H), np.float32)
    V = np.empty((w.B, w.L, w.H, w.dv), np.float32) if want_v else None
    for b in range(w.B):
        for h in range(w.H):
            k, be, gg, v = gen_head(w, b, h, C=C, want_v=want_v)
            K[b, :, h] = k
            beta[b, :, h] = be
            g[b, :, h] = gg
            if want_v:
                V[b, :, h] = v
    return K, beta, g, V


def tile_index(w: Workload, b: int, h: int, chunk: int, C: Optional[int] = None) -> int:
    """Position of the (b, h, chunk) tile in the [B, H, L/C, C, C] layout."""
    C = w.C if C is None else C
    return (b * w.H + h) * (w.L // C) + chunk


def tile_coords(w: Workload, t: int, C: Optional[int] = None) -> Tuple[int, int, int]:
    C = w.C if C is None else C
    nc = w.L // C
    bh, chunk = divmod(t, nc)
    b, h = divmod(bh, w.H)
    return b, h, chunk


# ----------------------------------------------------------------------------
# stress inputs (tests and error grids only)


def gen_stress_head(L: int, dk: int, C: int, seed: int, dv: int = 0):
    """A harder-than-default head: keys share a common direction
    (normalize(u + 0.5 z)), gates decay slowly (-softplus(x - 4)), so
    |A| entries reach ~0.5 and the inverse has sizeable deep sub-diagonals.
    Returns float32 K [L, dk], beta [L], g [L], V [L, dv] (or None)."""
    rng = np.random.default_rng([seed, 7777])
    u = rng.standard_normal(dk)
    z = rng.standard_normal((L, dk))
    k = u[None, :] + 0.5 * z
    k = k / np.linalg.norm(k, axis=1, keepdims=True)
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal(L)))
    inc = -_softplus(rng.standard_normal(L) - 4.0)
    g = chunk_cumsum(inc, C)
    v = rng.standard_normal((L, dv)) if dv else None
    return (k.astype(np.float32), beta.astype(np.float32), g.astype(np.float32),
            None if v is None else v.astype(np.float32))


def as_blhd(*heads):
    """Stack per-head arrays ([L, d] or [L]) of one batch into [1, L, H, d]
    or [1, L, H]."""
    return np.stack(heads, axis=1)[None]


# ----------------------------------------------------------------------------
# packed variable-length sequences (serving)


def varlen_lengths(total: int, seed: int = 3000, lo: int = 1, hi: int = 4096):
    """Sequence lengths of a serving mix: log-uniform in [lo, hi], drawn until
    they add up to `total` (the last one cut to fit)."""
    rng = np.random.default_rng([seed, 5])
    out = []
    left = total
    while left > 0:
        n = int(np.exp(rng.uniform(np.log(lo), np.log(hi + 1))))
        n = max(lo, min(n, hi, left))
        out.append(n)
        left -= n
    return out


def gen_varlen(w: Workload, lengths, C: Optional[int] = None, want_q: bool = False):
    """Packed inputs of sequences with the given lengths: K [1, T, H, dk],
    beta, g [1, T, H], V [1, T, H, dv] (and Q [1, T, H, dk] when asked),
    cu_seqlens [n + 1] int32.  Sequence s, head h draws from
    default_rng([seed, 2, s, h]) in the order K, beta, decay increments, V,
    Q, with the workload's distributions; g is the within-chunk cumulative
    sum with chunks restarting at every sequence start."""
    C = w.C if C is None else C
    lengths = [int(x) for x in lengths]
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    T = int(cu[-1])
    K = np.zeros((1, T, w.H, w.dk), np.float32)
    V = np.zeros((1, T, w.H, w.dv), np.float32)
    Q = np.zeros((1, T, w.H, w.dk), np.float32) if want_q else None
    beta = np.zeros((1, T, w.H), np.float32)
    g = np.zeros((1, T, w.H), np.float32)
    for s, n in enumerate(lengths):
        if n == 0:
            continue
        t0 = int(cu[s])
        for h in range(w.H):
            rng = np.random.default_rng([w.seed, 2, s, h])
            z = rng.standard_normal((n, w.dk))
            k = z / np.linalg.norm(z, axis=1, keepdims=True)
            be = 1.0 / (1.0 + np.exp(-rng.standard_normal(n)))
            x = rng.standard_normal(n)
            inc = -_softplus(x + 3.0) if w.gate == "default" else -_softplus(2.0 * x + 1.0)
            gg = np.empty(n)
            for a in range(0, n, C):
                gg[a:a + C] = np.cumsum(inc[a:a + C])
            v = rng.standard_normal((n, w.dv))
            K[0, t0:t0 + n, h] = _store(k, w.dtype)
            V[0, t0:t0 + n, h] = _store(v, w.dtype)
            beta[0, t0:t0 + n, h] = be
            g[0, t0:t0 + n, h] = gg
            if want_q:
                z = rng.standard_normal((n, w.dk))
                Q[0, t0:t0 + n, h] = _store(z / np.linalg.norm(z, axis=1, keepdims=True), w.dtype)
    out = (K, beta, g, V, cu)
    return out + (Q,) if want_q else out
