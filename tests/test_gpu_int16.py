"""Bit-exact parity of the INT16 path (through the C ABI) with the integer
oracle at 16-bit codes.

As for INT8: both sides start from the same float32 A tiles, so the
quantiser takes every rounding decision on the same values, and from there
on everything is integer arithmetic; codes and exponents must agree exactly.
The GPU forms each product of 16-bit codes from four int8 MFMAs over the
codes' limbs and keeps products and sums as fp64 integers; the oracle uses
int64.  Cases cover the limb boundaries (codes around multiples of 256 and
the range ends +-32639) besides the workload distributions.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn
from oracle import int8 as oi

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu

SPEC = oi.SPEC16
ORDERS = {16: [(3, 2), (0, 3), (2, 0), (1, 1), (5, 4)],
          32: [(3, 4), (0, 2), (3, 0), (2, 7), (6, 3)],
          64: [(3, 8), (0, 5), (3, 0), (3, 15), (7, 7), (1, 2)]}


def f32_tiles(C, L=None, H=2, gate="wide", stress=False, seed=0):
    """float32 A tiles [n, C, C] of the low-bit workload's distributions."""
    w = wl.workload("int8")
    L = L or 4 * max(C, 64)
    if stress:
        heads = [wl.gen_stress_head(L, w.dk, C, seed=seed + h) for h in range(H)]
    else:
        w = w.with_(L=L, H=H, B=1, gate=gate)
        heads = [wl.gen_head(w, 0, h, C=C, want_v=False) for h in range(H)]
    K = wl.as_blhd(*[x[0] for x in heads])
    beta = wl.as_blhd(*[x[1] for x in heads])
    g = wl.as_blhd(*[x[2] for x in heads])
    return gdn.tiles_flat(gdn.build_A(K, beta, g, C)).astype(np.float32)


def random_codes(n, C, seed, density=1.0, emin=None, emax=None, limb_edges=False):
    """Random strictly lower int16 codes (dense, sparse, or drawn from values
    next to the limb boundaries) and exponents.  Dense tiles take exponents at
    which every row of |A| sums below 1 (32639 2^e C < 1: the Neumann series
    of Section 3.1 converges, Lemma 2), sparse ones a wide range."""
    if emax is None:
        emax = -(15 + int(np.log2(C)) + 1) if density >= 0.5 else 2
    if emin is None:
        emin = emax - 12 if density >= 0.5 else -30
    rng = np.random.default_rng([seed, C, 16])
    if limb_edges:
        base = 256 * rng.integers(-127, 128, size=(n, C, C))
        q = np.clip(base + rng.choice([-129, -128, -127, -1, 0, 1, 127, 128], size=(n, C, C)),
                    -32639, 32639)
        q = np.where(rng.random((n, C, C)) < 0.05, rng.choice([-32639, 32639], (n, C, C)), q)
    else:
        q = rng.integers(-32639, 32640, size=(n, C, C))
    if density < 1.0:
        q = np.where(rng.random((n, C, C)) < density, q, 0)
    q = np.tril(q, -1)
    e = rng.integers(emin, emax + 1, size=n)
    return q.astype(np.int64), e.astype(np.int64)


def to_dev(x, dt):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dt).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def run_engine(qA, eA, N, S, want_deq=True, plain=False):
    out = G.gdn_chunk_inverse_neumann_i16(to_dev(qA, torch.int16), to_dev(eA, torch.int32),
                                          N, S, want_deq=want_deq, plain=plain)
    return [host(t) for t in out]


def check_deq(Td, rq, re, plain=False):
    """Tdeq against the oracle's codes: equal wherever T_hat is finite in
    fp32, and infinite where its value overflows fp32 (random codes with
    large exponents)."""
    with np.errstate(over="ignore"):
        ref = (oi.dequant(rq, re) if plain else oi.dequant_unit(rq, re)).astype(np.float32)
    fin = np.isfinite(ref)
    assert np.array_equal(Td[fin], ref[fin])
    assert np.array_equal(Td[~fin], ref[~fin])
    return fin.mean()


def check_engine(qA, eA, N, S, label, plain=False):
    print(f"i16 engine {label}{' plain' if plain else ''} N={N} S={S} n={qA.shape[0]}",
          flush=True)
    qT, eT, Td = run_engine(qA, eA, N, S, plain=plain)
    rq, re, _ = oi.neumann_inverse_int16(qA, eA, N, S, plain=plain)
    bad = np.flatnonzero(np.any(qT.astype(np.int64) != rq, axis=(-1, -2)) |
                         (eT.astype(np.int64) != re))
    print(f"  mismatching tiles={bad.size}", flush=True)
    assert bad.size == 0, (label, N, S, bad[:8])
    check_deq(Td, rq, re, plain)


# ---------------------------------------------------------------------------
# quantiser


@pytest.mark.parametrize("C", [16, 32, 64])
@pytest.mark.parametrize("src", ["workload", "default_gate", "stress"])
def test_quantize_i16_bit_exact(C, src):
    A = f32_tiles(C, stress=(src == "stress"), gate="default" if src == "default_gate" else "wide")
    print(f"i16 quantize C={C} {src} n={A.shape[0]}", flush=True)
    Aq, eA = G.gdn_quantize_tiles_i16(to_dev(A, torch.float32))
    rq, re = oi.quantize(A, SPEC)
    assert np.array_equal(host(Aq).astype(np.int64), rq)
    assert np.array_equal(host(eA).astype(np.int64), re)


def test_quantize_i16_edge_values():
    """Zero tiles, a max on a power of two, a max just past 32639 at the
    first exponent, half-way codes, tiny and large magnitudes, and an upper
    triangle of junk that must be ignored."""
    C = 16
    tiles = np.zeros((6, C, C), np.float32)
    tiles[1, 5, 2] = 1.0
    tiles[2, 9, 0] = 32639.6 / 32768.0        # needs the next exponent
    tiles[2, 3, 1] = 0.5 / 32768.0
    tiles[3, 1, 0] = 32639.0
    tiles[3, 2, 0] = 2.5                      # half-way code at e = 0 -> 2
    tiles[3, 2, 1] = -3.5                     # -> -4
    tiles[4, 7, 3] = 3e-30
    tiles[4, 8, 3] = -1.7e-30
    tiles[5, 15, 0] = 6e30
    tiles[5, 15, 14] = 1e29
    junk = tiles + np.triu(np.full((C, C), 1e35, np.float32))
    Aq, eA = G.gdn_quantize_tiles_i16(to_dev(junk, torch.float32))
    rq, re = oi.quantize(tiles, SPEC)
    assert np.array_equal(host(Aq).astype(np.int64), rq)
    assert np.array_equal(host(eA).astype(np.int64), re)
    assert host(eA)[0] == 0 and np.all(host(Aq)[0] == 0)
    assert host(Aq)[3, 1, 0] == 32639 and host(eA)[3] == 0


# ---------------------------------------------------------------------------
# integer inverse


@pytest.mark.parametrize("C", [16, 32, 64])
@pytest.mark.parametrize("src", ["workload", "stress", "random_dense", "random_sparse",
                                 "limb_edges"])
def test_neumann_i16_bit_exact(C, src):
    if src.startswith("random") or src == "limb_edges":
        qA, eA = random_codes(32, C, seed={"random_dense": 11, "random_sparse": 12}.get(src, 13),
                              density=0.08 if src == "random_sparse" else 1.0,
                              limb_edges=(src == "limb_edges"))
    else:
        qA, eA = oi.quantize(f32_tiles(C, stress=(src == "stress")), SPEC)
    for N, S in ORDERS[C]:
        check_engine(qA, eA, N, S, f"C={C} {src}")


def test_neumann_i16_extreme_orders():
    for C in (16, 32, 64):
        qA, eA = oi.quantize(f32_tiles(C, stress=True, H=1), SPEC)
        for N, S in [(C - 1, 0), (0, C - 1), (C - 1, C - 1)]:
            check_engine(qA, eA, N, S, f"C={C} extreme")


def test_neumann_i16_edge_tiles():
    for C in (16, 32, 64):
        qA = np.zeros((5, C, C), np.int64)
        eA = np.zeros(5, np.int64)
        qA[1, C - 1, 0] = 32639               # one deep entry only
        eA[1] = -3
        qA[2, 1, 0] = -32639                  # one sub-diagonal entry
        qA[3] = np.tril(np.full((C, C), 32639), -1)   # all-max codes
        eA[3] = -20
        qA[4] = np.tril(np.full((C, C), -1), -1)
        eA[4] = 40
        for N, S in [(3, 2), (0, 1), (3, 0)]:
            check_engine(qA, eA, N, S, f"C={C} edge")
        qT, eT, Td = run_engine(qA[:1], eA[:1], 3, 2)
        assert np.all(qT == 0) and eT[0] == 0 and np.array_equal(Td[0], np.eye(C, dtype=np.float32))


@pytest.mark.parametrize("C", [16, 32, 64])
@pytest.mark.parametrize("src", ["workload", "stress", "random_dense"])
def test_neumann_i16_plain_bit_exact(C, src):
    """The plain form (GDN_INT_PLAIN: the unit diagonal inside every tensor's
    codes) against the oracle's plain form."""
    if src.startswith("random"):
        qA, eA = random_codes(32, C, seed=13)
    else:
        qA, eA = oi.quantize(f32_tiles(C, stress=(src == "stress")), SPEC)
    for N, S in ORDERS[C][:4]:
        check_engine(qA, eA, N, S, f"C={C} {src}", plain=True)


def test_neumann_i16_plain_identity():
    """A = 0 in plain form: T_hat = I with 1 at the finest scale that holds
    it (2^(qbits - 1) at exponent 1 - qbits)."""
    qb = 15
    for C in (16, 32, 64):
        qA = np.zeros((2, C, C), np.int64)
        qT, eT, Td = run_engine(qA, np.zeros(2, np.int64), 3, 2, plain=True)
        assert np.all(eT == 1 - qb)
        assert np.array_equal(qT[0].astype(np.int64), np.eye(C, dtype=np.int64) << (qb - 1))
        assert np.array_equal(Td[1], np.eye(C, dtype=np.float32))


def test_i16_pipeline_many_tiles_odd_count():
    """Quantiser then engine on 67 tiles, both on the GPU, as one chain."""
    A = f32_tiles(64, L=67 * 64, H=1)
    assert A.shape[0] == 67
    Aq, eA = G.gdn_quantize_tiles_i16(to_dev(A, torch.float32))
    qT, eT = G.gdn_chunk_inverse_neumann_i16(Aq, eA, 3, 8)
    rqA, reA = oi.quantize(A, SPEC)
    rq, re, _ = oi.neumann_inverse_int16(rqA, reA, 3, 8)
    assert np.array_equal(host(qT).astype(np.int64), rq)
    assert np.array_equal(host(eT).astype(np.int64), re)


def test_i16_deterministic_and_without_dequant():
    qA, eA = random_codes(40, 64, seed=21)
    a = run_engine(qA, eA, 3, 8)
    b = run_engine(qA, eA, 3, 8, want_deq=False)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_i16_full_size_sampled():
    """Low-bit workload at full size (B=4, H=32, L=16384, C=64: 32768 tiles)
    in one launch of each kernel, compared tile by tile on a sample."""
    w = wl.workload("int8")
    C = w.C
    nc = w.L // C
    A = np.empty((w.B * w.H * nc, C, C), np.float32)
    for b in range(w.B):
        for h in range(w.H):
            K, beta, g, _ = wl.gen_head(w, b, h, want_v=False)
            t0 = wl.tile_index(w, b, h, 0)
            A[t0:t0 + nc] = gdn.tiles_flat(
                gdn.build_A(K[None, :, None], beta[None, :, None], g[None, :, None], C))
    print(f"int16 full size: {A.shape[0]} tiles generated", flush=True)
    Aq, eA = G.gdn_quantize_tiles_i16(to_dev(A, torch.float32))
    N, S = G.gdn_default_order(C)
    qT, eT, Td = G.gdn_chunk_inverse_neumann_i16(Aq, eA, N, S, want_deq=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(78)
    idx = np.sort(np.concatenate([[0, A.shape[0] - 1],
                                  rng.choice(A.shape[0], 254, replace=False)]))
    idx_t = torch.from_numpy(idx).to("cuda")
    rqA, reA = oi.quantize(A[idx], SPEC)
    assert np.array_equal(host(Aq[idx_t]).astype(np.int64), rqA)
    assert np.array_equal(host(eA[idx_t]).astype(np.int64), reA)
    rq, re, _ = oi.neumann_inverse_int16(rqA, reA, N, S)
    assert np.array_equal(host(qT[idx_t]).astype(np.int64), rq)
    assert np.array_equal(host(eT[idx_t]).astype(np.int64), re)
    assert np.array_equal(host(Td[idx_t]), oi.dequant_unit(rq, re).astype(np.float32))


# ---------------------------------------------------------------------------
# one launch from K: build A, quantise, integer inverse


def head_set(C, kdt, L=None, H=2, stress=False):
    w = wl.workload("int8").with_(dtype=kdt, L=L or 4 * max(C, 64), H=H, B=1)
    if stress:
        heads = [wl.gen_stress_head(w.L, w.dk, C, seed=60 + h) for h in range(H)]
        heads = [(wl.round_to_bf16(k) if kdt == "bf16" else k, b, g, v) for k, b, g, v in heads]
    else:
        heads = [wl.gen_head(w, 0, h, C=C, want_v=False) for h in range(H)]
    return tuple(wl.as_blhd(*[x[i] for x in heads]) for i in range(3))


def to_cuda(x, dt=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda").to(dt)


@pytest.mark.parametrize("kdt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64])
def test_i16_fused_matches_stages(C, kdt):
    """The fused launch equals gdn_build_A (fp32) -> quantiser -> integer
    inverse on the GPU, bit for bit."""
    K, beta, g = head_set(C, kdt, stress=(C == 32))
    dK = to_cuda(K, torch.bfloat16 if kdt == "bf16" else torch.float32)
    db, dg = to_cuda(beta), to_cuda(g)
    for N, S in ORDERS[C][:3]:
        print(f"i16 fused vs stages C={C} K={kdt} N={N} S={S}", flush=True)
        A = G.gdn_build_A(dK, db, dg, C, a_dtype=torch.float32)
        Aq, eA = G.gdn_quantize_tiles_i16(A)
        q1, e1, d1 = G.gdn_chunk_inverse_neumann_i16(Aq, eA, N, S, want_deq=True)
        q2, e2, d2 = G.gdn_chunk_inverse_neumann_i16_fused(dK, db, dg, C, N, S, want_deq=True)
        assert np.array_equal(host(q1).reshape(-1), host(q2).reshape(-1))
        assert np.array_equal(host(e1), host(e2))
        assert np.array_equal(host(d1).reshape(-1), host(d2).reshape(-1))


@pytest.mark.parametrize("C", [16, 32, 64])
def test_i16_fused_vs_oracle_and_float(C):
    """Against the integer oracle run from its own fp32 A (float64 build,
    rounded): the GPU forms A in fp32 arithmetic, so an entry a few ulp away
    can move a 16-bit code at a rounding boundary.  Measured: every tile of
    this sample bit-exact at C = 16, 32, 64; the bounds allow three tiles in
    64 to differ, by at most a few dozen quanta.  Against the float64
    T_hat(N, S) the INT16 result is within a small multiple of 2^-16 of
    max|T_hat - I| per tile."""
    K, beta, g = head_set(C, "bf16", L=16 * C, H=4)
    N, S = G.gdn_default_order(C)
    print(f"i16 fused vs oracle C={C}", flush=True)
    Tq, eT, Td = G.gdn_chunk_inverse_neumann_i16_fused(to_cuda(K, torch.bfloat16), to_cuda(beta),
                                                       to_cuda(g), C, N, S, want_deq=True)
    Af = gdn.tiles_flat(gdn.build_A(K, beta, g, C))
    qA, eA = oi.quantize(Af.astype(np.float32), SPEC)
    rq, re, _ = oi.neumann_inverse_int16(qA, eA, N, S)
    gq = host(Tq).reshape(rq.shape).astype(np.int64)
    ge = host(eT).astype(np.int64)
    same = np.all(gq == rq, axis=(-1, -2)) & (ge == re)
    got = host(Td).reshape(rq.shape).astype(np.float64)
    quanta = np.abs(got - oi.dequant_unit(rq, re)) / np.ldexp(1.0, re)[:, None, None]
    print(f"  {same.mean():.4f} of {same.size} tiles bit-exact, max {quanta.max():.1f} quanta",
          flush=True)
    assert same.mean() >= 0.95
    assert quanta.max() <= 64.0
    T = gdn.neumann_inverse(Af, N, S)
    scale = np.max(np.abs(T - np.eye(C)), axis=(-1, -2))
    err = np.max(np.abs(got - T), axis=(-1, -2))
    assert np.all(err <= 16 * 2.0 ** -16 * scale)


# ---------------------------------------------------------------------------
# the forward-substitution baseline on 16-bit codes


def check_fwdsub(qA, eA, label):
    print(f"i16 fwdsub {label} n={qA.shape[0]}", flush=True)
    qT, eT, Td = [host(t) for t in G.gdn_chunk_inverse_fwdsub_i16(
        to_dev(qA, torch.int16), to_dev(eA, torch.int32), want_deq=True)]
    rq, re = oi.fwdsub_inverse_int(qA, eA)
    bad = np.flatnonzero(np.any(qT.astype(np.int64) != rq, axis=(-1, -2)) |
                         (eT.astype(np.int64) != re))
    print(f"  mismatching tiles={bad.size}", flush=True)
    assert bad.size == 0, (label, bad[:8])
    check_deq(Td, rq, re)


@pytest.mark.parametrize("C", [16, 32, 64])
@pytest.mark.parametrize("src", ["workload", "stress", "random_dense", "random_sparse",
                                 "limb_edges"])
def test_fwdsub_i16_bit_exact(C, src):
    if src.startswith("random") or src == "limb_edges":
        qA, eA = random_codes(32, C, seed={"random_dense": 31, "random_sparse": 32}.get(src, 33),
                              density=0.08 if src == "random_sparse" else 1.0,
                              limb_edges=(src == "limb_edges"))
    else:
        qA, eA = oi.quantize(f32_tiles(C, stress=(src == "stress")), SPEC)
    check_fwdsub(qA, eA, f"C={C} {src}")


def test_fwdsub_i16_growth_and_edge_tiles():
    """Tiles whose inverse outgrows A (minus-ones: x_ij = 2^(i-j-1)), so the
    tile exponent grows row after row; all-max codes; zero and one-entry
    tiles; a large exponent."""
    for C in (16, 32, 64):
        qA = np.zeros((7, C, C), np.int64)
        eA = np.zeros(7, np.int64)
        qA[1, C - 1, 0] = 32639
        eA[1] = -3
        qA[2, 1, 0] = -32639
        qA[3] = np.tril(np.full((C, C), 32639), -1)
        eA[3] = -20
        qA[4] = np.tril(np.full((C, C), -1), -1)
        eA[4] = 40
        qA[5] = np.tril(np.full((C, C), -16384), -1)    # A = -1: x_ij = 2^(i-j-1)
        eA[5] = -14
        qA[6] = np.tril(np.full((C, C), -24575), -1)    # A ~ -0.75, growth with rounding
        eA[6] = -15
        check_fwdsub(qA, eA, f"C={C} growth/edge")
        qT, eT = [host(t) for t in G.gdn_chunk_inverse_fwdsub_i16(
            to_dev(qA[:1], torch.int16), to_dev(eA[:1], torch.int32))]
        assert np.all(qT == 0) and eT[0] == 0


def test_fwdsub_i16_many_tiles_and_accuracy():
    """Quantiser then integer forward substitution on 131 workload tiles, on
    the GPU; bit-exact, and within a few 16-bit quanta of the exact
    inverse."""
    A = f32_tiles(64, L=131 * 64, H=1)
    Aq, eA = G.gdn_quantize_tiles_i16(to_dev(A, torch.float32))
    qT, eT, Td = G.gdn_chunk_inverse_fwdsub_i16(Aq, eA, want_deq=True)
    rqA, reA = oi.quantize(A, SPEC)
    rq, re = oi.fwdsub_inverse_int(rqA, reA)
    assert np.array_equal(host(qT).astype(np.int64), rq)
    assert np.array_equal(host(eT).astype(np.int64), re)
    X = gdn.forward_substitution_inverse(A.astype(np.float64))
    scale = np.max(np.abs(X - np.eye(64)), axis=(-1, -2))
    err = np.max(np.abs(host(Td).astype(np.float64) - X), axis=(-1, -2))
    assert np.all(err <= 8 * 2.0 ** -15 * scale)
