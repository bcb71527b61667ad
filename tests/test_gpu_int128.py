"""Bit-exact parity of the integer paths at C = 128 (block-wise, three
exponents per tile; through the C ABI) with the integer oracle, at 8- and
16-bit codes.

Both sides start from the same float32 A tiles, so the quantiser takes every
rounding decision on the same values; from there on everything is integer
arithmetic, and codes and exponents must agree exactly.  Cases: the workload
distributions (default and wide gates, stress tiles), random codes with
independent block exponents (every rebase path of the merge's sums), tiles
with zero blocks (absent terms), compile-time and run-time orders, many tiles
with a ragged count, and the low-bit workload at full size, sampled.

The one-launch path from K (gdn_chunk_inverse_neumann_i8/_i16_fused at
C = 128) forms A in fp32 on the GPU: it must equal the three launches
(gdn_build_A, the quantiser, the inverse) bit for bit, and the integer oracle
run from its own fp32 A within a few quanta (an A entry one rounding apart
can move a code).
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn
from oracle import int8 as oi

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu

C = 128
WIDTHS = {
    "i8": (oi.SPEC8, torch.int8, G.gdn_quantize_tiles_i8, G.gdn_chunk_inverse_neumann_i8),
    "i16": (oi.SPEC16, torch.int16, G.gdn_quantize_tiles_i16, G.gdn_chunk_inverse_neumann_i16),
}


def f32_tiles(L=512, H=2, gate="wide", stress=False, seed=0):
    """float32 A tiles [n, 128, 128] of the low-bit workload's distributions."""
    w = wl.workload("int8")
    if stress:
        heads = [wl.gen_stress_head(L, w.dk, C, seed=seed + h) for h in range(H)]
    else:
        w = w.with_(L=L, H=H, B=1, gate=gate, seed=w.seed + seed)
        heads = [wl.gen_head(w, 0, h, C=C, want_v=False) for h in range(H)]
    K = wl.as_blhd(*[x[0] for x in heads])
    beta = wl.as_blhd(*[x[1] for x in heads])
    g = wl.as_blhd(*[x[2] for x in heads])
    return gdn.tiles_flat(gdn.build_A(K, beta, g, C)).astype(np.float32)


def random_codes(n, spec, seed, density=1.0, emin=-30, emax=2):
    """Random codes in the block layout (strictly lower diagonal blocks, full
    block 21, zero block 12) with independent exponents per block."""
    rng = np.random.default_rng([seed, spec.qmax])
    q = rng.integers(-spec.qmax, spec.qmax + 1, size=(n, C, C))
    if density < 1.0:
        q = np.where(rng.random((n, C, C)) < density, q, 0)
    q = np.tril(q, -1)
    e = rng.integers(emin, emax + 1, size=(n, 3))
    return q.astype(np.int64), e.astype(np.int64)


def to_dev(x, dt):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dt).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def check_inverse(width, qA, eA, N, S, label):
    spec, cdt, _, inv = WIDTHS[width]
    print(f"{width} C=128 inverse {label} N={N} S={S} n={qA.shape[0]}", flush=True)
    qT, eT, Td = (host(t) for t in inv(to_dev(qA, cdt), to_dev(eA, torch.int32), N, S,
                                        want_deq=True))
    rq, re = oi.neumann_inverse_int_blocked(qA, eA, N, S, spec)
    assert eT.shape == (qA.shape[0], 3)
    for t in range(qA.shape[0]):
        assert np.array_equal(qT[t].astype(np.int64), rq[t]), f"codes of tile {t}"
        assert np.array_equal(eT[t].astype(np.int64), re[t]), f"exponents of tile {t}"
    assert np.array_equal(Td, oi.dequant_unit_blocked(rq, re).astype(np.float32))


@pytest.mark.parametrize("width", ["i8", "i16"])
@pytest.mark.parametrize("src", ["default", "wide", "stress"])
def test_quantize_blocked_bit_exact(width, src):
    spec, cdt, quant, _ = WIDTHS[width]
    A = f32_tiles(gate="default" if src == "default" else "wide", stress=src == "stress")
    A[1, 64:, :64] = 0.0   # a zero block 21
    A[2, :64, :64] = 0.0   # a zero block 11
    # entries on and above the diagonal are ignored
    junk = A + np.triu(np.full((C, C), 1e30, np.float32))
    print(f"{width} C=128 quantise {src} n={A.shape[0]}", flush=True)
    qd, ed = quant(to_dev(junk, torch.float32))
    rq, re = oi.quantize_blocked(A, spec)
    assert np.array_equal(host(qd).astype(np.int64), rq)
    assert np.array_equal(host(ed).astype(np.int64), re)


@pytest.mark.parametrize("width", ["i8", "i16"])
@pytest.mark.parametrize("src", ["default", "wide", "stress"])
def test_inverse_blocked_bit_exact(width, src):
    spec = WIDTHS[width][0]
    A = f32_tiles(gate="default" if src == "default" else "wide", stress=src == "stress",
                  seed=3)
    qA, eA = oi.quantize_blocked(A, spec)
    check_inverse(width, qA, eA, 3, 8, src)


@pytest.mark.parametrize("width", ["i8", "i16"])
@pytest.mark.parametrize("N,S", [(3, 8), (0, 5), (3, 0), (2, 3), (7, 7)])
def test_inverse_blocked_orders_random_codes(width, N, S):
    spec = WIDTHS[width][0]
    qA, eA = random_codes(6, spec, seed=N * 16 + S, density=0.3)
    # the diagonal blocks in the convergent regime (every row of |A_ww| sums
    # below 1, Lemma 2), A21 anywhere; block exponents far apart in both
    # directions between A21 and the diagonal blocks
    dhi = -(spec.qbits + 6 + 1)
    eA[:, 0] = np.minimum(eA[:, 0], dhi)
    eA[:, 2] = np.minimum(eA[:, 2], dhi)
    eA[0] = [dhi - 6, 3, dhi - 6]
    eA[1] = [dhi, -25, dhi]
    check_inverse(width, qA, eA, N, S, "random")


@pytest.mark.parametrize("width", ["i8", "i16"])
def test_inverse_blocked_zero_blocks(width):
    spec = WIDTHS[width][0]
    A = f32_tiles(H=1, L=768, seed=5)  # 6 tiles
    A[0] = 0.0                       # all zero: X = I
    A[1, 64:, :64] = 0.0             # A21 = 0: X21 = 0
    A[2, :64, :64] = 0.0             # A11 = 0: X11 = I
    A[3, 64:, 64:] = 0.0             # A22 = 0: X22 = I
    A[4, :64, :64] = 0.0
    A[4, 64:, 64:] = 0.0             # only A21: X21 = -A21
    A[5] = np.tril(np.ones((C, C), np.float32), -1)  # all ones: X = I - Z
    qA, eA = oi.quantize_blocked(A, spec)
    check_inverse(width, qA, eA, 3, 8, "zero blocks")
    _, cdt, _, inv = WIDTHS[width]
    qT, eT = (host(t) for t in inv(to_dev(qA, cdt), to_dev(eA, torch.int32), 3, 8))
    assert not np.any(qT[0]) and not np.any(eT[0])
    assert np.array_equal(qT[4, 64:, :64].astype(np.int64), -qA[4, 64:, :64])
    if width == "i16":
        # 16 bits keep the band of each block's quantised power sum, so the
        # all-ones tile comes out exact across the block boundary (8 bits
        # lose it to the unmasked powers' outliers; the oracle pins both)
        assert np.array_equal(oi.dequant_unit_blocked(qT[5:6], eT[5:6])[0],
                              np.eye(C) - np.eye(C, k=-1))


@pytest.mark.parametrize("width", ["i8", "i16"])
def test_blocked_many_tiles_odd_count_and_without_dequant(width):
    spec, cdt, quant, inv = WIDTHS[width]
    A = f32_tiles(H=3, L=1280, seed=7)[:29]
    print(f"{width} C=128 pipeline n={A.shape[0]}", flush=True)
    qd, ed = quant(to_dev(A, torch.float32))
    qT, eT = inv(qd, ed, 3, 8)
    qT2, eT2, _ = inv(qd, ed, 3, 8, want_deq=True)
    rq, re = oi.quantize_blocked(A, spec)
    rT, rE = oi.neumann_inverse_int_blocked(rq, re, 3, 8, spec)
    assert np.array_equal(host(qT).astype(np.int64), rT)
    assert np.array_equal(host(eT).astype(np.int64), rE)
    assert torch.equal(qT, qT2) and torch.equal(eT, eT2)


@pytest.fixture(scope="module")
def full_size_tiles():
    """The low-bit workload at C = 128 and full size (B=4, H=32, L=16384:
    16384 tiles), float32 A built by the oracle head by head."""
    w = wl.workload("int8").with_(C=C)
    nc = w.L // C
    A = np.empty((w.B * w.H * nc, C, C), np.float32)
    for b in range(w.B):
        for h in range(w.H):
            K, beta, g, _ = wl.gen_head(w, b, h, C=C, want_v=False)
            t0 = (b * w.H + h) * nc
            A[t0:t0 + nc] = gdn.tiles_flat(
                gdn.build_A(K[None, :, None], beta[None, :, None], g[None, :, None], C))
    print(f"C=128 full size: {A.shape[0]} tiles generated", flush=True)
    return A


@pytest.mark.parametrize("width", ["i8", "i16"])
def test_blocked_full_size_sampled(width, full_size_tiles):
    """One launch of each kernel over all 16384 tiles; a sample of tiles (the
    first, the last and 126 drawn) compared with the oracle."""
    spec, cdt, quant, inv = WIDTHS[width]
    A = full_size_tiles
    qd, ed = quant(to_dev(A, torch.float32))
    qT, eT, Td = inv(qd, ed, 3, 8, want_deq=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(128)
    idx = np.sort(np.concatenate([[0, A.shape[0] - 1],
                                  rng.choice(np.arange(1, A.shape[0] - 1), 126, replace=False)]))
    idx_t = torch.from_numpy(idx).to("cuda")
    rq, re = oi.quantize_blocked(A[idx], spec)
    assert np.array_equal(host(qd[idx_t]).astype(np.int64), rq)
    assert np.array_equal(host(ed[idx_t]).astype(np.int64), re)
    rT, rE = oi.neumann_inverse_int_blocked(rq, re, 3, 8, spec)
    assert np.array_equal(host(qT[idx_t]).astype(np.int64), rT)
    assert np.array_equal(host(eT[idx_t]).astype(np.int64), rE)
    assert np.array_equal(host(Td[idx_t]), oi.dequant_unit_blocked(rT, rE).astype(np.float32))


# ---------------------------------------------------------------------------
# one launch from K: build A, quantise block by block, integer inverse

FUSED = {"i8": G.gdn_chunk_inverse_neumann_i8_fused, "i16": G.gdn_chunk_inverse_neumann_i16_fused}


def head_set(kdt, L=512, H=2, dk=128, stress=False, seed=0):
    w = wl.workload("int8").with_(dtype=kdt, L=L, H=H, B=1, dk=dk, seed=1003 + seed)
    if stress:
        heads = [wl.gen_stress_head(L, dk, C, seed=90 + h) for h in range(H)]
        heads = [(wl.round_to_bf16(k) if kdt == "bf16" else k, b, g, v) for k, b, g, v in heads]
    else:
        heads = [wl.gen_head(w, 0, h, C=C, want_v=False) for h in range(H)]
    return tuple(wl.as_blhd(*[x[i] for x in heads]) for i in range(3))


def to_cuda(x, dt=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda").to(dt)


@pytest.mark.parametrize("width", ["i8", "i16"])
@pytest.mark.parametrize("kdt,dk,stress", [("bf16", 128, False), ("f32", 128, True),
                                           ("bf16", 64, True), ("f32", 64, False)])
def test_fused_matches_stages(width, kdt, dk, stress):
    """The one launch equals gdn_build_A (fp32) -> block-wise quantiser ->
    block-wise integer inverse on the GPU, bit for bit (the same fp32 A
    values, hence the same codes)."""
    _, _, quant, inv = WIDTHS[width]
    K, beta, g = head_set(kdt, dk=dk, stress=stress, H=3)
    dK = to_cuda(K, torch.bfloat16 if kdt == "bf16" else torch.float32)
    db, dg = to_cuda(beta), to_cuda(g)
    for N, S in [(3, 8), (2, 3)]:
        print(f"{width} C=128 fused vs stages K={kdt} dk={dk} N={N} S={S}", flush=True)
        A = G.gdn_build_A(dK, db, dg, C, a_dtype=torch.float32)
        Aq, eA = quant(A)
        q1, e1, d1 = inv(Aq, eA, N, S, want_deq=True)
        q2, e2, d2 = FUSED[width](dK, db, dg, C, N, S, want_deq=True)
        assert e2.shape == (q2.shape[0] * q2.shape[1] * q2.shape[2], 3)
        assert np.array_equal(host(q1).reshape(-1), host(q2).reshape(-1))
        assert np.array_equal(host(e1), host(e2))
        assert np.array_equal(host(d1).reshape(-1), host(d2).reshape(-1))


@pytest.mark.parametrize("width", ["i8", "i16"])
def test_fused_vs_oracle_and_float(width):
    """Against the integer oracle run from its own fp32 A (float64 build,
    rounded): the GPU forms A in fp32 arithmetic, so an entry a few ulp away
    can move a code at a rounding boundary; the dequantised results stay
    within a few dozen quanta of each block's exponent, and both are close
    to the float64 block-wise T_hat(3, 8)."""
    spec = WIDTHS[width][0]
    K, beta, g = head_set("bf16", L=2048, H=4)
    print(f"{width} C=128 fused vs oracle", flush=True)
    Tq, eT, Td = FUSED[width](to_cuda(K, torch.bfloat16), to_cuda(beta), to_cuda(g), C, 3, 8,
                              want_deq=True)
    Af = gdn.tiles_flat(gdn.build_A(K, beta, g, C))
    qA, eA = oi.quantize_blocked(Af.astype(np.float32), spec)
    rq, re = oi.neumann_inverse_int_blocked(qA, eA, 3, 8, spec)
    gq = host(Tq).reshape(rq.shape).astype(np.int64)
    ge = host(eT).astype(np.int64)
    same = np.all(gq == rq, axis=(-1, -2)) & np.all(ge == re, axis=-1)
    got = host(Td).reshape(rq.shape).astype(np.float64)
    ref = oi.dequant_unit_blocked(rq, re)
    quantum = np.ones(rq.shape)
    for k, (rs, cs) in enumerate([(slice(0, 64), slice(0, 64)), (slice(64, 128), slice(0, 64)),
                                  (slice(64, 128), slice(64, 128))]):
        quantum[:, rs, cs] = np.ldexp(1.0, re[:, k])[:, None, None]
    quanta = np.abs(got - ref) / quantum
    print(f"  {same.mean():.4f} of {same.size} tiles bit-exact, max {quanta.max():.1f} quanta",
          flush=True)
    assert quanta.max() <= 64.0
    T = gdn.neumann_inverse_blocked(Af, 3, 8)
    scale = np.max(np.abs(T - np.eye(C)), axis=(-1, -2))
    err = np.max(np.abs(got - T), axis=(-1, -2))
    bits = 8 if width == "i8" else 16
    assert np.all(err <= 16 * 2.0 ** -bits * scale)


@pytest.mark.parametrize("width", ["i8", "i16"])
def test_fused_full_size_sampled(width):
    """The one launch at the size bench.py times (low-bit workload at C = 128:
    B=4, H=32, L=16384, bf16 K; 16384 tiles): equal to the three launches on
    the GPU bit for bit everywhere, and on a sample of tiles within a few
    quanta of the integer oracle run from its own fp32 A (an A entry a
    rounding apart can move a code)."""
    spec, _, quant, inv = WIDTHS[width]
    w = wl.workload("int8").with_(C=C)
    K, beta, g, _ = wl.gen_inputs(w, C=C, want_v=False)
    print(f"{width} C=128 fused full size: {w.B * w.H * (w.L // C)} tiles", flush=True)
    dK, db, dg = to_cuda(K, torch.bfloat16), to_cuda(beta), to_cuda(g)
    q2, e2, d2 = FUSED[width](dK, db, dg, C, 3, 8, want_deq=True)
    A = G.gdn_build_A(dK, db, dg, C, a_dtype=torch.float32)
    Aq, eA = quant(A)
    del A
    q1, e1 = inv(Aq, eA, 3, 8)
    assert torch.equal(q1, q2) and torch.equal(e1, e2)
    del q1, e1, Aq, eA
    nc = w.L // C
    rng = np.random.default_rng(1280)
    picks = [(0, 0, 0), (w.B - 1, w.H - 1, nc - 1)] + [
        (int(rng.integers(w.B)), int(rng.integers(w.H)), int(rng.integers(nc))) for _ in range(30)]
    for b, h, ck in picks:
        sl = slice(ck * C, (ck + 1) * C)
        Af = gdn.tiles_flat(gdn.build_A(K[b:b + 1, sl, h:h + 1], beta[b:b + 1, sl, h:h + 1],
                                        g[b:b + 1, sl, h:h + 1], C))
        qA, eAr = oi.quantize_blocked(Af.astype(np.float32), spec)
        rq, re = oi.neumann_inverse_int_blocked(qA, eAr, 3, 8, spec)
        t = (b * w.H + h) * nc + ck
        got = host(d2.reshape(-1, C, C)[t]).astype(np.float64)
        ref = oi.dequant_unit_blocked(rq, re)[0]
        quantum = np.ones((C, C))
        for k, (rs, cs) in enumerate([(slice(0, 64), slice(0, 64)), (slice(64, 128), slice(0, 64)),
                                      (slice(64, 128), slice(64, 128))]):
            quantum[rs, cs] = np.ldexp(1.0, re[0, k])
        assert np.max(np.abs(got - ref) / quantum) <= 64.0, (b, h, ck)
