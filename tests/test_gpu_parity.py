"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Inputs are seeded (workloads); the oracle computes from exactly the values
the GPU sees (rounded to the storage dtype, upcast to float64).  Tolerances
are the stated ones: max abs error <= 1e-5 in fp32 mode and <= 2e-2 in bf16
mode; W and U scale them by max(1, max |ref|).
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def dev(x, dt="f32"):
    x = np.asarray(x, dtype=np.float32)
    if dt == "bf16":
        x = wl.round_to_bf16(x)
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(TDT[dt])


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def stored(x, dt):
    """The values a tensor of dtype dt holds, as float64."""
    x = np.asarray(x, dtype=np.float32)
    return (wl.round_to_bf16(x) if dt == "bf16" else x).astype(np.float64)


def gdn_tiles(C, n_heads=2, L=None, stress=False, seed=0):
    """A tiles [n, C, C] (float64) from the tiny workload or the stress set."""
    w = wl.workload("tiny")
    L = L or 4 * max(C, 64)
    if stress:
        heads = [wl.gen_stress_head(L, w.dk, C, seed=seed + h) for h in range(n_heads)]
    else:
        heads = [wl.gen_head(w.with_(L=L), 0, h, C=C, want_v=False) for h in range(n_heads)]
    K = wl.as_blhd(*[x[0] for x in heads])
    beta = wl.as_blhd(*[x[1] for x in heads])
    g = wl.as_blhd(*[x[2] for x in heads])
    return gdn.tiles_flat(gdn.build_A(K, beta, g, C))


def maxerr(a, b):
    return float(np.max(np.abs(a - b))) if a.size else 0.0


# ---------------------------------------------------------------------------
# approximate inverse


ORDERS = {16: [(3, 2), (3, 1), (3, 3), (0, 5), (2, 0)],
          32: [(3, 4), (3, 1), (3, 7), (1, 3)],
          64: [(3, 8), (3, 1), (3, 15), (4, 3), (0, 2)],
          128: [(3, 8), (3, 1), (3, 15)]}


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
@pytest.mark.parametrize("stress", [False, True])
def test_neumann_matches_oracle(C, dt, stress):
    A = stored(gdn_tiles(C, stress=stress), dt)
    dA = dev(A, dt)
    for N, S in ORDERS[C]:
        T = host(G.gdn_chunk_inverse_neumann(dA, N, S))
        if C == 128:
            ref = gdn.neumann_inverse_blocked(A, N, S)
        else:
            ref = gdn.neumann_inverse(A, N, S)
        err = maxerr(T, ref)
        # stress tiles leave the workload range (|T| up to ~7): bf16 rounding
        # then scales with the magnitude of the result
        tol = TOL[dt] * (max(1.0, np.max(np.abs(ref))) if stress else 1.0)
        print(f"C={C} {dt} stress={stress} N={N} S={S} n={A.shape[0]} max|err|={err:.3e} "
              f"tol={tol:.1e}", flush=True)
        assert err <= tol, (N, S, err)
        # structure is exact
        assert np.all(np.triu(T, 1) == 0)
        assert np.all(np.diagonal(T, axis1=-2, axis2=-1) == 1)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_neumann_orders_past_one_block(dt):
    # N >= 16: T0's band reaches past the first sub-diagonal 16-block (the
    # general band path of the engine); workload tiles, both dtypes
    for C, (N, S) in [(32, (17, 2)), (64, (20, 3)), (64, (40, 1)), (128, (20, 2))]:
        A = stored(gdn_tiles(C), dt)
        T = host(G.gdn_chunk_inverse_neumann(dev(A, dt), N, S))
        ref = gdn.neumann_inverse_blocked(A, N, S) if C == 128 else gdn.neumann_inverse(A, N, S)
        err = maxerr(T, ref)
        print(f"C={C} {dt} N={N} S={S} max|err|={err:.3e}", flush=True)
        assert err <= TOL[dt], (C, N, S, err)


def test_neumann_exact_orders_reach_inverse():
    """(S + 1)(N + 1) >= C makes T_hat the exact inverse: compare with X."""
    for C, (N, S) in [(16, (3, 3)), (32, (3, 7)), (64, (3, 15))]:
        A = stored(gdn_tiles(C, stress=True), "f32")
        T = host(G.gdn_chunk_inverse_neumann(dev(A), N, S))
        X = gdn.forward_substitution_inverse(A)
        assert maxerr(T, X) <= 1e-5


def test_neumann_many_tiles_odd_count():
    """67 tiles (not a multiple of anything) of the bf16 Qwen3.5 workload."""
    w = wl.workload("qwen35_prefill")
    K, beta, g, _ = wl.gen_inputs(w.with_(L=67 * 64, H=1), want_v=False)
    A = stored(gdn.tiles_flat(gdn.build_A(K, beta, g, 64)), "bf16")
    assert A.shape[0] == 67
    T = host(G.gdn_chunk_inverse_neumann(dev(A, "bf16"), 3, 8))
    assert maxerr(T, gdn.neumann_inverse(A, 3, 8)) <= TOL["bf16"]


def test_neumann_edge_cases():
    for C in (16, 32, 64, 128):
        # A = 0 -> identity, exactly
        Z = torch.zeros((3, C, C), device="cuda")
        assert np.array_equal(host(G.gdn_chunk_inverse_neumann(Z, 3, 8 if C > 16 else 2)),
                              np.broadcast_to(np.eye(C), (3, C, C)))
        # all-ones strictly lower (GDN sign): exact bidiagonal inverse
        A1 = np.tril(np.ones((2, C, C)), -1)
        T = host(G.gdn_chunk_inverse_neumann(dev(A1), 3, 4))
        assert np.array_equal(T, np.broadcast_to(np.eye(C) - np.eye(C, k=-1), (2, C, C)))
        # entries on and above the diagonal are ignored
        A = stored(gdn_tiles(C, n_heads=1), "f32")
        junk = A + np.triu(np.random.default_rng(C).uniform(-5, 5, A.shape))
        for dt in ("f32", "bf16"):
            a = host(G.gdn_chunk_inverse_neumann(dev(stored(A, dt), dt), 3, 4))
            b = host(G.gdn_chunk_inverse_neumann(dev(stored(junk, dt), dt), 3, 4))
            assert np.array_equal(a, b)
    # extreme orders
    A = stored(gdn_tiles(64), "f32")
    for N, S in [(63, 0), (0, 63), (63, 63), (1, 1), (0, 0)]:
        T = host(G.gdn_chunk_inverse_neumann(dev(A), N, S))
        assert maxerr(T, gdn.neumann_inverse(A, N, S)) <= 1e-5, (N, S)
    # on the stress set the full-order sums cancel powers up to ~1e3 x |T|
    # (Section 3.2): fp32 error is relative to the largest power
    A = stored(gdn_tiles(64, stress=True), "f32")
    P = np.broadcast_to(np.eye(64), A.shape).copy()
    big = 1.0
    for _ in range(63):
        P = P @ -A
        big = max(big, np.max(np.abs(P)))
    for N, S in [(63, 0), (0, 63)]:
        T = host(G.gdn_chunk_inverse_neumann(dev(A), N, S))
        assert maxerr(T, gdn.neumann_inverse(A, N, S)) <= 64 * 2.0 ** -24 * 64 * big, (N, S)


def test_neumann_deterministic():
    A = dev(stored(gdn_tiles(64, stress=True), "bf16"), "bf16")
    a = G.gdn_chunk_inverse_neumann(A, 3, 8)
    b = G.gdn_chunk_inverse_neumann(A, 3, 8)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# ---------------------------------------------------------------------------
# exact inverse by forward substitution


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_fwdsub_matches_exact(C, dt):
    for stress in (False, True):
        A = stored(gdn_tiles(C, stress=stress), dt)
        T = host(G.gdn_chunk_inverse_fwdsub(dev(A, dt)))
        X = gdn.forward_substitution_inverse(A)
        tol = TOL[dt] if dt == "bf16" else 1e-5 * max(1.0, np.max(np.abs(X)))
        err = maxerr(T, X)
        print(f"fwdsub C={C} {dt} stress={stress} max|err|={err:.3e}", flush=True)
        assert err <= tol
        assert np.all(np.triu(T, 1) == 0) and np.all(np.diagonal(T, axis1=-2, axis2=-1) == 1)


# ---------------------------------------------------------------------------
# build A, WY, fused


def head_inputs(w, C, n_heads, dt):
    heads = [wl.gen_head(w, 0, h, C=C) for h in range(n_heads)]
    K = wl.as_blhd(*[x[0] for x in heads])
    beta = wl.as_blhd(*[x[1] for x in heads])
    g = wl.as_blhd(*[x[2] for x in heads])
    V = wl.as_blhd(*[x[3] for x in heads])
    return K, beta, g, V


@pytest.mark.parametrize("kdt,adt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_build_A(C, kdt, adt):
    w = wl.workload("tiny").with_(dtype=kdt, L=4 * max(C, 64))
    K, beta, g, _ = head_inputs(w, C, 3, kdt)
    ref = gdn.build_A(K, beta, g, C)
    A = host(G.gdn_build_A(dev(K, kdt), dev(beta), dev(g), C, a_dtype=TDT[adt]))
    assert A.shape == ref.shape
    tol = 1e-5 if adt == "f32" else TOL["bf16"]
    err = maxerr(A, ref)
    print(f"build_A C={C} K={kdt} A={adt} max|err|={err:.3e}", flush=True)
    assert err <= tol
    assert np.all(np.triu(A) == 0)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_wy_apply(C, dt):
    w = wl.workload("tiny").with_(dtype=dt, L=4 * max(C, 64))
    K, beta, g, V = head_inputs(w, C, 2, dt)
    A = gdn.build_A(K, beta, g, C)
    T = stored(gdn.forward_substitution_inverse(A), dt)
    Wr, Ur = gdn.wy_apply(T, K, V, beta, C)
    W, U = G.gdn_wy_apply(dev(T, dt), dev(K, dt), dev(V, dt), dev(beta), C)
    W, U = host(W), host(U)
    for got, ref in ((W, Wr), (U, Ur)):
        tol = TOL[dt] * max(1.0, np.max(np.abs(ref)))
        err = maxerr(got, ref)
        print(f"wy C={C} {dt} max|err|={err:.3e} tol={tol:.1e}", flush=True)
        assert err <= tol


# ---------------------------------------------------------------------------
# exact block-wise inverse


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
@pytest.mark.parametrize("stress", [False, True])
def test_blockwise_matches_exact_inverse(C, dt, stress):
    A = stored(gdn_tiles(C, stress=stress), dt)
    X = gdn.forward_substitution_inverse(A)
    T = host(G.gdn_chunk_inverse_blockwise(dev(A, dt)))
    tol = TOL[dt] * (max(1.0, np.max(np.abs(X))) if stress else 1.0)
    err = maxerr(T, X)
    print(f"blockwise C={C} {dt} stress={stress} n={A.shape[0]} max|err|={err:.3e} tol={tol:.1e}",
          flush=True)
    assert err <= tol
    assert np.all(np.triu(T, 1) == 0)
    assert np.all(np.diagonal(T, axis1=-2, axis2=-1) == 1)


def test_blockwise_edge_cases():
    for C in (16, 32, 64, 128):
        Z = torch.zeros((3, C, C), device="cuda")
        assert np.array_equal(host(G.gdn_chunk_inverse_blockwise(Z)),
                              np.broadcast_to(np.eye(C), (3, C, C)))
        # all-ones strictly lower (GDN sign): the bidiagonal inverse; every
        # intermediate is an integer below 2^24, so fp32 reaches it exactly
        A1 = np.tril(np.ones((2, C, C)), -1)
        X1 = np.eye(C) - np.eye(C, k=-1)
        assert np.array_equal(host(G.gdn_chunk_inverse_blockwise(dev(A1))),
                              np.broadcast_to(X1, (2, C, C)))
        # entries on and above the diagonal are ignored
        A = gdn_tiles(C, n_heads=1)[:2]
        junk = A + np.triu(np.ones_like(A))
        assert np.array_equal(host(G.gdn_chunk_inverse_blockwise(dev(junk))),
                              host(G.gdn_chunk_inverse_blockwise(dev(A))))


def test_blockwise_many_tiles_full_size_sampled():
    """Sweep workload at C = 64 (32768 tiles) in one launch, sampled tiles
    against the oracle's exact inverse."""
    w = wl.workload("sweep")
    C = 64
    K, beta, g, _ = wl.gen_inputs(w.with_(H=4), C=C, want_v=False)
    A = stored(gdn.tiles_flat(gdn.build_A(K, beta, g, C)), "bf16")
    T = G.gdn_chunk_inverse_blockwise(dev(A, "bf16"))
    idx = np.random.default_rng(3).choice(A.shape[0], 64, replace=False)
    X = gdn.forward_substitution_inverse(A[idx])
    assert maxerr(host(T)[idx], X) <= TOL["bf16"]


def ref_inverse(A, N, S):
    """The oracle's T_hat(N, S); C = 128 by the two-block form."""
    if A.shape[-1] == 128:
        return gdn.neumann_inverse_blocked(A, N, S)
    return gdn.neumann_inverse(A, N, S)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_fused(C, dt):
    w = wl.workload("tiny").with_(dtype=dt, L=4 * max(C, 64))
    K, beta, g, V = head_inputs(w, C, 2, dt)
    N, S = gdn.default_order(C)
    A = gdn.build_A(K, beta, g, C)
    Tr = ref_inverse(A, N, S)
    Wr, Ur = gdn.wy_apply(Tr, K, V, beta, C)
    W, U, T = G.gdn_chunk_wy_fused(dev(K, dt), dev(V, dt), dev(beta), dev(g), C, N, S, want_T=True)
    T, W, U = host(T), host(W), host(U)
    assert maxerr(T, Tr) <= TOL[dt]
    for got, ref in ((W, Wr), (U, Ur)):
        tol = TOL[dt] * max(1.0, np.max(np.abs(ref)))
        err = maxerr(got, ref)
        print(f"fused C={C} {dt} max|err|={err:.3e} tol={tol:.1e}", flush=True)
        assert err <= tol
    # without the optional Tinv output
    W2, U2 = G.gdn_chunk_wy_fused(dev(K, dt), dev(V, dt), dev(beta), dev(g), C, N, S)
    assert np.array_equal(host(W2), W) and np.array_equal(host(U2), U)


FUSED_ORDERS = {16: [(0, 5), (2, 0)], 32: [(1, 3), (3, 7)], 64: [(4, 3), (3, 15), (0, 2)],
                128: [(3, 1), (4, 3), (3, 15)]}


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_fused_stress_and_orders(C, dt):
    """Stress heads (|A| up to ~0.5) at non-default orders, and dk = dv = 64."""
    for dk in (128, 64):
        heads = [wl.gen_stress_head(2 * max(C, 64), dk, C, seed=40 + h, dv=dk) for h in range(2)]
        K, beta, g, V = (stored(wl.as_blhd(*[x[i] for x in heads]), dt if i in (0, 3) else "f32")
                         for i in range(4))
        A = gdn.build_A(K, beta, g, C)
        for N, S in FUSED_ORDERS[C]:
            Tr = ref_inverse(A, N, S)
            Wr, Ur = gdn.wy_apply(Tr, K, V, beta, C)
            W, U, T = G.gdn_chunk_wy_fused(dev(K, dt), dev(V, dt), dev(beta), dev(g), C, N, S,
                                           want_T=True)
            scale = max(1.0, np.max(np.abs(Tr)))
            eT = maxerr(host(T), Tr)
            eW, eU = maxerr(host(W), Wr), maxerr(host(U), Ur)
            print(f"fused stress C={C} {dt} dk={dk} N={N} S={S} T {eT:.2e} W {eW:.2e} "
                  f"U {eU:.2e}", flush=True)
            assert eT <= TOL[dt] * scale
            assert eW <= TOL[dt] * scale * max(1.0, np.max(np.abs(Wr)))
            assert eU <= TOL[dt] * scale * max(1.0, np.max(np.abs(Ur)))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_fused_blockwise_exact(C, dt):
    """Fused path with the exact block-wise inverse: W, U, Tinv against the
    oracle's exact inverse X (workload and stress heads, dk = dv = 128 / 64)."""
    for stress, dk in ((False, 128), (True, 128), (True, 64)):
        if stress:
            heads = [wl.gen_stress_head(2 * max(C, 64), dk, C, seed=70 + h, dv=dk)
                     for h in range(2)]
            K, beta, g, V = (stored(wl.as_blhd(*[x[i] for x in heads]),
                                    dt if i in (0, 3) else "f32") for i in range(4))
        else:
            w = wl.workload("tiny").with_(dtype=dt, L=4 * max(C, 64))
            K, beta, g, V = head_inputs(w, C, 2, dt)
        X = gdn.forward_substitution_inverse(gdn.build_A(K, beta, g, C))
        Wr, Ur = gdn.wy_apply(X, K, V, beta, C)
        W, U, T = G.gdn_chunk_wy_fused_blockwise(dev(K, dt), dev(V, dt), dev(beta), dev(g), C,
                                                 want_T=True)
        scale = max(1.0, np.max(np.abs(X)))
        eT, eW, eU = maxerr(host(T), X), maxerr(host(W), Wr), maxerr(host(U), Ur)
        print(f"fused exact C={C} {dt} stress={stress} dk={dk} T {eT:.2e} W {eW:.2e} U {eU:.2e}",
              flush=True)
        assert eT <= TOL[dt] * scale
        assert eW <= TOL[dt] * scale * max(1.0, np.max(np.abs(Wr)))
        assert eU <= TOL[dt] * scale * max(1.0, np.max(np.abs(Ur)))
        W2, U2 = G.gdn_chunk_wy_fused_blockwise(dev(K, dt), dev(V, dt), dev(beta), dev(g), C)
        assert np.array_equal(host(W2), host(W)) and np.array_equal(host(U2), host(U))


@pytest.mark.parametrize("exact", [False, True])
@pytest.mark.parametrize("H", [16, 32])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_fused_grouped_heads(C, H, exact):
    """Head counts at which one workgroup takes the chunks of neighbouring
    heads of a chunk row (two per workgroup when 16 divides H, four at
    C <= 64 when 32 does): every tile's W, U and Tinv against the oracle, and
    the outputs without Tinv equal to those with it."""
    dt = "bf16"
    w = wl.workload("tiny").with_(dtype=dt, L=2 * max(C, 64), H=H)
    K, beta, g, V = head_inputs(w, C, H, dt)
    A = gdn.build_A(K, beta, g, C)
    if exact:
        Tr = gdn.forward_substitution_inverse(A)
        run = lambda want: G.gdn_chunk_wy_fused_blockwise(dev(K, dt), dev(V, dt), dev(beta),
                                                           dev(g), C, want_T=want)
    else:
        N, S = gdn.default_order(C)
        Tr = ref_inverse(A, N, S)
        run = lambda want: G.gdn_chunk_wy_fused(dev(K, dt), dev(V, dt), dev(beta), dev(g), C, N,
                                                S, want_T=want)
    Wr, Ur = gdn.wy_apply(Tr, K, V, beta, C)
    W, U, T = (host(x) for x in run(True))
    eT, eW, eU = maxerr(T, Tr), maxerr(W, Wr), maxerr(U, Ur)
    print(f"fused grouped C={C} H={H} exact={exact} tiles={A.shape[0]} T {eT:.2e} W {eW:.2e} "
          f"U {eU:.2e}", flush=True)
    assert eT <= TOL[dt]
    assert eW <= TOL[dt] * max(1.0, np.max(np.abs(Wr)))
    assert eU <= TOL[dt] * max(1.0, np.max(np.abs(Ur)))
    W2, U2 = run(False)
    assert np.array_equal(host(W2), W) and np.array_equal(host(U2), U)


@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_deterministic_and_launch_shape_independent(C):
    """A tile's result depends on that tile alone: repeated launches give the
    same bits, a tile inverted within a batch starting at another offset (so
    sharing its wave or workgroup with other tiles) gives the same bits, and
    a chunk computed by the fused kernel inside a workgroup of neighbouring
    heads (H = 16) equals the same chunk computed alone (H = 2)."""
    dt = "bf16"
    N, S = gdn.default_order(C)
    w = wl.workload("tiny").with_(dtype=dt, L=2 * max(C, 64), H=16)
    K, beta, g, V = head_inputs(w, C, 16, dt)
    A = stored(gdn.tiles_flat(gdn.build_A(K, beta, g, C)), dt)
    dA = dev(A, dt)
    for inv in (lambda a: G.gdn_chunk_inverse_neumann(a, N, S),
                lambda a: G.gdn_chunk_inverse_blockwise(a)):
        T1, T2 = host(inv(dA)), host(inv(dA))
        assert np.array_equal(T1, T2)
        for lo, hi in ((5, 12), (1, 2), (3, A.shape[0])):
            assert np.array_equal(host(inv(dA[lo:hi].contiguous())), T1[lo:hi]), (lo, hi)
    for fused in (lambda k, v, b, gg: G.gdn_chunk_wy_fused(k, v, b, gg, C, N, S, want_T=True),
                  lambda k, v, b, gg: G.gdn_chunk_wy_fused_blockwise(k, v, b, gg, C, want_T=True)):
        full = [host(x) for x in fused(dev(K, dt), dev(V, dt), dev(beta), dev(g))]
        again = [host(x) for x in fused(dev(K, dt), dev(V, dt), dev(beta), dev(g))]
        assert all(np.array_equal(a, b) for a, b in zip(full, again))
        for h0 in (0, 6):
            sub = [host(x) for x in fused(dev(K[:, :, h0:h0 + 2], dt), dev(V[:, :, h0:h0 + 2], dt),
                                          dev(beta[:, :, h0:h0 + 2]), dev(g[:, :, h0:h0 + 2]))]
            nc = K.shape[1] // C
            assert np.array_equal(sub[0], full[0][:, :, h0:h0 + 2])  # W
            assert np.array_equal(sub[1], full[1][:, :, h0:h0 + 2])  # U
            # Tinv tiles [B, H, L / C, C, C] of those heads
            Tf = full[2].reshape(1, 16, nc, C, C)[:, h0:h0 + 2]
            assert np.array_equal(sub[2].reshape(Tf.shape), Tf)


def test_fused_matches_unfused_composition():
    """build_A -> neumann -> wy_apply equals the fused kernel (fp32)."""
    C = 64
    w = wl.workload("tiny")
    K, beta, g, V = head_inputs(w, C, 2, "f32")
    dK, dV, db, dg = dev(K), dev(V), dev(beta), dev(g)
    A = G.gdn_build_A(dK, db, dg, C)
    T = G.gdn_chunk_inverse_neumann(A, 3, 8)
    W1, U1 = G.gdn_wy_apply(T, dK, dV, db, C)
    W2, U2, T2 = G.gdn_chunk_wy_fused(dK, dV, db, dg, C, 3, 8, want_T=True)
    assert maxerr(host(T), host(T2)) <= 1e-5
    assert maxerr(host(W1), host(W2)) <= 1e-5
    assert maxerr(host(U1), host(U2)) <= 1e-5


# ---------------------------------------------------------------------------
# full-size workloads, sampled tiles


def _sampled_check(wname, C=None, n_sample=16, seed=0):
    """Fused launch over the whole workload; the oracle recomputes sampled
    tiles from their heads' inputs (regenerated per head)."""
    w = wl.workload(wname)
    C = C or w.C
    N, S = gdn.default_order(C)
    dt = w.dtype
    K, beta, g, V = wl.gen_inputs(w, C=C)
    dK, dV = dev(K, dt), dev(V, dt)
    del K, V
    W, U, T = G.gdn_chunk_wy_fused(dK, dV, dev(beta), dev(g), C, N, S, want_T=True)
    torch.cuda.synchronize()
    del dK, dV
    rng = np.random.default_rng(seed)
    n = w.B * w.H * (w.L // C)
    picks = sorted(set(rng.integers(0, n, n_sample).tolist()) | {0, n - 1})
    worst = 0.0
    for t in picks:
        b, h, c = wl.tile_coords(w, t, C)
        sl = slice(c * C, (c + 1) * C)
        Kh, bh, gh, Vh = wl.gen_head(w, b, h, C=C)
        Kt, bt, gt, Vt = (x[sl][None, :, None] for x in (Kh, bh, gh, Vh))
        A = gdn.build_A(Kt, bt, gt, C)
        Tr = ref_inverse(A, N, S)
        Wr, Ur = gdn.wy_apply(Tr, Kt, Vt, bt, C)
        Tg = T.view(-1, C, C)[t].float().cpu().numpy()
        Wg = W[b, sl, h].float().cpu().numpy()
        Ug = U[b, sl, h].float().cpu().numpy()
        assert maxerr(Tg, Tr[0, 0, 0]) <= TOL[dt]
        for got, ref in ((Wg, Wr[0, :, 0]), (Ug, Ur[0, :, 0])):
            e = maxerr(got, ref)
            worst = max(worst, e)
            assert e <= TOL[dt] * max(1.0, np.max(np.abs(ref))), (t, e)
    print(f"{wname} C={C}: {len(picks)} sampled tiles, worst W/U err {worst:.3e}", flush=True)


def test_qwen35_prefill_full_size_sampled():
    """The benchmarked workload (2048 tiles), in the launch the bench times."""
    _sampled_check("qwen35_prefill")


def test_sweep_c128_full_size_sampled():
    """Chunk-size sweep at C = 128 (B=4, H=32, L=16384: 16384 tiles), fused."""
    _sampled_check("sweep", C=128)


@pytest.mark.parametrize("C", [16, 32, 64])
def test_sweep_full_size_sampled(C):
    """Chunk-size sweep at C = 16, 32, 64 (B=4, H=32, L=16384: 131072,
    65536, 32768 tiles), fused, at each chunk size's default order; then the
    standalone T_hat and forward substitution on the same A tiles (the
    kernels the bench times per chunk size; at C = 16, 32 several tiles per
    wave), sampled against the oracle."""
    _sampled_check("sweep", C=C, seed=C)
    w = wl.workload("sweep").with_(C=C)
    N, S = gdn.default_order(C)
    n = w.B * w.H * (w.L // C)
    K, beta, g, _ = wl.gen_inputs(w, C=C, want_v=False)
    dA = G.gdn_build_A(dev(K, "bf16"), dev(beta), dev(g), C, a_dtype=torch.bfloat16)
    del K
    T = G.gdn_chunk_inverse_neumann(dA, N, S)
    X = G.gdn_chunk_inverse_fwdsub(dA)
    torch.cuda.synchronize()
    rng = np.random.default_rng(100 + C)
    # every tile slot of a wave (t % (64 / C)) and both ends
    picks = sorted(set(rng.integers(0, n, 16).tolist()) | {0, 1, 2, 3, n - 2, n - 1})
    Av = dA.view(-1, C, C)
    for t in picks:
        A = Av[t].float().cpu().numpy().astype(np.float64)[None]
        assert maxerr(host(T.view(-1, C, C)[t])[None], gdn.neumann_inverse(A, N, S)) <= TOL["bf16"], t
        assert maxerr(host(X.view(-1, C, C)[t])[None],
                      gdn.forward_substitution_inverse(A)) <= TOL["bf16"], t
    print(f"sweep C={C} standalone inverses: {len(picks)} sampled tiles", flush=True)


def test_long_context_full_size_sampled():
    """The long-context workload the bench times (B=1, H=32, L=131072, C=64,
    bf16: 65536 tiles) in one fused launch, sampled tiles against the oracle;
    then the inverse alone, the exact block-wise inverse and forward
    substitution on the same 65536 A tiles (the same-shape comparison the
    bench reports), sampled against the oracle's T_hat and exact inverse."""
    _sampled_check("long_context", n_sample=24, seed=4)
    w = wl.workload("long_context")
    C = w.C
    n = w.B * w.H * (w.L // C)
    rng = np.random.default_rng(5)
    picks = sorted(set(rng.integers(0, n, 16).tolist()) | {0, n - 1})
    K, beta, g, _ = wl.gen_inputs(w, C=C, want_v=False)
    dA = G.gdn_build_A(dev(K, "bf16"), dev(beta), dev(g), C, a_dtype=torch.bfloat16)
    del K
    T = G.gdn_chunk_inverse_neumann(dA, 3, 8)
    X = G.gdn_chunk_inverse_fwdsub(dA)
    Xb = G.gdn_chunk_inverse_blockwise(dA)
    torch.cuda.synchronize()
    Av = dA.view(-1, C, C)
    for t in picks:
        A = Av[t].float().cpu().numpy().astype(np.float64)[None]
        assert maxerr(host(T.view(-1, C, C)[t])[None], gdn.neumann_inverse(A, 3, 8)) <= TOL["bf16"]
        Xr = gdn.forward_substitution_inverse(A)
        assert maxerr(host(X.view(-1, C, C)[t])[None], Xr) <= TOL["bf16"], t
        assert maxerr(host(Xb.view(-1, C, C)[t])[None], Xr) <= TOL["bf16"], t
    print(f"long_context same-shape inverses: {len(picks)} sampled tiles", flush=True)


# ---------------------------------------------------------------------------
# non-finite inputs


def test_nonfinite_inputs_stay_in_their_tile():
    """A NaN or an infinity in the strictly lower part of a tile of A makes
    that tile's inverse non-finite at the same position (T_ij carries -A_ij
    through T0 on the band i - j <= N, through E beyond it) and leaves every
    other tile exactly as it is without it; NaN/Inf above the diagonal are
    never read.  The same holds for forward substitution and the exact
    block-wise inverse."""
    bad = [(0, None, None, np.nan), (1, 5, 2, np.inf), (2, 3, 1, -np.inf)]
    for C in (16, 32, 64, 128):
        A = stored(gdn_tiles(C, n_heads=1), "f32")[:6]
        B = A.copy()
        cells = []
        for k, i, j, v in bad:
            i = C - 1 if i is None else i
            j = 0 if j is None else j
            B[k, i, j] = v
            cells.append((k, i, j))
        B[3, 0, C - 1] = np.nan  # above the diagonal: ignored
        for dt in ("f32", "bf16"):
            for name, fn in (("neumann", lambda x: G.gdn_chunk_inverse_neumann(x, 3, 2 if C == 16 else 8)),
                             ("fwdsub", G.gdn_chunk_inverse_fwdsub),
                             ("blockwise", G.gdn_chunk_inverse_blockwise)):
                clean = host(fn(dev(A, dt) if dt == "f32" else dev(stored(A, dt), dt)))
                got = host(fn(dev(B, dt) if dt == "f32" else dev(B, dt)))
                for k, i, j in cells:
                    assert not np.isfinite(got[k, i, j]), (C, dt, name, k)
                assert np.array_equal(got[3:], clean[3:]), (C, dt, name)
    # the fused path: a NaN in one token's key reaches W and U of its own
    # chunk and head only
    C = 64
    w = wl.workload("tiny").with_(B=1, L=4 * C, H=2, dtype="bf16")
    K, beta, g, V = wl.gen_inputs(w, C=C)
    Kb = K.copy()
    Kb[0, C + 5, 1, 7] = np.nan  # chunk 1 of head 1
    outs = []
    for KK in (K, Kb):
        W, U = G.gdn_chunk_wy_fused(dev(KK, "bf16"), dev(V, "bf16"), dev(beta), dev(g), C, 3, 8)
        outs.append((host(W), host(U)))
    (W0, U0), (W1, U1) = outs
    sl = slice(C, 2 * C)
    assert not np.all(np.isfinite(W1[0, sl, 1])) and not np.all(np.isfinite(U1[0, sl, 1]))
    mask = np.ones(W0.shape[:3], bool)
    mask[0, sl, 1] = False
    assert np.array_equal(W1[mask], W0[mask]) and np.array_equal(U1[mask], U0[mask])


def test_binding_rejects_wrong_sizes():
    """Caller-supplied tensors of the wrong element count never reach a kernel."""
    A = torch.zeros((4, 64, 64), device="cuda")
    with pytest.raises(ValueError, match="Tinv"):
        G.gdn_chunk_inverse_neumann(A, 3, 8, Tinv=torch.empty((3, 64, 64), device="cuda"))
    with pytest.raises(ValueError, match="Tinv"):
        G.gdn_chunk_inverse_fwdsub(A, Tinv=torch.empty((5, 64, 64), device="cuda"))
    K = torch.zeros((1, 128, 2, 128), device="cuda", dtype=torch.bfloat16)
    b = torch.zeros((1, 128, 2), device="cuda")
    with pytest.raises(ValueError, match="beta"):
        G.gdn_build_A(K, b[:, :64], b, 64)
    with pytest.raises(ValueError, match="W"):
        G.gdn_chunk_wy_fused(K, K, b, b, 64, 3, 8, W=torch.empty_like(K)[:, :64])
    with pytest.raises(ValueError, match="eA"):
        G.gdn_quantize_tiles_i8(A, eA=torch.empty(3, dtype=torch.int32, device="cuda"))
    Aq, eA = G.gdn_quantize_tiles_i8(A)
    with pytest.raises(ValueError, match="Tq"):
        G.gdn_chunk_inverse_neumann_i8(Aq, eA, 3, 8, Tq=Aq[:2])
    torch.cuda.synchronize()
