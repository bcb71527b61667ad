"""Parity of the layer forward (gdn_chunk_forward, through the C ABI) with
the float64 forward oracle.

The oracle runs on exactly the values the GPU reads (inputs rounded to the
storage dtype, upcast to float64) with the same inverse (exact, or T_hat(N,
S) at the order the GPU uses).  Tolerance: max |O - O_ref| and
max |S - S_ref| within TOL * max(1, max |ref|), TOL = 1e-5 in fp32 mode
and 2e-2 in bf16 mode, the bounds the inverse itself is held to; in bf16
every MFMA operand is rounded (W, U, P, the state where it multiplies W and
Q, V_new where it multiplies P and K^T), each a relative 2^-9, and the
output sums a handful of such products.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn, gdn_forward as fwd

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def dev(x, dt="f32"):
    x = np.asarray(x, dtype=np.float32)
    if dt == "bf16":
        x = wl.round_to_bf16(x)
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(TDT[dt])


def dev32(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def stored(x, dt):
    x = np.asarray(x, dtype=np.float32)
    return (wl.round_to_bf16(x) if dt == "bf16" else x).astype(np.float64)


def layer_inputs(C, dt, B=1, L=None, H=2, dk=128, dv=128, stress=False, seed=0):
    """Q, K, V, beta, g [B, L, H, *] (float64 holding stored values) and S0."""
    L = L or 4 * C
    w = wl.workload("tiny").with_(B=B, L=L, H=H, dk=dk, dv=dv, C=C, dtype=dt, seed=2000 + seed)
    if stress:
        rng = np.random.default_rng(seed)
        Q = np.empty((B, L, H, dk)); K = np.empty_like(Q); V = np.empty((B, L, H, dv))
        beta = np.empty((B, L, H)); g = np.empty_like(beta)
        for b in range(B):
            for h in range(H):
                k, be, gg, v = wl.gen_stress_head(L, dk, C, seed=seed * 100 + b * H + h, dv=dv)
                z = rng.standard_normal((L, dk))
                Q[b, :, h] = z / np.linalg.norm(z, axis=1, keepdims=True)
                K[b, :, h], V[b, :, h], beta[b, :, h], g[b, :, h] = k, v, be, gg
        Q, K, V = (stored(x, dt) for x in (Q, K, V))
        S0 = np.random.default_rng(seed + 1).standard_normal((B, H, dk, dv)).astype(np.float32)
    else:
        Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w)
        Q, K, V = (x.astype(np.float64) for x in (Q, K, V))
    return Q, K, V, beta.astype(np.float32), g.astype(np.float32), S0


def run_gpu(Q, K, V, beta, g, S0, C, dt, **kw):
    O, Sf = G.gdn_chunk_forward(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g), C,
                                S0=None if S0 is None else dev32(S0), **kw)
    return host(O), (None if Sf is None else host(Sf))


def run_ref(Q, K, V, beta, g, S0, C, N=None, S=None, exact=False, scale=None):
    dk = K.shape[-1]
    scale = dk ** -0.5 if scale is None else scale
    if exact:
        inv = gdn.forward_substitution_inverse
    else:
        dn, ds = gdn.default_order(C)
        N = dn if N is None else N
        S = ds if S is None else S
        inv = lambda A: gdn.neumann_inverse(A, N, S)
    return fwd.gdn_chunked(Q, K, V, beta.astype(np.float64), g.astype(np.float64), C,
                           None if S0 is None else S0.astype(np.float64), scale=scale, inverse=inv)


def check(got, ref, dt, what):
    tol = TOL[dt] * max(1.0, float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    print(f"  {what}: max err {err:.3e} (bound {tol:.3e})")
    assert err <= tol, f"{what}: max err {err:.3e} > {tol:.3e}"
    return err


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64])
@pytest.mark.parametrize("exact", [False, True])
def test_forward_matches_oracle(C, dt, exact):
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=2, L=3 * C + 64, H=3, seed=C)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt, exact=exact)
    Or, Sr = run_ref(Q, K, V, beta, g, S0, C, exact=exact)
    check(O, Or, dt, "O")
    check(Sf, Sr, dt, "S_final")


@pytest.mark.parametrize("dk,dv", [(64, 64), (64, 128), (128, 64)])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_forward_feature_widths(dk, dv, dt):
    C = 64
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=4 * C, H=2, dk=dk, dv=dv, seed=dk + dv)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt)
    Or, Sr = run_ref(Q, K, V, beta, g, S0, C)
    check(O, Or, dt, "O")
    check(Sf, Sr, dt, "S_final")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64])
def test_forward_stress_orders_and_scale(C, dt):
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=4 * C, H=2, stress=True, seed=7 + C)
    for N, S in [gdn.default_order(C), (3, 1), (1, 0), (4, 3)]:
        O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt, N=N, S=S, scale=0.75)
        Or, Sr = run_ref(Q, K, V, beta, g, S0, C, N=N, S=S, scale=0.75)
        check(O, Or, dt, f"O (N, S) = ({N}, {S})")
        check(Sf, Sr, dt, f"S_final (N, S) = ({N}, {S})")


def test_forward_matches_token_recurrence():
    # against the other coding of the oracle, the plain token recurrence
    C, dt = 32, "f32"
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=4 * C, H=2, seed=3)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt, exact=True, scale=0.5)
    Or, Sr = fwd.gdn_recurrent(Q, K, V, beta.astype(np.float64), g.astype(np.float64), C,
                               S0.astype(np.float64), scale=0.5)
    check(O, Or, dt, "O")
    check(Sf, Sr, dt, "S_final")


def test_forward_without_initial_state_and_without_final_state():
    C, dt = 64, "bf16"
    Q, K, V, beta, g, _ = layer_inputs(C, dt, B=1, L=2 * C, H=2, seed=4)
    O1, S1 = run_gpu(Q, K, V, beta, g, None, C, dt)
    O2, S2 = run_gpu(Q, K, V, beta, g, np.zeros((1, 2, 128, 128), np.float32), C, dt)
    assert np.array_equal(O1, O2) and np.array_equal(S1, S2)
    O3, S3 = run_gpu(Q, K, V, beta, g, None, C, dt, want_state=False)
    assert S3 is None and np.array_equal(O1, O3)
    Or, Sr = run_ref(Q, K, V, beta, g, None, C)
    check(O1, Or, dt, "O")
    check(S1, Sr, dt, "S_final")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_forward_state_hand_off_is_exact(dt):
    # the state leaves in fp32 exactly as it is carried between chunks, and
    # chunks are formed independently, so splitting a sequence at a chunk
    # boundary and handing the state over reproduces the one-call result bit
    # for bit
    C = 32
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=6 * C, H=2, seed=5)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt)
    cut = 2 * C
    Oa, Sa = run_gpu(Q[:, :cut], K[:, :cut], V[:, :cut], beta[:, :cut], g[:, :cut], S0, C, dt)
    Ob, Sb = run_gpu(Q[:, cut:], K[:, cut:], V[:, cut:], beta[:, cut:], g[:, cut:],
                     Sa.astype(np.float32), C, dt)
    assert np.array_equal(np.concatenate([Oa, Ob], axis=1), O)
    assert np.array_equal(Sb, Sf)


def test_forward_in_place_state():
    C, dt = 64, "bf16"
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=2 * C, H=2, seed=6)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt)
    s = dev32(S0)
    O2, S2 = G.gdn_chunk_forward(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g), C,
                                 S0=s, S_final=s)
    assert S2 is s
    assert np.array_equal(host(O2), O) and np.array_equal(host(s), Sf)


def test_forward_zero_length_copies_state():
    S0 = np.random.default_rng(0).standard_normal((2, 3, 128, 64)).astype(np.float32)
    e = torch.empty((2, 0, 3, 128), dtype=torch.bfloat16, device="cuda")
    ev = torch.empty((2, 0, 3, 64), dtype=torch.bfloat16, device="cuda")
    eb = torch.empty((2, 0, 3), dtype=torch.float32, device="cuda")
    _, Sf = G.gdn_chunk_forward(e, e, ev, eb, eb, 64, S0=dev32(S0))
    assert np.array_equal(host(Sf), S0.astype(np.float64))
    _, Sz = G.gdn_chunk_forward(e, e, ev, eb, eb, 64)
    assert not np.any(host(Sz))


def test_forward_single_chunk_and_odd_heads():
    C, dt = 16, "bf16"
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=3, L=C, H=5, seed=8)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt)
    Or, Sr = run_ref(Q, K, V, beta, g, S0, C)
    check(O, Or, dt, "O")
    check(Sf, Sr, dt, "S_final")


def test_forward_deterministic():
    C, dt = 64, "bf16"
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=4 * C, H=8, seed=9)
    a = run_gpu(Q, K, V, beta, g, S0, C, dt)
    b = run_gpu(Q, K, V, beta, g, S0, C, dt)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_forward_qwen35_prefill_full_size_sampled():
    # the full 8K-token, 16-head layer on the GPU; the oracle recomputes two
    # whole heads (every chunk of the sequence) and they are compared in full
    w = wl.workload("qwen35_prefill")
    dt, C = w.dtype, w.C
    Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt)
    for h in (0, 11):
        sl = slice(h, h + 1)
        Or, Sr = run_ref(Q[:, :, sl].astype(np.float64), K[:, :, sl].astype(np.float64),
                         V[:, :, sl].astype(np.float64), beta[:, :, sl], g[:, :, sl],
                         S0[:, sl], C)
        check(O[:, :, sl], Or, dt, f"O head {h}")
        check(Sf[:, sl], Sr, dt, f"S_final head {h}")


def test_forward_binding_and_workspace_checks():
    C, dt = 64, "bf16"
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=C, H=2, seed=10)
    q, k, v, b, gg = dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g)
    need = G.gdn_chunk_forward_workspace(1, C, 2, 128, 128, C, torch.bfloat16)
    small = torch.empty(need - 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(G.GdnError) as e:
        G.gdn_chunk_forward(q, k, v, b, gg, C, workspace=small)
    assert e.value.code == -9
    with pytest.raises(ValueError):
        G.gdn_chunk_forward(q, k, v[:, :, :1], b, gg, C)
    Q, K, V, beta, g, _ = layer_inputs(C, dt, B=1, L=2 * C, H=2, seed=11)
    with pytest.raises(G.GdnError) as e:  # C = 128 is not built for the forward
        G.gdn_chunk_forward(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g), 128)
    assert e.value.code == -8


@pytest.mark.parametrize("C", [16, 64])
def test_forward_two_phases_equal_one_call(C):
    dt = "bf16"
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=2, L=3 * C, H=4, seed=12)
    O, Sf = run_gpu(Q, K, V, beta, g, S0, C, dt, scale=0.3)
    q, k, v, b, gg = dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g)
    need = G.gdn_chunk_forward_workspace(2, 3 * C, 4, 128, 128, C, torch.bfloat16)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    G.gdn_chunk_forward_prepare(q, k, v, b, gg, C, ws)
    O2, S2 = G.gdn_chunk_forward_state(q, gg, C, ws, 128, S0=dev32(S0), scale=0.3)
    assert np.array_equal(host(O2), O) and np.array_equal(host(S2), Sf)
