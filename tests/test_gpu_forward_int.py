"""Parity of the layer forward with the integer inverse inside it
(gdn_chunk_forward / gdn_chunk_forward_varlen with inverse "int16" or
"int8", through the C ABI) with the float64 forward oracle whose inverse is
the integer T_hat(N, S) of the integer oracle, dequantised
(oracle/int8.py::dequantized_inverse): the quantised GDN layer of
Section 3.5 with the rest of the layer in the compute dtype.

Tolerances, relative to max(1, max |ref|): the bars of the float forward,
1e-5 in fp32 and 2e-2 in bf16.  Both sides take every quantisation
decision on fp32 values of A (GPU: MFMA sums; oracle: float64 rounded to
fp32), which agree to an ulp; a code flips only where an entry sits within
an ulp of a rounding boundary, and one flip would move one entry of T by a
quantum (2^-14 / 2^-6 of max |T - I|).  In these seeded cases no flip
reaches the outputs: the fp32 errors are at fp32 rounding level (~1e-8,
printed).
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn_forward as fwd
from oracle import int8 as oi
from oracle import varlen

import paper_2606_06034_amd as G

from test_gpu_forward import dev, dev32, host, layer_inputs

pytestmark = pytest.mark.gpu

SPEC = {"int16": oi.SPEC16, "int8": oi.SPEC8}
TOL = {("f32", "int16"): 1e-5, ("f32", "int8"): 1e-5,
       ("bf16", "int16"): 2e-2, ("bf16", "int8"): 2e-2}


def check(got, ref, dt, mode, what):
    tol = TOL[(dt, mode)] * max(1.0, float(np.max(np.abs(ref))))
    err = float(np.max(np.abs(got - ref)))
    print(f"  {what}: max err {err:.3e} (bound {tol:.3e})", flush=True)
    assert err <= tol, f"{what}: max err {err:.3e} > {tol:.3e}"


def inverse_of(mode, C):
    N, S = G.gdn_default_order(C)
    return lambda A: oi.dequantized_inverse(A, N, S, SPEC[mode], C=C)


@pytest.mark.parametrize("mode", ["int16", "int8"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64])
def test_forward_int_matches_oracle(C, dt, mode):
    print(f"forward {mode} C={C} {dt}", flush=True)
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=2, L=3 * C + 64, H=3, seed=C + 7)
    O, Sf = G.gdn_chunk_forward(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g), C,
                                S0=dev32(S0), inverse=mode)
    scale = K.shape[-1] ** -0.5
    Or, Sr = fwd.gdn_chunked(Q, K, V, beta.astype(np.float64), g.astype(np.float64), C,
                             S0.astype(np.float64), scale=scale, inverse=inverse_of(mode, C))
    check(host(O), Or, dt, mode, "O")
    check(host(Sf), Sr, dt, mode, "S_final")


@pytest.mark.parametrize("mode", ["int16", "int8"])
def test_forward_int_stress_and_split(mode):
    """Stress heads (larger |A|, longer residual chains), and the prepare /
    state phases run apart reproduce the one call bit for bit."""
    C, dt = 64, "bf16"
    print(f"forward {mode} stress", flush=True)
    Q, K, V, beta, g, S0 = layer_inputs(C, dt, B=1, L=4 * C, H=2, stress=True, seed=3)
    args = (dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g))
    O, Sf = G.gdn_chunk_forward(*args, C, S0=dev32(S0), inverse=mode)
    scale = K.shape[-1] ** -0.5
    Or, Sr = fwd.gdn_chunked(Q, K, V, beta.astype(np.float64), g.astype(np.float64), C,
                             S0.astype(np.float64), scale=scale, inverse=inverse_of(mode, C))
    check(host(O), Or, dt, mode, "O")
    check(host(Sf), Sr, dt, mode, "S_final")
    B, L, H, dk = K.shape
    ws = torch.empty(G.gdn_chunk_forward_workspace(B, L, H, dk, V.shape[-1], C, torch.bfloat16),
                     dtype=torch.uint8, device="cuda")
    G.gdn_chunk_forward_prepare(args[0], args[1], args[2], args[3], args[4], C, ws, inverse=mode)
    O2, S2 = G.gdn_chunk_forward_state(args[0], args[4], C, ws, V.shape[-1], S0=dev32(S0))
    assert torch.equal(O, O2) and torch.equal(Sf, S2)


@pytest.mark.parametrize("mode", ["int16", "int8"])
def test_forward_varlen_int_matches_oracle(mode):
    """Packed sequences with ragged last chunks: each partial chunk's m x m
    system is the C x C tile padded with tokens that write nothing, on which
    the integer recipe runs."""
    C, dt = 32, "bf16"
    lengths = [5, 0, 70, 64, 1, 33]
    print(f"forward varlen {mode} {lengths}", flush=True)
    rng = np.random.default_rng(5)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    T, H, dk, dv = int(cu[-1]), 2, 128, 128
    z = rng.standard_normal((1, T, H, dk))
    K = wl.round_to_bf16((z / np.linalg.norm(z, axis=-1, keepdims=True)).astype(np.float32))
    Q = wl.round_to_bf16((0.3 * rng.standard_normal((1, T, H, dk))).astype(np.float32))
    V = wl.round_to_bf16(rng.standard_normal((1, T, H, dv)).astype(np.float32))
    beta = rng.random((1, T, H)).astype(np.float32)
    g = varlen.varlen_cumsum(-0.1 * rng.random((T, H)), cu, C)[None].astype(np.float32)
    S0 = rng.standard_normal((len(lengths), H, dk, dv)).astype(np.float32)
    tables = G.gdn_varlen_tables(cu, C)
    O, Sf = G.gdn_chunk_forward_varlen(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g),
                                       tables, C, S0=dev32(S0), inverse=mode)
    Or, Sr = varlen.forward_varlen_chunked(Q, K, V, beta, g, cu, C, S0, dk ** -0.5,
                                           inverse=inverse_of(mode, C))
    check(host(O), Or, dt, mode, "O")
    check(host(Sf), Sr, dt, mode, "S_final")
