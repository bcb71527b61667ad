"""Parity of the layer forward over packed sequences (gdn_chunk_forward_varlen,
through the C ABI) with the packed forward oracle.

The oracle runs every sequence on its own from its own initial state, every
chunk on its m x m system, on exactly the values the GPU reads (storage
dtype, upcast to float64) and with the same inverse.  Tolerances as for the
fixed-length forward: max |O - O_ref| and max |S - S_ref| within
TOL * max(1, max |ref|), TOL = 1e-5 (fp32) and 2e-2 (bf16).
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn, varlen

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}
RAGGED = [1, 15, 16, 17, 63, 64, 65, 130, 0, 7, 200]


def dev(x, dt):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda").to(TDT[dt])


def dev32(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def inputs(lengths, C, dt, H=2, dk=128, dv=128, seed=0, gate="default"):
    w = wl.workload("tiny").with_(H=H, C=C, dtype=dt, dk=dk, dv=dv, seed=5000 + seed, gate=gate)
    K, beta, g, V, cu, Q = wl.gen_varlen(w, lengths, C=C, want_q=True)
    S0 = np.stack([np.stack([wl.gen_state(w, s, h) for h in range(H)]) for s in range(len(lengths))])
    return Q, K, V, beta, g, cu, S0


def inverse_for(C, exact, N=None, S=None):
    if exact:
        return gdn.forward_substitution_inverse
    dn, ds = gdn.default_order(C)
    n, s = (dn if N is None else N), (ds if S is None else S)
    return lambda A: gdn.neumann_inverse(A, n, s)


def check(lengths, C, dt, exact=False, N=None, S=None, H=2, dk=128, dv=128, seed=0,
          with_state=True, scale=0.3):
    Q, K, V, beta, g, cu, S0 = inputs(lengths, C, dt, H, dk, dv, seed)
    print(f"varlen forward C={C} {dt} exact={exact} N={N} S={S} lengths={lengths}", flush=True)
    tables = G.gdn_varlen_tables(cu, C)
    O, Sf = G.gdn_chunk_forward_varlen(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g),
                                       tables, C, S0=dev32(S0) if with_state else None, N=N, S=S,
                                       exact=exact, scale=scale)
    Or, Sr = varlen.forward_varlen_chunked(Q, K, V, beta, g, cu, C, S0 if with_state else None,
                                           scale, inverse_for(C, exact, N, S))
    tol = TOL[dt]
    eo = np.max(np.abs(host(O) - Or)) if Or.size else 0.0
    es = np.max(np.abs(host(Sf) - Sr))
    print(f"  O err {eo:.2e} (max |O| {np.max(np.abs(Or)) if Or.size else 0:.2f}), "
          f"S err {es:.2e}", flush=True)
    assert eo <= tol * max(1.0, np.max(np.abs(Or)) if Or.size else 1.0)
    assert es <= tol * max(1.0, np.max(np.abs(Sr)))
    return O, Sf


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64])
def test_forward_varlen_matches_oracle(C, dt):
    check(RAGGED, C, dt, seed=C)


@pytest.mark.parametrize("C", [32, 64])
def test_forward_varlen_exact_inverse_and_other_orders(C):
    check(RAGGED, C, "bf16", exact=True, seed=1)
    check([5, 40, 99], C, "f32", N=2, S=3, dk=64, dv=128, seed=2)


def test_forward_varlen_without_initial_state_and_with_one_sequence():
    check([300], 64, "bf16", with_state=False, seed=3)
    check([64 * 3], 64, "f32", seed=4)


def test_forward_varlen_equal_lengths_match_fixed_length_bit_for_bit():
    """Sequences of equal length, a multiple of C, packed one after another
    are the [B, L, H, d] layout of gdn_chunk_forward: O and the final states
    agree bit for bit."""
    C, dt, B, L, H = 64, "bf16", 3, 256, 4
    w = wl.workload("qwen35_prefill").with_(B=B, L=L, H=H)
    Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w)
    dQ, dK, dV, db, dg, dS0 = dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g), dev32(S0)
    Of, Sff = G.gdn_chunk_forward(dQ, dK, dV, db, dg, C, S0=dS0, scale=0.1)
    pack = lambda t: t.reshape((1, B * L) + tuple(t.shape[2:]))
    tables = G.gdn_varlen_tables(list(range(0, B * L + 1, L)), C)
    Ov, Sfv = G.gdn_chunk_forward_varlen(pack(dQ), pack(dK), pack(dV), pack(db), pack(dg), tables,
                                         C, S0=dS0, scale=0.1)
    torch.cuda.synchronize()
    assert torch.equal(pack(Of), Ov)
    assert torch.equal(Sff, Sfv)


def test_forward_varlen_rows_written_in_place_state_and_empty():
    C, dt = 32, "f32"
    lengths = [3, 0, 33, 0]
    Q, K, V, beta, g, cu, S0 = inputs(lengths, C, dt, seed=5)
    T = int(cu[-1])
    Obuf = torch.full((1, T + 2, 2, 128), 7.0, device="cuda")
    O = Obuf[:, :T]
    assert O.is_contiguous()
    St = dev32(S0)
    tables = G.gdn_varlen_tables(cu, C)
    G.gdn_chunk_forward_varlen(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g), tables,
                               C, S0=St, S_final=St, O=O, scale=0.5)
    Or, Sr = varlen.forward_varlen_chunked(Q, K, V, beta, g, cu, C, S0, 0.5)
    assert not np.any(host(O) == 7.0) and np.all(host(Obuf[:, T:]) == 7.0)
    assert np.max(np.abs(host(O) - Or)) <= 1e-5 * max(1.0, np.max(np.abs(Or)))
    assert np.max(np.abs(host(St) - Sr)) <= 1e-5 * max(1.0, np.max(np.abs(Sr)))
    assert np.array_equal(host(St)[1], S0[1]) and np.array_equal(host(St)[3], S0[3])
    # only empty sequences: the states pass through
    z = torch.zeros((1, 0, 2, 128), device="cuda")
    zb = torch.zeros((1, 0, 2), device="cuda")
    S2 = dev32(S0[:2])
    _, Sf = G.gdn_chunk_forward_varlen(z, z, z, zb, zb, G.gdn_varlen_tables([0, 0, 0], C), C,
                                       S0=S2)
    assert torch.equal(Sf, S2)


def test_forward_varlen_serving_mix_full_size():
    """The serving mix at the prefill's size (8192 tokens, 16 heads, bf16),
    every token of every head checked."""
    C, dt = 64, "bf16"
    lengths = wl.varlen_lengths(8192)
    w = wl.workload("qwen35_prefill")
    K, beta, g, V, cu, Q = wl.gen_varlen(w, lengths, C=C, want_q=True)
    S0 = np.stack([np.stack([wl.gen_state(w, s, h) for h in range(w.H)]) for s in range(len(lengths))])
    print(f"serving mix: {len(lengths)} sequences, {int(cu[-1])} tokens", flush=True)
    tables = G.gdn_varlen_tables(cu, C)
    O, Sf = G.gdn_chunk_forward_varlen(dev(Q, dt), dev(K, dt), dev(V, dt), dev32(beta), dev32(g),
                                       tables, C, S0=dev32(S0))
    Or, Sr = varlen.forward_varlen_chunked(Q, K, V, beta, g, cu, C, S0, 128 ** -0.5,
                                           inverse_for(C, False))
    assert np.max(np.abs(host(O) - Or)) <= TOL[dt] * max(1.0, np.max(np.abs(Or)))
    assert np.max(np.abs(host(Sf) - Sr)) <= TOL[dt] * max(1.0, np.max(np.abs(Sr)))
