"""Pins of the float64 forward oracle (oracle/gdn_forward.py).

The two codings in the oracle (token recurrence, chunk-wise form) check each
other; beyond that, each coding is held to properties of the gated delta rule
that follow from its definition, not from either coding:

* with beta = 1 and unit keys, reading the state with the key just written
  returns the value just written, whatever the decay and the old state;
* with beta = 0 the state only decays: o_t = exp(G_t) S0^T q_t, G the
  running sum of the log-decays since the start of the sequence;
* with orthonormal keys the delta rule reduces to gated linear attention
  plus the erasure of the old state along the keys written so far,
  o_t = sum_{j <= t} exp(G_t - G_j) beta_j (q_t . k_j) v_j
  + exp(G_t) S0^T (I - sum_{j <= t} beta_j k_j k_j^T) q_t
  (the projectors k_j k_j^T commute and annihilate each other);
* the state and the output are linear in (V, S0) jointly;
* the chunk length is a choice of evaluation order, not of the result.
"""

import numpy as np
import pytest

import workloads as wl
from oracle import gdn, gdn_forward as fwd


def _rand_inputs(B, L, H, dk, dv, C, seed, gate_shift=3.0, stress=False):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((B, L, H, dk))
    if stress:
        z = z + 2.0 * rng.standard_normal((1, 1, H, dk))
    K = z / np.linalg.norm(z, axis=-1, keepdims=True)
    z = rng.standard_normal((B, L, H, dk))
    Q = z / np.linalg.norm(z, axis=-1, keepdims=True)
    V = rng.standard_normal((B, L, H, dv))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((B, L, H))))
    inc = -np.logaddexp(0.0, rng.standard_normal((B, L, H)) + gate_shift)
    g = wl.chunk_cumsum(inc, C, axis=1)
    S0 = rng.standard_normal((B, H, dk, dv))
    return Q, K, V, beta, g, S0, inc


@pytest.mark.parametrize("C", [16, 32, 64])
@pytest.mark.parametrize("stress", [False, True])
def test_chunked_equals_recurrent(C, stress):
    Q, K, V, beta, g, S0, _ = _rand_inputs(2, 4 * C, 2, 32, 24, C, seed=C, stress=stress,
                                           gate_shift=-1.0 if stress else 3.0)
    Or, Sr = fwd.gdn_recurrent(Q, K, V, beta, g, C, S0, scale=0.7)
    Oc, Sc = fwd.gdn_chunked(Q, K, V, beta, g, C, S0, scale=0.7)
    assert np.max(np.abs(Oc - Or)) < 1e-11 * max(1.0, np.max(np.abs(Or)))
    assert np.max(np.abs(Sc - Sr)) < 1e-11 * max(1.0, np.max(np.abs(Sr)))


def test_chunk_length_does_not_change_result():
    C0 = 16
    Q, K, V, beta, _, S0, inc = _rand_inputs(1, 128, 2, 32, 32, C0, seed=11, gate_shift=0.0)
    outs = []
    for C in (16, 32, 64, 128):
        g = wl.chunk_cumsum(inc, C, axis=1)
        outs.append(fwd.gdn_chunked(Q, K, V, beta, g, C, S0))
    for O, S in outs[1:]:
        assert np.max(np.abs(O - outs[0][0])) < 1e-11 * np.max(np.abs(outs[0][0]))
        assert np.max(np.abs(S - outs[0][1])) < 1e-11 * np.max(np.abs(outs[0][1]))


def test_token_log_decay_inverts_chunk_cumsum():
    rng = np.random.default_rng(3)
    inc = -rng.random((2, 64, 3))
    g = wl.chunk_cumsum(inc, 16, axis=1)
    assert np.allclose(fwd.token_log_decay(g, 16), inc, rtol=0, atol=1e-14)


@pytest.mark.parametrize("coding", ["recurrent", "chunked"])
def test_delta_rule_write_is_exact_at_beta_one(coding):
    # S_t^T k_t = a_t (1 - beta_t) S_{t-1}^T k_t + beta_t v_t = v_t when beta_t = 1
    C = 16
    Q, K, V, beta, g, S0, _ = _rand_inputs(1, 2 * C, 2, 16, 8, C, seed=5, gate_shift=-1.0)
    beta = np.ones_like(beta)
    run = fwd.gdn_recurrent if coding == "recurrent" else fwd.gdn_chunked
    O, _ = run(K, K, V, beta, g, C, S0)  # queries = keys
    assert np.max(np.abs(O - V)) < 1e-12


@pytest.mark.parametrize("coding", ["recurrent", "chunked"])
def test_beta_zero_is_pure_decay(coding):
    C = 16
    Q, K, V, beta, g, S0, inc = _rand_inputs(2, 3 * C, 2, 16, 8, C, seed=6, gate_shift=1.0)
    beta = np.zeros_like(beta)
    run = fwd.gdn_recurrent if coding == "recurrent" else fwd.gdn_chunked
    O, S = run(Q, K, V, beta, g, C, S0, scale=1.3)
    G = np.cumsum(inc, axis=1)  # [B, L, H]
    ref = 1.3 * np.exp(G)[..., None] * np.einsum("bhkv,blhk->blhv", S0, Q)
    assert np.max(np.abs(O - ref)) < 1e-12
    assert np.max(np.abs(S - np.exp(G[:, -1])[..., None, None] * S0)) < 1e-12


@pytest.mark.parametrize("coding", ["recurrent", "chunked"])
def test_orthogonal_keys_reduce_to_gated_linear_attention(coding):
    C, L, dk, dv = 16, 32, 32, 8
    rng = np.random.default_rng(8)
    Qm, _ = np.linalg.qr(rng.standard_normal((dk, dk)))  # orthonormal columns
    K = Qm.T[None, :, None, :]  # token t has key column t of Qm: k_i . k_j = delta_ij
    Q = rng.standard_normal((1, L, 1, dk))
    V = rng.standard_normal((1, L, 1, dv))
    beta = rng.random((1, L, 1))
    inc = -rng.random((1, L, 1))
    g = wl.chunk_cumsum(inc, C, axis=1)
    S0 = rng.standard_normal((1, 1, dk, dv))
    run = fwd.gdn_recurrent if coding == "recurrent" else fwd.gdn_chunked
    O, _ = run(Q, K, V, beta, g, C, S0)
    G = np.cumsum(inc[0, :, 0])
    ref = np.zeros((L, dv))
    for t in range(L):
        erase = np.eye(dk) - sum(beta[0, j, 0] * np.outer(K[0, j, 0], K[0, j, 0])
                                 for j in range(t + 1))
        ref[t] = np.exp(G[t]) * (S0[0, 0].T @ (erase @ Q[0, t, 0]))
        for j in range(t + 1):
            ref[t] += np.exp(G[t] - G[j]) * beta[0, j, 0] * (Q[0, t, 0] @ K[0, j, 0]) * V[0, j, 0]
    assert np.max(np.abs(O[0, :, 0] - ref)) < 1e-12


@pytest.mark.parametrize("coding", ["recurrent", "chunked"])
def test_linear_in_values_and_initial_state(coding):
    C = 16
    Q, K, V1, beta, g, S1, _ = _rand_inputs(1, 2 * C, 2, 16, 8, C, seed=9)
    _, _, V2, _, _, S2, _ = _rand_inputs(1, 2 * C, 2, 16, 8, C, seed=10)
    run = fwd.gdn_recurrent if coding == "recurrent" else fwd.gdn_chunked
    Oa, Sa = run(Q, K, V1, beta, g, C, S1)
    Ob, Sb = run(Q, K, V2, beta, g, C, S2)
    Oc, Sc = run(Q, K, 2.0 * V1 - 3.0 * V2, beta, g, C, 2.0 * S1 - 3.0 * S2)
    assert np.max(np.abs(Oc - (2.0 * Oa - 3.0 * Ob))) < 1e-11
    assert np.max(np.abs(Sc - (2.0 * Sa - 3.0 * Sb))) < 1e-11


def test_no_initial_state_means_zero_state():
    C = 16
    Q, K, V, beta, g, S0, _ = _rand_inputs(1, 2 * C, 2, 16, 8, C, seed=12)
    for run in (fwd.gdn_recurrent, fwd.gdn_chunked):
        O1, S1 = run(Q, K, V, beta, g, C)
        O2, S2 = run(Q, K, V, beta, g, C, np.zeros_like(S0))
        assert np.array_equal(O1, O2) and np.array_equal(S1, S2)


def test_approximate_inverse_error_reaches_output_bounded():
    # with T_hat(N, S) in place of the exact inverse the chunk-wise form
    # departs from the recurrence by no more than the inverse's own error
    # allows; at the default order on these gates the two are equal to
    # rounding
    C = 64
    Q, K, V, beta, g, S0, _ = _rand_inputs(1, 2 * C, 1, 32, 16, C, seed=13)
    N, S = gdn.default_order(C)
    Oe, _ = fwd.gdn_chunked(Q, K, V, beta, g, C, S0)
    Oa, _ = fwd.gdn_chunked(Q, K, V, beta, g, C, S0,
                            inverse=lambda A: gdn.neumann_inverse(A, N, S))
    assert np.max(np.abs(Oa - Oe)) < 1e-12 * np.max(np.abs(Oe))
    # a deliberately low order leaves a visible error
    Ol, _ = fwd.gdn_chunked(Q, K, V, beta, g, C, S0,
                            inverse=lambda A: gdn.neumann_inverse(A, 1, 0))
    assert np.max(np.abs(Ol - Oe)) > 1e-6 * np.max(np.abs(Oe))


def test_workload_queries_do_not_change_other_draws():
    w = wl.workload("tiny", L=256)
    k, b, g, v = wl.gen_head(w, 0, 1)
    q2, k2, v2, b2, g2 = wl.gen_head_qkv(w, 0, 1)
    assert np.array_equal(k, k2) and np.array_equal(v, v2)
    assert np.array_equal(b, b2) and np.array_equal(g, g2)
    assert np.allclose(np.linalg.norm(q2, axis=1), 1.0, atol=1e-6)
    assert not np.allclose(q2, k2)
