"""Pins of the packed variable-length oracle (oracle/varlen.py).

* equal sequence lengths that are multiples of C reproduce the fixed-length
  oracle (batch of sequences) exactly;
* a partial chunk of m tokens gives the first m rows of W, U that the full
  chunk gives with any continuation (T is lower triangular, so row i depends
  on the chunk's tokens up to i only), and the first m x m block of its
  inverse;
* padding a partial chunk with tokens that write nothing (beta = 0) gives the
  same inverse with the identity on the padded rows and columns;
* the chunk table covers every token once, and single-token chunks reduce to
  W = beta k;
* the layer forward over packed sequences: its chunk-wise form equals the
  token recurrence run on every sequence alone (ragged last chunks, empty
  sequences, one state per sequence), equal lengths reproduce the
  fixed-length forward, sequences do not interact, and a sequence split at
  a chunk boundary continues from the first piece's final state.
"""

import numpy as np
import pytest

import workloads as wl
from oracle import gdn, gdn_forward, varlen


def test_chunk_table_covers_tokens_once():
    lengths = [0, 1, 63, 64, 65, 130, 0, 7]
    cu = np.concatenate([[0], np.cumsum(lengths)])
    table = varlen.chunk_table(cu, 64)
    seen = np.zeros(cu[-1], int)
    for s, t, m in table:
        assert 1 <= m <= 64 and cu[s] <= t and t + m <= cu[s + 1]
        seen[t:t + m] += 1
    assert np.all(seen == 1)
    off = varlen.chunk_offsets(cu, 64)
    assert off[-1] == len(table)
    assert list(np.diff(off)) == [0, 1, 1, 1, 2, 3, 0, 1]


@pytest.mark.parametrize("C", [16, 64])
def test_equal_lengths_reduce_to_fixed_length(C):
    w = wl.workload("tiny").with_(B=3, L=2 * C, H=2, dk=32, dv=16, C=C)
    K, beta, g, V = wl.gen_inputs(w)
    cu = np.arange(0, 3 * 2 * C + 1, 2 * C)
    pack = lambda x: x.reshape((1, -1) + x.shape[2:])
    Wv, Uv, Tv = varlen.wy_varlen(pack(K), pack(V), pack(beta), pack(g), cu, C)
    Tf = gdn.forward_substitution_inverse(gdn.build_A(K, beta, g, C))  # [B, H, nc, C, C]
    Wf, Uf = gdn.wy_apply(Tf, K, V, beta, C)
    assert np.allclose(Wv, pack(Wf), rtol=0, atol=1e-12)
    assert np.allclose(Uv, pack(Uf), rtol=0, atol=1e-12)
    # tiles: [H, n_chunks] with chunks of sequence b at b * nc + c
    nc = 2
    for b in range(3):
        for h in range(2):
            for c in range(nc):
                assert np.allclose(Tv[h, b * nc + c], Tf[b, h, c], rtol=0, atol=1e-12)


@pytest.mark.parametrize("m", [1, 5, 31])
def test_partial_chunk_is_prefix_of_full_chunk(m):
    C = 32
    rng = np.random.default_rng(m)
    z = rng.standard_normal((1, C, 1, 16))
    K = z / np.linalg.norm(z, axis=-1, keepdims=True)
    V = rng.standard_normal((1, C, 1, 8))
    beta = rng.random((1, C, 1))
    g = np.cumsum(-rng.random((1, C, 1)), axis=1)
    Wp, Up, Tp = varlen.wy_varlen(K[:, :m], V[:, :m], beta[:, :m], g[:, :m], [0, m], C)
    Wf, Uf, Tf = varlen.wy_varlen(K, V, beta, g, [0, C], C)
    assert np.allclose(Wp[0], Wf[0, :m], rtol=0, atol=1e-12)
    assert np.allclose(Up[0], Uf[0, :m], rtol=0, atol=1e-12)
    assert np.allclose(Tp[0, 0, :m, :m], Tf[0, 0, :m, :m], rtol=0, atol=1e-12)
    assert np.array_equal(Tp[0, 0, m:, :], np.eye(C)[m:])
    assert np.array_equal(Tp[0, 0, :, m:], np.eye(C)[:, m:])


def test_padding_with_silent_tokens_gives_same_inverse():
    C, m = 64, 23
    rng = np.random.default_rng(2)
    z = rng.standard_normal((1, C, 1, 32))
    K = z / np.linalg.norm(z, axis=-1, keepdims=True)
    beta = rng.random((1, C, 1))
    g = np.cumsum(-rng.random((1, C, 1)), axis=1)
    beta[:, m:] = 0.0
    Tpad = gdn.forward_substitution_inverse(gdn.build_A(K, beta, g, C))[0, 0, 0]
    _, _, Tv = varlen.wy_varlen(K[:, :m], K[:, :m, :, :4], beta[:, :m], g[:, :m], [0, m], C)
    # rows past m of the padded system: beta = 0 writes nothing, so they are
    # unit rows of (I + A); the top-left block is the m x m inverse
    assert np.allclose(Tpad[:m, :m], Tv[0, 0, :m, :m], rtol=0, atol=1e-12)
    assert np.allclose(Tpad[m:, m:], np.eye(C - m), rtol=0, atol=1e-12)


def test_single_token_chunks():
    rng = np.random.default_rng(3)
    K = rng.standard_normal((1, 3, 2, 8))
    V = rng.standard_normal((1, 3, 2, 4))
    beta = rng.random((1, 3, 2))
    g = -rng.random((1, 3, 2))
    W, U, T = varlen.wy_varlen(K, V, beta, g, [0, 1, 2, 3], 16)
    assert np.allclose(W, beta[..., None] * K, rtol=0, atol=1e-15)
    assert np.allclose(U, beta[..., None] * V, rtol=0, atol=1e-15)
    assert T.shape == (2, 3, 16, 16) and np.array_equal(T[0, 0], np.eye(16))


def test_neumann_on_partial_chunks_equals_padded_neumann():
    # T_hat(N, S) of an m x m system equals the top-left block of T_hat(N, S)
    # of the system padded with silent tokens (every power is block diagonal)
    C, m = 64, 40
    rng = np.random.default_rng(4)
    z = rng.standard_normal((1, C, 1, 32)) + 2.0 * rng.standard_normal((1, 1, 1, 32))
    K = z / np.linalg.norm(z, axis=-1, keepdims=True)
    beta = rng.random((1, C, 1))
    beta[:, m:] = 0.0
    g = np.cumsum(-0.02 * rng.random((1, C, 1)), axis=1)
    A = gdn.build_A(K, beta, g, C)[0, 0, 0]
    Tpad = gdn.neumann_inverse(A[None], 3, 2)[0]
    Tm = gdn.neumann_inverse(A[None, :m, :m], 3, 2)[0]
    assert np.allclose(Tpad[:m, :m], Tm, rtol=0, atol=1e-13)
    assert np.allclose(Tpad[m:, m:], np.eye(C - m), rtol=0, atol=1e-13)
    assert np.abs(Tm - gdn.forward_substitution_inverse(A[None, :m, :m])[0]).max() > 1e-9


def test_varlen_generator_layout():
    w = wl.workload("qwen35_prefill").with_(H=2)
    K, beta, g, V, cu = wl.gen_varlen(w, [5, 0, 70], C=64)
    assert list(cu) == [0, 5, 5, 75]
    assert K.shape == (1, 75, 2, 128) and V.shape == (1, 75, 2, 128)
    # g restarts at the sequence start and at every chunk of C tokens
    assert np.all(g[0, :, 0] < 0) and np.all(np.diff(g[0, :5, 0]) < 0)
    assert g[0, 5, 0] > g[0, 4, 0]  # sequence 2 starts a new chunk
    assert np.allclose(varlen.varlen_cumsum(
        np.concatenate([[g[0, 0, 0]], np.diff(g[0, :5, 0])]), [0, 5], 64), g[0, :5, 0])
    assert g[0, 5 + 64, 0] > g[0, 5 + 63, 0]  # a new chunk starts at token 64 of sequence 2


# ---------------------------------------------------------------------------
# the layer forward over packed sequences


def _fwd_inputs(lengths, C, H=2, dk=16, dv=8, seed=0):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    T = int(cu[-1])
    z = rng.standard_normal((1, T, H, dk))
    K = z / np.linalg.norm(z, axis=-1, keepdims=True)
    Q = rng.standard_normal((1, T, H, dk))
    V = rng.standard_normal((1, T, H, dv))
    beta = rng.random((1, T, H))
    g = varlen.varlen_cumsum(-0.3 * rng.random((T, H)), cu, C)[None]
    S0 = rng.standard_normal((len(lengths), H, dk, dv))
    return Q, K, V, beta, g, cu, S0


@pytest.mark.parametrize("C", [8, 16])
def test_forward_varlen_chunked_equals_recurrence(C):
    """The chunk-wise form over packed sequences (ragged last chunks, empty
    sequences, a state per sequence) equals the token recurrence run on
    every sequence alone."""
    Q, K, V, beta, g, cu, S0 = _fwd_inputs([5, 0, 70, 2 * C, 1, C + 1], C)
    O1, S1 = varlen.forward_varlen_recurrent(Q, K, V, beta, g, cu, C, S0, 0.5)
    O2, S2 = varlen.forward_varlen_chunked(Q, K, V, beta, g, cu, C, S0, 0.5)
    assert np.allclose(O1, O2, rtol=0, atol=1e-12)
    assert np.allclose(S1, S2, rtol=0, atol=1e-12)
    assert np.array_equal(S2[1], S0[1])  # the empty sequence keeps its state


def test_forward_varlen_equal_lengths_reduce_to_fixed_length():
    C, B, L = 16, 3, 48
    w = wl.workload("tiny").with_(B=B, L=L, H=2, dk=16, dv=8, C=C)
    Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w, C=C)
    Of, Sf = gdn_forward.gdn_chunked(Q, K, V, beta, g, C, S0, 0.25)
    pack = lambda x: x.reshape((1, -1) + x.shape[2:])
    Ov, Sv = varlen.forward_varlen_chunked(pack(Q), pack(K), pack(V), pack(beta), pack(g),
                                           np.arange(0, B * L + 1, L), C, S0.reshape(B * 2, 16, 8)
                                           .reshape(B, 2, 16, 8), 0.25)
    assert np.allclose(Ov, pack(Of), rtol=0, atol=1e-12)
    assert np.allclose(Sv, Sf, rtol=0, atol=1e-12)


def test_forward_varlen_sequences_are_independent_and_split_at_chunks():
    """Changing one sequence leaves the others' outputs and states alone;
    running a sequence as two pieces split at a chunk boundary, the second
    starting from the first's final state, gives the one-piece result."""
    C = 8
    Q, K, V, beta, g, cu, S0 = _fwd_inputs([13, 24, 9], C, seed=1)
    O, S = varlen.forward_varlen_chunked(Q, K, V, beta, g, cu, C, S0)
    V2 = V.copy()
    V2[:, cu[1]:cu[2]] *= -3.0
    O2, S2 = varlen.forward_varlen_chunked(Q, K, V2, beta, g, cu, C, S0)
    for s in (0, 2):
        assert np.array_equal(O[:, cu[s]:cu[s + 1]], O2[:, cu[s]:cu[s + 1]])
        assert np.array_equal(S[s], S2[s])
    # sequence 1 (24 tokens) as 16 + 8 tokens
    cut = [0, 13, 29, 37, 46]
    Oa, Sa = varlen.forward_varlen_chunked(Q, K, V, beta, g, cut, C, np.stack([S0[0], S0[1], S0[1], S0[2]]))
    Ob, Sb = varlen.forward_varlen_chunked(Q[:, 29:37], K[:, 29:37], V[:, 29:37], beta[:, 29:37],
                                           g[:, 29:37], [0, 8], C, Sa[1:2])
    assert np.allclose(Ob, O[:, 29:37], rtol=0, atol=1e-12)
    assert np.allclose(Sb[0], S[1], rtol=0, atol=1e-12)
