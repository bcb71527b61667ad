"""Parity of the fused path over packed variable-length sequences
(gdn_chunk_wy_fused_varlen, through the C ABI) with the packed oracle.

The oracle solves every chunk on its own m x m system from exactly the
values the GPU reads (storage dtype, upcast to float64), with the same
inverse (exact, or T_hat(N, S) at the GPU's order).  Tolerances as for the
fixed-length fused path: max abs error <= 1e-5 (fp32) and 2e-2 (bf16),
scaled by max(1, max |ref|) for W and U.
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


def dev(x, dt):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda").to(TDT[dt])


def dev32(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def run(lengths, C, dt, exact=False, N=None, S=None, H=3, seed=0, dk=128, dv=128):
    w = wl.workload("tiny").with_(H=H, C=C, dtype=dt, dk=dk, dv=dv, seed=4000 + seed)
    K, beta, g, V, cu = wl.gen_varlen(w, lengths, C=C)
    tables = G.gdn_varlen_tables(cu, C)
    Wg, Ug, Tg = G.gdn_chunk_wy_fused_varlen(dev(K, dt), dev(V, dt), dev32(beta), dev32(g), tables,
                                             C, N=N, S=S, exact=exact, want_T=True)
    Wr, Ur, Tr = varlen.wy_varlen(K, V, beta, g, cu, C, inverse=oracle_inverse(C, exact, N, S))
    return (host(Wg), host(Ug), host(Tg)), (Wr, Ur, Tr), cu


def padded(inv, C):
    """An m x m inverse taken as the top left of `inv` on the system padded
    to C x C with tokens that write nothing (zero rows and columns)."""
    def f(A):
        m = A.shape[-1]
        P = np.zeros(A.shape[:-2] + (C, C))
        P[..., :m, :m] = A
        return inv(P)[..., :m, :m]
    return f


def oracle_inverse(C, exact, N=None, S=None):
    if exact:
        return gdn.forward_substitution_inverse
    dn, ds = gdn.default_order(C)
    n, s = (dn if N is None else N), (ds if S is None else S)
    if C == 128:  # the two 64 x 64 blocks of the fixed-length C = 128 path
        return padded(lambda A: gdn.neumann_inverse_blocked(A, n, s), C)
    return lambda A: gdn.neumann_inverse(A, n, s)


def check(got, ref, dt):
    (Wg, Ug, Tg), (Wr, Ur, Tr) = got, ref
    assert Tg.shape == Tr.shape
    tol = TOL[dt]
    assert np.max(np.abs(Tg - Tr)) <= tol
    assert np.max(np.abs(Wg - Wr)) <= tol * max(1.0, np.max(np.abs(Wr)))
    assert np.max(np.abs(Ug - Ur)) <= tol * max(1.0, np.max(np.abs(Ur)))


RAGGED = [1, 15, 16, 17, 63, 64, 65, 130, 0, 7, 200]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
@pytest.mark.parametrize("exact", [False, True])
def test_varlen_matches_oracle(C, dt, exact):
    got, ref, _ = run(RAGGED, C, dt, exact=exact, seed=C)
    check(got, ref, dt)


RAGGED128 = [1, 63, 64, 65, 127, 128, 129, 0, 200, 256, 300]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_varlen_c128_half_boundaries(dt):
    # partial chunks with no token in the second half (m <= 64), tokens in
    # both halves, and full chunks
    got, ref, _ = run(RAGGED128, 128, dt, seed=7)
    check(got, ref, dt)


@pytest.mark.parametrize("C", [64, 128])
def test_varlen_batch_of_equal_ragged_lengths(C):
    # a [B, L] batch with L % C != 0 as B packed sequences of L tokens
    got, ref, _ = run([100, 100, 100], C, "bf16", seed=21 + C)
    check(got, ref, "bf16")


def test_varlen_c128_other_orders_and_widths():
    got, ref, _ = run([5, 100, 190], 128, "f32", N=2, S=3, dk=64, dv=128, seed=12)
    check(got, ref, "f32")
    got, ref, _ = run([70, 33], 128, "f32", N=16, S=2, dk=128, dv=64, seed=13)
    check(got, ref, "f32")


@pytest.mark.parametrize("C", [16, 64])
def test_varlen_other_orders_and_widths(C):
    got, ref, _ = run([5, 40, 99], C, "f32", N=2, S=3, dk=64, dv=128, seed=11)
    check(got, ref, "f32")


def test_varlen_equal_lengths_match_fixed_length_path_bit_for_bit():
    # sequences of equal length, a multiple of C, packed one after another are
    # the [B, L, H, d] layout of the fixed-length path; only the tile order
    # of Tinv differs ([H, chunks] against [B, H, L / C])
    C, dt, B, L, H = 64, "bf16", 3, 256, 4
    w = wl.workload("qwen35_prefill").with_(B=B, L=L, H=H)
    K, beta, g, V = wl.gen_inputs(w)
    dK, dV, db, dg = dev(K, dt), dev(V, dt), dev32(beta), dev32(g)
    Wf, Uf, Tf = G.gdn_chunk_wy_fused(dK, dV, db, dg, C, 3, 8, want_T=True)
    pack = lambda t: t.reshape((1, B * L) + tuple(t.shape[2:]))
    tables = G.gdn_varlen_tables(list(range(0, B * L + 1, L)), C)
    Wv, Uv, Tv = G.gdn_chunk_wy_fused_varlen(pack(dK), pack(dV), pack(db), pack(dg), tables, C,
                                             want_T=True)
    assert torch.equal(pack(Wf), Wv) and torch.equal(pack(Uf), Uv)
    nc = L // C
    assert torch.equal(Tf.permute(1, 0, 2, 3, 4).reshape(H, B * nc, C, C), Tv)


@pytest.mark.parametrize("C", [64, 128])
def test_varlen_serving_mix_full_size(C):
    # the serving mix at the prefill's size: 8192 tokens, 16 heads, bf16;
    # every chunk of every head checked
    dt = "bf16"
    lengths = wl.varlen_lengths(8192)
    w = wl.workload("qwen35_prefill")
    K, beta, g, V, cu = wl.gen_varlen(w, lengths, C=C)
    tables = G.gdn_varlen_tables(cu, C)
    Wg, Ug = G.gdn_chunk_wy_fused_varlen(dev(K, dt), dev(V, dt), dev32(beta), dev32(g), tables, C)
    Wr, Ur, _ = varlen.wy_varlen(K, V, beta, g, cu, C, inverse=oracle_inverse(C, False))
    assert np.max(np.abs(host(Wg) - Wr)) <= TOL[dt] * max(1.0, np.max(np.abs(Wr)))
    assert np.max(np.abs(host(Ug) - Ur)) <= TOL[dt] * max(1.0, np.max(np.abs(Ur)))


def test_varlen_rows_of_every_token_written_and_nothing_else():
    C, dt = 32, "f32"
    lengths = [3, 0, 33]
    w = wl.workload("tiny").with_(H=2, C=C, dtype=dt)
    K, beta, g, V, cu = wl.gen_varlen(w, lengths, C=C)
    T = int(cu[-1])
    # two extra token rows past the packed sequences, filled with a marker
    Wbuf = torch.full((1, T + 2, 2, 128), 7.0, device="cuda")
    Ubuf = torch.full((1, T + 2, 2, 128), 7.0, device="cuda")
    tables = G.gdn_varlen_tables(cu, C)
    W, U = Wbuf[:, :T], Ubuf[:, :T]  # contiguous views into the larger buffers
    assert W.is_contiguous() and U.is_contiguous()
    G.gdn_chunk_wy_fused_varlen(dev(K, dt), dev(V, dt), dev32(beta), dev32(g), tables, C, W=W, U=U)
    assert not np.any(host(W) == 7.0) and not np.any(host(U) == 7.0)
    assert np.all(host(Wbuf[:, T:]) == 7.0) and np.all(host(Ubuf[:, T:]) == 7.0)


def test_varlen_empty_and_degenerate():
    C, dt = 16, "f32"
    # only empty sequences: nothing to do
    K = torch.zeros((1, 0, 2, 128), device="cuda")
    b = torch.zeros((1, 0, 2), device="cuda")
    tables = G.gdn_varlen_tables([0, 0, 0], C)
    W, U = G.gdn_chunk_wy_fused_varlen(K, K, b, b, tables, C)
    assert W.numel() == 0
    # single-token sequences: W = beta k
    got, ref, _ = run([1, 1, 1, 2], C, dt, seed=3)
    check(got, ref, dt)
    assert np.allclose(got[2][:, 0], np.eye(C)[None].repeat(3, 0), atol=0)
