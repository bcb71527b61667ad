"""Maximum-size launches: tensors past 4 GiB of byte offsets.

A few seeded tiles (or chunks) are repeated on the device (torch's repeat:
plumbing) until every tensor of the launch spans more than 2^32 bytes; the
outputs at the first, middle and last positions must equal the oracle's
result for the corresponding base tile, so any 32-bit offset arithmetic in
the kernels would show.  Tolerances as in the parity tests.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import gdn
from oracle import int8 as oi

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def base_tiles(C, n=16, seed=0):
    w = wl.workload("tiny").with_(L=n * C, H=1, B=1, C=C, seed=6000 + seed)
    K, beta, g, _ = wl.gen_inputs(w, C=C, want_v=False)
    A = gdn.tiles_flat(gdn.build_A(K, beta, g, C))
    return wl.round_to_bf16(A.astype(np.float32)).astype(np.float64)


def test_neumann_inverse_past_4GiB():
    C, nb = 64, 16
    A0 = base_tiles(C, nb)
    reps = (1 << 32) // (C * C * 2) // nb + 2          # bf16 tiles: just past 2^32 bytes
    n = nb * reps
    print(f"neumann past 4 GiB: {n} tiles, {n * C * C * 2 / 2**30:.2f} GiB per tensor", flush=True)
    dA = torch.from_numpy(A0.astype(np.float32)).to("cuda").to(torch.bfloat16).repeat(reps, 1, 1)
    T = G.gdn_chunk_inverse_neumann(dA, 3, 8)
    ref = gdn.neumann_inverse(A0, 3, 8)
    for start in (0, (reps // 2) * nb, n - nb):
        got = host(T[start:start + nb])
        assert np.max(np.abs(got - ref)) <= 2e-2, start
    del dA, T
    torch.cuda.empty_cache()


def test_int16_inverse_past_4GiB():
    C, nb = 64, 16
    A0 = base_tiles(C, nb, seed=1).astype(np.float32)
    qA, eA = oi.quantize(A0, oi.SPEC16)
    reps = (1 << 32) // (C * C * 2) // nb + 2
    n = nb * reps
    print(f"int16 past 4 GiB: {n} tiles", flush=True)
    dq = torch.from_numpy(qA.astype(np.int16)).to("cuda").repeat(reps, 1, 1)
    de = torch.from_numpy(eA.astype(np.int32)).to("cuda").repeat(reps)
    Tq, eT = G.gdn_chunk_inverse_neumann_i16(dq, de, 3, 8)
    rq, re, _ = oi.neumann_inverse_int16(qA, eA, 3, 8)
    torch.cuda.synchronize()
    for start in (0, (reps // 2) * nb, n - nb):
        assert np.array_equal(Tq[start:start + nb].cpu().numpy().astype(np.int64), rq), start
        assert np.array_equal(eT[start:start + nb].cpu().numpy().astype(np.int64), re), start
    del dq, de, Tq, eT
    torch.cuda.empty_cache()


def test_fused_path_past_4GiB():
    """K, V, W, U of [1, L, H, 128] bf16 past 2^32 bytes each: one seeded
    chunk of 64 tokens (64 heads) repeated along L."""
    C, H = 64, 64
    w = wl.workload("tiny").with_(B=1, L=C, H=H, C=C, dtype="bf16", seed=6100)
    K, beta, g, V = wl.gen_inputs(w, C=C)
    chunks = (1 << 32) // (C * H * 128 * 2) + 2
    L = chunks * C
    print(f"fused past 4 GiB: L={L}, {L * H * 128 * 2 / 2**30:.2f} GiB per tensor", flush=True)
    dev = lambda x, t: torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).to("cuda").to(t)
    dK = dev(K, torch.bfloat16).repeat(1, chunks, 1, 1)
    dV = dev(V, torch.bfloat16).repeat(1, chunks, 1, 1)
    db = dev(beta, torch.float32).repeat(1, chunks, 1)
    dg = dev(g, torch.float32).repeat(1, chunks, 1)
    W, U = G.gdn_chunk_wy_fused(dK, dV, db, dg, C, 3, 8)
    Kf, Vf = (np.asarray(x, np.float64) for x in (K, V))
    T = gdn.neumann_inverse(gdn.build_A(Kf, beta, g, C), 3, 8)
    Wr, Ur = gdn.wy_apply(T, Kf, Vf, beta, C)
    for ck in (0, chunks // 2, chunks - 1):
        sl = slice(ck * C, (ck + 1) * C)
        assert np.max(np.abs(host(W[:, sl]) - Wr)) <= 2e-2 * max(1.0, np.max(np.abs(Wr))), ck
        assert np.max(np.abs(host(U[:, sl]) - Ur)) <= 2e-2 * max(1.0, np.max(np.abs(Ur))), ck
    del dK, dV, db, dg, W, U
    torch.cuda.empty_cache()


def test_int16_blockwise_c128_past_4GiB():
    """The block-wise integer inverse at C = 128 (three exponents per tile)
    with int16 codes past 2^32 bytes: 8 seeded tiles repeated."""
    C, nb = 128, 8
    A0 = base_tiles(C, nb, seed=2).astype(np.float32)
    qA, eA = oi.quantize_blocked(A0, oi.SPEC16)
    reps = (1 << 32) // (C * C * 2) // nb + 2
    n = nb * reps
    print(f"int16 C=128 past 4 GiB: {n} tiles, {n * C * C * 2 / 2**30:.2f} GiB of codes",
          flush=True)
    dq = torch.from_numpy(qA.astype(np.int16)).to("cuda").repeat(reps, 1, 1)
    de = torch.from_numpy(eA.astype(np.int32)).to("cuda").repeat(reps, 1)
    Tq, eT = G.gdn_chunk_inverse_neumann_i16(dq, de, 3, 8)
    rq, re = oi.neumann_inverse_int_blocked(qA, eA, 3, 8, oi.SPEC16)
    torch.cuda.synchronize()
    for start in (0, (reps // 2) * nb, n - nb):
        assert np.array_equal(Tq[start:start + nb].cpu().numpy().astype(np.int64), rq), start
        assert np.array_equal(eT[start:start + nb].cpu().numpy().astype(np.int64), re), start
    del dq, de, Tq, eT
    torch.cuda.empty_cache()
