"""The allocation-free layer forward (gdn_chunk_forward_noalloc) through the
C ABI, against the layer forward with a caller's workspace
(gdn_chunk_forward) on the same inputs: two calls in a row, the second on a
smaller input than the first, each equal bit for bit (both calls run the
same kernels; only where the workspace lives differs).  The scratch keeps
the first call's contents when the second starts."""

import numpy as np
import pytest
import torch

import workloads as wl

import paper_2606_06034_amd as G

pytestmark = pytest.mark.gpu


def _inputs(w, C, dt):
    Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w, C=C)
    dev = lambda x, t: torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(t)
    return (dev(Q, dt), dev(K, dt), dev(V, dt), dev(beta, torch.float32),
            dev(g, torch.float32), dev(S0, torch.float32))


def _compare(w, C, dt, inverse):
    Q, K, V, beta, g, S0 = _inputs(w, C, dt)
    print(f"noalloc vs workspace: B={w.B} H={w.H} L={w.L} C={C} {dt} {inverse}", flush=True)
    O1, S1 = G.gdn_chunk_forward(Q, K, V, beta, g, C, S0=S0, inverse=inverse)
    O2 = torch.full_like(V, float("nan"))
    S2 = torch.full_like(S0, float("nan"))
    G.gdn_chunk_forward_noalloc(Q, K, V, beta, g, C, O2, S0=S0, S_final=S2, inverse=inverse)
    torch.cuda.synchronize()
    assert torch.equal(O1, O2)
    assert torch.equal(S1, S2)
    assert torch.isfinite(O2.float()).all() and torch.isfinite(S2).all()


@pytest.mark.parametrize("inverse", ["neumann", "int16"])
def test_noalloc_two_calls_second_smaller(inverse):
    # the first call: 16 heads x 4096 tokens (1024 chunk tiles of 64, bf16;
    # 54 MiB of scratch), then 2 heads x 512 tokens (16 tiles)
    big = wl.workload("qwen35_prefill").with_(L=4096)
    small = wl.workload("qwen35_prefill").with_(L=512, H=2)
    _compare(big, 64, torch.bfloat16, inverse)
    _compare(small, 64, torch.bfloat16, inverse)


def test_noalloc_fp32_and_other_chunk_sizes():
    for C in (16, 32):
        w = wl.workload("tiny").with_(L=512, H=2, C=C)
        _compare(w, C, torch.float32, "neumann")


def test_noalloc_rejects_sizes_past_the_scratch():
    # 2428 bf16 tiles of C = 64, dk = dv = 128 need more than 128 MiB
    need = G.gdn_chunk_forward_workspace(1, 64 * 2428, 1, 128, 128, 64, torch.bfloat16)
    assert need > G.GDN_FORWARD_SCRATCH_BYTES
    w = wl.workload("qwen35_prefill").with_(L=64 * 2428, H=1)
    K = torch.zeros((1, w.L, 1, 128), dtype=torch.bfloat16, device="cuda")
    beta = torch.zeros((1, w.L, 1), dtype=torch.float32, device="cuda")
    with pytest.raises(G.GdnError) as ei:
        G.gdn_chunk_forward_noalloc(K, K, K, beta, beta, 64, torch.empty_like(K))
    assert ei.value.code == -9  # GDN_ERR_WORKSPACE
