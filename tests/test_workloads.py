"""Seeded input generator: storage rounding and reproducibility."""

import numpy as np
import torch

import workloads as wl


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-30, 30, 100000))).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0, -3.5]
    ours = wl.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_heads_are_independent_and_reproducible():
    w = wl.workload("tiny")
    a = wl.gen_head(w, 0, 2)
    b = wl.gen_head(w, 0, 2)
    c = wl.gen_head(w, 0, 3)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    assert not np.array_equal(a[0], c[0])
    K, beta, g, V = wl.gen_inputs(w.with_(L=128))
    assert np.array_equal(K[0, :, 2], wl.gen_head(w.with_(L=128), 0, 2)[0])


def test_distributions():
    w = wl.workload("qwen35_prefill").with_(L=1024)
    k, beta, g, v = wl.gen_head(w, 0, 0)
    assert np.allclose(np.linalg.norm(k.astype(np.float64), axis=1), 1.0, atol=1e-2)
    assert np.all((beta > 0) & (beta < 1))
    gc = g.reshape(-1, w.C)
    assert np.all(np.diff(gc, axis=1) < 0)  # strictly decaying within a chunk
    assert np.array_equal(wl.round_to_bf16(k), k)  # already bf16 values
