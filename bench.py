"""Benchmark of the chunk-wise Gated DeltaNet inverse path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--C C]
                    [--path fused|inverse|fwdsub|unfused] [--no-cpu-baseline]

A step is one pass of the hot path over one batch of synthetic inputs
already resident in HBM.  The default workload is the Qwen3.5-shaped prefill
(B=1, H=16, L=8192, C=64, dk=dv=128, bf16; 2048 chunk tiles) and the default
path is the fused kernel: build A -> MatMul-only inverse T_hat(3, 8) -> W, U.

Prints ONE JSON line: throughput in chunk inverses per second, the roofline
of the dominant kernel (timed with HIP events on the stream it runs on), and
the CPU oracle timed on a bounded sample of the same workload together with
the GPU's max abs error against it on that sample.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0   # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3    # dense fp32 MFMA
METRIC = "C×C chunk inverses/sec + TFLOP/s vs MFMA peak; max abs err vs fp64 oracle"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="qwen35_prefill", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--C", type=int, default=None)
    ap.add_argument("--N", type=int, default=None)
    ap.add_argument("--S", type=int, default=None)
    ap.add_argument("--path", default="fused", choices=["fused", "inverse", "fwdsub", "unfused"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tiles", type=int, default=512)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run 10 device-to-device copies of 512 MiB (to scale HBM "
                         "byte counters) and exit")
    return ap.parse_args()


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU; --gpus {a.gpus} is not supported "
              "(tiles are independent: a multi-GPU run would shard heads, see DESIGN.md)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if a.copy_calibration:
        src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_per_copy": 512 << 20, "copies": 10}))
        return

    import paper_2606_06034_amd as G

    w = wl.workload(a.workload)
    C = a.C or w.C
    w = w.with_(C=C)
    N0, S0 = G.gdn_default_order(C)
    N = N0 if a.N is None else a.N
    S = S0 if a.S is None else a.S
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4
    n_tiles = w.B * w.H * (w.L // C)

    # ---- inputs, resident in HBM before timing
    want_v = a.path in ("fused", "unfused")
    K, beta, g, V = wl.gen_inputs(w, C=C, want_v=want_v)
    if V is None:
        V = np.zeros((w.B, w.C, w.H, w.dv), np.float32)  # unused by the timed path
    dev = lambda x, t: torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(t)
    dK, dV = dev(K, dt), dev(V, dt)
    db, dg = dev(beta, torch.float32), dev(g, torch.float32)
    dW, dU = torch.empty_like(dK), torch.empty_like(dV)
    dT = torch.empty((w.B, w.H, w.L // C, C, C), dtype=dt, device="cuda")
    dA = G.gdn_build_A(dK, db, dg, C, a_dtype=dt)
    stream = torch.cuda.current_stream()

    if a.path == "fused":
        step = lambda: G.gdn_chunk_wy_fused(dK, dV, db, dg, C, N, S, W=dW, U=dU)
    elif a.path == "unfused":
        def step():
            G.gdn_build_A(dK, db, dg, C, A=dA)
            G.gdn_chunk_inverse_neumann(dA, N, S, Tinv=dT)
            G.gdn_wy_apply(dT, dK, dV, db, C, W=dW, U=dU)
    elif a.path == "inverse":
        step = lambda: G.gdn_chunk_inverse_neumann(dA, N, S, Tinv=dT)
    else:
        step = lambda: G.gdn_chunk_inverse_fwdsub(dA, Tinv=dT)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(a.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = e0.elapsed_time(e1) / a.steps  # HIP-event time per step (one launch for fused/inverse/fwdsub)
    ms_per_step = wall * 1e3 / a.steps
    value = n_tiles / (ms_per_step * 1e-3)

    # ---- algorithmic work per launch (measurement section)
    f_inv = (N + S) * 2 * C ** 3 * n_tiles  # dense-equivalent, the paper's product count
    if C == 128:
        f_inv = (2 * (N + S) + 2) * 2 * 64 ** 3 * n_tiles
    tok = w.B * w.L * w.H
    if a.path == "fused":
        bytes_ = tok * (w.dk + w.dv) * es * 2 + tok * 8
        flops = f_inv + n_tiles * (2 * C * C * w.dk + 2 * C * C * (w.dk + w.dv))
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = "k_fused"
    elif a.path == "inverse":
        bytes_ = n_tiles * C * C * es * 2
        flops = f_inv
        peak_f = BF16_PEAK_TFLOPS if es == 2 else FP32_PEAK_TFLOPS
        ai_ridge = peak_f * 1e12 / (HBM_PEAK_GBS * 1e9)
        if flops / bytes_ >= ai_ridge:
            bound, peak, unit = "mfma", peak_f, "TFLOP/s"
            achieved = flops / (ev_ms * 1e-3) / 1e12
        else:
            bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
            achieved = bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = "k_neumann"
    elif a.path == "fwdsub":
        bytes_ = n_tiles * C * C * es * 2
        flops = n_tiles * (C ** 3 - C) // 3  # sum over i > j of (i - j) FMAs = (C^3 - C) / 6
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = "k_fwdsub"
    else:
        bytes_ = None
        flops = f_inv
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", float("nan")
        kernel = "k_build_A+k_neumann+k_wy"

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "chunk inverses/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L": w.L, "H": w.H, "C": C, "dk": w.dk,
                   "dv": w.dv, "N": N, "S": S, "tiles": n_tiles, "path": a.path,
                   "parallelism": "none (1 GPU)"},
        "tflops_dense_equiv": round(f_inv / (ev_ms * 1e-3) / 1e12, 2),
        "tflops_vs_bf16_peak": round(f_inv / (ev_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
        "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                     "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(a.path, w.name, C, N, S, (N0, S0)),
                     "kernel": kernel,
                     "kernel_ms": round(ev_ms, 6),
                     "algorithmic_bytes": bytes_, "algorithmic_flops": flops},
    }

    if not a.no_cpu_baseline and want_v:
        out["cpu_baseline"] = cpu_baseline(w, C, N, S, a, (K, beta, g, V), dK, dV, db, dg,
                                             torch, G)
    print(json.dumps(out), flush=True)


# committed rocprofv3 summaries carrying measured HBM traffic per launch
PROFILES = {("fused", "qwen35_prefill", 64): ("k_fused_qwen35_prefill.md", "pipeline.hip"),
            ("inverse", "sweep", 64): ("k_neumann_sweep_c64.md", "neumann.hip")}


def measured_traffic(path, workload, C, N, S, default_order):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary,
    or None if there is none for this launch or the kernel source changed
    since the counters were taken."""
    key = PROFILES.get((path, workload, C))
    if key is None or (N, S) != default_order:
        return None
    fname, src = key
    try:
        from paper_2606_06034_amd.csrc import build as B
        txt = open(os.path.join(ROOT, "profiles", fname)).read()
        vals = dict(l.split(": ", 1) for l in txt.splitlines()
                    if l.startswith(("traffic_bytes_per_launch:", "source_digest:")))
        if vals.get("source_digest", "").strip() != B._digest(os.path.join(B.HERE, src)):
            return None
        return int(float(vals["traffic_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None


def cpu_baseline(w, C, N, S, a, host_inputs, dK, dV, db, dg, torch, G):
    """The oracle (float64 numpy) on a bounded sample of the same workload:
    the first `cpu_sample_tiles` tiles of head (0, 0), ... ; also the GPU's
    max abs error against it on those tiles (fused path outputs)."""
    from oracle import gdn

    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    nc = w.L // C
    want = max(1, a.cpu_sample_tiles)
    heads = []
    n = 0
    for b in range(w.B):
        for h in range(w.H):
            if n >= want:
                break
            heads.append((b, h))
            n += nc
    K, beta, g, V = host_inputs
    t0 = time.perf_counter()
    Ks = np.stack([K[b, :, h] for b, h in heads], 1)[None]
    bs = np.stack([beta[b, :, h] for b, h in heads], 1)[None]
    gs = np.stack([g[b, :, h] for b, h in heads], 1)[None]
    Vs = np.stack([V[b, :, h] for b, h in heads], 1)[None]
    A = gdn.build_A(Ks, bs, gs, C)
    T = gdn.neumann_inverse_blocked(A, N, S) if C == 128 else gdn.neumann_inverse(A, N, S)
    Wr, Ur = gdn.wy_apply(T, Ks, Vs, bs, C)
    secs = time.perf_counter() - t0
    tiles = A.shape[1] * A.shape[2]
    # GPU outputs of the same tiles
    W, U, Tg = G.gdn_chunk_wy_fused(dK, dV, db, dg, C, N, S, want_T=True) if C != 128 else (None, None, None)
    err = None
    if W is not None:
        torch.cuda.synchronize()
        Wg = np.stack([W[b, :, h].float().cpu().numpy() for b, h in heads], 1)[None]
        Ug = np.stack([U[b, :, h].float().cpu().numpy() for b, h in heads], 1)[None]
        Tgs = np.stack([Tg[b, h].float().cpu().numpy() for b, h in heads], 0)[None]
        err = {"T": float(np.max(np.abs(Tgs - T))), "W": float(np.max(np.abs(Wg - Wr))),
               "U": float(np.max(np.abs(Ug - Ur)))}
    return {"value": round(tiles / secs, 1), "unit": "chunk inverses/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{tiles} tiles ({len(heads)} heads x {nc} chunks) of {w.name}: "
                      f"build A + T_hat({N},{S}) + W/U in float64 numpy, {secs:.2f} s",
            "max_abs_err_gpu_vs_oracle": err}


if __name__ == "__main__":
    main()
