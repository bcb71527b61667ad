"""Benchmark of the chunk-wise Gated DeltaNet inverse path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--C C]
                    [--path fused|fused_blockwise|inverse|fwdsub|blockwise|unfused|int8|int16|
                            forward]
                    [--no-cpu-baseline]

A step is one pass of the hot path over one batch of synthetic inputs
already resident in HBM.  The default workload is the long-context stress
shape (B=1, H=32, L=131072, C=64, dk=dv=128, bf16; 65536 chunk tiles), the
largest single-GPU configuration, and the default path is the fused kernel:
build A -> MatMul-only inverse T_hat(3, 8) -> W, U.  On the fused path the
inverse alone (T_hat), the exact block-wise inverse and the forward-
substitution baseline are also timed on the same tiles (Section 4.3 compares
the inverse against forward substitution kernel for kernel).

Prints ONE JSON line: throughput in chunk inverses per second, the roofline
of the dominant kernel (timed with HIP events on the stream it runs on), and
the CPU oracle timed on one host thread on a bounded sample of the same
workload (T_hat and forward substitution; the T_hat pass also with the host
pools' default thread count) together with the GPU's max abs error against
it on that sample.

--path forward runs the whole chunk-wise Gated DeltaNet layer forward
(gdn_chunk_forward: per-chunk factors, then the state recurrence and the
output), times its two launches apart and, for context, the inverse alone
(T_hat and forward substitution) on the same chunks, so the inverse's share
of the layer can be read off.

--varlen runs the fused path (or, with --path forward, the layer forward)
over packed sequences of the serving mix: the workload's token count split
into sequences of log-uniform lengths, chunks restarting at every sequence.

--path int8 runs the low-bit path (default workload "int8": B=4, H=32,
L=16384, C=64, wide gates) in one launch: build A in fp32 -> per-tile INT8
quantiser -> integer inverse T_hat(3, 8); the same path as three launches
is timed beside it for context.  --path int16 does the same with 16-bit
codes (each product four int8 MFMAs over the codes' limbs).
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
INT8_PEAK_TOPS = 5000.0     # dense int8 MFMA
METRIC = "C×C chunk inverses/sec + TFLOP/s vs MFMA peak; max abs err vs fp64 oracle"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="long_context", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--C", type=int, default=None)
    ap.add_argument("--N", type=int, default=None)
    ap.add_argument("--S", type=int, default=None)
    ap.add_argument("--path", default="fused", choices=["fused", "fused_blockwise", "inverse", "fwdsub", "blockwise",
                             "unfused", "int8", "int16", "forward"])
    ap.add_argument("--exact", action="store_true",
                    help="--path forward / --varlen: the exact block-wise inverse instead of T_hat(N, S)")
    ap.add_argument("--inverse", default=None, choices=["neumann", "exact", "int16", "int8"],
                    help="--path forward: the inverse inside the layer (int16 / int8: the "
                         "integer T_hat(N, S), the quantised GDN layer)")
    ap.add_argument("--varlen", action="store_true",
                    help="--path fused over packed sequences of a serving mix of lengths "
                         "(log-uniform 1..4096, B*L tokens in total, ragged last chunks)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-same-shape", action="store_true",
                    help="fused path: skip timing the inverse-only kernels on the same tiles")
    ap.add_argument("--cpu-sample-tiles", type=int, default=2048,
                    help="tiles of the workload the CPU oracle runs on (whole heads)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat oracle passes over the sample until this much time has passed")
    ap.add_argument("--error-grid", action="store_true",
                    help="instead of timing: max |T_hat(N, S) - X| and per-tile SNR for "
                         "N = 1..6, S = 0..16 against the exact inverse X (fp64 triangular "
                         "solve on the host), workload and stress tiles; fp32, bf16 and the "
                         "integer modes (split and plain forms)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run 10 device-to-device copies of 512 MiB (to scale HBM "
                         "byte counters) and exit")
    return ap.parse_args()


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py: runs on exactly one GPU; --gpus {a.gpus} is not supported "
              "(tiles are independent: several GPUs would each take a share of the heads)",
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

    if a.error_grid:
        print(json.dumps(error_grid(a, G, torch)), flush=True)
        return

    low = a.path in ("int8", "int16")
    if low and "--workload" not in sys.argv:
        a.workload = "int8"
    w = wl.workload(a.workload)
    C = a.C or w.C
    w = w.with_(C=C)
    N0, S0 = G.gdn_default_order(C)
    N = N0 if a.N is None else a.N
    S = S0 if a.S is None else a.S
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4
    n_tiles = w.B * w.H * (w.L // C)

    if a.path == "forward" and a.varlen:
        return bench_forward_varlen(a, w, C, N, S, G, torch)
    if a.path == "forward":
        return bench_forward(a, w, C, N, S, (N0, S0), G, torch)
    if a.varlen:
        return bench_varlen(a, w, C, N, S, G, torch)

    # ---- inputs, resident in HBM before timing
    want_v = a.path in ("fused", "fused_blockwise", "unfused")
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
    elif a.path == "fused_blockwise":
        step = lambda: G.gdn_chunk_wy_fused_blockwise(dK, dV, db, dg, C, W=dW, U=dU)
    elif a.path == "unfused":
        def step():
            G.gdn_build_A(dK, db, dg, C, A=dA)
            G.gdn_chunk_inverse_neumann(dA, N, S, Tinv=dT)
            G.gdn_wy_apply(dT, dK, dV, db, C, W=dW, U=dU)
    elif a.path == "inverse":
        step = lambda: G.gdn_chunk_inverse_neumann(dA, N, S, Tinv=dT)
    elif low:
        qdt, sfx = (torch.int8, "i8") if a.path == "int8" else (torch.int16, "i16")
        dTq = torch.empty((w.B, w.H, w.L // C, C, C), dtype=qdt, device="cuda")
        fused = getattr(G, f"gdn_chunk_inverse_neumann_{sfx}_fused")
        # C = 128: block-wise, three exponents per tile
        deT = torch.empty((n_tiles, 3) if C == 128 else n_tiles, dtype=torch.int32, device="cuda")
        step = lambda: fused(dK, db, dg, C, N, S, Tq=dTq, eT=deT)
    elif a.path == "blockwise":
        step = lambda: G.gdn_chunk_inverse_blockwise(dA, Tinv=dT)
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
    if low:  # context: the same path as three launches
        quant = getattr(G, f"gdn_quantize_tiles_{sfx}")
        inv = getattr(G, f"gdn_chunk_inverse_neumann_{sfx}")
        dA32 = G.gdn_build_A(dK, db, dg, C, a_dtype=torch.float32)
        dAq = torch.empty(dA32.shape, dtype=qdt, device="cuda")
        deA = torch.empty((n_tiles, 3) if C == 128 else n_tiles, dtype=torch.int32, device="cuda")
        dTq2, deT2 = torch.empty_like(dAq), torch.empty_like(deA)
        stages = [lambda: G.gdn_build_A(dK, db, dg, C, A=dA32),
                  lambda: quant(dA32, Aq=dAq, eA=deA),
                  lambda: inv(dAq, deA, N, S, Tq=dTq2, eT=deT2)]
        if C < 128:
            # the integer forward-substitution baseline on the same codes
            fwd_int = getattr(G, f"gdn_chunk_inverse_fwdsub_{sfx}")
            dTq3, deT3 = torch.empty_like(dAq), torch.empty_like(deA)
            stages.append(lambda: fwd_int(dAq, deA, Tq=dTq3, eT=deT3))
        stage_ms = []
        for fn in stages:
            fn()
            e0.record(stream)
            for _ in range(a.steps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            stage_ms.append(e0.elapsed_time(e1) / a.steps)
        del dA32, dAq

    # ---- algorithmic work per launch: the per-tile bytes and operations of each kernel
    f_inv = (N + S) * 2 * C ** 3 * n_tiles  # dense-equivalent, the paper's product count
    f_useful = (N + S) * C * (C + 1) * (C + 2) // 3 * n_tiles
    if C == 128:
        f_inv = (2 * (N + S) + 2) * 2 * 64 ** 3 * n_tiles
        # two 64-blocks, then the merge's two products of a full and a lower 64-block
        f_useful = (2 * (N + S) * 64 * 65 * 66 // 3 + 2 * 64 * 64 * 65) * n_tiles
    tok = w.B * w.L * w.H
    if a.path in ("fused", "fused_blockwise"):
        bytes_ = tok * (w.dk + w.dv) * es * 2 + tok * 8
        flops = f_inv + n_tiles * (2 * C * C * w.dk + 2 * C * C * (w.dk + w.dv))
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = "k_fused" if C < 128 else "k_fused128"
    elif a.path == "inverse":
        # The bound is chosen from the method's own work: the non-zero
        # (lower-triangular) part of its N + S products.  At C = 64 that is
        # 61 FLOP per byte of bf16 tile IO, below the bf16 ridge (312), so
        # the inverse alone is HBM-bound; the dense-equivalent rate is
        # reported beside it, labelled as such.
        bytes_ = n_tiles * C * C * es * 2
        flops = f_useful
        peak_f = BF16_PEAK_TFLOPS if es == 2 else FP32_PEAK_TFLOPS
        ai_ridge = peak_f * 1e12 / (HBM_PEAK_GBS * 1e9)
        if flops / bytes_ >= ai_ridge:
            bound, peak, unit = "mfma", peak_f, "TFLOP/s"
            achieved = flops / (ev_ms * 1e-3) / 1e12
        else:
            bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
            achieved = bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = "k_neumann" if C < 128 else "k_neumann128"
    elif a.path in ("fwdsub", "blockwise"):
        # the exact inverse: tile in, tile out; the arithmetic of substitution
        bytes_ = n_tiles * C * C * es * 2
        flops = n_tiles * (C ** 3 - C) // 3  # sum over i > j of (i - j) FMAs = (C^3 - C) / 6
        bound, peak, unit, achieved = "hbm", HBM_PEAK_GBS, "GB/s", bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = "k_fwdsub" if a.path == "fwdsub" else "k_blockwise"
    elif low:
        # K (dk per token) and beta, g in; T_hat codes and exponents out.  An
        # INT16 product is four int8 MFMA products over the codes' limbs.
        # C = 128: three exponents per tile, 2 (N + S) + 2 products of 64-blocks.
        # The bound is chosen from the method's own work, as for the float
        # inverse: the non-zero part of the N + S products, in int8 MFMA
        # operations (an INT16 product is four limb products).  At C = 64
        # that is 48 (INT8) and 160 (INT16) operations per byte, below the
        # int8 ridge (625): HBM-bound.
        qb = 1 if a.path == "int8" else 2
        bytes_ = tok * (w.dk * es + 8) + n_tiles * (C * C * qb + 4 * (3 if C == 128 else 1))
        flops = f_useful * qb * qb
        if flops / bytes_ >= INT8_PEAK_TOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
            bound, peak, unit = "mfma", INT8_PEAK_TOPS, "TOP/s"
            achieved = flops / (ev_ms * 1e-3) / 1e12
        else:
            bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
            achieved = bytes_ / (ev_ms * 1e-3) / 1e9
        kernel = f"k_inverse_{sfx}_fused" if C < 128 else "k_inverse_int128_fused"
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
        # the method's own work: the non-zero (lower-triangular) part of the
        # N + S products, per tile and as a rate of the timed kernel; the
        # dense-equivalent count (every product a full C x C x C one) beside it
        "flop_per_tile": {"useful": f_useful // n_tiles, "dense_equiv": f_inv // n_tiles},
        "tflops_useful": round(f_useful / (ev_ms * 1e-3) / 1e12, 2),
        "tflops_useful_vs_bf16_peak": round(f_useful / (ev_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
        "tflops_dense_equiv": round(f_inv / (ev_ms * 1e-3) / 1e12, 2),
        "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                     "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(a.path, w.name, C, N, S, (N0, S0)),
                     "kernel": kernel,
                     "kernel_ms": round(ev_ms, 6),
                     "algorithmic_bytes": bytes_, "algorithmic_flops": flops},
    }

    if a.path in ("fused", "fused_blockwise") and not a.no_same_shape:
        out["same_shape_inverse"] = same_shape_inverse(a, G, torch, stream, dA, dT, n_tiles, C, N,
                                                       S, es, f_useful)
    if low:
        # int8 MFMA operations: useful (the non-zero part of the N + S
        # products, the roofline's count) and dense-equivalent
        dense = f_inv * qb * qb
        out["int8_ops_per_tile"] = {"useful": flops // n_tiles, "dense_equiv": dense // n_tiles}
        out["tops_useful"] = round(flops / (ev_ms * 1e-3) / 1e12, 2)
        out["tops_useful_vs_int8_peak"] = round(flops / (ev_ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4)
        out["tops_dense_equiv"] = round(dense / (ev_ms * 1e-3) / 1e12, 2)
        for k in ("flop_per_tile", "tflops_useful", "tflops_useful_vs_bf16_peak",
                  "tflops_dense_equiv"):
            del out[k]
        out["config"]["three_launch_ms"] = {"build_A_f32": round(stage_ms[0], 6),
                                            "quantize": round(stage_ms[1], 6),
                                            "inverse_" + sfx: round(stage_ms[2], 6)}
        if C < 128:
            out["config"]["fwdsub_" + sfx + "_ms"] = round(stage_ms[3], 6)
        out["dtype"] = sfx
        if not a.no_cpu_baseline:
            out["cpu_baseline"] = cpu_baseline_int(w, C, N, S, a, (K, beta, g), dTq, deT,
                                                   torch, G, sfx)
    elif not a.no_cpu_baseline and a.path in ("fused", "unfused"):
        out["cpu_baseline"] = cpu_baseline(w, C, N, S, a, (K, beta, g, V), dK, dV, db, dg,
                                             torch, G)
    print(json.dumps(out), flush=True)


def same_shape_inverse(a, G, torch, stream, dA, dT, n_tiles, C, N, S, es, f_useful):
    """The inverse alone on the step's own tiles (A built once in the IO
    dtype): T_hat(N, S), the exact block-wise inverse and the forward-
    substitution baseline, each timed per launch without the host's launch
    overhead (_kernel_time); tile IO bytes and the useful product work per
    launch."""
    steps = max(1, a.steps // 2)
    res = {}
    for name, fn in (("neumann", lambda: G.gdn_chunk_inverse_neumann(dA, N, S, Tinv=dT)),
                     ("blockwise", lambda: G.gdn_chunk_inverse_blockwise(dA, Tinv=dT)),
                     ("fwdsub", lambda: G.gdn_chunk_inverse_fwdsub(dA, Tinv=dT))):
        ms, how = _kernel_time(fn, dT, steps, stream, torch)
        gbs = n_tiles * C * C * es * 2 / (ms * 1e-3) / 1e9
        res[name] = {"ms": round(ms, 6), "chunk_inverses_per_s": round(n_tiles / (ms * 1e-3), 1),
                     "GB/s": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                     "timing": how}
    res["neumann"]["tflops_useful"] = round(f_useful / (res["neumann"]["ms"] * 1e-3) / 1e12, 2)
    res["fwdsub_time_over_neumann"] = round(res["fwdsub"]["ms"] / res["neumann"]["ms"], 3)
    res["blockwise_time_over_neumann"] = round(res["blockwise"]["ms"] / res["neumann"]["ms"], 3)
    return res


def _kernel_time(fn, out, steps, stream, torch):
    """Time per launch (ms) of fn, whose result lands in `out`, without the
    host's per-call launch overhead (which exceeds a launch of a few
    thousand tiles): `steps` calls captured in one HIP graph, replayed and
    timed with HIP events.  Two replays, each with eager work after it, are
    first checked bit for bit against an eager call's result; if capture
    fails or a replay differs, the eager per-call time (_time) is returned
    instead.  Returns (ms, "graph" | "eager")."""
    fn()
    torch.cuda.synchronize()
    ref = out.clone()
    try:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            for _ in range(steps):
                fn()
        for _ in range(2):
            out.zero_()
            g.replay()
            torch.cuda.synchronize()
            if not torch.equal(out, ref):
                raise RuntimeError("a graph replay differs from the eager call")
            fn()
            torch.cuda.synchronize()
        cur = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        g.replay()
        e1.record(cur)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps, "graph"
    except Exception:  # noqa: BLE001 -- any capture problem: time eagerly
        torch.cuda.synchronize()
        return _time(fn, steps, stream, torch), "eager"


def _time(fn, steps, stream, torch):
    """HIP-event time per call (ms) on `stream`, after one untimed call."""
    fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def bench_forward(a, w, C, N, S, default_order, G, torch):
    """The layer forward (gdn_chunk_forward) on the workload's sizes."""
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4
    n_tiles = w.B * w.H * (w.L // C)
    tok = w.B * w.L * w.H
    Q, K, V, beta, g, S0 = wl.gen_forward_inputs(w, C=C)
    dev = lambda x, t: torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(t)
    dQ, dK, dV = dev(Q, dt), dev(K, dt), dev(V, dt)
    db, dg, dS0 = dev(beta, torch.float32), dev(g, torch.float32), dev(S0, torch.float32)
    host = (Q, K, V, beta, g, S0) if not a.no_cpu_baseline else None
    del Q, K, V
    dO = torch.empty_like(dV)
    dSf = torch.empty_like(dS0)
    ws = torch.empty(G.gdn_chunk_forward_workspace(w.B, w.L, w.H, w.dk, w.dv, C, dt),
                     dtype=torch.uint8, device="cuda")
    scale = w.dk ** -0.5
    stream = torch.cuda.current_stream()
    inv_mode = a.inverse or ("exact" if a.exact else "neumann")
    step = lambda: G.gdn_chunk_forward(dQ, dK, dV, db, dg, C, S0=dS0, N=N, S=S,
                                       inverse=inv_mode, scale=scale, O=dO, S_final=dSf,
                                       workspace=ws)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(a.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = e0.elapsed_time(e1) / a.steps
    ms_per_step = wall * 1e3 / a.steps
    # the two launches apart, and the inverse alone on the same chunks
    prep_ms = _time(lambda: G.gdn_chunk_forward_prepare(dQ, dK, dV, db, dg, C, ws, N=N, S=S,
                                                        inverse=inv_mode), a.steps, stream, torch)
    state_ms = _time(lambda: G.gdn_chunk_forward_state(dQ, dg, C, ws, w.dv, S0=dS0, scale=scale,
                                                       O=dO, S_final=dSf), a.steps, stream, torch)
    # how far the layer's output moves from the layer with the exact inverse
    # (the effect of the approximation, and of the integer codes, on O)
    dev_vs_exact = None
    if inv_mode != "exact":
        Oe, Se = G.gdn_chunk_forward(dQ, dK, dV, db, dg, C, S0=dS0, inverse="exact", scale=scale,
                                     workspace=ws)
        torch.cuda.synchronize()
        dev_vs_exact = {"O": float(((dO.float() - Oe.float()).abs().max() /
                                    Oe.float().abs().max()).item()),
                        "S_final": float(((dSf - Se).abs().max() / Se.abs().max()).item())}
        del Oe, Se
    del ws
    dA = G.gdn_build_A(dK, db, dg, C, a_dtype=dt)
    dT = torch.empty_like(dA)
    inv_ms, inv_how = _kernel_time(lambda: G.gdn_chunk_inverse_neumann(dA, N, S, Tinv=dT), dT,
                                   a.steps, stream, torch)
    fws_ms, _ = _kernel_time(lambda: G.gdn_chunk_inverse_fwdsub(dA, Tinv=dT), dT,
                             max(1, a.steps // 4), stream, torch)
    del dA, dT
    # algorithmic bytes per launch
    # workspace: W, U, K^T and the masked Q K^T per chunk, written once, read once
    ws_b = G.gdn_chunk_forward_workspace(w.B, w.L, w.H, w.dk, w.dv, C, dt)
    prep_bytes = tok * (2 * w.dk + w.dv) * es + tok * 8 + ws_b
    state_bytes = ws_b + tok * (w.dk + w.dv) * es + tok * 4 + 2 * w.B * w.H * w.dk * w.dv * 4
    if state_ms >= prep_ms:
        kernel, kms, kbytes = "k_fwd_state", state_ms, state_bytes
    else:
        kernel, kms, kbytes = "k_fwd_chunk", prep_ms, prep_bytes
    achieved = kbytes / (kms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(n_tiles / (ms_per_step * 1e-3), 1),
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
                   "dv": w.dv, "N": N, "S": S, "tiles": n_tiles, "path": "forward",
                   "inverse": {"exact": "exact block-wise", "neumann": f"T_hat({N},{S})",
                               "int16": f"INT16 T_hat({N},{S})",
                               "int8": f"INT8 T_hat({N},{S})"}[inv_mode],
                   "parallelism": "none (1 GPU)"},
        "tokens_per_s": round(w.B * w.L / (ms_per_step * 1e-3), 1),
        "layer_ms": round(ev_ms, 6),
        "prepare_ms": round(prep_ms, 6),
        "state_ms": round(state_ms, 6),
        "inverse_alone_ms": round(inv_ms, 6),
        "inverse_alone_timing": inv_how,
        "fwdsub_alone_ms": round(fws_ms, 6),
        "inverse_share_of_layer": round(inv_ms / ev_ms, 4),
        "fwdsub_share_if_swapped_in": round(fws_ms / (ev_ms - inv_ms + fws_ms), 4),
        "rel_dev_vs_exact_inverse_layer": dev_vs_exact,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": (measured_traffic("forward", w.name, C, N, S, default_order)
                                 if kernel == "k_fwd_state" and inv_mode == "neumann" else None),
                     "kernel": kernel, "kernel_ms": round(kms, 6),
                     "algorithmic_bytes": kbytes},
    }
    if host is not None:
        out["cpu_baseline"] = cpu_baseline_forward(w, C, N, S, a, host, dO, dSf, scale, inv_mode)
    print(json.dumps(out), flush=True)


def bench_forward_varlen(a, w, C, N, S, G, torch):
    """The layer forward over packed sequences (gdn_chunk_forward_varlen) on
    the serving mix of the workload's token count."""
    inv_mode = a.inverse or ("exact" if a.exact else "neumann")
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4
    lengths = wl.varlen_lengths(w.B * w.L)
    wv = w.with_(B=1)
    K, beta, g, V, cu, Q = wl.gen_varlen(wv, lengths, C=C, want_q=True)
    S0 = np.stack([np.stack([wl.gen_state(wv, s, h) for h in range(w.H)])
                   for s in range(len(lengths))])
    T = int(cu[-1])
    dev = lambda x, t: torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(t)
    dQ, dK, dV = dev(Q, dt), dev(K, dt), dev(V, dt)
    db, dg, dS0 = dev(beta, torch.float32), dev(g, torch.float32), dev(S0, torch.float32)
    tables = G.gdn_varlen_tables(cu, C)
    n_chunks = tables[2]
    n_tiles = n_chunks * w.H
    dO, dSf = torch.empty_like(dV), torch.empty_like(dS0)
    ws = torch.empty(G.gdn_chunk_forward_workspace(1, n_chunks * C, w.H, w.dk, w.dv, C, dt),
                     dtype=torch.uint8, device="cuda")
    scale = w.dk ** -0.5
    stream = torch.cuda.current_stream()
    step = lambda: G.gdn_chunk_forward_varlen(dQ, dK, dV, db, dg, tables, C, S0=dS0, N=N, S=S,
                                              inverse=inv_mode, scale=scale, O=dO, S_final=dSf,
                                              workspace=ws)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(a.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = e0.elapsed_time(e1) / a.steps
    ms_per_step = wall * 1e3 / a.steps
    tok = T * w.H
    ws_b = G.gdn_chunk_forward_workspace(1, n_chunks * C, w.H, w.dk, w.dv, C, dt)
    layer_bytes = (tok * (2 * w.dk + w.dv) * es + tok * 8 + 2 * ws_b + tok * (w.dk + w.dv) * es
                   + tok * 4 + 2 * len(lengths) * w.H * w.dk * w.dv * 4)
    achieved = layer_bytes / (ev_ms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(n_tiles / (ms_per_step * 1e-3), 1),
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
        "config": {"workload": w.name + " serving mix", "tokens": T, "sequences": len(lengths),
                   "ragged_sequences": int(sum(1 for x in lengths if x % C)), "H": w.H, "C": C,
                   "dk": w.dk, "dv": w.dv, "N": N, "S": S, "tiles": n_tiles,
                   "path": "forward varlen",
                   "inverse": {"exact": "exact block-wise", "neumann": f"T_hat({N},{S})",
                               "int16": f"INT16 T_hat({N},{S})",
                               "int8": f"INT8 T_hat({N},{S})"}[inv_mode],
                   "parallelism": "none (1 GPU)"},
        "tokens_per_s": round(T / (ms_per_step * 1e-3), 1),
        "layer_ms": round(ev_ms, 6),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "k_fwd_chunk + k_fwd_state (one call)",
                     "kernel_ms": round(ev_ms, 6), "algorithmic_bytes": layer_bytes},
    }
    if not a.no_cpu_baseline:
        from oracle import gdn, varlen
        from oracle import int8 as oi
        inv = {"exact": gdn.forward_substitution_inverse,
               "neumann": lambda A: gdn.neumann_inverse(A, N, S),
               "int16": lambda A: oi.dequantized_inverse(A, N, S, oi.SPEC16, C=C),
               "int8": lambda A: oi.dequantized_inverse(A, N, S, oi.SPEC8, C=C)}[inv_mode]
        ns, chunks, t_end = 0, 0, 0
        while ns < len(lengths) and chunks < max(1, a.cpu_sample_tiles // w.H):
            chunks += -(-lengths[ns] // C)
            t_end = int(cu[ns + 1])
            ns += 1
        sub = lambda x: x[:, :t_end]
        cu_s = cu[:ns + 1]
        with _one_thread():
            passes, t0 = 0, time.perf_counter()
            while True:
                Or, Sr = varlen.forward_varlen_chunked(sub(Q), sub(K), sub(V), sub(beta), sub(g),
                                                       cu_s, C, S0[:ns], scale, inv)
                passes += 1
                secs = time.perf_counter() - t0
                if secs >= a.cpu_seconds:
                    break
        torch.cuda.synchronize()
        Og = dO[:, :t_end].float().cpu().numpy()
        Sg = dSf[:ns].cpu().numpy()
        out["cpu_baseline"] = {
            "value": round(chunks * w.H * passes / secs, 1), "unit": "chunk inverses/s",
            "cores": 1, "kind": "oracle", "cpu_model": _cpu_model(),
            "sample": f"the first {ns} sequences ({t_end} tokens, {chunks} chunks per head, "
                      f"{w.H} heads), {passes} passes of the packed chunk-wise forward in "
                      f"float64 numpy on one thread ({inv_mode} inverse), {secs:.2f} s",
            "max_abs_err_gpu_vs_oracle": {"O": float(np.max(np.abs(Og - Or))),
                                          "S_final": float(np.max(np.abs(Sg - Sr)))}}
    print(json.dumps(out), flush=True)


def bench_varlen(a, w, C, N, S, G, torch):
    """The fused path over packed sequences (gdn_chunk_wy_fused_varlen)."""
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4
    lengths = wl.varlen_lengths(w.B * w.L)
    K, beta, g, V, cu = wl.gen_varlen(w.with_(B=1), lengths, C=C)
    T = int(cu[-1])
    dev = lambda x, t: torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(t)
    dK, dV, db, dg = dev(K, dt), dev(V, dt), dev(beta, torch.float32), dev(g, torch.float32)
    tables = G.gdn_varlen_tables(cu, C)
    n_chunks = tables[2]
    n_tiles = n_chunks * w.H
    dW, dU = torch.empty_like(dK), torch.empty_like(dV)
    stream = torch.cuda.current_stream()
    step = lambda: G.gdn_chunk_wy_fused_varlen(dK, dV, db, dg, tables, C, N=N, S=S,
                                               exact=a.exact, W=dW, U=dU)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(a.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = e0.elapsed_time(e1) / a.steps
    ms_per_step = wall * 1e3 / a.steps
    tok = T * w.H
    bytes_ = tok * (w.dk + w.dv) * es * 2 + tok * 8  # K, V in; W, U out; beta, g
    achieved = bytes_ / (ev_ms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(n_tiles / (ms_per_step * 1e-3), 1),
        "unit": "chunk inverses/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name + " packed serving mix", "sequences": len(lengths),
                   "tokens": T, "H": w.H, "C": C, "dk": w.dk, "dv": w.dv, "N": N, "S": S,
                   "chunks": n_chunks, "ragged_chunks": int(sum(1 for x in lengths if x % C)),
                   "tiles": n_tiles, "path": "fused_varlen",
                   "inverse": "exact block-wise" if a.exact else f"T_hat({N},{S})",
                   "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": ("k_fused128" if C == 128 else "k_fused") + " (packed)",
                     "kernel_ms": round(ev_ms, 6),
                     "algorithmic_bytes": bytes_},
    }
    if not a.no_cpu_baseline:
        from oracle import gdn, varlen

        # whole sequences from the start up to ~cpu_sample_tiles chunk tiles
        nseq, tiles = 0, 0
        while nseq < len(lengths) and tiles < a.cpu_sample_tiles:
            tiles += -(-lengths[nseq] // C) * w.H
            nseq += 1
        te = int(cu[nseq])
        def blocked_padded(A):
            # C = 128: the two 64-blocks of the tile padded with tokens that
            # write nothing, the m x m inverse in its top left
            m = A.shape[-1]
            P = np.zeros(A.shape[:-2] + (C, C))
            P[..., :m, :m] = A
            return gdn.neumann_inverse_blocked(P, N, S)[..., :m, :m]

        inv = (gdn.forward_substitution_inverse if a.exact else
               blocked_padded if C == 128 else (lambda A: gdn.neumann_inverse(A, N, S)))
        with _one_thread():
            passes, t0 = 0, time.perf_counter()
            while True:
                Wr, Ur, _ = varlen.wy_varlen(K[:, :te], V[:, :te], beta[:, :te], g[:, :te],
                                             cu[:nseq + 1], C, inverse=inv)
                passes += 1
                secs = time.perf_counter() - t0
                if secs >= a.cpu_seconds:
                    break
        torch.cuda.synchronize()
        err = {"W": float(np.max(np.abs(dW[:, :te].float().cpu().numpy() - Wr))),
               "U": float(np.max(np.abs(dU[:, :te].float().cpu().numpy() - Ur)))}
        out["cpu_baseline"] = {"value": round(tiles * passes / secs, 1), "unit": "chunk inverses/s",
                               "cores": 1, "kind": "oracle", "cpu_model": _cpu_model(),
                               "sample": f"the first {nseq} sequences ({te} tokens, {tiles} chunk "
                                         f"tiles), {passes} passes in float64 numpy on one "
                                         f"thread, {secs:.2f} s",
                               "max_abs_err_gpu_vs_oracle": err}
    print(json.dumps(out), flush=True)


def cpu_baseline_forward(w, C, N, S, a, host, dO, dSf, scale, inv_mode="neumann"):
    """The forward oracle (float64 numpy, chunk-wise form) on whole heads of
    the same workload, passes repeated until `cpu_seconds` have elapsed, and
    the GPU's max abs error against it on those heads."""
    from oracle import gdn, gdn_forward as fwd

    Q, K, V, beta, g, S0 = host
    nc = w.L // C
    heads = [(b, h) for b in range(w.B) for h in range(w.H)][:max(1, a.cpu_sample_tiles // nc)]
    pick = lambda x: np.stack([x[b, :, h] for b, h in heads], 1)[None].astype(np.float64)
    Qs, Ks, Vs, bs, gs = (pick(x) for x in (Q, K, V, beta, g))
    S0s = np.stack([S0[b, h] for b, h in heads], 0)[None].astype(np.float64)
    from oracle import int8 as oi
    inv = {"exact": gdn.forward_substitution_inverse,
           "neumann": lambda A: gdn.neumann_inverse(A, N, S),
           "int16": lambda A: oi.dequantized_inverse(A, N, S, oi.SPEC16),
           "int8": lambda A: oi.dequantized_inverse(A, N, S, oi.SPEC8)}[inv_mode]
    with _one_thread():
        passes, t0 = 0, time.perf_counter()
        while True:
            Or, Sr = fwd.gdn_chunked(Qs, Ks, Vs, bs, gs, C, S0s, scale=scale, inverse=inv)
            passes += 1
            secs = time.perf_counter() - t0
            if secs >= a.cpu_seconds:
                break
    tiles = len(heads) * nc * passes
    Og = np.stack([dO[b, :, h].float().cpu().numpy() for b, h in heads], 1)[None]
    Sg = np.stack([dSf[b, h].float().cpu().numpy() for b, h in heads], 0)[None]
    return {"value": round(tiles / secs, 1), "unit": "chunk inverses/s", "cores": 1,
            "kind": "oracle", "cpu_model": _cpu_model(),
            "sample": f"{len(heads)} heads x {nc} chunks of {w.name}, {passes} passes of the "
                      f"chunk-wise forward in float64 numpy on one thread ({inv_mode} "
                      f"inverse), {secs:.2f} s",
            "max_abs_err_gpu_vs_oracle": {"O": float(np.max(np.abs(Og - Or))),
                                          "S_final": float(np.max(np.abs(Sg - Sr)))}}


# committed rocprofv3 summaries carrying measured HBM traffic per launch
PROFILES = {("fused", "qwen35_prefill", 64): ("k_fused_qwen35_prefill.md", "pipeline.hip"),
            ("fused", "long_context", 64): ("k_fused_long_context.md", "pipeline.hip"),
            ("fused", "sweep", 128): ("k_fused128_sweep_c128.md", "pipeline.hip"),
            ("inverse", "sweep", 64): ("k_neumann_sweep_c64.md", "neumann.hip"),
            ("int8", "int8", 64): ("k_inverse_i8_fused_int8.md", "int8.hip"),
            ("int16", "int8", 64): ("k_inverse_i16_fused_int8.md", "int16.hip"),
            ("int8", "int8", 128): ("k_inverse_int128_fused_i8_int8.md", "int8.hip"),
            ("int16", "int8", 128): ("k_inverse_int128_fused_i16_int8.md", "int16.hip"),
            ("forward", "qwen35_prefill", 64): ("k_fwd_state_qwen35_prefill.md", "forward.hip")}


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
    whole heads (0, 0), (0, 1), ... up to `cpu_sample_tiles` tiles, passes
    repeated until `cpu_seconds` have elapsed; also the GPU's max abs error
    against it on those tiles (fused path outputs)."""
    from oracle import gdn

    cores = _threads()
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
    Ks = np.stack([K[b, :, h] for b, h in heads], 1)[None]
    bs = np.stack([beta[b, :, h] for b, h in heads], 1)[None]
    gs = np.stack([g[b, :, h] for b, h in heads], 1)[None]
    Vs = np.stack([V[b, :, h] for b, h in heads], 1)[None]

    def one_pass():
        A = gdn.build_A(Ks, bs, gs, C)
        T = gdn.neumann_inverse_blocked(A, N, S) if C == 128 else gdn.neumann_inverse(A, N, S)
        Wr, Ur = gdn.wy_apply(T, Ks, Vs, bs, C)
        return A, T, Wr, Ur

    with _one_thread():
        passes, t0 = 0, time.perf_counter()
        while True:
            A, T, Wr, Ur = one_pass()
            passes += 1
            secs = time.perf_counter() - t0
            if secs >= a.cpu_seconds:
                break
    tiles = A.shape[1] * A.shape[2] * passes
    n_sample = A.shape[1] * A.shape[2]

    def rate(fn, seconds):
        k, t1 = 0, time.perf_counter()
        while True:
            fn()
            k += 1
            dt_ = time.perf_counter() - t1
            if dt_ >= seconds:
                return round(n_sample * k / dt_, 1), k, dt_
    # the same sample with the host pools' default thread count, and the
    # exact inverse by forward substitution (the baseline the paper compares
    # against) on one thread
    all_threads = rate(one_pass, a.cpu_seconds / 2)
    with _one_thread():
        fws = rate(lambda: gdn.forward_substitution_inverse(A), a.cpu_seconds / 2)
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
    return {"value": round(tiles / secs, 1), "unit": "chunk inverses/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{len(heads)} heads x {nc} chunks of {w.name} ({tiles // passes} "
                      f"tiles), {passes} passes: build A + T_hat({N},{S}) + W/U in float64 "
                      f"numpy on one thread, {secs:.2f} s",
            "cpu_model": _cpu_model(),
            "all_threads": {"value": all_threads[0], "threads": cores,
                            "passes": all_threads[1], "seconds": round(all_threads[2], 2)},
            "fwdsub_oracle": {"value": fws[0], "cores": 1, "passes": fws[1],
                              "seconds": round(fws[2], 2),
                              "what": "exact inverse by forward substitution on the same A"},
            "max_abs_err_gpu_vs_oracle": err}


def _one_thread():
    """Host BLAS/OpenMP pools limited to one thread: the oracle's products
    are small (C x C tiles), so extra threads add nothing, and one thread is
    the core count it is reported with."""
    from threadpoolctl import threadpool_limits
    return threadpool_limits(limits=1)


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return None


def error_grid(a, G, torch):
    """Approximation error of T_hat(N, S) against X = (I + A)^-1 per order.

    Tiles: the first two heads of the sweep workload at each C, and two
    stress heads (shared key direction, slow decay; |A| up to ~0.5).  A is
    built on the GPU in fp32; X is its exact inverse from an fp64
    triangular solve on the host (scipy, per tile); bf16 mode inverts A
    rounded to bf16; int16 / int8 quantise A (per tile, per block at
    C = 128) and run the integer inverse, dequantised, in the split form
    (unit diagonal outside the codes, Section 3.2's mitigation of the
    powers' dynamic range) and, at C <= 64, the plain form (diagonal inside
    every tensor: "int16_plain", "int8_plain").  Per (C, set, dtype, N, S):
    max abs error over tiles and the per-tile SNR
    10 log10(|X|_F^2 / |X - T_hat|_F^2), mean and worst."""
    from scipy.linalg import solve_triangular
    Cs = [a.C] if a.C else [16, 32, 64, 128]
    out = {"metric": "approximation error of T_hat(N, S) vs exact inverse", "grid": []}
    for C in Cs:
        w = wl.workload("sweep").with_(C=C, B=1, H=2)
        sets = {"workload": wl.gen_inputs(w, C=C, want_v=False)[:3]}
        heads = [wl.gen_stress_head(4096, w.dk, C, seed=900 + h) for h in range(2)]
        sets["stress"] = tuple(wl.as_blhd(*[x[i] for x in heads]) for i in range(3))
        lim = (64 if C == 128 else C) - 1
        for name, (K, beta, g) in sets.items():
            dK = torch.from_numpy(np.ascontiguousarray(K)).to("cuda")
            db = torch.from_numpy(np.ascontiguousarray(beta)).to("cuda")
            dg = torch.from_numpy(np.ascontiguousarray(g)).to("cuda")
            A32 = G.gdn_build_A(dK, db, dg, C, a_dtype=torch.float32)
            Ah = A32.cpu().double().numpy().reshape(-1, C, C)
            eye = np.eye(C)
            Xh = np.stack([solve_triangular(eye + t, eye, lower=True, unit_diagonal=True)
                           for t in Ah])
            X = torch.from_numpy(Xh.reshape(A32.shape)).to("cuda")
            xn = (X ** 2).sum(dim=(-1, -2))
            # the integer modes: quantised per tile (per block at C = 128), the
            # integer T_hat(N, S), dequantised
            def int_inverse(quant, inv, plain=False):
                qA, eA = quant(A32)
                return lambda N, S: inv(qA, eA, N, S, want_deq=True, plain=plain)[2].double()
            modes = [("f32", lambda N, S: G.gdn_chunk_inverse_neumann(A32, N, S).double()),
                     ("bf16", lambda N, S: G.gdn_chunk_inverse_neumann(
                         A32.to(torch.bfloat16), N, S).double()),
                     ("int16", int_inverse(G.gdn_quantize_tiles_i16,
                                           G.gdn_chunk_inverse_neumann_i16)),
                     ("int8", int_inverse(G.gdn_quantize_tiles_i8,
                                          G.gdn_chunk_inverse_neumann_i8))]
            if C <= 64:
                modes += [("int16_plain", int_inverse(G.gdn_quantize_tiles_i16,
                                                      G.gdn_chunk_inverse_neumann_i16, True)),
                          ("int8_plain", int_inverse(G.gdn_quantize_tiles_i8,
                                                     G.gdn_chunk_inverse_neumann_i8, True))]
            for dtn, inverse in modes:
                for N in range(1, 7):
                    for S in range(0, 17):
                        if N > lim or S > lim:
                            continue
                        T = inverse(N, S)
                        d = T - X
                        en = (d ** 2).sum(dim=(-1, -2))
                        snr = 10 * torch.log10(xn / en.clamp_min(1e-300))
                        out["grid"].append({
                            "C": C, "set": name, "dtype": dtn, "N": N, "S": S,
                            "tiles": int(T.numel() // (C * C)),
                            "max_abs_err": float(d.abs().max()),
                            "snr_db_mean": round(float(snr.mean()), 2),
                            "snr_db_worst": round(float(snr.min()), 2)})
    return out


def _threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def cpu_baseline_int(w, C, N, S, a, host_inputs, dTq, deT, torch, G, sfx):
    """The integer oracle on whole heads up to `cpu_sample_tiles` tiles,
    passes repeated until `cpu_seconds` have elapsed: build A in float64,
    round to float32, quantise, integer T_hat.  Reports the GPU's
    dequantised T_hat against it (the GPU builds A in fp32 itself, so an
    A entry a rounding apart can move a code: this is an error figure, the
    bit-exact checks live in the tests) and both against the exact inverse."""
    from oracle import gdn
    from oracle import int8 as oi

    spec = oi.SPEC8 if sfx == "i8" else oi.SPEC16
    nc = w.L // C
    want = max(1, a.cpu_sample_tiles)
    heads = [(b, h) for b in range(w.B) for h in range(w.H)][:max(1, -(-want // nc))]
    K, beta, g = host_inputs
    Ks = np.stack([K[b, :, h] for b, h in heads], 1)[None]
    bs = np.stack([beta[b, :, h] for b, h in heads], 1)[None]
    gs = np.stack([g[b, :, h] for b, h in heads], 1)[None]
    with _one_thread():
        passes, t0 = 0, time.perf_counter()
        while True:
            A = gdn.build_A(Ks, bs, gs, C).astype(np.float32)
            if C == 128:
                qA, eA = oi.quantize_blocked(A, spec)
                qT, eT = oi.neumann_inverse_int_blocked(qA, eA, N, S, spec)
            else:
                qA, eA = oi.quantize(A, spec)
                qT, eT, _ = oi.neumann_inverse_int8(qA, eA, N, S, spec)
            passes += 1
            secs = time.perf_counter() - t0
            if secs >= a.cpu_seconds:
                break
    deq = oi.dequant_unit_blocked if C == 128 else oi.dequant_unit
    Tr = deq(qT, eT)[0]
    X = gdn.forward_substitution_inverse(A.astype(np.float64))[0]
    extra = {}
    if C < 128:
        # accuracy of the integer forward substitution on the same codes
        qF, eF = oi.fwdsub_inverse_int(qA, eA, spec)
        extra["fwdsub_" + sfx + "_oracle"] = float(np.max(np.abs(oi.dequant_unit(qF, eF)[0] - X)))
    torch.cuda.synchronize()
    eview = deT.view(w.B, w.H, nc, 3) if C == 128 else deT.view(w.B, w.H, nc)
    Tg = np.stack([deq(dTq[b, h].cpu().numpy().astype(np.int64),
                       eview[b, h].cpu().numpy().astype(np.int64))
                   for b, h in heads], 0)
    tiles = Tr.shape[0] * Tr.shape[1]
    return {"value": round(tiles * passes / secs, 1), "unit": "chunk inverses/s",
            "cores": 1, "kind": "oracle", "cpu_model": _cpu_model(),
            "sample": f"{len(heads)} heads x {nc} chunks of {w.name} ({tiles} tiles), {passes} "
                      f"passes: build A + {sfx.upper().replace('I', 'INT')} quantiser + "
                      f"integer T_hat({N},{S})"
                      f"{' (block-wise, C = 128)' if C == 128 else ''}, numpy on one thread, "
                      f"{secs:.2f} s",
            "max_abs_err_gpu_vs_oracle": {"T": float(np.max(np.abs(Tg - Tr)))},
            "max_abs_err_vs_exact_inverse": {"gpu": float(np.max(np.abs(Tg - X))),
                                             "oracle": float(np.max(np.abs(Tr - X))),
                                             **extra}}


if __name__ == "__main__":
    main()
