"""Benchmark of the ternary x int8 mpGEMM hot path on one MI355X.

One step = one pass of the hot path over one batch of synthetic input for every linear of the workload:
per-token int8 quantisation of each activation group (q/k/v share one input, gate/up share one) and the
ternary mpGEMM with its fused epilogue for each linear.  Weights are ternarised and packed once before
timing (offline preprocessing); the packed copies rotate so that every step streams its weights from
HBM rather than from the 256 MB Infinity Cache.

Prints one JSON line.  `value` is the packed-weight bandwidth of the step (GB/s); `roofline` describes
the dominant kernel (the mpGEMM) from HIP events around a graph of its launches back to back;
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, GB/s
INT8_PEAK_TOPS = 5000.0          # MI355X dense int8 MFMA, TOP/s
ROT_BYTES = 512 << 20            # rotate through at least 2x the Infinity Cache


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", type=int, default=1)
    p.add_argument("--tokens", type=int, default=None)
    p.add_argument("--layout", default="i2s", choices=["i2s", "tl2"])
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-parity", action="store_true")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2502_11880_amd as B
    from paper_2502_11880_amd import inputs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    spec = inputs.WORKLOADS[args.workload]
    M = args.tokens if args.tokens is not None else spec["tokens"][0]
    layout = args.layout
    linears = [(name, K, N) for name, K, N, _ in spec["linears"]]
    by_name = {name: (K, N) for name, K, N in linears}

    # ---- offline: generate, ternarise and pack every weight on the GPU ----
    packed, scales = {}, {}
    for i, (name, K, N) in enumerate(linears):
        W = inputs.weight_f32(N, K, seed=inputs.seed_for(args.workload, i)).to(dev)
        pk = torch.empty(B.bitnet_packed_bytes(layout, N, K), dtype=torch.uint8, device=dev)
        sc = torch.empty(1, dtype=torch.float32, device=dev)
        pws = torch.empty(B.bitnet_pack_workspace_bytes(N, K), dtype=torch.uint8, device=dev)
        B.bitnet_pack_weights(layout, W, pk, sc, pws)
        packed[name], scales[name] = pk, sc
        del W
    torch.cuda.synchronize()
    step_weight_bytes = sum(p.numel() for p in packed.values())
    copies = max(1, math.ceil(ROT_BYTES / step_weight_bytes))
    rot = [packed] + [{k: v.clone() for k, v in packed.items()} for _ in range(copies - 1)]

    groups = [[n for n in g if n in by_name] for g in inputs.ACTIVATION_GROUPS]
    groups = [g for g in groups if g]
    xs, xqs, sxs = [], [], []
    for gi, g in enumerate(groups):
        K = by_name[g[0]][0]
        xs.append(inputs.activation_f32(M, K, seed=inputs.seed_for(args.workload, 100 + gi)).to(dev))
        xqs.append(torch.empty((M, K), dtype=torch.int8, device=dev))
        sxs.append(torch.empty(M, dtype=torch.float32, device=dev))
    ys = {n: torch.empty((M, by_name[n][1]), dtype=torch.float32, device=dev) for n in by_name}
    wss = {n: torch.zeros(max(16, B.bitnet_mpgemm_workspace_bytes(layout, M, by_name[n][1], by_name[n][0])),
                          dtype=torch.uint8, device=dev) for n in by_name}
    stream = torch.cuda.Stream()
    sptr = stream.cuda_stream

    def step(i, quantize=True):
        pk = rot[i % copies]
        for gi, g in enumerate(groups):
            if quantize:
                B.bitnet_quantize_act(xs[gi], xqs[gi], sxs[gi], sptr)
            for n in g:
                K, N = by_name[n]
                B.bitnet_mpgemm(layout, pk[n], scales[n], N, K, xqs[gi], sxs[gi], ys[n], None, wss[n], sptr)

    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step(i)
    torch.cuda.synchronize()

    # The K timed steps are captured once as a HIP graph and replayed, so the GPU runs them back to back
    # (host-side launch overhead would otherwise dominate kernels this short).  A second graph holds only
    # the mpGEMM launches of the same K steps, back to back: its time per launch is the dominant kernel's
    # launch duration (including the short gap between graph nodes).
    g_steps = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_steps, stream=stream):
        for i in range(args.steps):
            step(args.warmup + i)
    g_gemm = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_gemm, stream=stream):
        for i in range(args.steps):
            step(args.warmup + i, quantize=False)
    with torch.cuda.stream(stream):
        g_steps.replay()
        g_gemm.replay()
    torch.cuda.synchronize()

    # ---- timed region: one replay of the K-step graph, then one of the mpGEMM-only graph ----
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    w0 = time.perf_counter()
    with torch.cuda.stream(stream):
        ev[0].record(stream)
        g_steps.replay()
        ev[1].record(stream)
        g_gemm.replay()
        ev[2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    gpu_ms = ev[0].elapsed_time(ev[1])
    ms_per_step = gpu_ms / args.steps
    gemm_total_ms = ev[1].elapsed_time(ev[2])
    launches = args.steps * len(linears)

    per_launch_bytes = {n: packed[n].numel() + M * by_name[n][0] + 4 * M * by_name[n][1] for n in by_name}
    avg_bytes = sum(per_launch_bytes.values()) / len(per_launch_bytes)
    avg_launch_ms = gemm_total_ms / launches
    achieved = avg_bytes / (avg_launch_ms * 1e-3) / 1e9

    value = step_weight_bytes / (ms_per_step * 1e-3) / 1e9
    tokens_per_s = M / (ms_per_step * 1e-3)

    parity = None
    if not args.no_parity:
        parity = parity_spot_check(args, layout, M, linears, packed, scales, xs, groups, by_name, dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, M, linears, groups, by_name, step_weight_bytes)

    out = {
        "metric": "decode GEMV weight GB/s (% HBM peak) + tokens/s; prefill int8 TOPS (% MFMA peak)",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": spec["name"], "tokens": M, "layout": layout,
                   "linears": [f"{n}:{K}x{N}" for n, K, N in linears],
                   "packed_weight_bytes_per_step": step_weight_bytes, "rotating_copies": copies},
        "tokens_per_s": round(tokens_per_s, 1),
        "hbm_frac_step": round(value / HBM_PEAK_GBS, 4),
        "wall_s": round(wall, 3),
        "roofline": {"bound": "hbm", "kernel": "bitnet_mpgemm (decode GEMV)", "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None, "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                     "avg_algorithmic_bytes": int(avg_bytes), "launches": launches},
        "cpu_baseline": cpu,
        "parity": parity,
    }
    print(json.dumps(out), flush=True)


def parity_spot_check(args, layout, M, linears, packed, scales, xs, groups, by_name, dev):
    """Bit-exact check of the benchmark's own first linear against the oracle."""
    import numpy as np
    import torch

    import paper_2502_11880_amd as B
    from oracle import bitnet_oracle as O
    from paper_2502_11880_amd import inputs

    name, K, N = linears[0]
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(args.workload, 0))
    x = xs[0].cpu()
    xq = torch.empty((M, K), dtype=torch.int8, device=dev)
    s = torch.empty(M, dtype=torch.float32, device=dev)
    B.bitnet_quantize_act(xs[0], xq, s)
    y = torch.empty((M, N), dtype=torch.float32, device=dev)
    acc = torch.empty((M, N), dtype=torch.int32, device=dev)
    ws = torch.zeros(max(16, B.bitnet_mpgemm_workspace_bytes(layout, M, N, K)), dtype=torch.uint8, device=dev)
    B.bitnet_mpgemm(layout, packed[name], scales[name], N, K, xq, s, y, acc, ws)
    torch.cuda.synchronize()
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    exact = bool(np.array_equal(acc.cpu().numpy(), acc_ref))
    rel = float(np.max(np.abs(y.cpu().numpy().astype(np.float64) - y_ref) / np.maximum(np.abs(y_ref), 1e-30)))
    return {"linear": f"{name}:{K}x{N}", "acc_bit_exact": exact, "y_max_rel_err": rel}


def cpu_baseline(args, M, linears, groups, by_name, step_weight_bytes):
    """Time the oracle (quantise + exact integer accumulation + epilogue) on the host for ~cpu_seconds."""
    import numpy as np
    import torch

    from oracle import bitnet_oracle as O
    from paper_2502_11880_amd import inputs

    torch.set_num_threads(1)
    ts, betas = {}, {}
    for i, (name, K, N) in enumerate(linears):
        W = inputs.weight_f32(N, K, seed=inputs.seed_for(args.workload, i)).numpy()
        ts[name], betas[name] = O.ternarize(W)
    xs = [inputs.activation_f32(M, by_name[g[0]][0], seed=inputs.seed_for(args.workload, 100 + gi)).numpy()
          for gi, g in enumerate(groups)]
    t0 = time.perf_counter()
    steps = 0
    while True:
        for gi, g in enumerate(groups):
            xq, s = O.quantize_act(xs[gi])
            for n in g:
                O.epilogue(O.mad_gemm(xq, ts[n]), betas[n], s)
        steps += 1
        el = time.perf_counter() - t0
        if el >= args.cpu_seconds:
            break
    per_step = el / steps
    return {"value": round(step_weight_bytes / per_step / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{steps} full steps of the same workload (all {len(linears)} linears, M={M}) in {el:.1f} s; "
                      "numpy int64 matmul, single thread",
            "tokens_per_s": round(M / per_step, 3)}


if __name__ == "__main__":
    main()
