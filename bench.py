"""Benchmark of the ternary x int8 mpGEMM hot path on one MI355X.

One step = one pass of the hot path over one batch of synthetic input through every linear of the
workload, in layer order: the q/k/v group, o, the gate/up group, down (for a stack of layers, every layer in
turn; the layers hold copies of one packed layer in separate HBM buffers, so every byte is streamed).  Each group quantises its input
activation per token (int8, absmax) and multiplies it by the group's packed ternary weights with the fused
dequantisation epilogue.  Each group is one bitnet_mpgemm_fused call: at one token a single launch that also
quantises; otherwise the quantiser, then one launch for all the group's weights (the decode GEMV for M <= 16,
the MFMA GEMM over the weights' concatenated row tiles for M > 16).  Decode also times the separate-call path
(bitnet_quantize_act + one bitnet_mpgemm per weight) and reports it beside the value; prefill times the fused
GEMM launches alone (on the already quantised activations) for its roofline.  Weights are ternarised and packed
once before timing (offline preprocessing); packed copies rotate so every step streams its weights from HBM
rather than from the 256 MB Infinity Cache.

The K timed steps are captured once in a HIP graph and replayed, so the GPU runs them back to back.
The default workload is the largest single-GPU one: the 56-layer 100B-class stack (hidden 12288, FFN 33024) at one
token, I2_S.  Prints one JSON line.  Decode: `value` = packed weight bytes per step / step time (GB/s), `roofline`
bound "hbm".  Prefill: `value` = int8 TOP/s of the step (2*M*N*K per linear), `roofline` bound "mfma".
`gweights_per_s` counts ternary weights per second (I2_S and TL2 on one scale); `ms_per_step_spread` gives the
10th/50th/90th percentile of the per-step time over ten replays of the same graph (the first is the timed one).
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload, with every host thread and with one.
`parity` checks the timed launches themselves (the first activation group's fused call, in the first, middle and
last layer) on every output against the oracle.  The default run also measures the 8B-class layer set at 2048 tokens
(I2_S prefill) in a child process started first and adds it as `prefill_extra` (`--no-extra` skips it).
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
DECODE_MAX_TOKENS = 16
SMALL_BATCH_MAX = 112            # 17..112 tokens: the decode GEMV in token slices (I2_S, TL1)
CPU_ROWS = 512                   # oracle timing sample per weight for stacks of layers
METRIC = "decode GEMV weight GB/s (% HBM peak) + tokens/s; prefill int8 TOPS (% MFMA peak)"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", type=int, default=4)
    p.add_argument("--tokens", type=int, default=None)
    p.add_argument("--layout", default="i2s", choices=["i2s", "tl2", "tl1", "c4g2", "c5g2", "c3g5", "tl2_0", "tl1_0"])
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extra", action="store_true",
                   help="skip the 2048-token prefill figure that the default run adds to its line")
    p.add_argument("--no-parity", action="store_true")
    p.add_argument("--replays", type=int, default=10, help="replays of the timed graph for the spread figure")
    return p.parse_args()


def log(msg):
    """A progress line on stderr (the JSON result is the only line on stdout)."""
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


LOSSY = {"tl2_0": "tl2_elut_decode_kernel", "tl1_0": "tl1_elut_decode_kernel"}   # layout -> kernel
INT_BETA = 0.02                  # per-tensor scale given with the integer-weight layouts' weights
INT_C = {"c4g2": 4, "c5g2": 5, "c3g5": 3}


def int_layout(layout):
    return layout in INT_C


def bench_weight(args, inputs, layout, i, N, K):
    """The benchmark's weight i: fp32 N(0, 0.02) for the ternary layouts (ternarised by the packer), seeded integers
    of the layout's set for the integer-weight layouts."""
    seed = inputs.seed_for(args.workload, i)
    if int_layout(layout):
        return inputs.int_weights(N, K, INT_C[layout], seed=seed)
    return inputs.weight_f32(N, K, seed=seed)


def activation_groups(by_name, inputs):
    """Linears that read the same input, in layer order; any linear not in a listed group stands alone."""
    groups = [[n for n in g if n in by_name] for g in inputs.ACTIVATION_GROUPS]
    groups = [g for g in groups if g]
    listed = {n for g in groups for n in g}
    return groups + [[n] for n in by_name if n not in listed]


def prefill_extra(args):
    """The default run also reports the 8B-class layer set at 2048 tokens (I2_S prefill), measured by this script in
    a child process started before this one touches the GPU; None when skipped or when the child fails."""
    if args.no_extra or args.workload != 4 or args.tokens is not None or args.layout != "i2s":
        return None
    import subprocess

    log("prefill figure (8B-class layer set, 2048 tokens) in a child process")
    cmd = [sys.executable, os.path.abspath(__file__), "--workload", "3", "--tokens", "2048", "--no-cpu-baseline",
           "--no-extra"]
    if args.no_parity:
        cmd.append("--no-parity")
    try:
        res = subprocess.run(cmd, stdout=subprocess.PIPE, text=True, timeout=600)
        line = [ln for ln in res.stdout.splitlines() if ln.startswith("{")][-1] if res.returncode == 0 else None
    except (subprocess.TimeoutExpired, IndexError):
        line = None
    if line is None:
        log("prefill figure: child run failed; reported as null")
        return None
    d = json.loads(line)
    r = d["roofline"]
    return {"workload": d["config"]["workload"], "tokens": d["config"]["tokens"], "layout": d["config"]["layout"],
            "value": d["value"], "unit": d["unit"], "ms_per_step": d["ms_per_step"],
            "gemm_only_ms_per_step": d.get("gemm_only_ms_per_step"),
            "roofline": {k: r.get(k) for k in ("bound", "kernel", "achieved", "peak", "unit", "frac", "traffic")},
            "parity_pass": (d.get("parity") or {}).get("pass")}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    extra = prefill_extra(args)

    import torch

    import paper_2502_11880_amd as B
    from paper_2502_11880_amd import inputs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    spec = inputs.WORKLOADS[args.workload]
    M = args.tokens if args.tokens is not None else spec["tokens"][0]
    decode = M <= DECODE_MAX_TOKENS
    layout = args.layout
    linears = [(name, K, N) for name, K, N, _ in spec["linears"]]
    by_name = {name: (K, N) for name, K, N in linears}
    n_layers = spec.get("layers", 1)
    if not decode or n_layers > 1:
        args.steps = max(1, min(args.steps, 20))
        args.warmup = max(1, min(args.warmup, 3))

    # ---- offline: generate, ternarise and pack every weight on the GPU ----
    log(f"workload {args.workload} ({spec['name']}), {M} token(s), {layout}: packing {len(linears)} weights")
    packed, scales = {}, {}
    for i, (name, K, N) in enumerate(linears):
        W = bench_weight(args, inputs, layout, i, N, K).to(dev)
        nbytes = B.bitnet_packed_bytes(layout, N, K)
        if nbytes == 0:
            print(f"layout {layout} does not take a {N} x {K} weight", file=sys.stderr)
            sys.exit(2)
        pk = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        if int_layout(layout):
            sc = torch.full((1,), INT_BETA, dtype=torch.float32, device=dev)
            B.bitnet_pack_int_weights(layout, W, pk)
        else:
            sc = torch.empty(1, dtype=torch.float32, device=dev)
            pws = torch.empty(B.bitnet_pack_workspace_bytes(N, K), dtype=torch.uint8, device=dev)
            B.bitnet_pack_weights(layout, W, pk, sc, pws)
        packed[name], scales[name] = pk, sc
        del W
    torch.cuda.synchronize()
    layer_weight_bytes = sum(p.numel() for p in packed.values())
    step_weight_bytes = layer_weight_bytes * n_layers
    copies = max(1, math.ceil(ROT_BYTES / step_weight_bytes)) if decode else 1
    # rot[c][l]: packed weights of layer l in rotating copy c (layers past the first are copies of it)
    rot = [[packed if (c, l) == (0, 0) else {k: v.clone() for k, v in packed.items()} for l in range(n_layers)]
           for c in range(copies)]

    log(f"{copies} rotating copies of {n_layers} layer(s), {step_weight_bytes / 1e9:.2f} GB of packed weights per step")
    groups = activation_groups(by_name, inputs)
    xs, xqs, sxs, rss = [], [], [], []
    for gi, g in enumerate(groups):
        K = by_name[g[0]][0]
        xs.append(inputs.activation_f32(M, K, seed=inputs.seed_for(args.workload, 100 + gi)).to(dev))
        xqs.append(torch.empty((M, K), dtype=torch.int8, device=dev))
        sxs.append(torch.empty(M, dtype=torch.float32, device=dev))
        rss.append(torch.empty(M, dtype=torch.int32, device=dev))
    ys = {n: torch.empty((M, by_name[n][1]), dtype=torch.float32, device=dev) for n in by_name}
    ws_bytes = max(B.bitnet_mpgemm_workspace_bytes(layout, M, N, K) for _, K, N in linears)
    ws_bytes = max([ws_bytes] + [B.bitnet_mpgemm_fused_workspace_bytes(layout, [by_name[n][1] for n in g],
                                                                       by_name[g[0]][0], M) for g in groups])
    ws = torch.zeros(max(16, ws_bytes), dtype=torch.uint8, device=dev)
    fargs = [[[B.FusedArgs([rot[c][l][n] for n in g], [scales[n] for n in g], [ys[n] for n in g]) for g in groups]
              for l in range(n_layers)] for c in range(copies)]
    stream = torch.cuda.Stream()
    sptr = stream.cuda_stream
    # the set-up above ran on the default stream: the side stream starts after all of it
    torch.cuda.synchronize()
    stream.wait_stream(torch.cuda.current_stream())

    def step(i, path, quantize=True):
        c = i % copies
        for l in range(n_layers):
            for gi, g in enumerate(groups):
                if path == "fused":
                    # quantize=False: the products alone, on the activation the warm-up steps quantised
                    B.bitnet_mpgemm_fused(layout, None, None, xs[gi] if quantize else None, xqs[gi], sxs[gi], rss[gi],
                                          None, ws, sptr, args=fargs[c][l][gi])
                    continue
                if quantize:
                    B.bitnet_quantize_act(xs[gi], xqs[gi], sxs[gi], rss[gi], sptr)
                for n in g:
                    K, N = by_name[n]
                    B.bitnet_mpgemm(layout, rot[c][l][n], scales[n], N, K, xqs[gi], sxs[gi], ys[n], None, ws, sptr,
                                    x_rowsum=rss[gi])

    def capture(fn):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(args.steps):
                fn(args.warmup + i)
        return g

    main_path = "fused"
    log(f"warm-up ({args.warmup} steps), then {args.steps} steps captured in a graph")
    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step(i, main_path)
            if decode:
                step(i, "separate")
    torch.cuda.synchronize()

    # Graphs: the K steps on the main path, the same steps on the separate-call path (decode), or the
    # fused GEMM launches alone (prefill: the dominant kernel).
    g_main = capture(lambda i: step(i, main_path))
    g_second = capture(lambda i: step(i, "separate")) if decode else \
        capture(lambda i: step(i, "fused", quantize=False))
    with torch.cuda.stream(stream):
        g_main.replay()
        g_second.replay()
    torch.cuda.synchronize()

    # ---- timed region ----
    log("timed replay")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    w0 = time.perf_counter()
    with torch.cuda.stream(stream):
        ev[0].record(stream)
        g_main.replay()
        ev[1].record(stream)
        g_second.replay()
        ev[2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_per_step = ev[0].elapsed_time(ev[1]) / args.steps
    second_ms = ev[1].elapsed_time(ev[2]) / args.steps
    # spread: the same K steps replayed again, each replay timed on its own (outside the timed region above)
    reps = [ms_per_step]
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.replays) - 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g_main.replay()
            e1.record(stream)
            e1.synchronize()
            reps.append(e0.elapsed_time(e1) / args.steps)
    reps.sort()
    spread = {"replays": len(reps), "p10": round(reps[len(reps) // 10], 5), "p50": round(reps[len(reps) // 2], 5),
              "p90": round(reps[min(len(reps) - 1, (9 * len(reps)) // 10)], 5)}

    flops = sum(2.0 * M * N * K for _, K, N in linears)
    step_weights = sum(N * K for _, K, N in linears) * n_layers   # ternary weights read per step
    if decode:
        value = step_weight_bytes / (ms_per_step * 1e-3) / 1e9
        unit = "GB/s"
        launches = len(groups) * n_layers
        grp_bytes = [sum(packed[n].numel() + 4 * M * by_name[n][1] for n in g) + 5 * M * by_name[g[0]][0] + 8 * M
                     for g in groups]
        avg_bytes = sum(grp_bytes) * n_layers / launches
        avg_launch_ms = ms_per_step / launches
        achieved = avg_bytes / (avg_launch_ms * 1e-3) / 1e9
        words = " on TL1 words" if layout == "tl1" else ""
        if int_layout(layout):
            kernel = f"elut_generic_kernel ({layout} table lookups) per weight, after quantize_rows_reg per group"
        elif layout in LOSSY:
            kernel = f"{LOSSY[layout]} (int8-quantised tables) per weight, after quantize_rows_reg per group"
        elif layout == "tl2" and M == 1:
            kernel = "tl2_mfma_decode_kernel (bitnet_mpgemm_fused, one token: quantiser fused)"
        elif layout == "tl2":
            kernel = "bitnet_mpgemm_fused on TL2: quantize_rows_reg + tl2_mfma_decode_kernel per group"
        elif M == 1:
            kernel = f"i2s_gemv1_stream_kernel{words} (bitnet_mpgemm_fused, one token: quantiser fused)"
        else:
            kernel = f"bitnet_mpgemm_fused: quantize_rows_reg + i2s_decode_stream_kernel{words} per group"
        traffic = measured_traffic(*TRAFFIC[key]) if (key := (args.workload, M, layout)) in TRAFFIC else None
        roofline = {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                    "traffic_unit": "bytes per launch (FETCH_SIZE x copy factor + WRITE_SIZE)" if traffic else None,
                    "avg_launch_us": round(avg_launch_ms * 1e3, 3), "avg_algorithmic_bytes": int(avg_bytes),
                    "launches_per_step": launches}
    else:
        value = flops / (ms_per_step * 1e-3) / 1e12
        unit = "TOP/s"
        launches = len(groups) * n_layers
        avg_launch_ms = second_ms / launches
        sliced = M <= SMALL_BATCH_MAX and layout in ("i2s", "tl1")
        if sliced:
            kernel = (f"i2s_decode_stream_kernel{' on TL1 words' if layout == 'tl1' else ''} in token slices "
                      "(bitnet_mpgemm_fused, 17-112 tokens: one launch per activation group)")
        elif int_layout(layout):
            kernel = f"elut_generic_kernel ({layout} table lookups) per weight"
        elif layout in LOSSY:
            kernel = f"{LOSSY[layout]} (int8-quantised tables) in 8-token slices per weight"
        else:
            kernel = "i2s_prefill_kernel (bitnet_mpgemm_fused, M > 16: one launch per activation group)"
            if layout != "i2s":
                kernel = f"{layout}_to_i2s transcoding per group + " + kernel
        # the roofline that binds: HBM for the weight stream (packed weights, the codes read, the fp32 outputs
        # written) or int8 MFMA, whichever takes longer at its peak
        gemm_bytes = sum(sum(packed[n].numel() + 4 * M * by_name[n][1] for n in g) + M * by_name[g[0]][0]
                         for g in groups) * n_layers
        hbm_bound = gemm_bytes / (HBM_PEAK_GBS * 1e9) > flops / (INT8_PEAK_TOPS * 1e12)
        traffic = measured_traffic(*TRAFFIC[key]) if (key := (args.workload, M, layout)) in TRAFFIC else None
        if hbm_bound:
            achieved = (gemm_bytes / launches) / (avg_launch_ms * 1e-3) / 1e9
            roofline = {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                        "traffic_unit": "bytes per launch (FETCH_SIZE x copy factor + WRITE_SIZE)" if traffic else None,
                        "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                        "avg_algorithmic_bytes": int(gemm_bytes / launches), "launches_per_step": launches}
        else:
            achieved = (flops / launches) / (avg_launch_ms * 1e-3) / 1e12
            roofline = {"bound": "mfma", "kernel": kernel,
                        "achieved": round(achieved, 1), "peak": INT8_PEAK_TOPS, "unit": "TFLOP/s",
                        "frac": round(achieved / INT8_PEAK_TOPS, 4), "traffic": traffic,
                        "traffic_unit": "bytes per launch (FETCH_SIZE x copy factor + WRITE_SIZE)" if traffic else None,
                        "avg_launch_us": round(avg_launch_ms * 1e3, 3), "avg_algorithmic_ops": int(flops / launches),
                        "launches_per_step": launches}
    tokens_per_s = M / (ms_per_step * 1e-3)

    parity = None
    log(f"{ms_per_step:.5f} ms per step; parity of the timed launches against the oracle")
    if not args.no_parity:
        parity = parity_check(args, layout, M, linears, groups, by_name, xs, ys, fargs, n_layers, ws, stream)
    cpu = None
    if not args.no_cpu_baseline:
        log("CPU oracle timing")
        cpu = cpu_baseline(args, M, linears, groups, by_name, step_weight_bytes, flops, decode)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": spec["name"], "tokens": M, "layout": layout, "path": main_path, "layers": n_layers,
                   "linears": [f"{n}:{K}x{N}" for n, K, N in linears],
                   "packed_weight_bytes_per_step": step_weight_bytes, "rotating_copies": copies},
        "tokens_per_s": round(tokens_per_s, 1),
        "gweights_per_s": round(step_weights / (ms_per_step * 1e-3) / 1e9, 2),
        "ms_per_step_spread": spread,
        "hbm_frac_step": round(step_weight_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "mfma_frac_step": round(flops / (ms_per_step * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4),
        ("separate_path_ms_per_step" if decode else "gemm_only_ms_per_step"): round(second_ms, 5),
        "wall_s": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity": parity,
    }
    if extra is not None:
        out["prefill_extra"] = extra
    print(json.dumps(out), flush=True)


# committed counter summaries (HBM bytes per launch) and the kernel sources they were taken on
# (workload, tokens, layout) -> (summary, kernel sources)
TRAFFIC = {
    (4, 1, "i2s"): ("profiles/decode_i2s_100b_m1_hbm_traffic.md",
                    ("paper_2502_11880_amd/csrc/k_decode_i2s.hip", "paper_2502_11880_amd/csrc/bitnet_internal.hpp")),
    (1, 1, "i2s"): ("profiles/decode_i2s_bitnet3b_m1_hbm_traffic.md",
                    ("paper_2502_11880_amd/csrc/k_decode_i2s.hip", "paper_2502_11880_amd/csrc/bitnet_internal.hpp")),
    (3, 2048, "i2s"): ("profiles/prefill_i2s_llama8b_m2048_hbm_traffic.md",
                       ("paper_2502_11880_amd/csrc/k_prefill_i2s.hip", "paper_2502_11880_amd/csrc/bitnet_internal.hpp")),
}


def code_only(text):
    """Source text without // comments, trailing blanks and empty lines (comment edits keep the hash)."""
    lines = (line.split("//", 1)[0].rstrip() for line in text.splitlines())
    return "\n".join(line for line in lines if line)


def measured_traffic(profile, sources):
    """HBM bytes per launch from a committed counter summary, or None when the kernel sources no longer hash to
    the ones the counters were taken on."""
    import hashlib
    import os

    root = os.path.dirname(os.path.abspath(__file__))
    try:
        text = open(os.path.join(root, profile)).read()
        h = hashlib.sha256()
        for f in sources:
            h.update(code_only(open(os.path.join(root, f)).read()).encode())
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines() if line.count(": ") == 1 and " " not in line.split(": ")[0])
    if fields.get("source_sha256", "").strip() != h.hexdigest():
        return None
    return int(fields["traffic_bytes_per_launch"])


def parity_check(args, layout, M, linears, groups, by_name, xs, ys, fargs, n_layers, ws, stream):
    """Every output of the first activation group's fused call -- the launch the timed step makes, with the same
    arguments -- against the oracle, in the first, middle and last layer (rotating copy 0)."""
    import numpy as np
    import torch

    import paper_2502_11880_amd as B
    from oracle import bitnet_oracle as O
    from paper_2502_11880_amd import inputs

    g = groups[0]
    K = by_name[g[0]][0]
    index = {name: i for i, (name, _, _) in enumerate(linears)}
    xq_ref, s_ref = O.quantize_act(xs[0].cpu().numpy())
    refs = {}
    for n in g:
        N = by_name[n][1]
        W = bench_weight(args, inputs, layout, index[n], N, K).numpy()
        t_ref, beta = (W, np.float32(INT_BETA)) if int_layout(layout) else O.ternarize(W)
        acc_ref = oracle_acc(O, layout, xq_ref, t_ref)
        refs[n] = (acc_ref, O.epilogue(acc_ref, beta, s_ref))
        del t_ref
    dev = xs[0].device
    xq = torch.empty((M, K), dtype=torch.int8, device=dev)
    s = torch.empty(M, dtype=torch.float32, device=dev)
    rs = torch.empty(M, dtype=torch.int32, device=dev)
    layers = sorted({0, n_layers // 2, n_layers - 1})
    codes_ok, zeros_ok, worst, outputs = True, True, 0.0, 0
    for l in layers:
        for n in g:
            ys[n].fill_(float("nan"))
        with torch.cuda.stream(stream):
            B.bitnet_mpgemm_fused(layout, None, None, xs[0], xq, s, rs, None, ws, stream.cuda_stream,
                                  args=fargs[0][l][0])
        torch.cuda.synchronize()
        codes_ok = codes_ok and bool(np.array_equal(xq.cpu().numpy(), xq_ref)) and bool(
            np.array_equal(s.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))) and bool(
            np.array_equal(rs.cpu().numpy(), xq_ref.astype(np.int64).sum(1)))
        for n in g:
            acc_ref, y_ref = refs[n]
            yg = ys[n].cpu().numpy().astype(np.float64)
            err = np.abs(yg - y_ref) / np.maximum(np.abs(y_ref), 1e-30)
            err[acc_ref == 0] = 0.0
            worst = max(worst, float(np.nan_to_num(err, nan=np.inf).max()))
            zeros_ok = zeros_ok and bool(np.all(yg[acc_ref == 0] == 0.0))
            outputs += yg.size
    return {"group": ",".join(g) + f":{K}x[" + ",".join(str(by_name[n][1]) for n in g) + "]",
            "call": "bitnet_mpgemm_fused, the timed launch and arguments", "layers_checked": layers,
            "rows_checked": M, "outputs_checked": outputs, "codes_bit_exact": codes_ok,
            "y_max_rel_err": worst, "zeros_exact": zeros_ok,
            "pass": bool(codes_ok and zeros_ok and worst <= 1e-5)}


def oracle_acc(O, layout, xq, t):
    """The oracle's accumulators for a layout: the exact integer products, or for the lossy layouts the lookups on
    int8-quantised tables over the oracle's own packing."""
    N, K = t.shape
    if layout == "tl2_0":
        return O.elut_gemm_lossy(xq, O.pack_tl2(t), N, K)
    if layout == "tl1_0":
        return O.elut_gemm_tl1_lossy(xq, O.pack_tl1(t), N, K)
    return O.mad_gemm(xq, t)


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def host_threads():
    """Threads this process may run on (its CPU affinity), else the host's CPU count."""
    try:
        return len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        return os.cpu_count() or 1


def cpu_baseline(args, M, linears, groups, by_name, step_weight_bytes, flops, decode):
    """Time the oracle (quantise + exact integer accumulation + epilogue) on the host for ~cpu_seconds, once with
    every host thread and once with one (the oracle's matrix product is a BLAS call; the rest is numpy)."""
    import torch
    from threadpoolctl import threadpool_limits

    from oracle import bitnet_oracle as O
    from paper_2502_11880_amd import inputs

    n_layers = inputs.WORKLOADS[args.workload].get("layers", 1)
    # very large layers: the first CPU_ROWS output rows of each weight stand in for all of them
    row_cap = CPU_ROWS if n_layers > 1 else None
    ts, betas, packs = {}, {}, {}
    sample_bytes = 0
    for i, (name, K, N) in enumerate(linears):
        Ns = N if row_cap is None else min(N, row_cap)
        W = bench_weight(args, inputs, args.layout, i, Ns, K).numpy()
        ts[name], betas[name] = (W, INT_BETA) if int_layout(args.layout) else O.ternarize(W)
        if args.layout in LOSSY:
            packs[name] = (O.pack_tl2 if args.layout == "tl2_0" else O.pack_tl1)(ts[name])
        sample_bytes += Ns * K // 4
    # prefill: a bounded sample of token rows stands in for the full M
    Mc = M if decode else min(M, 4)
    xs = [inputs.activation_f32(M, by_name[g[0]][0], seed=inputs.seed_for(args.workload, 100 + gi)).numpy()[:Mc]
          for gi, g in enumerate(groups)]

    def timed(threads):
        torch.set_num_threads(threads)
        with threadpool_limits(limits=threads):
            t0 = time.perf_counter()
            steps = 0
            while True:
                for gi, g in enumerate(groups):
                    xq, s = O.quantize_act(xs[gi])
                    for n in g:
                        if args.layout == "tl2_0":
                            acc = O.elut_gemm_lossy(xq, packs[n], *ts[n].shape)
                        elif args.layout == "tl1_0":
                            acc = O.elut_gemm_tl1_lossy(xq, packs[n], *ts[n].shape)
                        else:
                            acc = O.mad_gemm(xq, ts[n])
                        O.epilogue(acc, betas[n], s)
                steps += 1
                el = time.perf_counter() - t0
                if el >= args.cpu_seconds / 2:
                    return steps, el

    legs = {}
    for threads in (host_threads(), 1):
        steps, el = timed(threads)
        per_step = el / steps
        if decode and row_cap is not None:
            rate = sample_bytes / per_step            # packed-equivalent weight bytes per second
            legs[threads] = {"value": round(rate / 1e9, 4), "unit": "GB/s", "cores": threads,
                             "sample": f"{steps} passes over the first {row_cap} output rows of each of the "
                                       f"{len(linears)} linears of one layer (M={M}) in {el:.1f} s",
                             "tokens_per_s": round(M * rate / step_weight_bytes, 6)}
        elif decode:
            legs[threads] = {"value": round(step_weight_bytes / per_step / 1e9, 4), "unit": "GB/s", "cores": threads,
                             "sample": f"{steps} full steps of the same workload (all {len(linears)} linears, M={M}) "
                                       f"in {el:.1f} s", "tokens_per_s": round(M / per_step, 3)}
        else:
            legs[threads] = {"value": round(flops * Mc / M / per_step / 1e12, 6), "unit": "TOP/s", "cores": threads,
                             "sample": f"{steps} steps of the same linears on {Mc} of the {M} token rows in {el:.1f} s",
                             "tokens_per_s": round(Mc / per_step, 3)}
    allc = legs[host_threads()]
    one = legs[1]
    how = ("; numpy quantiser and epilogue, float64 BLAS matrix product (exact for these integers)"
           if args.layout not in LOSSY else "; numpy quantiser, table build, int8 table quantisation, lookups and "
           "epilogue (the packing is done beforehand)")
    return {**allc, "kind": "oracle", "sample": allc["sample"] + how, "cpu_model": cpu_model(),
            "host_threads": host_threads(),
            "single_thread": {k: one[k] for k in ("value", "unit", "cores", "sample", "tokens_per_s")}}


if __name__ == "__main__":
    main()
