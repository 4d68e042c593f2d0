#!/usr/bin/env python3
"""Benchmark: tile-major GEMM on one MI355X.

One step = one decode pass over a Llama-3.1-70B-shaped layer at M = 8 tokens:
the four projections (QKV 8192->10240, O 8192->8192, gate+up 8192->57344,
down 28672->8192) through tl_gemm with bf16 weights stored tile-major
(G = 4096 B, 32 x 64-element memory tiles), block-granular fetch, fp32 out.
The layer holds 1.71 GB of weights, far above the 256 MB last-level cache, so
every call streams its weight from HBM.  The timed region launches K steps
eagerly on one stream; the same step captured as a HIP graph and replayed K
times is timed too and reported beside it.

value = algorithmic bytes (2NK + 2MK + 4MN summed over the four GEMMs) per
second over the K timed steps, in GB/s.  Also reported: prefill TFLOP/s at
M = 2048 (tiles 256x256x64, 256x128x64 and 128x128x64, bf16 out), read amplification of
the decode compute tile and of the paper's 128 x 256 tile, repack GB/s, the
decode kernel's roofline, and the CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
METRIC = "tile-major GEMM HBM GB/s (% peak) at M=8; prefill TFLOP/s; read-amp factor"
DECODE_M = 8
G, BR = 4096, 32


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_04031_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def profiled_traffic(kernel_hash):
    """HBM bytes per decode launch from the committed rocprofv3 --pmc summary,
    if it was taken on the current decode kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "decode_llama70b_m8_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_sha256_16") != kernel_hash:
        return None
    return d.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the path is single-GPU; see the sharding notes in the design document)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_04031_amd as tl
    from paper_2607_04031_amd import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    tl.load_library()
    dev = torch.device("cuda:0")
    # all work on one side stream (default priority): graphs cannot be
    # captured on the null stream
    stream = torch.cuda.Stream(device=dev)
    torch.cuda.set_stream(stream)

    # ---------------- weights: seeded, row-major, repacked on the GPU --------
    desc = tl.layout(G=G, block_rows=BR)
    weights, weights_rm_host = [], []
    repack_ms, repack_bytes = 0.0, 0
    for i, (name, N, K) in enumerate(synth.LLAMA70B):
        log(f"generating {name} [{N},{K}]")
        bits = synth.normal_bf16((N, K), seed=synth.llama_weight_seed(i), sigma=synth.W_SIGMA)
        W = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)
        Wt = torch.empty_like(W)
        tl.tl_repack(W, Wt, N, K, 2, G, BR)          # warm
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        tl.tl_repack(W, Wt, N, K, 2, G, BR)
        e1.record(stream)
        torch.cuda.synchronize()
        repack_ms += e0.elapsed_time(e1)
        repack_bytes += 2 * N * K * 2
        del W
        weights.append((name, N, K, Wt))
        if not args.no_cpu_baseline:
            weights_rm_host.append(bits)
        else:
            del bits
    acts = []
    for i, (name, N, K, _) in enumerate(weights):
        a = synth.normal_bf16((DECODE_M, K), seed=synth.llama_decode_act_seed(i, DECODE_M))
        acts.append((a, torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)))
    outs = [torch.empty((DECODE_M, N), dtype=torch.float32, device=dev) for (_, N, _, _) in weights]
    step_bytes = sum(2 * N * K + 2 * DECODE_M * K + 4 * DECODE_M * N for (_, N, K, _) in weights)

    def step(events=None):
        for j, ((name, N, K, Wt), (_, A), C) in enumerate(zip(weights, acts, outs)):
            if events is not None:
                events[j][0].record(stream)
            tl.tl_gemm(A, Wt, C, DECODE_M, N, K, desc, tl.TL_FETCH_BLOCK)
            if events is not None:
                events[j][1].record(stream)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---------------- timed region: K eager steps ----------------
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall_s = t1 - t0
    ms_per_step = wall_s * 1e3 / args.steps
    value_gbs = step_bytes * args.steps / wall_s / 1e9

    # the same step captured once as a HIP graph and replayed K times (the
    # library's workspace already exists, so capture records kernels only);
    # reported beside the eager number
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        step()
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    graph_gbs = step_bytes * args.steps / (time.perf_counter() - t0) / 1e9

    # per-launch durations from HIP events recorded on the launch stream around
    # each tl_gemm call (a separate pass over the same launches)
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
           for _ in weights] for _ in range(args.steps)]
    for s in range(args.steps):
        step(ev[s])
    torch.cuda.synchronize()
    per_shape_ms = [0.0] * len(weights)
    for s in range(args.steps):
        for j in range(len(weights)):
            per_shape_ms[j] += ev[s][j][0].elapsed_time(ev[s][j][1])
    per_shape_ms = [x / args.steps for x in per_shape_ms]
    launch_bytes = [2 * N * K + 2 * DECODE_M * K + 4 * DECODE_M * N for (_, N, K, _) in weights]
    achieved = sum(launch_bytes) / (sum(per_shape_ms) * 1e-3) / 1e9
    per_shape = {name: {"us": round(ms * 1e3, 2), "GB/s": round(b / (ms * 1e-3) / 1e9, 1),
                        "frac_hbm_peak": round(b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "split_k": tl.tl_gemm_plan(DECODE_M, N, K, desc)["split_k"]}
                 for (name, N, K, _), ms, b in zip(weights, per_shape_ms, launch_bytes)}
    log(f"decode layer M={DECODE_M}: eager {value_gbs:.1f} GB/s, graph replay {graph_gbs:.1f} GB/s, "
        f"kernels {achieved:.1f} GB/s")

    # ---------------- read amplification ----------------
    plan = tl.tl_gemm_plan(DECODE_M, 8192, 8192, desc, tl.TL_FETCH_BLOCK)
    amp_tile = tl.tl_read_amp(DECODE_M, 8192, 8192, plan["tile_m"], plan["tile_n"], plan["tile_k"], desc, G)
    rm = tl.layout(kind=tl.TL_LAYOUT_NK_ROW)
    amp_rm = tl.tl_read_amp(DECODE_M, 8192, 8192, plan["tile_m"], plan["tile_n"], plan["tile_k"], rm, G)
    kn = tl.layout(kind=tl.TL_LAYOUT_KN_ROW)
    req_kn = tl.tl_read_amp(1, 2048, 2048, 1, 256, 128, kn, G)["max_blocks_per_tile"]
    req_tm = tl.tl_read_amp(1, 2048, 2048, 1, 256, 128, desc, G)["max_blocks_per_tile"]
    read_amp = {
        "decode_tile": [plan["tile_m"], plan["tile_n"], plan["tile_k"]],
        "tile_major": amp_tile["amp"],
        "row_major_same_tile": amp_rm["amp"],
        "requests_per_128x256_tile_row_major": req_kn,
        "requests_per_128x256_tile_tile_major": req_tm,
        "waste_frac_block_fetch": 1.0 - 1.0 / amp_tile["amp"],
    }

    # ---------------- prefill (M = 2048) ----------------
    prefill = None
    if not args.no_prefill:
        prefill = {}
        Mp = synth.LLAMA_PREFILL_M
        pacts = []
        for i, (name, N, K, _) in enumerate(weights):
            a = synth.normal_bf16((Mp, K), seed=synth.llama_prefill_act_seed(i))
            pacts.append(torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev))
        pouts = [torch.empty((Mp, N), dtype=torch.bfloat16, device=dev) for (_, N, _, _) in weights]
        flops = sum(2.0 * Mp * N * K for (_, N, K, _) in weights)
        for tm, tn in ((256, 256), (256, 128), (128, 128)):
            pd = tl.layout(G=G, block_rows=BR, tile_m=tm, tile_n=tn, out_dtype=tl.TL_OUT_BF16)
            for _ in range(2):
                for (name, N, K, Wt), A, C in zip(weights, pacts, pouts):
                    tl.tl_gemm(A, Wt, C, Mp, N, K, pd, tl.TL_FETCH_BLOCK)
            torch.cuda.synchronize()
            reps = 3
            pev = [[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in weights]
            tot = [0.0] * len(weights)
            for _ in range(reps):
                for j, ((name, N, K, Wt), A, C) in enumerate(zip(weights, pacts, pouts)):
                    pev[j][0].record(stream)
                    tl.tl_gemm(A, Wt, C, Mp, N, K, pd, tl.TL_FETCH_BLOCK)
                    pev[j][1].record(stream)
                torch.cuda.synchronize()
                for j in range(len(weights)):
                    tot[j] += pev[j][0].elapsed_time(pev[j][1])
            ms = sum(tot) / reps
            tf = flops / (ms * 1e-3) / 1e12
            prefill[f"tile_{tm}x{tn}x64"] = {
                "TFLOP/s": round(tf, 1), "frac_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4),
                "layer_ms": round(ms, 3),
                "per_shape_TFLOP/s": {name: round(2.0 * Mp * N * K / (t / reps * 1e-3) / 1e12, 1)
                                      for (name, N, K, _), t in zip(weights, tot)}}
            log(f"prefill tile {tm}x{tn}: {tf:.1f} TFLOP/s")
        del pacts, pouts

    # ---------------- HBM copy calibration (for rocprofv3 counters) ---------
    calib_bytes = 1 << 30
    src = torch.empty(calib_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst

    # ---------------- CPU oracle baseline ----------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        log(f"cpu oracle: full decode layer at M={DECODE_M}, {threads} threads")
        t0 = time.perf_counter()
        for bits, (a_bits, _) in zip(weights_rm_host, acts):
            oracle.gemm_f64(a_bits, bits)
        dt = time.perf_counter() - t0
        cpu = {"value": round(step_bytes / dt / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
               "sample": f"one full decode layer (4 GEMMs, M={DECODE_M}, row-major weights), fp64, "
                         f"{dt:.2f} s"}

    kernel_hash = source_hash("tl_decode.hip")
    traffic = profiled_traffic(kernel_hash)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "decode_kernel (tile-major, M=8; a split_k > 1 call includes its reduce kernel)",
                "per_shape": per_shape}

    out = {
        "metric": METRIC,
        "value": round(value_gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama-3.1-70b-shaped decode layer (qkv, o, gate_up, down), M=8, "
                               "bf16 weights tile-major G=4096 B 32x64 memory tiles, block fetch, fp32 out",
                   "M": DECODE_M, "G": G, "block_rows": BR, "weight_bytes": sum(2 * N * K for (_, N, K, _) in weights)},
        "frac_hbm_peak": round(value_gbs / HBM_PEAK_GBS, 4),
        "graph_replay_GB/s": round(graph_gbs, 1),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "prefill": prefill,
        "read_amp": read_amp,
        "repack_GB/s": round(repack_bytes / (repack_ms * 1e-3) / 1e9, 1),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
