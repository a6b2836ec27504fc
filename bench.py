"""Throughput of one GPU's share of the block join-agg hot path on MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload qkv]

Workload "qkv": the LLaMA-7B QKV projection, one GPU's 1/8 column share:
'tj,jk->tk' bf16 with t = 4096 tokens (2 x 2048), j = 4096, k = 1536, blocks
512 x 512, x ~ N(0,1), W ~ N(0, 0.02); the join-agg (192 tuples in 24 output
groups, SUM of 8 partial products per output block) followed by the
repartition of its output from 512 x 512 blocks to per-head 4096 x 128 blocks.
One step = that join-agg + that repartition; inputs are resident in HBM
before the timed region.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E


def _events_ms(fn, n):
    """Average duration of fn() over n launches, timed with HIP events on the
    current stream (the stream libea launches on)."""
    import torch

    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    for _ in range(n):
        s.record()
        fn()
        e.record()
        e.synchronize()
        times.append(s.elapsed_time(e))
    return sum(times) / len(times)


def qkv_workload():
    import torch

    import synth
    from paper_2609_03905_amd import ea

    w = synth.qkv_projection()
    X = ea.from_dense(torch.from_numpy(w["X"].view("int16")).cuda(), "bf16", w["pX"])
    W = ea.from_dense(torch.from_numpy(w["W"].view("int16")).cuda(), "bf16", w["pW"])
    Y = ea.Relation((4096, 1536), "bf16", w["pY"])
    Yh = ea.Relation((4096, 1536), "bf16", w["pHead"])

    def gemm():
        ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)

    def repart():
        ea.repartition(Y, Yh)

    def step():
        gemm()
        repart()

    flops = 2.0 * 4096 * 4096 * 1536
    repart_bytes = 2 * 4096 * 1536 * 2
    comps = {
        "joinagg_gemm": dict(fn=gemm, flops=flops, bound="mfma"),
        "repartition": dict(fn=repart, bytes=repart_bytes, bound="hbm"),
    }
    return dict(step=step, flops=flops, comps=comps, dominant="joinagg_gemm",
                config={"workload": "qkv_projection_share", "spec": "tj,jk->tk", "t": 4096, "j": 4096, "k": 1536,
                        "block": 512, "repartition": "512x512 -> 4096x128 per-head blocks", "dtype": "bf16"})


def cpu_baseline_qkv(target_s: float = 10.0):
    """The oracle's dense fp64 product on a bounded sample of output rows of
    the same workload, scaled to TFLOP/s."""
    import numpy as np

    import oracle
    import synth

    w = synth.qkv_projection()
    x = synth.to_f64(w["X"], "bf16")
    wt = synth.to_f64(w["W"], "bf16")
    rows = 16
    while True:
        t0 = time.perf_counter()
        oracle.matmul(x[:rows], wt)
        dt = time.perf_counter() - t0
        if dt > target_s / 4 or rows >= 4096:
            break
        rows = min(4096, int(rows * max(2.0, target_s / 4 / max(dt, 1e-3))))
    flops = 2.0 * rows * 4096 * 1536
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"fp64 oracle matmul of {rows} of 4096 output rows x 1536 columns, K=4096 ({dt:.1f} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qkv", choices=["qkv"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs one GPU's share on one GPU; --gpus {args.gpus} is not supported "
              "(the multi-GPU exchange is outside this build)", file=sys.stderr)
        sys.exit(2)

    import torch

    torch.cuda.set_device(0)
    wl = qkv_workload()
    step = wl["step"]
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(args.steps):
        step()
    e.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = s.elapsed_time(e) / args.steps

    comps = {}
    for name, c in wl["comps"].items():
        ms = _events_ms(c["fn"], max(args.steps, 20))
        d = {"ms": ms}
        if "flops" in c:
            d["tflops"] = c["flops"] / ms / 1e9
            d["frac_mfma_peak"] = d["tflops"] / PEAK_BF16_TFLOPS
        if "bytes" in c:
            d["gbs"] = c["bytes"] / ms / 1e6
            d["frac_hbm_peak"] = d["gbs"] / PEAK_HBM_GBS
        comps[name] = d
    dom = wl["comps"][wl["dominant"]]
    dms = comps[wl["dominant"]]["ms"]
    if dom["bound"] == "mfma":
        achieved = dom["flops"] / dms / 1e9
        roof = {"kernel": wl["dominant"], "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None}
    else:
        achieved = dom["bytes"] / dms / 1e6
        roof = {"kernel": wl["dominant"], "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None}

    value = wl["flops"] / ms_per_step / 1e9
    out = {
        "metric": "join-agg TFLOP/s (%MFMA peak), norm/repartition GB/s (%HBM), ms per LLaMA block",
        "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1) activations, N(0,0.02) weights)",
        "config": wl["config"], "roofline": roof, "components": comps, "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_qkv()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
