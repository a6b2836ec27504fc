"""Throughput of one GPU's share of the block join-agg hot path on MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload block|qkv|attention|packed_gqa|reductions|repartition|w1_block|w1_1k|w1_8k|w1_128k|w1_128x1k|chains]

Default workload "block": one GPU's share of a LLaMA-65B-shape transformer
block (hidden 8192, 8 of 64 heads of dim 128, SwiGLU FFN 2752 = 22016/8,
batch 1 x seq 2048, bf16, seeded N(0,1) activations, N(0,0.02) weights,
U(0.5,1.5) norm weights).  One step = the whole chain: RMSNorm join-agg, QKV
block-GEMM join-agg, repartition to per-head blocks, causal attention join-agg
(online-softmax aggregation over 128-key blocks), repartition back, O-proj
join-agg with fused residual, RMSNorm, SwiGLU join-agg, down join-agg with
fused residual.  The join of every stage is resolved once (plan cache) before
the timed region; inputs are resident in HBM.  `value` = the step's
algorithmic FLOPs (423.06 GFLOP) / step time.

Other workloads (not the default line): "qkv" = the LLaMA-7B QKV projection
share 'tj,jk->tk' 4096x4096x1536 in 512x512 blocks plus its repartition to
per-head 4096x128 blocks; "attention" = causal attention B2 H4 S2048 D128;
"reductions" = RMSNorm over x[4096, 4096] in 8 column blocks and causal
softmax over s[4, 2048, 2048] in 256-key blocks; "repartition" = a 256 MiB
bf16 relation re-blocked from 512x512 to 128-row blocks (a pure copy).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 / fp16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
METRIC = "join-agg TFLOP/s (%MFMA peak), norm/repartition GB/s (%HBM), ms per LLaMA block"


def _events_ms(fn, n, warm=3):
    """Average GPU duration of fn() over n back-to-back launches, measured
    with HIP events on the current stream (the stream libea launches on).
    The launches are queued behind a bounded spin kernel, so the events see
    them run back to back even where one host call takes longer than its
    kernel; the spin is doubled until the start event is still pending once
    every launch is queued."""
    import torch

    for _ in range(warm):
        fn()
    spin = 1 << 22
    for _ in range(6):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        torch.cuda._sleep(spin)
        s.record()
        for _ in range(n):
            fn()
        e.record()
        queued_in_time = not s.query()
        e.synchronize()
        if queued_in_time:
            break
        spin *= 2
    return s.elapsed_time(e) / n


def _host_us_per_call(fn, n):
    """Host time of one call of fn() (marshalling, plan lookup, launch)."""
    import torch

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n):
        fn()
    t = (time.perf_counter() - t0) / n * 1e6
    torch.cuda.synchronize()
    return t


def _profiled_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from its committed counter summary
    (profiles/<kernel>_traffic.txt: FETCH_SIZE and WRITE_SIZE per dispatch,
    scaled by the readings of a copy of known size), or None when there is no
    summary or the kernel's sources have changed since it was taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"{kernel}_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        k, sep, v = line.partition(":")
        if sep and " " not in k.strip():
            rec[k.strip()] = v.strip()
    h = hashlib.sha256()
    for src in ("ea_gemm.hip", "ea_host.cpp", "ea_internal.h"):
        with open(os.path.join(ROOT, "paper_2609_03905_amd", "csrc", src), "rb") as f:
            h.update(f.read())
    if rec.get("kernel_source_sha256") != h.hexdigest() or "traffic_bytes" not in rec:
        return None
    return float(rec["traffic_bytes"])


def _dev(a):
    import numpy as np
    import torch

    return torch.from_numpy(a.view(np.int16)).cuda()


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------
def block_workload():
    import synth
    from paper_2609_03905_amd.block import LlamaBlockShare

    w = synth.llama_block()
    blk = LlamaBlockShare(w["t"], w["hidden"], w["heads"], w["d_head"], w["ffn"], block=w["block"], eps=w["eps"])
    blk.load({k: _dev(w[k]) for k in ("x", "n1", "n2", "wqkv", "wo", "wg", "wu", "wd")})
    work = blk.work()
    stages = blk.stages()
    comps = {name: dict(fn=fn, same_buffers=True, **work[name]) for name, fn in stages}
    flops = sum(c.get("flops", 0) for c in comps.values())
    return dict(step=blk.forward, flops=flops, comps=comps, dominant="swiglu_gemm",
                config={"workload": "llama65b_block_share", "hidden": 8192, "heads": "8 of 64", "d_head": 128,
                        "ffn": 2752, "tokens": 2048, "batch": 1, "block": 512, "dtype": "bf16",
                        "chain": [n for n, _ in stages]},
                cpu=cpu_baseline_block)


ROTATE_BYTES = 1 << 30


class _Rotation:
    """Round-robin over copies of a workload's buffers, placed at different
    addresses: consecutive calls use different copies, and the copies together
    (>= 1 GiB) exceed the 256 MB Infinity Cache, so a timed call reads its
    inputs from HBM rather than from what the previous call left cached."""

    def __init__(self, sets):
        self.sets, self.i = sets, -1

    def next(self):
        self.i = (self.i + 1) % len(self.sets)
        return self.sets[self.i]


def _buffer_sets(make_set, set_bytes: int):
    return [make_set(i) for i in range(max(1, -(-ROTATE_BYTES // set_bytes)))]


def _copy(rel, ea):
    """Relation with the same partition and contents in a new allocation."""
    return ea.Relation(rel.shape, rel.dtype, rel.partition, data=rel.bytes().clone())


def qkv_workload():
    import synth
    from paper_2609_03905_amd import ea

    w = synth.qkv_projection()
    X0 = ea.from_dense(_dev(w["X"]), "bf16", w["pX"])
    W0 = ea.from_dense(_dev(w["W"]), "bf16", w["pW"])

    def make_set(i):
        X, W = (X0, W0) if i == 0 else (_copy(X0, ea), _copy(W0, ea))
        return X, W, ea.Relation((4096, 1536), "bf16", w["pY"]), ea.Relation((4096, 1536), "bf16", w["pHead"])

    set_bytes = 4096 * 4096 * 2 + 3 * 4096 * 1536 * 2
    sets = _buffer_sets(make_set, set_bytes)
    rot, rot_g, rot_r = (_Rotation(sets) for _ in range(3))
    run_gemm = lambda X, W, Y: ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    gemm = lambda: run_gemm(*rot_g.next()[:3])
    # standalone, nothing reads the head-blocked output, so it is streamed
    # (the output store policy; in the block chain attention reads it and the
    # store stays cached)
    run_repart = lambda Y, Yh: ea.repartition(Y, Yh, store=ea.STORE_STREAM)
    repart = lambda: (lambda st: run_repart(st[2], st[3]))(rot_r.next())

    def step():
        X, W, Y, Yh = rot.next()
        run_gemm(X, W, Y)
        run_repart(Y, Yh)

    flops = 2.0 * 4096 * 4096 * 1536
    comps = {"joinagg_gemm": dict(fn=gemm, flops=flops), "repartition": dict(fn=repart, bytes=2 * 4096 * 1536 * 2)}
    return dict(step=step, flops=flops, comps=comps, dominant="joinagg_gemm",
                config={"workload": "llama7b_qkv_projection_share", "spec": "tj,jk->tk", "t": 4096, "j": 4096,
                        "k": 1536, "block": 512, "repartition": "512x512 -> 4096x128", "dtype": "bf16",
                        "buffer_sets": len(rot.sets)},
                cpu=cpu_baseline_qkv)


def attention_workload():
    import synth
    from paper_2609_03905_amd import ea

    w = synth.attention()
    base = [ea.from_dense(_dev(w[n]), "bf16", w["pq"]) for n in "qkv"]

    def make_set(i):
        qkv = base if i == 0 else [_copy(r, ea) for r in base]
        return qkv + [ea.Relation((2, 4, 2048, 128), "bf16", w["pq"])]

    rot = _Rotation(_buffer_sets(make_set, 4 * 2 * 4 * 2048 * 128 * 2))

    def fn():
        Q, K, V, O = rot.next()
        ea.joinagg("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O, scale=w["scale"], causal=True)

    flops = 4.0 * 128 * 2 * 4 * 2048 * 2049 / 2
    return dict(step=fn, flops=flops, comps={"attention": dict(fn=fn, flops=flops)}, dominant="attention",
                config={"workload": "llama7b_causal_attention_share", "batch": 2, "heads": 4, "seq": 2048,
                        "d_head": 128, "q_block": 128, "k_block": 128, "dtype": "bf16",
                        "buffer_sets": len(rot.sets)}, cpu=None)


def packed_gqa_workload():
    import synth
    from paper_2609_03905_amd import ea

    w = synth.packed_gqa_attention()
    Q0 = ea.from_dense(_dev(w["q"]), "bf16", w["pq"])
    K0, V0 = (ea.from_dense(_dev(w[n]), "bf16", w["pk"]) for n in "kv")
    hq, s = w["q"].shape[1], w["q"].shape[2]

    def make_set(i):
        qkv = [Q0, K0, V0] if i == 0 else [_copy(r, ea) for r in (Q0, K0, V0)]
        return qkv + [ea.Relation((1, hq, s, 128), "bf16", w["pq"])]

    rot = _Rotation(_buffer_sets(make_set, (2 * hq + 2) * s * 128 * 2))

    def fn():
        Q, K, V, O = rot.next()
        ea.joinagg("bhqd,bgkd,bgkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O, scale=w["scale"],
                   causal=True, gqa_group=w["gqa"], seq_ends=w["ends"])

    L = w["ends"][0]
    flops = 4.0 * 128 * hq * len(w["ends"]) * L * (L + 1) / 2
    return dict(step=fn, flops=flops, comps={"attention": dict(fn=fn, flops=flops)}, dominant="attention",
                config={"workload": "packed_gqa_attention_share", "sequences": len(w["ends"]), "seq_len": L,
                        "heads_q": hq, "heads_kv": w["k"].shape[1], "d_head": 128, "q_block": 128, "k_block": 128,
                        "causal": True, "dtype": "bf16", "buffer_sets": len(rot.sets)}, cpu=None)


def w1_block_workload(t=8192, seq_len=1024):
    """One GPU's 8-way head share of the paper's W1 block on t tokens packed
    as sequences of seq_len (seq_len == t: one sequence)."""
    import synth
    from paper_2609_03905_amd.block import LlamaBlockShare

    w = synth.w1_block(t=t, seq_len=seq_len)
    blk = LlamaBlockShare(w["t"], w["hidden"], w["heads"], w["d_head"], w["ffn"], block=w["block"], eps=w["eps"],
                          heads_kv=w["heads_kv"], seq_ends=w["seq_ends"])
    blk.load({k: _dev(w[k]) for k in ("x", "n1", "n2", "wqkv", "wo", "wg", "wu", "wd")})
    work = blk.work()
    stages = blk.stages()
    comps = {name: dict(fn=fn, same_buffers=True, **work[name]) for name, fn in stages}
    flops = sum(c.get("flops", 0) for c in comps.values())
    n_seq = t // seq_len
    dominant = max(("swiglu_gemm", "attention"), key=lambda k: comps[k]["flops"])
    name = "w1_block_share" if (t, seq_len) == (8192, 1024) else f"w1_block_share_{n_seq}x{seq_len}"
    return dict(step=blk.forward, flops=flops, comps=comps, dominant=dominant,
                config={"workload": name, "hidden": 4096, "heads_q": "4 of 32", "heads_kv": "1 of 8",
                        "d_head": 128, "ffn": "1792 of 14336", "tokens": t,
                        "sequences": f"{n_seq} x {seq_len} packed" if n_seq > 1 else f"one of {seq_len}",
                        "block": 512, "dtype": "bf16", "chain": [n for n, _ in stages]},
                cpu=None)


def chains_workload():
    import synth
    from paper_2609_03905_amd import chain

    chains, comps, total = {}, {}, 0.0
    for name in sorted(synth.CHAINS):
        dims, tree = synth.CHAINS[name]
        ch = chain.MatrixChain(dims, tree)
        for i in range(len(dims) - 1):
            std = 1.0 if i == 0 else 1.0 / dims[i] ** 0.5
            ch.load(i, synth.chain_matrix_device((dims[i], dims[i + 1]), 900 + 20 * "ABCDE".index(name) + i, std))
        chains[name] = ch
        fl = chain.flops(dims, tree)
        comps[f"chain_{name}"] = dict(fn=ch.run, flops=fl)
        total += fl

    def step():
        for ch in chains.values():
            ch.run()

    return dict(step=step, flops=total, comps=comps, dominant="chain_E",
                data="synthetic (seeded on the device: first matrix N(0,1), matrix i N(0,1/d_i))",
                config={"workload": "matrix_chains_A_to_E", "chains": "A,B,C,D,E (Section 6 dims, fixed trees)",
                        "block": 512, "dtype": "bf16", "products": sum(len(chain.products(t)) for _, t in
                                                                     synth.CHAINS.values())},
                cpu=None)


def matmul_fp32_workload():
    """The 256^3 fp32 matmul join-agg 'ij,jk->ik', each input 4x4 blocks of
    64x64 (SUM of 4 partials per output key); 2 MiB of buffers, rotated
    through 1 GiB of copies like the other workloads."""
    import numpy as np
    import torch

    import synth
    from paper_2609_03905_amd import ea

    w = synth.matmul_256_fp32()
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    A0 = ea.from_dense(dev(w["A"]), "f32", w["pA"])
    B0 = ea.from_dense(dev(w["B"]), "f32", w["pB"])

    def make_set(i):
        A, B = (A0, B0) if i == 0 else (_copy(A0, ea), _copy(B0, ea))
        return A, B, ea.Relation((256, 256), "f32", w["pC"])

    rot = _Rotation(_buffer_sets(make_set, 3 * 256 * 256 * 4))

    def fn():
        A, B, C = rot.next()
        ea.joinagg(w["spec"], ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)

    flops = 2.0 * 256 ** 3
    return dict(step=fn, flops=flops, comps={"matmul_fp32": dict(fn=fn, flops=flops)}, dominant="matmul_fp32",
                config={"workload": "matmul_256_fp32", "spec": "ij,jk->ik", "blocks": "4x4 of 64x64", "dtype": "f32",
                        "buffer_sets": len(rot.sets)}, cpu=None)


def reductions_workload():
    import synth
    from paper_2609_03905_amd import ea

    w = synth.reductions()
    X0 = ea.from_dense(_dev(w["x"]), "bf16", w["px"])
    Wt = ea.from_dense(_dev(w["w"]), "bf16", w["pw"])
    S0 = ea.from_dense(_dev(w["s"]), "bf16", w["ps"])

    def make_set(i):
        X, S = (X0, S0) if i == 0 else (_copy(X0, ea), _copy(S0, ea))
        return X, ea.Relation((4096, 4096), "bf16", w["px"]), S, ea.Relation((4, 2048, 2048), "bf16", w["ps"])

    set_bytes = 2 * 4096 * 4096 * 2 + 2 * 4 * 2048 * 2048 * 2
    sets = _buffer_sets(make_set, set_bytes)
    rot, rot_r, rot_s = (_Rotation(sets) for _ in range(3))
    # standalone operators whose outputs nothing reads next: streamed stores
    st = ea.STORE_STREAM
    run_rms = lambda X, Y: ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=w["eps"], store=st)
    run_sm = lambda S, P: ea.joinagg("hqk->hqk", ea.OP_SOFTMAX, ea.AGG_LSE, [S], P, causal=True, store=st)
    rms = lambda: (lambda b: run_rms(b[0], b[1]))(rot_r.next())
    sm = lambda: (lambda b: run_sm(b[2], b[3]))(rot_s.next())

    def step():
        X, Y, S, P = rot.next()
        run_rms(X, Y)
        run_sm(S, P)

    rms_bytes = 2 * 4096 * 4096 * 2 + 4096 * 2
    sm_bytes = 4 * (2048 * 2049 // 2) * 2 + 4 * 2048 * 2048 * 2
    return dict(step=step, flops=0.0, comps={"rmsnorm": dict(fn=rms, bytes=rms_bytes),
                                            "causal_softmax": dict(fn=sm, bytes=sm_bytes)},
                dominant="rmsnorm", bytes=rms_bytes + sm_bytes,
                config={"workload": "reductions", "rmsnorm": "x[4096,4096] bf16, 8 column blocks",
                        "softmax": "s[4,2048,2048] bf16 causal, 256-key blocks", "dtype": "bf16",
                        "store": "stream", "buffer_sets": len(rot.sets)}, cpu=None)


def repartition_workload():
    """Local repartition at HBM scale: a [8192, 16384] bf16 relation (256 MiB,
    larger than the 256 MB Infinity Cache) re-blocked from 512x512 blocks to
    128-row blocks of full width.  A pure copy with a known byte count; its
    FETCH_SIZE / WRITE_SIZE readings are the scale factor for counter-derived
    traffic of the other kernels."""
    import torch

    import synth
    from paper_2609_03905_amd import ea

    shape = (8192, 16384)
    src = ea.Relation(shape, "bf16", [synth.splits(8192, 512), synth.splits(16384, 512)])
    dst = ea.Relation(shape, "bf16", [synth.splits(8192, 128), synth.whole(16384)])
    g = torch.Generator(device="cuda")
    g.manual_seed(601)
    src.bytes().copy_(torch.randint(0, 256, (src.nbytes,), dtype=torch.uint8, device="cuda", generator=g))
    fn = lambda: ea.repartition(src, dst, store=ea.STORE_STREAM)  # 256 MiB: larger than the caches
    nbytes = 2 * shape[0] * shape[1] * 2
    return dict(step=fn, flops=0.0, bytes=nbytes, comps={"repartition": dict(fn=fn, bytes=nbytes)},
                dominant="repartition",
                config={"workload": "repartition_256MiB", "shape": list(shape), "dtype": "bf16",
                        "from": "512x512 blocks", "to": "128 x 16384 blocks", "store": "stream"}, cpu=None)


# ---------------------------------------------------------------------------
# Every single-operator configuration of the target, measured next to the
# headline block step: time, rate, fraction of the bound's peak and the bar
# (>= 60% of bf16 MFMA peak for block GEMMs, >= 70% of HBM for the
# memory-bound operators; C1 and attention carry no bar).
# ---------------------------------------------------------------------------
PEAK_FP32_TFLOPS = 157.3  # MI355X fp32 (matrix) peak


def _rate(c, ms, peak_tflops=PEAK_BF16_TFLOPS):
    d = {"us": round(ms * 1e3, 3)}
    if "flops" in c:
        d["tflops"] = c["flops"] / ms / 1e9
        d["frac_peak"] = d["tflops"] / peak_tflops
    if "bytes" in c:
        d["gbs"] = c["bytes"] / ms / 1e6
        d["frac_peak"] = d["gbs"] / PEAK_HBM_GBS
    return d


def copy_ceiling_us(nbytes: int, n: int):
    """Practical ceiling of a memory-bound operator moving nbytes each way:
    the faster of a device-to-device copy (torch copy_, the runtime's copy
    kernel) and the library's own repartition between two one-block relations
    (a contiguous copy), with buffers rotated through >= 1 GiB like the
    operators' own workloads.  Returns (us, which)."""
    import torch

    from paper_2609_03905_amd import ea

    m = nbytes // 2
    sets = [(torch.empty(nbytes, dtype=torch.uint8, device="cuda"), torch.empty(nbytes, dtype=torch.uint8, device="cuda"))
            for _ in range(max(1, -(-ROTATE_BYTES // (2 * nbytes))))]
    rels = [(ea.Relation((m,), "bf16", [[0, m]], data=a), ea.Relation((m,), "bf16", [[0, m]], data=b)) for a, b in sets]
    rot_t, rot_r = _Rotation(sets), _Rotation(rels)
    t_copy = _events_ms(lambda: (lambda ab: ab[1].copy_(ab[0]))(rot_t.next()), n) * 1e3
    t_own = _events_ms(lambda: (lambda ab: ea.repartition(ab[0], ab[1], store=ea.STORE_STREAM))(rot_r.next()), n) * 1e3
    return (t_copy, "device copy") if t_copy <= t_own else (t_own, "library repartition")


def config_rows(n):
    import gc

    import torch

    rows = {}
    spec = [("C1_matmul_fp32_256", matmul_fp32_workload, "matmul_fp32", None, PEAK_FP32_TFLOPS),
            ("C2_qkv_gemm", qkv_workload, "joinagg_gemm", 0.60, PEAK_BF16_TFLOPS),
            ("C2_repartition", qkv_workload, "repartition", 0.70, None),
            ("C3_rmsnorm", reductions_workload, "rmsnorm", 0.70, None),
            ("C3_causal_softmax", reductions_workload, "causal_softmax", 0.70, None),
            ("C4_causal_attention", attention_workload, "attention", None, PEAK_BF16_TFLOPS)]
    built = {}
    for name, make, comp, bar, peak in spec:
        if make not in built:
            built.clear()
            gc.collect()
            torch.cuda.empty_cache()
            built[make] = make()
        wl = built[make]
        c = wl["comps"][comp]
        ms = _events_ms(c["fn"], n)
        d = _rate(c, ms, peak or PEAK_BF16_TFLOPS)
        d["workload"] = wl["config"]["workload"]
        if "buffer_sets" in wl["config"]:
            d["buffer_sets"] = wl["config"]["buffer_sets"]
        if bar is not None:
            d["bar_frac"] = bar
            d["meets_bar"] = bool(d["frac_peak"] >= bar)
        if "bytes" in c:  # memory-bound: against a copy moving the same bytes
            cu, how = copy_ceiling_us(int(c["bytes"]) // 2, n)
            d["copy_ceiling_us"] = round(cu, 3)
            d["copy_ceiling"] = how
            d["within_10pct_of_copy"] = bool(d["us"] <= 1.1 * cu)
        rows[name] = d
    built.clear()
    gc.collect()
    torch.cuda.empty_cache()
    return rows


def oracle_single_thread():
    """The oracle on one thread, timed on the two small configurations: the
    256^3 fp32 matmul and the QKV share's 12 MiB repartition (512x512 blocks
    to per-head 4096x128 blocks)."""
    import numpy as np

    import oracle
    import synth

    n0 = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        w = synth.matmul_256_fp32()
        a, b = synth.to_f64(w["A"], "f32"), synth.to_f64(w["B"], "f32")
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 1.0 or reps < 3:
            oracle.matmul(a, b)
            reps += 1
        c1 = (time.perf_counter() - t0) / reps
        q = synth.qkv_projection()
        y = np.random.default_rng(5).integers(0, 1 << 16, (4096, 1536), dtype=np.uint16)
        blocked = oracle.pack(y, q["pY"])
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 2.0 or reps < 3:
            oracle.repartition(blocked, q["pY"], q["pHead"], np.uint16)
            reps += 1
        c2 = (time.perf_counter() - t0) / reps
    finally:
        oracle.set_num_threads(n0)
    return {"C1_matmul_fp32_256": {"ms": c1 * 1e3, "gflops": 2.0 * 256 ** 3 / c1 / 1e9, "threads": 1},
            "C2_repartition": {"ms": c2 * 1e3, "gbs": 2 * 4096 * 1536 * 2 / c2 / 1e9, "threads": 1}}


# ---------------------------------------------------------------------------
# CPU baselines: the oracle, untuned, on a bounded sample of the workload
# ---------------------------------------------------------------------------
def _adaptive(run, first, cap, target_s):
    """Grow the sample (rows of the workload) until one run takes about a
    third of target_s, or the whole workload; then time as many runs of it
    as cover at least 10 s.  Returns (rows, repetitions, seconds of the
    timed repetitions)."""
    n = first
    while True:
        t0 = time.perf_counter()
        run(n)
        dt = time.perf_counter() - t0
        if dt >= target_s / 3 or n >= cap:
            break
        n = min(cap, max(2 * n, int(n * target_s / 3 / max(dt, 1e-3))))
    reps = max(1, -int(-10.0 // max(dt, 1e-3)))
    t0 = time.perf_counter()
    for _ in range(reps):
        run(n)
    return n, reps, time.perf_counter() - t0


def cpu_baseline_block(target_s: float = 12.0):
    import numpy as np

    import oracle
    import synth

    w = synth.llama_block()
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    run = lambda rows: oracle.llama_block(f["x"][:rows], f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"],
                                          f["n2"], heads=8, d_head=128, eps=1e-6)
    rows, reps, dt = _adaptive(run, 16, 2048, target_s)
    dense = 2 * rows * (8192 * 3072 + 1024 * 8192 + 2 * 8192 * 2752 + 2752 * 8192)
    attn = 4 * 128 * 8 * rows * (rows + 1) // 2
    return {"value": (dense + attn) * reps / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"fp64 oracle block chain on the first {rows} of 2048 tokens (causal prefix), "
                      f"{reps} run(s) in {dt:.1f} s"}


def cpu_baseline_qkv(target_s: float = 12.0):
    import oracle
    import synth

    w = synth.qkv_projection()
    x, wt = synth.to_f64(w["X"], "bf16"), synth.to_f64(w["W"], "bf16")
    rows, reps, dt = _adaptive(lambda r: oracle.matmul(x[:r], wt), 16, 4096, target_s)
    return {"value": 2.0 * rows * 4096 * 1536 * reps / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": f"fp64 oracle matmul of {rows} of 4096 output rows, {reps} run(s) in {dt:.1f} s"}


WORKLOADS = {"block": block_workload, "qkv": qkv_workload, "attention": attention_workload,
             "packed_gqa": packed_gqa_workload, "w1_block": w1_block_workload, "w1_1k": lambda: w1_block_workload(1024, 1024),
             "w1_8k": lambda: w1_block_workload(8192, 8192), "w1_128k": lambda: w1_block_workload(131072, 131072),
             "w1_128x1k": lambda: w1_block_workload(131072, 1024), "chains": chains_workload,
             "reductions": reductions_workload, "matmul_fp32": matmul_fp32_workload,
             "repartition": repartition_workload}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="block", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the single-operator configuration rows")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share on one GPU; --gpus {args.gpus} is not supported "
              "(exchanges between GPUs are outside this build)", file=sys.stderr)
        sys.exit(2)

    import torch

    torch.cuda.set_device(0)
    wl = WORKLOADS[args.workload]()
    step = wl["step"]
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Events only at the boundaries of a few batches of steps: a timing event
    # recorded between two steps leaves the GPU idle for about 6 us (measured
    # in a kernel trace of the block chain), which per-step events would add
    # to every step.  The 95% interval comes from the batch means.
    n_batch = min(5, args.steps)
    bounds = [round(b * args.steps / n_batch) for b in range(n_batch + 1)]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_batch + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for b in range(n_batch):
        for _ in range(bounds[b + 1] - bounds[b]):
            step()
        ev[b + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = ev[0].elapsed_time(ev[-1]) / args.steps
    per = [ev[b].elapsed_time(ev[b + 1]) / (bounds[b + 1] - bounds[b]) for b in range(n_batch)]
    sd = (sum((x - ms_per_step) ** 2 for x in per) / max(1, len(per) - 1)) ** 0.5
    ci95 = 1.96 * sd / max(1, len(per)) ** 0.5  # normal approximation of the mean's 95% interval

    comps = {}
    for name, c in wl["comps"].items():
        ms = _events_ms(c["fn"], max(args.steps, 20))
        d = {"ms": round(ms, 5), "host_us": round(_host_us_per_call(c["fn"], 20), 2)}
        if "flops" in c:
            d["tflops"] = c["flops"] / ms / 1e9
            d["frac_mfma_peak"] = d["tflops"] / PEAK_BF16_TFLOPS
        if "bytes" in c:
            d["gbs"] = c["bytes"] / ms / 1e6
            d["frac_hbm_peak"] = d["gbs"] / PEAK_HBM_GBS
            if c.get("same_buffers"):
                # a chain stage re-run on its own buffers: inputs under 256 MB
                # stay in the Infinity Cache between launches, so this is not
                # an HBM rate (the configs rows rotate buffers for that)
                d["same_buffers"] = True
                d["rate_note"] = "repeated launches on one buffer set; inputs may be served by the Infinity Cache"
        comps[name] = d
    dom = wl["comps"][wl["dominant"]]
    dms = comps[wl["dominant"]]["ms"]
    if "flops" in dom:
        achieved = dom["flops"] / dms / 1e9
        roof = {"kernel": wl["dominant"], "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": _profiled_traffic(wl["dominant"])}
    else:
        achieved = dom["bytes"] / dms / 1e6
        roof = {"kernel": wl["dominant"], "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None}

    if wl["flops"]:
        value, unit = wl["flops"] / ms_per_step / 1e9, "TFLOP/s"
    else:
        value, unit = wl["bytes"] / ms_per_step / 1e6, "GB/s"
    out = {
        "metric": METRIC, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "ms_per_step_ci95": [ms_per_step - ci95, ms_per_step + ci95],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": wl.get("data", "synthetic (seeded N(0,1) activations, N(0,0.02) weights, random init)"),
        "config": wl["config"], "roofline": roof, "components": comps, "wall_s": round(wall, 4),
    }
    if args.workload == "block" and not args.no_configs:
        out["configs"] = config_rows(max(args.steps, 20))
    if not args.no_cpu_baseline and out["config"]["workload"] == "llama65b_block_share":
        out["cpu_baseline"] = cpu_baseline_block()
        out["cpu_single_thread"] = oracle_single_thread()
    elif not args.no_cpu_baseline and wl.get("cpu"):
        out["cpu_baseline"] = wl["cpu"]()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
