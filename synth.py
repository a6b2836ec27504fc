"""Seeded synthetic inputs and workload recipes.

This module is shared by the oracle side (tests, CPU baseline) and the GPU side
(bench, smoke, GPU tests).  It holds no arithmetic of the join-agg method: it
only draws random numbers, stores them in the workload's dtype, and describes
shapes and block partitions.

Generator: numpy PCG64 (``numpy.random.default_rng(seed)``).  Normal draws are
taken in fp64, scaled by the standard deviation, cast to fp32, and, for bf16
tensors, rounded to bf16 with torch's round-to-nearest-even cast.  bf16 tensors
are carried as uint16 bit patterns; ``to_f64`` widens them exactly.
"""
from __future__ import annotations

import numpy as np
import torch

ELEM_SIZE = {"f32": 4, "bf16": 2, "f16": 2}


# --------------------------------------------------------------------------
# storage conversions (exact widening; rounding only through torch's cast)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of a stored tensor."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    if dtype == "f16":
        return np.asarray(a).view(np.float16).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp32/fp64 values -> stored representation of ``dtype``."""
    x = np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f16":
        return x.astype(np.float16).view(np.uint16)
    return np.ascontiguousarray(x)


# --------------------------------------------------------------------------
# draws
# --------------------------------------------------------------------------
def normal(shape, seed: int, std: float = 1.0, dtype: str = "bf16") -> np.ndarray:
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(size=shape) * std).astype(np.float32)
    return store(x, dtype)


def uniform(shape, seed: int, lo: float, hi: float, dtype: str = "bf16") -> np.ndarray:
    rng = np.random.default_rng(seed)
    x = rng.uniform(lo, hi, size=shape).astype(np.float32)
    return store(x, dtype)


def integers(shape, seed: int, lo: int, hi: int, dtype: str = "bf16") -> np.ndarray:
    """Small integers in [lo, hi], exactly representable in every dtype here."""
    rng = np.random.default_rng(seed)
    x = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    return store(x, dtype)


# --------------------------------------------------------------------------
# partitions: one list of split points per dim
# --------------------------------------------------------------------------
def splits(extent: int, block: int) -> list[int]:
    """[0, block, 2*block, ..., extent]; the last interval may be shorter."""
    pts = list(range(0, extent, block)) + [extent]
    return pts


def random_splits(extent: int, nblocks: int, rng: np.random.Generator, quantum: int = 1) -> list[int]:
    """Random non-uniform split points, each a multiple of ``quantum``."""
    units = extent // quantum
    nblocks = max(1, min(nblocks, units))
    cuts = sorted(rng.choice(np.arange(1, units), size=nblocks - 1, replace=False).tolist()) if nblocks > 1 else []
    return [0] + [c * quantum for c in cuts] + [extent]


def whole(extent: int) -> list[int]:
    return [0, extent]


# --------------------------------------------------------------------------
# the five workloads (shapes, partitions, distributions, seeds)
# --------------------------------------------------------------------------
def matmul_256_fp32():
    """Single matmul join-agg 'ij,jk->ik', fp32, 256^3, 4x4 blocks of 64x64."""
    A = normal((256, 256), 101, 1.0, "f32")
    B = normal((256, 256), 102, 1.0, "f32")
    p = [splits(256, 64), splits(256, 64)]
    return dict(spec="ij,jk->ik", A=A, B=B, pA=p, pB=p, pC=p, dtype="f32")


def qkv_projection(t=4096, j=4096, k=1536, block=512, head=128):
    """LLaMA-7B QKV projection, one GPU's 1/8 column share, bf16, 512^2 blocks,
    then repartition of the output to per-head [t, 128] blocks."""
    X = normal((t, j), 201, 1.0, "bf16")
    W = normal((j, k), 202, 0.02, "bf16")
    pX = [splits(t, block), splits(j, block)]
    pW = [splits(j, block), splits(k, block)]
    pY = [splits(t, block), splits(k, block)]
    pHead = [whole(t), splits(k, head)]
    return dict(spec="tj,jk->tk", X=X, W=W, pX=pX, pW=pW, pY=pY, pHead=pHead, dtype="bf16")


def reductions(t=4096, c=4096, cblock=512, heads=4, seq=2048, kblock=256):
    """RMSNorm over x[t, c] in 8 column blocks; causal softmax over scores
    [heads, seq, seq] in key blocks of 256."""
    x = normal((t, c), 301, 1.0, "bf16")
    w = uniform((c,), 302, 0.5, 1.5, "bf16")
    s = normal((heads, seq, seq), 303, 1.0, "bf16")
    px = [whole(t), splits(c, cblock)]
    pw = [splits(c, cblock)]
    ps = [splits(heads, 1), whole(seq), splits(seq, kblock)]
    return dict(x=x, w=w, s=s, px=px, pw=pw, ps=ps, eps=1e-6)


def attention(b=2, h=4, s=2048, d=128, qblock=128, kblock=128):
    """Causal attention, one GPU's head share of LLaMA-7B, bf16."""
    q = normal((b, h, s, d), 401, 1.0, "bf16")
    k = normal((b, h, s, d), 402, 1.0, "bf16")
    v = normal((b, h, s, d), 403, 1.0, "bf16")
    pq = [splits(b, 1), splits(h, 1), splits(s, qblock), whole(d)]
    pk = [splits(b, 1), splits(h, 1), splits(s, kblock), whole(d)]
    return dict(q=q, k=k, v=v, pq=pq, pk=pk, scale=1.0 / np.sqrt(d))


def packed_gqa_attention(n_seq=8, seq_len=1024, heads_q=4, heads_kv=1, d=128, block=128):
    """Causal attention over packed sequences with grouped-query heads: one
    GPU's head share (4 query heads over 1 key/value head = 32 over 8 split
    eight ways) of a 4096-wide, 32-head LLaMA-style model on a batch of eight
    1K-token sequences packed end to end, bf16."""
    s = n_seq * seq_len
    q = normal((1, heads_q, s, d), 411, 1.0, "bf16")
    k = normal((1, heads_kv, s, d), 412, 1.0, "bf16")
    v = normal((1, heads_kv, s, d), 413, 1.0, "bf16")
    pq = [[0, 1], splits(heads_q, 1), splits(s, block), whole(d)]
    pk = [[0, 1], splits(heads_kv, 1), splits(s, block), whole(d)]
    ends = [seq_len * (i + 1) for i in range(n_seq)]
    return dict(q=q, k=k, v=v, pq=pq, pk=pk, ends=ends, scale=1.0 / np.sqrt(d), gqa=heads_q // heads_kv)


def _right_nested(first: int, last: int):
    """(first, (first + 1, ( ... (last - 1, last))))."""
    return last if first == last else (first, _right_nested(first + 1, last))


# The matrix chains of Section 6: dims (matrix i is [dims[i], dims[i+1]]) and
# parenthesization (nested pairs of 0-based matrix indices); each multiply
# averages about 8192^3 scalar multiplies
CHAINS = {
    # nine matrices, dims alternating 16,384 and 6,144 between ends of 10,240:
    # (M1 M2) (((M3 M4) ((M5 M6) (M7 M8))) M9)
    "A": ([10240, 16384, 6144, 16384, 6144, 16384, 6144, 16384, 6144, 10240],
          ((0, 1), (((2, 3), ((4, 5), (6, 7))), 8))),
    # five matrices, dims alternating 20,480 and 5,120 between ends of 9,216:
    # (M1 M2) ((M3 M4) M5)
    "B": ([9216, 20480, 5120, 20480, 5120, 9216], ((0, 1), ((2, 3), 4))),
    # three matrices, right-associated: M1 (M2 M3)
    "C": ([10240, 12288, 32768, 2048], (0, (1, 2))),
    # nine matrices, ends 24,576, necks 1,536, interior 20,480:
    # M1 ((M2 (M3 (M4 (M5 (M6 (M7 M8)))))) M9)
    "D": ([24576, 1536] + [20480] * 6 + [1536, 24576], (0, (_right_nested(1, 7), 8))),
    # thirteen matrices, ends 49,152, necks 1,024, interior 20,480:
    # M1 ((M2 (M3 ( ... (M11 M12)))) M13)
    "E": ([49152, 1024] + [20480] * 10 + [1024, 49152], (0, (_right_nested(1, 11), 12))),
}


def w1_block(t=8192, hidden=4096, heads=4, heads_kv=1, d_head=128, ffn=1792, block=512, seq_len=1024):
    """One GPU's head share (8-way) of the paper's LLaMA-scale block: model
    dim 4096, 32 query heads over 8 key/value heads of dim 128, FFN 14336,
    on a batch of eight 1K-token sequences packed end to end."""
    qkv = (heads + 2 * heads_kv) * d_head
    hd = heads * d_head
    x = normal((t, hidden), 521, 1.0, "bf16")
    wqkv = normal((hidden, qkv), 522, 0.02, "bf16")
    wo = normal((hd, hidden), 523, 0.02, "bf16")
    wg = normal((hidden, ffn), 524, 0.02, "bf16")
    wu = normal((hidden, ffn), 525, 0.02, "bf16")
    wd = normal((ffn, hidden), 526, 0.02, "bf16")
    n1 = uniform((hidden,), 527, 0.5, 1.5, "bf16")
    n2 = uniform((hidden,), 528, 0.5, 1.5, "bf16")
    return dict(x=x, wqkv=wqkv, wo=wo, wg=wg, wu=wu, wd=wd, n1=n1, n2=n2, t=t, hidden=hidden, heads=heads,
                heads_kv=heads_kv, d_head=d_head, ffn=ffn, block=block, eps=1e-6,
                seq_ends=list(range(seq_len, t + 1, seq_len)))


def chain_matrices(dims, seed: int, div: int = 1):
    """Matrices of a matrix chain (dims divided by `div`), bf16, host: matrix
    i is [d_i, d_(i+1)] with N(0, 1/d_i) entries (N(0, 1) for the first), so
    every product of the chain stays of order one."""
    d = [x // div for x in dims]
    return [normal((d[i], d[i + 1]), seed + i, 1.0 if i == 0 else 1.0 / np.sqrt(d[i]), "bf16")
            for i in range(len(d) - 1)], d


def chain_matrix_device(shape, seed: int, std: float, device="cuda"):
    """One full-size chain matrix drawn on the device (torch's seeded
    generator, N(0, std^2), fp32 then RNE to bf16), for runs with no oracle
    check: full-size chains hold up to 7.5 GB of inputs."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std).to(torch.bfloat16)


def llama_block(t=2048, hidden=8192, heads=8, d_head=128, ffn=2752, block=512):
    """One GPU's share of a LLaMA-65B-shape block: hidden 8192, 8 of 64 heads,
    SwiGLU FFN 2752 = 22016/8, batch 1 x seq 2048."""
    qkv = 3 * heads * d_head
    hd = heads * d_head
    x = normal((t, hidden), 501, 1.0, "bf16")
    wqkv = normal((hidden, qkv), 502, 0.02, "bf16")
    wo = normal((hd, hidden), 503, 0.02, "bf16")
    wg = normal((hidden, ffn), 504, 0.02, "bf16")
    wu = normal((hidden, ffn), 505, 0.02, "bf16")
    wd = normal((ffn, hidden), 506, 0.02, "bf16")
    n1 = uniform((hidden,), 507, 0.5, 1.5, "bf16")
    n2 = uniform((hidden,), 508, 0.5, 1.5, "bf16")
    return dict(x=x, wqkv=wqkv, wo=wo, wg=wg, wu=wu, wd=wd, n1=n1, n2=n2,
                t=t, hidden=hidden, heads=heads, d_head=d_head, ffn=ffn, block=block, eps=1e-6)
