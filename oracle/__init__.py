"""CPU oracle for the block join-agg hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never loads it, and
it imports nothing from the product package: the two share no code.  The only
module both sides use is ``synth`` (seeded input generators, no arithmetic of
the method).

Each function computes the plain dense definition of a result in fp64 (C loops
in ``ea_oracle.c``, OpenMP over output rows).  Blocks appear only where they are
the result itself: the block layout, the join's tuple table and the
repartition.  Citations refer to "Every Kernel Is a Join" (Einsummable): its
sections, definitions and examples.

Partitions are given as a list with one entry per dim, each entry the split
points ``[0, s1, ..., extent]`` of that dim (non-uniform splits allowed).

Pin status (what each function is checked against, in tests/test_oracle_pins.py):
  rne_bf16 ......... torch's round-to-nearest-even cast (library routine)
  layout/pack ...... 1-block identity, explicit small-case byte positions
  repartition ...... round trips, dense-view equality, the overlay example
  join ............. the paper's worked matmul example (Section 3.2/3.3),
                     the product-of-intervals count rule, causal closed-form count
  einsum ........... numpy.einsum (library), brute-force max, decomposition
                     invariance with integer data (bit-exact)
  matmul ........... numpy.matmul (library), identity/zero closed forms
  rmsnorm .......... torch rms_norm (library), constant-row closed form
  softmax .......... torch softmax (library), constant-row 1/(q+1) closed form
  attention ........ torch scaled_dot_product_attention (library), equal-V and
                     zero-K closed forms; grouped-query heads against SDPA on
                     K/V heads repeated per group, packed sequences against
                     SDPA run on each sequence alone
  join (attention predicates) grouped-query and packed-sequence tuple counts
                     in closed form (the paper's three-sequence example)
  llama_block ...... composition of the pinned parts only: the paper does not
                     define the block, so its chain is "parity unpinned" beyond
                     that composition
"""
from __future__ import annotations

import ctypes
import itertools
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ea_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

JOIN_MUL, JOIN_ADD = 0, 1
AGG_NONE, AGG_SUM, AGG_MAX = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C, OpenMP, no BLAS)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        i64p = ctypes.POINTER(ctypes.c_int64)
        dp = ctypes.POINTER(ctypes.c_double)
        L.or_num_threads.restype = ctypes.c_int
        L.or_set_num_threads.argtypes = [ctypes.c_int]
        L.or_rne_bf16.argtypes = [ctypes.c_int64, dp, dp]
        L.or_layout.argtypes = [ctypes.c_int, i64p, i64p, ctypes.c_int64, i64p, i64p]
        L.or_pack.argtypes = [ctypes.c_int, i64p, i64p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        L.or_unpack.argtypes = L.or_pack.argtypes
        L.or_join.restype = ctypes.c_int64
        L.or_join.argtypes = [ctypes.c_char_p, i64p, i64p, ctypes.c_char_p, ctypes.c_char, ctypes.c_char,
                              ctypes.POINTER(ctypes.c_int32), ctypes.c_int64, i64p, ctypes.c_int64, i64p]
        L.or_join_ex.restype = ctypes.c_int64
        L.or_join_ex.argtypes = [ctypes.c_char_p, i64p, i64p, ctypes.c_char_p, ctypes.c_char, ctypes.c_char,
                                 ctypes.c_int, ctypes.c_int64, i64p, ctypes.c_int64, ctypes.c_char, ctypes.c_char,
                                 ctypes.POINTER(ctypes.c_int32), ctypes.c_int64, i64p, ctypes.c_int64, i64p]
        L.or_einsum.argtypes = [ctypes.c_char_p, ctypes.c_int, ctypes.c_int, i64p,
                                ctypes.POINTER(dp), dp]
        L.or_matmul.argtypes = [ctypes.c_int64] * 3 + [dp, dp, dp]
        L.or_rmsnorm.argtypes = [ctypes.c_int64, ctypes.c_int64, dp, dp, ctypes.c_double, dp]
        L.or_softmax.argtypes = [ctypes.c_int64] * 3 + [dp, ctypes.c_int, dp]
        L.or_attention.argtypes = [ctypes.c_int64] * 4 + [dp, dp, dp, ctypes.c_int, ctypes.c_double, dp]
        L.or_attention_ex.argtypes = [ctypes.c_int64] * 5 + [dp, dp, dp, ctypes.c_int, ctypes.c_double,
                                                            ctypes.c_int64, i64p, dp]
        L.or_silu_mul.argtypes = [ctypes.c_int64, dp, dp, dp]
        L.or_add.argtypes = [ctypes.c_int64, dp, dp, dp]
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().or_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (timing only)."""
    lib().or_set_num_threads(int(n))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _i64p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with code {rc}")


# --------------------------------------------------------------------------
# rounding
# --------------------------------------------------------------------------
def rne_bf16(x) -> np.ndarray:
    """fp64 -> bf16 round-to-nearest-even, returned as fp64 values."""
    x = _f64(x)
    y = np.empty_like(x)
    _check(lib().or_rne_bf16(x.size, _dp(x), _dp(y)), "rne_bf16")
    return y


# --------------------------------------------------------------------------
# relation layout (Section 3.1 tensor types / tilings; Section 1 relations)
# --------------------------------------------------------------------------
def _flat_partition(partition):
    nb = _i64([len(s) - 1 for s in partition])
    sp = _i64([p for s in partition for p in s])
    return nb, sp


def layout(partition, elem_size: int):
    """Byte offset of every block (row-major block order) and total bytes."""
    nb, sp = _flat_partition(partition)
    n = int(np.prod(nb))
    offs = np.empty(n, dtype=np.int64)
    nbytes = np.zeros(1, dtype=np.int64)
    _check(lib().or_layout(len(partition), _i64p(nb), _i64p(sp), elem_size, _i64p(offs), _i64p(nbytes)),
           "layout")
    return offs, int(nbytes[0])


def pack(dense: np.ndarray, partition) -> np.ndarray:
    """Dense row-major tensor -> block-major relation bytes (uint8)."""
    dense = np.ascontiguousarray(dense)
    shape = tuple(s[-1] for s in partition)
    if dense.shape != shape:
        raise ValueError(f"dense shape {dense.shape} does not match partition extents {shape}")
    es = dense.dtype.itemsize
    _, nbytes = layout(partition, es)
    out = np.zeros(nbytes, dtype=np.uint8)
    nb, sp = _flat_partition(partition)
    _check(lib().or_pack(len(partition), _i64p(nb), _i64p(sp), es, dense.ctypes.data, out.ctypes.data), "pack")
    return out


def unpack(blocked: np.ndarray, partition, dtype) -> np.ndarray:
    """Block-major relation bytes -> dense row-major tensor of ``dtype``."""
    dtype = np.dtype(dtype)
    shape = tuple(s[-1] for s in partition)
    _, nbytes = layout(partition, dtype.itemsize)
    blocked = np.ascontiguousarray(blocked).view(np.uint8)
    if blocked.size < nbytes:
        raise ValueError("relation buffer smaller than its layout")
    out = np.empty(shape, dtype=dtype)
    nb, sp = _flat_partition(partition)
    _check(lib().or_unpack(len(partition), _i64p(nb), _i64p(sp), dtype.itemsize, blocked.ctypes.data,
                           out.ctypes.data), "unpack")
    return out


def repartition(blocked: np.ndarray, src_partition, dst_partition, dtype) -> np.ndarray:
    """The same dense tensor under a new partition: dst block b, element r is
    dense[lo_b + r] (Section 5.3: decompose into atoms, recompose)."""
    return pack(unpack(blocked, src_partition, dtype), dst_partition)


# --------------------------------------------------------------------------
# join (Section 3.2 Definitions "Join-agg spec" and "Implementation" step 1)
# --------------------------------------------------------------------------
def join(spec: str, partitions, group: str | None = None, causal: tuple[str, str] | None = None,
         positions: tuple[str, str] | None = None, seq_ends=None, gqa: tuple[int, str, str] | None = None):
    """Brute-force join of block relations.

    partitions: one partition per operand (inputs, then the output).
    group: letters whose block coordinates form the group key (default: the
    output letters).  causal: (q_letter, k_letter) keeps a tuple iff some q
    position of its q block is at or after some k position of its k block.
    Attention predicates (Section 3.3, Example "Flash attention"):
    positions (q_letter, k_letter) with seq_ends, the ends of packed
    sequences, keep a tuple iff some q position and some k position of its
    blocks lie in one sequence (and satisfy causal order, if causal);
    gqa (G, h_letter, g_letter) keeps it iff every query head h of its
    h block reads key/value head h // G inside its g block.
    Returns (tuples int32 [n, 1 + n_in] = (out_block, in_blocks...), group_off int64).
    """
    out_letters = spec.split("->")[1]
    if group is None:
        group = out_letters
    nb = _i64([len(s) - 1 for part in partitions for s in part])
    sp = _i64([p for part in partitions for s in part for p in s])
    n_in = len(spec.split("->")[0].split(","))
    ng = np.zeros(1, dtype=np.int64)
    pos = causal or positions
    pq = pos[0].encode() if pos else b"\0"
    pk = pos[1].encode() if pos else b"\0"
    ends = _i64(seq_ends if seq_ends is not None else [0])
    n_seq = 0 if seq_ends is None else len(seq_ends)
    G, gh, gg = (gqa[0], gqa[1].encode(), gqa[2].encode()) if gqa else (1, b"\0", b"\0")
    L = lib()

    def call(tp, cap, go, gcap):
        return L.or_join_ex(spec.encode(), _i64p(nb), _i64p(sp), group.encode(), pq, pk, int(causal is not None),
                            n_seq, _i64p(ends), G, gh, gg, tp, cap, go, gcap, _i64p(ng))

    n = call(None, 0, None, 0)
    if n < 0:
        raise ValueError(f"oracle join failed with code {n}")
    tuples = np.zeros((max(n, 1), n_in + 1), dtype=np.int32)
    goff = np.zeros(int(ng[0]) + 1, dtype=np.int64)
    n2 = call(tuples.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), tuples.shape[0], _i64p(goff), goff.size)
    if n2 != n:
        raise ValueError(f"oracle join failed with code {n2}")
    return tuples[:n], goff


# --------------------------------------------------------------------------
# dense numerics (fp64)
# --------------------------------------------------------------------------
def einsum(spec: str, inputs, join_op: int = JOIN_MUL, agg_op: int = AGG_SUM, out_shape=None) -> np.ndarray:
    """Dense join-agg: out[o] = AGG over contracted letters of JOIN(inputs)."""
    ins = [_f64(a) for a in inputs]
    lhs, rhs = spec.split("->")
    in_specs = lhs.split(",")
    if len(in_specs) != len(ins):
        raise ValueError("input count does not match the spec")
    sizes = {}
    for s, a in zip(in_specs, ins):
        for l, n in zip(s, a.shape):
            sizes[l] = n
    oshape = tuple(sizes[l] for l in rhs) if out_shape is None else tuple(out_shape)
    out = np.empty(oshape, dtype=np.float64)
    shapes = _i64([n for a in ins for n in a.shape] + list(oshape))
    arr = (ctypes.POINTER(ctypes.c_double) * len(ins))(*[_dp(a) for a in ins])
    _check(lib().or_einsum(spec.encode(), join_op, agg_op, _i64p(shapes), arr, _dp(out)), "einsum")
    return out


def matmul(a, b) -> np.ndarray:
    a, b = _f64(a), _f64(b)
    M, K = a.shape
    K2, N = b.shape
    if K != K2:
        raise ValueError("inner dims differ")
    c = np.empty((M, N), dtype=np.float64)
    _check(lib().or_matmul(M, K, N, _dp(a), _dp(b), _dp(c)), "matmul")
    return c


def rmsnorm(x, w, eps: float) -> np.ndarray:
    x, w = _f64(x), _f64(w)
    T, C = x.shape
    y = np.empty_like(x)
    _check(lib().or_rmsnorm(T, C, _dp(x), _dp(w), eps, _dp(y)), "rmsnorm")
    return y


def softmax(s, causal: bool) -> np.ndarray:
    s = _f64(s)
    H, Q, K = s.shape
    p = np.empty_like(s)
    _check(lib().or_softmax(H, Q, K, _dp(s), int(causal), _dp(p)), "softmax")
    return p


def attention(q, k, v, causal: bool, scale: float) -> np.ndarray:
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, S, D = q.shape
    o = np.empty_like(q)
    _check(lib().or_attention(B, H, S, D, _dp(q), _dp(k), _dp(v), int(causal), scale, _dp(o)), "attention")
    return o


def attention_ex(q, k, v, causal: bool, scale: float, seq_ends=None) -> np.ndarray:
    """Attention with grouped-query heads (k, v [B, Hkv, S, D], query head h
    reading key/value head h // (Hq // Hkv)) and packed sequences ending at
    seq_ends (None: one sequence); Section 3.3, Example "Flash attention"."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    ends = _i64(seq_ends if seq_ends is not None else [S])
    o = np.empty_like(q)
    _check(lib().or_attention_ex(B, Hq, Hkv, S, D, _dp(q), _dp(k), _dp(v), int(causal), scale,
                                 0 if seq_ends is None else len(ends), _i64p(ends), _dp(o)), "attention_ex")
    return o


def silu_mul(g, u) -> np.ndarray:
    g, u = _f64(g), _f64(u)
    y = np.empty_like(g)
    _check(lib().or_silu_mul(g.size, _dp(g), _dp(u), _dp(y)), "silu_mul")
    return y


def add(a, b) -> np.ndarray:
    a, b = _f64(a), _f64(b)
    y = np.empty_like(a)
    _check(lib().or_add(a.size, _dp(a), _dp(b), _dp(y)), "add")
    return y


# --------------------------------------------------------------------------
# composite: one GPU's share of a pre-norm LLaMA-shaped block
# --------------------------------------------------------------------------
def llama_block(x, n1, wqkv, wo, wg, wu, wd, n2, heads: int, d_head: int, eps: float, heads_kv: int | None = None,
                seq_ends=None):
    """The block chain with a bf16 round-to-nearest-even at every relation
    boundary (each arrow of the chain below stores a bf16 relation):

      h1 = RMSNorm(x; n1) -> qkv = h1 W_qkv -> attn = CausalAttn(q, k, v)
      -> x2 = x + attn W_o -> h2 = RMSNorm(x2; n2)
      -> a = SiLU(h2 W_g) * (h2 W_u) -> y = x2 + a W_d

    qkv's columns are [Q heads | K heads | V heads], head h of each taking
    columns [h*d_head, (h+1)*d_head) of its part; with heads_kv < heads the K
    and V parts have heads_kv heads (grouped-query attention), and seq_ends
    packs independent sequences along the tokens.  RoPE is not part of the chain.  Causal
    attention makes row t of every output depend only on rows <= t of x, so a
    prefix of x yields the same prefix of y.  All inputs are fp64 values.
    Returns every boundary relation as a dict of dense fp64 arrays.
    """
    r = rne_bf16
    T = x.shape[0]
    hkv = heads if heads_kv is None else heads_kv
    hd, kvd = heads * d_head, hkv * d_head
    h1 = r(rmsnorm(x, n1, eps))
    qkv = r(matmul(h1, wqkv))

    def heads_view(cols, n):
        return np.ascontiguousarray(cols.reshape(T, n, d_head).transpose(1, 0, 2))[None]

    q = heads_view(qkv[:, 0:hd], heads)
    k = heads_view(qkv[:, hd:hd + kvd], hkv)
    v = heads_view(qkv[:, hd + kvd:hd + 2 * kvd], hkv)
    if hkv == heads and seq_ends is None:
        o = r(attention(q, k, v, True, 1.0 / np.sqrt(d_head)))
    else:
        o = r(attention_ex(q, k, v, True, 1.0 / np.sqrt(d_head), seq_ends=seq_ends))
    attn = np.ascontiguousarray(o[0].transpose(1, 0, 2).reshape(T, hd))
    x2 = r(add(x, matmul(attn, wo)))
    h2 = r(rmsnorm(x2, n2, eps))
    a = r(silu_mul(matmul(h2, wg), matmul(h2, wu)))
    y = r(add(x2, matmul(a, wd)))
    return dict(h1=h1, qkv=qkv, attn=attn, x2=x2, h2=h2, a=a, y=y)


def attention_rows(q, k, v, rows, scale: float, seq_ends=None) -> np.ndarray:
    """Causal attention evaluated at the query positions ``rows`` only.

    q [Hq, S, D]; k and v [Hkv, S, D], query head h reading key/value head
    h // (Hq // Hkv); seq_ends: ends of packed sequences along S (None: one
    sequence).  Query t of head h takes the softmax of its scaled scores
    against the keys of its own sequence at positions <= t and returns the
    weighted sum of their values (Section 3.3, Example "Flash attention";
    the per-row formula attention_ex evaluates at every row).  Ends at or
    below 0 are ignored, so a window that starts inside the tokens can pass
    ends shifted by its start.  Returns [len(rows), Hq, D]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    Hq, S, D = q.shape
    group = Hq // k.shape[0]
    rows = np.asarray(rows, dtype=np.int64)
    ends = np.asarray(seq_ends if seq_ends is not None else [S], dtype=np.int64)
    o = np.empty((len(rows), Hq, D))
    for i, t in enumerate(rows):
        before = ends[ends <= t]
        s0 = int(before.max()) if before.size and before.max() > 0 else 0
        for h in range(Hq):
            m = h // group
            sc = (k[m, s0:t + 1] @ q[h, t]) * scale
            pr = np.exp(sc - sc.max())
            o[i, h] = (pr @ v[m, s0:t + 1]) / pr.sum()
    return o


def llama_block_rows(x, n1, wqkv, wo, wg, wu, wd, n2, heads: int, d_head: int, eps: float, rows,
                     heads_kv: int | None = None, seq_ends=None):
    """Rows `rows` of llama_block's boundary relations, for sequences too long
    for the whole chain in fp64 on the CPU.  h1 and qkv are computed for the
    tokens the rows read (from the start of the earliest row's sequence to
    the last row).  Attention is then evaluated only at the sampled query
    rows: query t of head h takes the softmax of its scaled scores against
    the keys of key/value head h // (heads // heads_kv) from the start of
    its sequence through t, and returns the weighted sum of their values
    (Section 3.3, Example "Flash attention"; the per-row formula that
    attention_ex evaluates at every row).  The remaining stages are
    row-wise.  The same bf16 rounding is applied at every relation boundary.
    Returns a dict of [len(rows), ...] fp64 arrays, rows in ascending order."""
    r = rne_bf16
    x = _f64(x)
    T = x.shape[0]
    hkv = heads if heads_kv is None else heads_kv
    hd, kvd = heads * d_head, hkv * d_head
    ends = np.asarray(seq_ends if seq_ends is not None else [T], dtype=np.int64)
    rows = np.unique(np.asarray(rows, dtype=np.int64))
    starts = np.array([int(ends[ends <= t].max()) if np.any(ends <= t) else 0 for t in rows], dtype=np.int64)
    lo, hi = int(starts.min()), int(rows.max()) + 1
    h1 = r(rmsnorm(x[lo:hi], n1, eps))
    qkv = r(matmul(h1, wqkv))

    def heads_of(cols, n):  # [n, hi - lo, d_head]
        return cols.reshape(hi - lo, n, d_head).transpose(1, 0, 2)

    q = heads_of(qkv[:, 0:hd], heads)
    k = heads_of(qkv[:, hd:hd + kvd], hkv)
    v = heads_of(qkv[:, hd + kvd:hd + 2 * kvd], hkv)
    o = attention_rows(q, k, v, rows - lo, 1.0 / np.sqrt(d_head), seq_ends=ends - lo).reshape(len(rows), hd)
    attn = r(o)
    x2 = r(add(x[rows], matmul(attn, wo)))
    h2 = r(rmsnorm(x2, n2, eps))
    a = r(silu_mul(matmul(h2, wg), matmul(h2, wu)))
    y = r(add(x2, matmul(a, wd)))
    return dict(h1=h1[rows - lo], qkv=qkv[rows - lo], attn=attn, x2=x2, h2=h2, a=a, y=y)


# --------------------------------------------------------------------------
# logical optimization (Section 4): brute force over every combination of
# join-agg specs, pure Python (small cases only)
# --------------------------------------------------------------------------
def _letters(spec: str):
    out = []
    for ch in spec.replace(",", "").replace("->", ""):
        if ch not in out:
            out.append(ch)
    return out


def logical_specs(spec: str, extents: dict, p: int, shardable=None):
    """Every join-agg spec of an operator over p processors (Section 4.2): an
    interval count per letter, 1 for letters that may not be split, each at
    most the letter's extent, multiplying to p."""
    letters = _letters(spec)
    out = []

    def rec(i, rem, cur):
        if i == len(letters):
            if rem == 1:
                out.append(dict(cur))
            return
        l = letters[i]
        if shardable is not None and l not in shardable:
            cur[l] = 1
            rec(i + 1, rem, cur)
            return
        for v in range(1, min(rem, extents[l]) + 1):
            if rem % v == 0:
                cur[l] = v
                rec(i + 1, rem // v, cur)

    rec(0, p, {})
    return out


def _intervals(n: int, c: int):
    pts = [(i * n) // c for i in range(c)] + [n]
    return [(pts[i], pts[i + 1]) for i in range(c)]


def logical_spec_cost(spec: str, extents: dict, counts: dict, input_tilings):
    """Cost (Section 4.3) of one operator's spec, by its definition: the
    function specifications are the cells of the interval grid; join adds
    the numbers in every cell's input blocks, aggregation (m - 1) times each
    distinct output block's numbers, repartition the whole input tensor for
    every input whose given tiling (a tuple of counts, None for a
    computation input) differs from the one the spec needs."""
    lhs, out = spec.split("->")
    ins = lhs.split(",")
    letters = _letters(spec)
    grids = [_intervals(extents[l], counts[l]) for l in letters]
    cost = 0
    out_seen = {}
    for cell in itertools.product(*grids):
        iv = dict(zip(letters, cell))
        for operand in ins:
            cost += int(np.prod([iv[l][1] - iv[l][0] for l in operand]))
        key = tuple(iv[l] for l in out)
        out_seen[key] = out_seen.get(key, 0) + 1
    for key, m in out_seen.items():
        cost += (m - 1) * int(np.prod([hi - lo for lo, hi in key]))
    for operand, t in zip(ins, input_tilings):
        if t is not None and tuple(t) != tuple(counts[l] for l in operand):
            cost += int(np.prod([extents[l] for l in operand]))
    return cost


def logical_plan_cost(ops, choice):
    """Total cost of a plan: ops are (spec, extents, inputs, shardable) with
    inputs naming producer indices (None: computation input); choice gives
    each operator's counts."""
    total = 0
    for (spec, extents, inputs, _), counts in zip(ops, choice):
        tilings = []
        for x in inputs:
            if x is None:
                tilings.append(None)
            else:
                pspec, _, _, _ = ops[x]
                tilings.append(tuple(choice[x][l] for l in pspec.split("->")[1]))
        total += logical_spec_cost(spec, extents, counts, tilings)
    return total


def logical_min_cost(ops, p: int):
    """The minimum total cost over every combination of specs (exhaustive)."""
    all_specs = [logical_specs(spec, ext, p, sh) for spec, ext, _, sh in ops]
    return min(logical_plan_cost(ops, combo) for combo in itertools.product(*all_specs))


# --------------------------------------------------------------------------
# exchange programs (Section 5.2, Definition "Closure; validity"), pure
# Python on structured programs with fixed sites
# --------------------------------------------------------------------------
def exprog_valid(ins, outs, actions):
    """ins: [(atom, site)]; outs: [(atoms, [sites])]; actions: [(atoms,
    [source sites], [[hop sites], ...])].  The closure: start from each IN
    atom at its site; an action at a source site is enabled when some
    aggregates present there are pairwise disjoint with union its atoms
    (tried over every subset of the present aggregates); firing adds the
    aggregate at the source and at every hop's sites.  Valid: every action
    fires at every source, and every OUT aggregate is at each of its sites."""
    state = set((frozenset([a]), s) for a, s in ins)
    pending = [(frozenset(x), s, hops) for x, srcs, hops in actions for s in srcs]
    fired = [False] * len(pending)

    def enabled(x, s):
        here = [a for a, t in state if t == s and a <= x]
        for n in range(1, len(here) + 1):
            for combo in itertools.combinations(here, n):
                if sum(len(c) for c in combo) == len(x) and frozenset().union(*combo) == x:
                    return True
        return False

    changed = True
    while changed:
        changed = False
        for i, (x, s, hops) in enumerate(pending):
            if not fired[i] and enabled(x, s):
                fired[i] = True
                changed = True
                state.add((x, s))
                for hop in hops:
                    for d in hop:
                        state.add((x, d))
    return all(fired) and all((frozenset(x), s) in state for x, sites in outs for s in sites)
