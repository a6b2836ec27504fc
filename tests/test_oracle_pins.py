"""Pins of the CPU oracle against things other than itself.

Each test checks an oracle function against a value the paper prints (golden
fixtures under tests/golden/), a closed form, an invariant, a library routine
the definition reduces to, or brute force on tiny inputs.  None of these
retypes the oracle's own formula.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# rounding
# ---------------------------------------------------------------------------
def test_rne_bf16_matches_torch_cast_on_fp32_values():
    rng = np.random.default_rng(7)
    x = np.concatenate([
        rng.standard_normal(200000) * 10.0 ** rng.integers(-30, 30, 200000),
        rng.standard_normal(1000) * 1e-39,  # bf16 subnormal range
    ]).astype(np.float32)
    # exact ties: halfway between adjacent bf16 values (low 16 bits = 0x8000)
    bits = (rng.integers(0, 2 ** 7, 5000).astype(np.uint32) << 16) | 0x8000   # 7 bf16 mantissa bits
    bits |= (rng.integers(0x30, 0x50, 5000).astype(np.uint32) << 23)         # exponent
    bits |= (rng.integers(0, 2, 5000).astype(np.uint32) << 31)               # sign
    x = np.concatenate([x, bits.view(np.float32), np.float32([0.0, -0.0, 1.0, -2.5])])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.rne_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_rne_bf16_is_nearest_on_fp64_values():
    rng = np.random.default_rng(8)
    x = rng.standard_normal(50000) * 10.0 ** rng.integers(-20, 20, 50000)
    y = oracle.rne_bf16(x)
    # y is a bf16 value: fp32-representable with the low 16 mantissa bits zero
    y32 = y.astype(np.float32)
    assert np.all(y32.astype(np.float64) == y)
    assert np.all((y32.view(np.uint32) & 0xFFFF) == 0)
    # and no other bf16 value is closer: compare with both bf16 neighbours
    up = (y32.view(np.uint32) + 0x10000).view(np.float32).astype(np.float64)
    dn = (y32.view(np.uint32) - 0x10000).view(np.float32).astype(np.float64)
    assert np.all(np.abs(y - x) <= np.abs(up - x))
    assert np.all(np.abs(y - x) <= np.abs(dn - x))


# ---------------------------------------------------------------------------
# layout, pack, repartition (Section 3.1 tilings; Section 5.3 atoms)
# ---------------------------------------------------------------------------
def test_layout_small_case_positions():
    # [3, 5] f32, rows {0,2,3}, cols {0,4,5}: blocks 2x4, 2x1, 1x4, 1x1, each
    # starting at a multiple of 256 bytes, in row-major block order.
    offs, nbytes = oracle.layout([[0, 2, 3], [0, 4, 5]], 4)
    assert offs.tolist() == [0, 256, 512, 768]
    assert nbytes == 768 + 4
    dense = np.arange(15, dtype=np.float32).reshape(3, 5)
    blk = oracle.pack(dense, [[0, 2, 3], [0, 4, 5]])
    f = blk.view(np.float32)
    assert f[0:8].tolist() == [0, 1, 2, 3, 5, 6, 7, 8]
    assert f[64:66].tolist() == [4, 9]
    assert f[128:132].tolist() == [10, 11, 12, 13]
    assert f[192:193].tolist() == [14]


def test_single_block_relation_is_the_dense_tensor():
    x = synth.normal((7, 9, 3), 1, dtype="f32")
    blk = oracle.pack(x, [[0, 7], [0, 9], [0, 3]])
    assert blk.tobytes() == x.tobytes()


@pytest.mark.parametrize("seed", range(5))
def test_pack_blocks_hold_dense_slices(seed):
    rng = np.random.default_rng(seed)
    shape = (int(rng.integers(1, 40)), int(rng.integers(1, 40)), int(rng.integers(1, 9)))
    part = [synth.random_splits(n, int(rng.integers(1, 5)), rng) for n in shape]
    x = synth.normal(shape, seed, dtype="bf16")
    blk = oracle.pack(x, part)
    offs, _ = oracle.layout(part, 2)
    for b, coords in enumerate(itertools.product(*[range(len(s) - 1) for s in part])):
        sl = tuple(slice(s[c], s[c + 1]) for s, c in zip(part, coords))
        piece = np.ascontiguousarray(x[sl])
        got = blk[offs[b]:offs[b] + piece.nbytes].view(np.uint16)
        np.testing.assert_array_equal(got, piece.ravel())
    np.testing.assert_array_equal(oracle.unpack(blk, part, np.uint16), x)


@pytest.mark.parametrize("seed", range(5))
def test_repartition_round_trip_is_identity(seed):
    rng = np.random.default_rng(100 + seed)
    shape = (int(rng.integers(1, 64)), int(rng.integers(1, 64)))
    p1 = [synth.random_splits(n, int(rng.integers(1, 6)), rng) for n in shape]
    p2 = [synth.random_splits(n, int(rng.integers(1, 6)), rng) for n in shape]
    x = synth.normal(shape, seed, dtype="f32")
    b1 = oracle.pack(x, p1)
    b2 = oracle.repartition(b1, p1, p2, np.float32)
    np.testing.assert_array_equal(oracle.unpack(b2, p2, np.float32), x)
    b1_again = oracle.repartition(b2, p2, p1, np.float32)
    assert b1_again.tobytes() == b1.tobytes()


def test_repartition_on_the_preamble_example():
    g = json.load(open(os.path.join(GOLDEN, "preamble_overlay_example.json")))
    n_rows, n_cols = g["shape"]
    prod = [g["producer_rows"], [0, n_cols]]
    cons = [g["consumer_rows"], [0, n_cols]]
    x = synth.normal((n_rows, n_cols), 3, dtype="bf16")
    bp = oracle.pack(x, prod)
    bc = oracle.repartition(bp, prod, cons, np.uint16)
    offs_p, _ = oracle.layout(prod, 2)
    offs_c, _ = oracle.layout(cons, 2)
    # every consumer block is one atom: a contiguous half of one producer block
    atom = 64 * n_cols * 2
    for c in range(g["n_atoms"]):
        p, half = divmod(c, g["atoms_per_producer_block"])
        src = bp[offs_p[p] + half * atom: offs_p[p] + (half + 1) * atom]
        dst = bc[offs_c[c]: offs_c[c] + atom]
        assert src.tobytes() == dst.tobytes()


# ---------------------------------------------------------------------------
# join (Section 3.2 Definitions "Join-agg spec" / "Implementation" step 1,
# Section 3.3 count of function specifications)
# ---------------------------------------------------------------------------
def _bounds(partition, block_index):
    nb = [len(s) - 1 for s in partition]
    coords = np.unravel_index(block_index, nb)
    return [s[c] for s, c in zip(partition, coords)], [s[c + 1] for s, c in zip(partition, coords)]


def test_join_reproduces_the_papers_matmul_example():
    g = json.load(open(os.path.join(GOLDEN, "matmul_join_agg_example.json")))
    for case in g["cases"]:
        P = case["partitions"]
        pA, pB, pC = [P["i"], P["j"]], [P["j"], P["k"]], [P["i"], P["k"]]
        tuples, goff = oracle.join(g["spec"], [pA, pB, pC])
        assert len(tuples) == case["n_function_specs"]
        distinct = sorted(set(tuples[:, 0].tolist()))
        assert len(distinct) == len(case["output_types"])
        for ob, want in zip(distinct, case["output_types"]):
            lo, hi = _bounds(pC, ob)
            assert lo == want["lower"] and hi == want["upper"]
            assert int(np.sum(tuples[:, 0] == ob)) == want["n_aggregated"]
            # the aggregated tuples differ exactly in their j interval
            js = sorted(_bounds(pA, int(t[1]))[0][1] for t in tuples[tuples[:, 0] == ob])
            assert js == P["j"][:-1]


@pytest.mark.parametrize("spec", ["ij,jk->ik", "ab,bc,cd->ad", "bij,bjk->bik", "ij,j->i", "ij->j"])
@pytest.mark.parametrize("seed", range(4))
def test_join_count_is_the_product_of_interval_counts(spec, seed):
    rng = np.random.default_rng(seed)
    lhs, out = spec.split("->")
    letters = sorted(set(lhs.replace(",", "")))
    size = {l: int(rng.integers(4, 40)) for l in letters}
    part = {l: synth.random_splits(size[l], int(rng.integers(1, 5)), rng) for l in letters}
    parts = [[part[l] for l in s] for s in lhs.split(",")] + [[part[l] for l in out]]
    tuples, goff = oracle.join(spec, parts)
    expect = int(np.prod([len(part[l]) - 1 for l in letters]))
    assert len(tuples) == expect
    # one group per output block, each with the product of contracted counts
    contracted = [l for l in letters if l not in out]
    per_group = int(np.prod([len(part[l]) - 1 for l in contracted])) if contracted else 1
    assert np.all(np.diff(goff) == per_group)
    # groups are keyed by output block, ascending
    assert np.all(np.diff(tuples[:, 0]) >= 0)


def test_join_causal_count_closed_form():
    # q and k blocks of 128 over 2048 positions, 2 batches x 4 heads:
    # group (b, h, qb) keeps key blocks 0..qb, so sum_{qb<16} (qb + 1) = 136 per (b, h).
    pq = [synth.splits(2, 1), synth.splits(4, 1), synth.splits(2048, 128), [0, 128]]
    tuples, goff = oracle.join("bhqd,bhkd,bhkd->bhqd", [pq, pq, pq, pq], group="bhqd", causal=("q", "k"))
    assert len(tuples) == 2 * 4 * 136
    sizes = np.diff(goff)
    assert sizes.tolist() == list(range(1, 17)) * 8


def test_join_drops_combinations_whose_shared_intervals_differ():
    # j split differently in the two inputs: only the interval [256, 512) matches.
    pA = [[0, 256], [0, 256, 512]]
    pB = [[0, 128, 256, 512], [0, 256]]
    tuples, _ = oracle.join("ij,jk->ik", [pA, pB, [[0, 256], [0, 256]]])
    assert tuples.tolist() == [[0, 1, 2]]


@pytest.mark.parametrize("seed", range(6))
def test_decomposition_invariance_integer_data(seed):
    """Definition "Implementation": join, aggregate by output type with +,
    recompose -- any valid decomposition reproduces the operator's output.
    Integer data keeps every sum exact, so a missing or duplicated tuple fails."""
    rng = np.random.default_rng(seed)
    I, J, K = (int(v) for v in rng.integers(8, 70, 3))
    pi = synth.random_splits(I, int(rng.integers(1, 5)), rng)
    pj = synth.random_splits(J, int(rng.integers(1, 5)), rng)
    pk = synth.random_splits(K, int(rng.integers(1, 5)), rng)
    A = synth.to_f64(synth.integers((I, J), seed, -2, 2, "f32"), "f32")
    B = synth.to_f64(synth.integers((J, K), seed + 50, -2, 2, "f32"), "f32")
    tuples, goff = oracle.join("ij,jk->ik", [[pi, pj], [pj, pk], [pi, pk]])
    C = np.zeros((I, K))
    for ob in range(len(goff) - 1):
        (i0, k0), (i1, k1) = _bounds([pi, pk], ob)
        acc = np.zeros((i1 - i0, k1 - k0))
        for t in tuples[goff[ob]:goff[ob + 1]]:
            (a_i0, a_j0), (a_i1, a_j1) = _bounds([pi, pj], int(t[1]))
            (b_j0, b_k0), (b_j1, b_k1) = _bounds([pj, pk], int(t[2]))
            acc += oracle.matmul(A[a_i0:a_i1, a_j0:a_j1], B[b_j0:b_j1, b_k0:b_k1])
        C[i0:i1, k0:k1] = acc
    exact = (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64)
    np.testing.assert_array_equal(C, exact)
    np.testing.assert_array_equal(oracle.matmul(A, B), exact)


# ---------------------------------------------------------------------------
# dense numerics
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("spec", ["ij,jk->ik", "bij,bjk->bik", "ij,ij->ij", "ijk->ik", "ij,j->i", "abc,cd,bd->ad"])
def test_einsum_mul_sum_matches_numpy(spec):
    rng = np.random.default_rng(11)
    lhs, out = spec.split("->")
    sizes = {l: int(rng.integers(2, 9)) for l in set(lhs.replace(",", ""))}
    ins = [rng.standard_normal([sizes[l] for l in s]) for s in lhs.split(",")]
    contracted = set(lhs.replace(",", "")) - set(out)
    agg = oracle.AGG_SUM if contracted else oracle.AGG_NONE
    got = oracle.einsum(spec, ins, oracle.JOIN_MUL, agg)
    np.testing.assert_allclose(got, np.einsum(spec, *ins), rtol=1e-12, atol=1e-12)


def test_einsum_max_product_is_brute_force_max():
    rng = np.random.default_rng(12)
    a = rng.standard_normal((5, 7))
    b = rng.standard_normal((7, 3))
    got = oracle.einsum("ij,jk->ik", [a, b], oracle.JOIN_MUL, oracle.AGG_MAX)
    np.testing.assert_array_equal(got, np.max(a[:, :, None] * b[None, :, :], axis=1))


def test_einsum_add_sum_closed_form():
    # sum_j (a[i,j] + b[j,k]) = rowsum(a)[i] + colsum(b)[k]
    a = synth.to_f64(synth.integers((6, 5), 1, -3, 3, "f32"), "f32")
    b = synth.to_f64(synth.integers((5, 4), 2, -3, 3, "f32"), "f32")
    got = oracle.einsum("ij,jk->ik", [a, b], oracle.JOIN_ADD, oracle.AGG_SUM)
    np.testing.assert_array_equal(got, a.sum(1)[:, None] + b.sum(0)[None, :])


def test_einsum_none_rejects_contraction():
    with pytest.raises(ValueError):
        oracle.einsum("ij,jk->ik", [np.ones((2, 2)), np.ones((2, 2))], oracle.JOIN_MUL, oracle.AGG_NONE)


def test_matmul_matches_numpy_and_closed_forms():
    rng = np.random.default_rng(13)
    a = rng.standard_normal((37, 53))
    b = rng.standard_normal((53, 29))
    np.testing.assert_allclose(oracle.matmul(a, b), a @ b, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(oracle.matmul(a, np.eye(53)), a)
    np.testing.assert_array_equal(oracle.matmul(a, np.zeros((53, 4))), np.zeros((37, 4)))


def test_rmsnorm_matches_torch_and_closed_forms():
    rng = np.random.default_rng(14)
    x = rng.standard_normal((33, 96))
    w = rng.uniform(0.5, 1.5, 96)
    eps = 1e-6
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(w), eps).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, w, eps), ref, rtol=1e-12, atol=1e-14)
    c = 0.37
    y = oracle.rmsnorm(np.full((2, 96), c), w, eps)
    np.testing.assert_allclose(y, np.tile(w * c / np.sqrt(c * c + eps), (2, 1)), rtol=1e-14)
    np.testing.assert_array_equal(oracle.rmsnorm(np.zeros((3, 96)), w, eps), np.zeros((3, 96)))


def test_softmax_matches_torch_and_closed_forms():
    rng = np.random.default_rng(15)
    s = rng.standard_normal((3, 40, 40)) * 3
    mask = np.tril(np.ones((40, 40), dtype=bool))
    ref = torch.softmax(torch.from_numpy(np.where(mask, s, -np.inf)), dim=-1).numpy()
    p = oracle.softmax(s, True)
    np.testing.assert_allclose(p, ref, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(oracle.softmax(s + rng.standard_normal((3, 40, 1)), True), p, rtol=1e-12, atol=1e-15)
    const = oracle.softmax(np.full((1, 40, 40), 2.0), True)
    q = np.arange(40)[:, None]
    np.testing.assert_allclose(const[0], np.where(mask, 1.0 / (q + 1), 0.0), rtol=1e-14)
    ref_nc = torch.softmax(torch.from_numpy(s), dim=-1).numpy()
    np.testing.assert_allclose(oracle.softmax(s, False), ref_nc, rtol=1e-12, atol=1e-15)


def test_attention_matches_torch_and_closed_forms():
    rng = np.random.default_rng(16)
    B, H, S, D = 2, 3, 37, 16
    q, k, v = (rng.standard_normal((B, H, S, D)) for _ in range(3))
    scale = 1.0 / np.sqrt(D)
    ref = F.scaled_dot_product_attention(torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
                                         is_causal=True, scale=scale).numpy()
    o = oracle.attention(q, k, v, True, scale)
    np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)
    # identical value rows give that row back
    vrow = rng.standard_normal(D)
    o_eq = oracle.attention(q, k, np.broadcast_to(vrow, (B, H, S, D)), True, scale)
    np.testing.assert_allclose(o_eq, np.broadcast_to(vrow, (B, H, S, D)), rtol=1e-13, atol=1e-13)
    # zero keys give the causal prefix mean of the values
    o_zero = oracle.attention(q, np.zeros_like(k), v, True, scale)
    prefix_mean = np.cumsum(v, axis=2) / np.arange(1, S + 1)[None, None, :, None]
    np.testing.assert_allclose(o_zero, prefix_mean, rtol=1e-12, atol=1e-13)
    # the first query sees only the first key
    np.testing.assert_allclose(o[:, :, 0], v[:, :, 0], rtol=1e-13, atol=1e-14)


def test_silu_mul_and_add_match_torch():
    rng = np.random.default_rng(17)
    g, u = rng.standard_normal(1000) * 4, rng.standard_normal(1000)
    ref = (F.silu(torch.from_numpy(g)) * torch.from_numpy(u)).numpy()
    np.testing.assert_allclose(oracle.silu_mul(g, u), ref, rtol=1e-13, atol=1e-15)
    np.testing.assert_array_equal(oracle.add(g, u), g + u)


def _torch_block(x, n1, wqkv, wo, wg, wu, wd, n2, heads, d_head, eps):
    """The same chain composed from torch library routines, rounding through
    torch's bf16 cast at the same boundaries."""
    t = lambda a: torch.from_numpy(a)
    r = lambda a: a.float().to(torch.bfloat16).double()
    T, Hd = x.shape
    hd = heads * d_head
    h1 = r(F.rms_norm(t(x), (Hd,), t(n1), eps))
    qkv = r(h1 @ t(wqkv))
    qh, kh, vh = (qkv[:, i * hd:(i + 1) * hd].reshape(T, heads, d_head).transpose(0, 1)[None] for i in range(3))
    o = r(F.scaled_dot_product_attention(qh, kh, vh, is_causal=True, scale=1.0 / np.sqrt(d_head)))
    attn = o[0].transpose(0, 1).reshape(T, hd)
    x2 = r(t(x) + attn @ t(wo))
    h2 = r(F.rms_norm(x2, (Hd,), t(n2), eps))
    a = r(F.silu(h2 @ t(wg)) * (h2 @ t(wu)))
    return r(x2 + a @ t(wd)).numpy()


def test_llama_block_composition_and_causal_prefix():
    w = synth.llama_block(t=48, hidden=64, heads=2, d_head=16, ffn=40)
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "wqkv", "wo", "wg", "wu", "wd", "n1", "n2")}
    args = (f["x"], f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"], f["n2"])
    out = oracle.llama_block(*args, heads=2, d_head=16, eps=1e-6)
    ref = _torch_block(*args, 2, 16, 1e-6)
    # rounding points match; rare one-ulp flips from fp32-vs-fp64 ties only
    diff = np.abs(out["y"] - ref)
    assert np.mean(diff > 0) < 0.01
    assert np.linalg.norm(out["y"] - ref) / np.linalg.norm(ref) < 1e-3
    # causal prefix: the first 20 rows of the output depend only on the first 20 rows of x
    pre = oracle.llama_block(f["x"][:20], *args[1:], heads=2, d_head=16, eps=1e-6)
    np.testing.assert_array_equal(pre["y"], out["y"][:20])


# ---------------------------------------------------------------------------
# grouped-query heads and packed sequences (Section 3.3, Example "Flash
# attention")
# ---------------------------------------------------------------------------
def _flash_example():
    with open(os.path.join(GOLDEN, "flash_attention_example.json")) as f:
        return json.load(f)


def _sdpa(q, k, v, causal, scale):
    return F.scaled_dot_product_attention(torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
                                          is_causal=causal, scale=scale).numpy()


@pytest.mark.parametrize("causal", [False, True])
def test_attention_ex_grouped_heads_match_sdpa_on_repeated_kv(causal):
    # Hq = 8 over Hkv = 2: query head h reads key/value head h // 4, the same
    # as plain attention with each key/value head repeated for its 4 query heads
    rng = np.random.default_rng(18)
    B, Hq, Hkv, S, D = 2, 8, 2, 29, 16
    q = rng.standard_normal((B, Hq, S, D))
    k, v = (rng.standard_normal((B, Hkv, S, D)) for _ in range(2))
    scale = 0.3
    ref = _sdpa(q, np.repeat(k, Hq // Hkv, axis=1), np.repeat(v, Hq // Hkv, axis=1), causal, scale)
    np.testing.assert_allclose(oracle.attention_ex(q, k, v, causal, scale), ref, rtol=1e-10, atol=1e-12)
    # one group: the plain definition
    ref1 = _sdpa(q, q, q, causal, scale)
    np.testing.assert_allclose(oracle.attention_ex(q, q, q, causal, scale), ref1, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_ex_packed_sequences_match_each_sequence_alone(causal):
    # attention never crosses a sequence end: packed, it equals attention run
    # on every sequence by itself (here with grouped heads too)
    rng = np.random.default_rng(19)
    B, Hq, Hkv, D = 1, 4, 2, 8
    ends = [7, 20, 21, 40]
    S = ends[-1]
    q = rng.standard_normal((B, Hq, S, D))
    k, v = (rng.standard_normal((B, Hkv, S, D)) for _ in range(2))
    o = oracle.attention_ex(q, k, v, causal, 0.5, seq_ends=ends)
    lo = 0
    for hi in ends:
        sl = slice(lo, hi)
        ref = _sdpa(q[:, :, sl], np.repeat(k[:, :, sl], 2, axis=1), np.repeat(v[:, :, sl], 2, axis=1), causal, 0.5)
        np.testing.assert_allclose(o[:, :, sl], ref, rtol=1e-10, atol=1e-12)
        lo = hi
    # a one-position sequence returns its own value row
    np.testing.assert_allclose(o[0, :, 20], np.repeat(v[0, :, 20], 2, axis=0), rtol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_join_packed_sequences_of_the_papers_example(causal):
    # ends 1024, 2560, 4096 in 128-blocks: sequences of 8, 12 and 12 blocks;
    # a query block keeps the key blocks of its own sequence (causal: those at
    # or before it), so sum n(n+1)/2 = 36 + 78 + 78 = 192 or sum n^2 = 352
    ex = _flash_example()
    S, ends = ex["sequence"], ex["ends"]
    p = [[0, 1], [0, 1], synth.splits(S, 128), [0, 128]]
    tuples, goff = oracle.join("bhqd,bhkd,bhkd->bhqd", [p, p, p, p], group="bhqd",
                               causal=("q", "k") if causal else None, positions=("q", "k"), seq_ends=ends)
    seq = np.searchsorted(ends, np.arange(0, S, 128), side="right")
    want = [(qb, kb) for qb in range(S // 128) for kb in range(S // 128)
            if seq[qb] == seq[kb] and (not causal or kb <= qb)]
    assert len(tuples) == (192 if causal else 352) == len(want)
    assert [(t[1], t[2]) for t in tuples.tolist()] == want
    assert np.all(tuples[:, 3] == tuples[:, 2])


def test_join_grouped_heads_of_the_papers_example():
    # 32 query heads over 8 key/value heads: query head h joins only key/value
    # head h // 4; with the query heads in blocks of 4, block m joins head m
    ex = _flash_example()
    Hq, Hkv = ex["heads_q"], ex["heads_kv"]
    G = Hq // Hkv
    pk = [[0, 1], synth.splits(Hkv, 1), [0, 256, 512], [0, 128]]
    for hb in (1, G):
        pq = [[0, 1], synth.splits(Hq, hb), [0, 256, 512], [0, 128]]
        tuples, _ = oracle.join("bhqd,bgkd,bgkd->bhqd", [pq, pk, pk, pq], group="bhqd", gqa=(G, "h", "g"))
        assert len(tuples) == (Hq // hb) * 2 * 2  # head blocks x query blocks x key blocks
        qhead = tuples[:, 1] // 2  # Q block index = head block * 2 query blocks + query block
        khead = tuples[:, 2] // 2
        assert np.all(khead == qhead * hb // G)
    # query-head blocks straddling two key/value heads join neither
    pq = [[0, 1], [0, 2, 6, 8], [0, 512], [0, 128]]
    tuples, _ = oracle.join("bhqd,bgkd,bgkd->bhqd", [pq, [[0, 1], [0, 1, 2], [0, 512], [0, 128]]] * 1 +
                            [[[0, 1], [0, 1, 2], [0, 512], [0, 128]], pq], group="bhqd", gqa=(4, "h", "g"))
    assert sorted(t[1] for t in tuples.tolist()) == [0, 2]


def test_llama_block_grouped_heads_and_packed_sequences():
    # grouped-query: the block with 4 query heads over 2 key/value heads equals
    # the (torch-pinned) plain block whose W_qkv repeats each K and V head for
    # its 2 query heads; packed: a later sequence's rows equal the block run on
    # that sequence alone (every step but attention is row by row)
    w = synth.llama_block(t=48, hidden=64, heads=4, d_head=16, ffn=40)
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "wqkv", "wo", "wg", "wu", "wd", "n1", "n2")}
    hd, kvd = 4 * 16, 2 * 16
    wqkv = f["wqkv"][:, :hd + 2 * kvd]
    rep = lambda cols: np.repeat(cols.reshape(64, 2, 16), 2, axis=1).reshape(64, hd)
    wqkv_mha = np.concatenate([wqkv[:, :hd], rep(wqkv[:, hd:hd + kvd]), rep(wqkv[:, hd + kvd:])], axis=1)
    rest = (f["wo"], f["wg"], f["wu"], f["wd"], f["n2"])
    gqa = oracle.llama_block(f["x"], f["n1"], wqkv, *rest, heads=4, d_head=16, eps=1e-6, heads_kv=2)
    mha = oracle.llama_block(f["x"], f["n1"], wqkv_mha, *rest, heads=4, d_head=16, eps=1e-6)
    diff = np.abs(gqa["y"] - mha["y"])
    assert np.mean(diff > 0) < 0.01
    assert np.linalg.norm(diff) / np.linalg.norm(mha["y"]) < 1e-3
    packed = oracle.llama_block(f["x"], f["n1"], wqkv, *rest, heads=4, d_head=16, eps=1e-6, heads_kv=2,
                                seq_ends=[20, 48])
    alone = oracle.llama_block(f["x"][20:], f["n1"], wqkv, *rest, heads=4, d_head=16, eps=1e-6, heads_kv=2,
                               seq_ends=[28])
    np.testing.assert_array_equal(packed["y"][20:], alone["y"])
    first = oracle.llama_block(f["x"][:20], f["n1"], wqkv, *rest, heads=4, d_head=16, eps=1e-6, heads_kv=2,
                               seq_ends=[20])
    np.testing.assert_array_equal(packed["y"][:20], first["y"])


@pytest.mark.parametrize("seq_ends", [None, [20, 48], [7, 31, 48]])
def test_llama_block_rows_equals_the_whole_chain_at_its_rows(seq_ends):
    # the sampled-rows block (attention written out per query row) against the
    # whole-chain oracle at the same rows, grouped heads, packed or single
    # sequence; boundaries round to bf16 on both sides, so an element may
    # differ by one bf16 step where fp64 summation order moves a value across
    # a rounding boundary
    w = synth.llama_block(t=48, hidden=64, heads=4, d_head=16, ffn=40)
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "wqkv", "wo", "wg", "wu", "wd", "n1", "n2")}
    wqkv = f["wqkv"][:, :4 * 16 + 2 * 2 * 16]
    args = (f["x"], f["n1"], wqkv, f["wo"], f["wg"], f["wu"], f["wd"], f["n2"])
    full = oracle.llama_block(*args, heads=4, d_head=16, eps=1e-6, heads_kv=2, seq_ends=seq_ends)
    rows = [0, 5, 19, 20, 21, 33, 47]
    part = oracle.llama_block_rows(*args, heads=4, d_head=16, eps=1e-6, rows=rows, heads_kv=2, seq_ends=seq_ends)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        ref = full[name][rows]
        got = part[name]
        assert got.shape == ref.shape
        close = np.isclose(got, ref, rtol=2.0 ** -7, atol=1e-30)
        assert close.all(), name
        assert np.mean(got == ref) > 0.98, name
    if seq_ends is None:
        # a history shifted by one token changes the row: the comparison can fail
        bad = oracle.llama_block_rows(f["x"][1:], *args[1:], heads=4, d_head=16, eps=1e-6, rows=[10], heads_kv=2)
        assert not np.allclose(bad["attn"], full["attn"][[10]])


@pytest.mark.parametrize("seq_ends", [None, [20, 48], [7, 31, 48]])
def test_attention_rows_equals_attention_ex_at_every_row(seq_ends):
    # the per-row evaluation against the whole-tensor oracle (itself pinned to
    # SDPA above), grouped heads: exact up to fp64 summation order
    rng = np.random.default_rng(77)
    q, k, v = rng.standard_normal((1, 4, 48, 16)), rng.standard_normal((1, 2, 48, 16)), rng.standard_normal((1, 2, 48, 16))
    full = oracle.attention_ex(q, k, v, True, 0.25, seq_ends=seq_ends)
    rows = np.arange(48)
    got = oracle.attention_rows(q[0], k[0], v[0], rows, 0.25, seq_ends=seq_ends)
    np.testing.assert_allclose(got, full[0].transpose(1, 0, 2), rtol=1e-12, atol=1e-12)
    # a window of tokens [20, 48) with its ends shifted by its start: the rows of
    # the second sequence are unchanged
    if seq_ends == [20, 48]:
        w = oracle.attention_rows(q[0][:, 20:], k[0][:, 20:], v[0][:, 20:], np.arange(28), 0.25,
                                  seq_ends=np.array(seq_ends) - 20)
        np.testing.assert_allclose(w, full[0][:, 20:].transpose(1, 0, 2), rtol=1e-12, atol=1e-12)
