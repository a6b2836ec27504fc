"""GPU parity of the join-agg kernels against the fp64 oracle.

Floating point: relative Frobenius error <= 1e-3 and max |diff| <= 2e-2 *
max |ref|; outputs stored as bf16 are compared with the oracle's value rounded
to bf16 the same way.  Integer-valued inputs make fp32 results exact for any
decomposition, so those cases are compared bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_close, empty, expected, upload, values
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------------
# fp32 block products and the generic einsum path
# ---------------------------------------------------------------------------
def test_matmul_fp32_256_in_64_blocks():
    w = synth.matmul_256_fp32()
    A, B = upload(w["A"], "f32", w["pA"]), upload(w["B"], "f32", w["pB"])
    C = empty((256, 256), "f32", w["pC"])
    ea.joinagg(w["spec"], ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)
    ref = oracle.matmul(synth.to_f64(w["A"], "f32"), synth.to_f64(w["B"], "f32"))
    assert_close(values(C), ref, what="C1")


@pytest.mark.parametrize("kmajor", [False, True])
@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_fp32_block_product_ragged_blocks(kmajor, out_dtype):
    # f32 'ij,jk->ik' / 'ij,kj->ik': 64 x 64 tiles of every output block, the
    # key's tuples summed in order; ragged blocks on every letter
    rng = np.random.default_rng(11)
    M, J, N = 200, 333, 150
    pm, pj, pn = (synth.random_splits(n, 3, rng) for n in (M, J, N))
    a = synth.normal((M, J), 12, dtype="f32")
    b = synth.normal((N, J) if kmajor else (J, N), 13, dtype="f32")
    A = upload(a, "f32", [pm, pj])
    B = upload(b, "f32", [pn, pj] if kmajor else [pj, pn])
    C = empty((M, N), out_dtype, [pm, pn])
    ea.joinagg("ij,kj->ik" if kmajor else "ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)
    fb = synth.to_f64(b, "f32")
    ref = oracle.matmul(synth.to_f64(a, "f32"), np.ascontiguousarray(fb.T) if kmajor else fb)
    assert_close(values(C), expected(ref, out_dtype), rel_fro=1e-5 if out_dtype == "f32" else 1e-3,
                 what=f"fp32 block product kmajor={kmajor} {out_dtype}")


@pytest.mark.parametrize("seed", range(4))
def test_generic_einsum_integer_data_bitexact(seed):
    rng = np.random.default_rng(seed)
    I, J, K = (int(v) for v in rng.integers(5, 70, 3))
    pi, pj, pk = (synth.random_splits(n, int(rng.integers(1, 5)), rng) for n in (I, J, K))
    a = synth.integers((I, J), seed, -3, 3, "f32")
    b = synth.integers((J, K), seed + 9, -3, 3, "f32")
    A, B = upload(a, "f32", [pi, pj]), upload(b, "f32", [pj, pk])
    fa, fb = synth.to_f64(a, "f32"), synth.to_f64(b, "f32")
    for join_op, agg_op in [(ea.JOIN_MUL, ea.AGG_SUM), (ea.JOIN_MUL, ea.AGG_MAX), (ea.JOIN_ADD, ea.AGG_SUM)]:
        C = empty((I, K), "f32", [pi, pk])
        ea.joinagg("ij,jk->ik", join_op, agg_op, [A, B], C)
        ref = oracle.einsum("ij,jk->ik", [fa, fb], join_op, agg_op)
        np.testing.assert_array_equal(values(C), ref)


@pytest.mark.parametrize("spec,shapes", [
    ("bij,bjk->bik", [(3, 20, 30), (3, 30, 12), (3, 20, 12)]),
    ("ij->j", [(50, 40), (40,)]),
    ("ij,ij->ij", [(33, 17), (33, 17), (33, 17)]),
    ("abc,cd,bd->ad", [(6, 7, 8), (8, 5), (7, 5), (6, 5)]),
])
def test_generic_einsum_specs(spec, shapes):
    rng = np.random.default_rng(3)
    lhs, rhs = spec.split("->")
    ops = lhs.split(",") + [rhs]
    size = {}
    for s, shp in zip(ops, shapes):
        size.update(dict(zip(s, shp)))
    part = {l: synth.random_splits(n, 3, rng) for l, n in size.items()}
    parts = [[part[l] for l in s] for s in ops]
    xs = [synth.normal(shp, 20 + i, dtype="bf16") for i, shp in enumerate(shapes[:-1])]
    ins = [upload(x, "bf16", p) for x, p in zip(xs, parts[:-1])]
    out = empty(shapes[-1], "f32", parts[-1])
    contracted = set(lhs.replace(",", "")) - set(rhs)
    agg = ea.AGG_SUM if contracted else ea.AGG_NONE
    ea.joinagg(spec, ea.JOIN_MUL, agg, ins, out)
    ref = oracle.einsum(spec, [synth.to_f64(x, "bf16") for x in xs], oracle.JOIN_MUL,
                        oracle.AGG_SUM if contracted else oracle.AGG_NONE)
    assert_close(values(out), ref, rel_fro=1e-5, what=spec)


# ---------------------------------------------------------------------------
# matrix-core block GEMM
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kmajor", [False, True])
@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_gemm_ragged_blocks(kmajor, out_dtype):
    rng = np.random.default_rng(5)
    T, J, K = 328, 272, 200  # several tiles, ragged tails in every dim
    pt = synth.random_splits(T, 3, rng)
    pj = synth.random_splits(J, 3, rng, quantum=8)
    pk = synth.random_splits(K, 2, rng)
    x = synth.normal((T, J), 31, dtype="bf16")
    w = synth.normal((K, J) if kmajor else (J, K), 32, 0.05, dtype="bf16")
    X = upload(x, "bf16", [pt, pj])
    W = upload(w, "bf16", [pk, pj] if kmajor else [pj, pk])
    Y = empty((T, K), out_dtype, [pt, pk])
    spec = "tj,kj->tk" if kmajor else "tj,jk->tk"
    ea.joinagg(spec, ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    fw = synth.to_f64(w, "bf16")
    ref = oracle.matmul(synth.to_f64(x, "bf16"), fw.T if kmajor else fw)
    assert_close(values(Y), expected(ref, out_dtype), what=f"gemm kmajor={kmajor} {out_dtype}")


@pytest.mark.parametrize("ragged", [False, True])
@pytest.mark.parametrize("out_dtype", ["f16", "f32"])
def test_gemm_f16_inputs(ragged, out_dtype):
    """fp16 operands take the same matrix-core paths as bf16 (f16 MFMA):
    32-aligned blocks the direct-to-LDS pipeline, ragged ones the register-
    staged one."""
    rng = np.random.default_rng(9)
    T, J, K = 320, 384, 264
    if ragged:
        pt = synth.random_splits(T, 3, rng)
        pj = synth.random_splits(J, 3, rng, quantum=8)
        pk = synth.random_splits(K, 2, rng, quantum=8)
    else:
        pt, pj, pk = synth.splits(T, 128), synth.splits(J, 128), [0, 128, 264]
    x = synth.normal((T, J), 35, dtype="f16")
    w = synth.normal((K, J), 36, 0.05, dtype="f16")
    X, W = upload(x, "f16", [pt, pj]), upload(w, "f16", [pk, pj])
    Y = empty((T, K), out_dtype, [pt, pk])
    ea.joinagg("tj,kj->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    ref = oracle.matmul(synth.to_f64(x, "f16"), synth.to_f64(w, "f16").T)
    assert_close(values(Y), expected(ref, out_dtype), what=f"f16 gemm ragged={ragged} -> {out_dtype}")


def test_swiglu_f16_inputs():
    T, H, F = 256, 384, 256
    pt, ph, pf = synth.splits(T, 128), synth.splits(H, 128), synth.splits(F, 128)
    x = synth.normal((T, H), 54, dtype="f16")
    wg = synth.normal((H, F), 55, 0.05, dtype="f16")
    wu = synth.normal((H, F), 56, 0.05, dtype="f16")
    X, G, U = upload(x, "f16", [pt, ph]), upload(wg, "f16", [ph, pf]), upload(wu, "f16", [ph, pf])
    A = empty((T, F), "f16", [pt, pf])
    ea.joinagg("tj,jk,jk->tk", ea.OP_SWIGLU, ea.AGG_SUM, [X, G, U], A)
    fx = synth.to_f64(x, "f16")
    ref = oracle.silu_mul(oracle.matmul(fx, synth.to_f64(wg, "f16")), oracle.matmul(fx, synth.to_f64(wu, "f16")))
    assert_close(values(A), expected(ref, "f16"), what="swiglu f16")


def test_gemm_many_split_parts_deterministic():
    # one 256x256 output tile over 8 contracted blocks: the key is split over
    # several workgroups (more than two parts: the part-order sum), merged by
    # the last to arrive; parity with the oracle, and the same bits every run
    T, J, K = 256, 4096, 256
    p = [synth.splits(T, 256), synth.splits(J, 512)]
    x = synth.normal((T, J), 45, dtype="bf16")
    w = synth.normal((J, K), 46, 0.05, dtype="bf16")
    X, W = upload(x, "bf16", p), upload(w, "bf16", [synth.splits(J, 512), synth.splits(K, 256)])
    pout = [synth.splits(T, 256), synth.splits(K, 256)]
    Y = empty((T, K), "f32", pout)
    ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    ref = oracle.matmul(synth.to_f64(x, "bf16"), synth.to_f64(w, "bf16"))
    assert_close(values(Y), ref, rel_fro=1e-5, what="gemm, many split parts")
    for _ in range(3):
        Y2 = empty((T, K), "f32", pout)
        ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y2)
        torch.cuda.synchronize()
        assert torch.equal(Y.bytes(), Y2.bytes())


def _sampled_rows(T, band=256, rng_seed=3):
    # a few rows of every 256-row tile band, its first and last among them
    rng = np.random.default_rng(rng_seed)
    rows = []
    for b0 in range(0, T, band):
        b1 = min(T, b0 + band)
        rows += [b0, b1 - 1] + list(rng.choice(np.arange(b0 + 1, b1 - 1), 2, replace=False))
    return np.array(sorted(set(rows)))


@pytest.mark.parametrize("swiglu", [False, True])
def test_gemm_block_share_shapes_full_size_sampled_rows(swiglu):
    # 2048 tokens x 8192 hidden in 512-blocks against a 3072-wide projection
    # (96 tiles, keys split in two) or SwiGLU's two 2752-wide weights (176
    # tiles, a ragged last column block): every tile is checked on sampled
    # rows, and repeated calls give the same bytes
    T, J, F = 2048, 8192, 2752 if swiglu else 3072
    pt, pj, pf = synth.splits(T, 512), synth.splits(J, 512), synth.splits(F, 512)
    x = synth.normal((T, J), 55, dtype="bf16")
    ws = [synth.normal((J, F), 56 + i, 0.02, dtype="bf16") for i in range(2 if swiglu else 1)]
    X = upload(x, "bf16", [pt, pj])
    Ws = [upload(w, "bf16", [pj, pf]) for w in ws]
    spec, op = ("tj,jk,jk->tk", ea.OP_SWIGLU) if swiglu else ("tj,jk->tk", ea.JOIN_MUL)
    Y = empty((T, F), "bf16", [pt, pf])
    ea.joinagg(spec, op, ea.AGG_SUM, [X] + Ws, Y)
    rows = _sampled_rows(T)
    fx = synth.to_f64(x, "bf16")[rows]
    prods = [oracle.matmul(fx, synth.to_f64(w, "bf16")) for w in ws]
    ref = oracle.silu_mul(*prods) if swiglu else prods[0]
    assert_close(values(Y)[rows], expected(ref, "bf16"), what="block-share GEMM, sampled rows")
    for _ in range(2):
        Y2 = empty((T, F), "bf16", [pt, pf])
        ea.joinagg(spec, op, ea.AGG_SUM, [X] + Ws, Y2)
        torch.cuda.synchronize()
        assert torch.equal(Y.bytes(), Y2.bytes())


@pytest.mark.parametrize("T,J,K", [(1, 32, 8), (3, 8, 8), (1, 64, 256), (5, 96, 40), (257, 32, 264)])
def test_gemm_tiny_and_single_row_shapes(T, J, K):
    # a single tile mostly masked: one row, one 8-wide column group, a
    # contracted extent of one MFMA step (direct path) or of 8 (register path)
    x = synth.normal((T, J), 47, dtype="bf16")
    w = synth.normal((J, K), 48, 0.1, dtype="bf16")
    pt, pj, pk = synth.whole(T), synth.whole(J), synth.whole(K)
    X, W = upload(x, "bf16", [pt, pj]), upload(w, "bf16", [pj, pk])
    Y = empty((T, K), "f32", [pt, pk])
    ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    ref = oracle.matmul(synth.to_f64(x, "bf16"), synth.to_f64(w, "bf16"))
    assert_close(values(Y), ref, rel_fro=1e-5, what=f"gemm {T}x{J}x{K}")


def test_gemm_integer_data_bitexact_and_residual():
    T, J, K = 256, 512, 384
    pt, pj, pk = synth.splits(T, 128), synth.splits(J, 128), synth.splits(K, 128)
    x = synth.integers((T, J), 41, -2, 2, "bf16")
    w = synth.integers((J, K), 42, -2, 2, "bf16")
    r = synth.integers((T, K), 43, -50, 50, "f32")
    X, W = upload(x, "bf16", [pt, pj]), upload(w, "bf16", [pj, pk])
    R = upload(r, "f32", [pt, pk])
    Y = empty((T, K), "f32", [pt, pk])
    ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y, residual=R)
    exact = synth.to_f64(x, "bf16") @ synth.to_f64(w, "bf16") + synth.to_f64(r, "f32")
    np.testing.assert_array_equal(values(Y), exact)


def test_gemm_identity_is_exact():
    x = synth.normal((256, 256), 44, dtype="bf16")
    eye = synth.store(np.eye(256), "bf16")
    p = [synth.splits(256, 128)] * 2
    X, I = upload(x, "bf16", p), upload(eye, "bf16", p)
    Y = empty((256, 256), "bf16", p)
    ea.joinagg("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [X, I], Y)
    np.testing.assert_array_equal(values(Y), synth.to_f64(x, "bf16"))


def test_gemm_qkv_projection_full_size_sampled_rows():
    w = synth.qkv_projection()
    X, W = upload(w["X"], "bf16", w["pX"]), upload(w["W"], "bf16", w["pW"])
    Y = empty((4096, 1536), "bf16", w["pY"])
    ea.joinagg(w["spec"], ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    got = values(Y)
    rows = np.random.default_rng(0).choice(4096, 96, replace=False)
    rows = np.concatenate([rows, [0, 511, 512, 4095]])
    ref = oracle.matmul(synth.to_f64(w["X"], "bf16")[rows], synth.to_f64(w["W"], "bf16"))
    assert_close(got[rows], expected(ref, "bf16"), what="QKV sampled rows")
    # determinism: a second run gives the same bytes (fixed aggregation order)
    Y2 = empty((4096, 1536), "bf16", w["pY"])
    ea.joinagg(w["spec"], ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y2)
    torch.cuda.synchronize()
    assert torch.equal(Y.bytes(), Y2.bytes())


def test_swiglu_ragged_ffn_blocks():
    T, H, F = 192, 512, 344
    pt, ph = synth.splits(T, 128), synth.splits(H, 128)
    pf = [0, 128, 256, 344]
    x = synth.normal((T, H), 51, dtype="bf16")
    wg = synth.normal((H, F), 52, 0.05, dtype="bf16")
    wu = synth.normal((H, F), 53, 0.05, dtype="bf16")
    X, G, U = upload(x, "bf16", [pt, ph]), upload(wg, "bf16", [ph, pf]), upload(wu, "bf16", [ph, pf])
    A = empty((T, F), "bf16", [pt, pf])
    ea.joinagg("tj,jk,jk->tk", ea.OP_SWIGLU, ea.AGG_SUM, [X, G, U], A)
    fx = synth.to_f64(x, "bf16")
    ref = oracle.silu_mul(oracle.matmul(fx, synth.to_f64(wg, "bf16")), oracle.matmul(fx, synth.to_f64(wu, "bf16")))
    assert_close(values(A), expected(ref, "bf16"), what="swiglu")


# ---------------------------------------------------------------------------
# row reductions
# ---------------------------------------------------------------------------
def test_rmsnorm_full_size_8_column_blocks():
    w = synth.reductions()
    X, Wt = upload(w["x"], "bf16", w["px"]), upload(w["w"], "bf16", w["pw"])
    Y = empty((4096, 4096), "bf16", w["px"])
    ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=w["eps"])
    ref = oracle.rmsnorm(synth.to_f64(w["x"], "bf16"), synth.to_f64(w["w"], "bf16"), w["eps"])
    assert_close(values(Y), expected(ref, "bf16"), what="rmsnorm")


@pytest.mark.parametrize("xdt,ydt", [("f32", "f32"), ("bf16", "f32"), ("f32", "bf16")])
def test_rmsnorm_ragged_blocks(xdt, ydt):
    rng = np.random.default_rng(8)
    T, C = 70, 300
    pt = synth.random_splits(T, 3, rng)
    pc = synth.random_splits(C, 4, rng)  # not 16-byte multiples: scalar path
    x = synth.normal((T, C), 61, dtype=xdt)
    wv = synth.uniform((C,), 62, 0.5, 1.5, dtype="bf16")
    X, Wt = upload(x, xdt, [pt, pc]), upload(wv, "bf16", [pc])
    Y = empty((T, C), ydt, [pt, pc])
    ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=1e-6)
    ref = oracle.rmsnorm(synth.to_f64(x, xdt), synth.to_f64(wv, "bf16"), 1e-6)
    assert_close(values(Y), expected(ref, ydt), what="rmsnorm ragged")


def test_rmsnorm_vector_path_f32_blocks():
    T, C = 64, 1024
    pt, pc = [0, 32, 64], synth.splits(C, 256)
    x = synth.normal((T, C), 63, dtype="f32")
    wv = synth.uniform((C,), 64, 0.5, 1.5, dtype="f32")
    X, Wt = upload(x, "f32", [pt, pc]), upload(wv, "f32", [pc])
    Y = empty((T, C), "f32", [pt, pc])
    ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=1e-6)
    ref = oracle.rmsnorm(synth.to_f64(x, "f32"), synth.to_f64(wv, "f32"), 1e-6)
    assert_close(values(Y), ref, rel_fro=1e-5, what="rmsnorm f32")


def test_causal_softmax_full_size_key_blocks():
    w = synth.reductions()
    S = upload(w["s"], "bf16", w["ps"])
    P = empty((4, 2048, 2048), "bf16", w["ps"])
    ea.joinagg("hqk->hqk", ea.OP_SOFTMAX, ea.AGG_LSE, [S], P, causal=True)
    ref = oracle.softmax(synth.to_f64(w["s"], "bf16"), True)
    got = values(P)
    assert_close(got, expected(ref, "bf16"), what="causal softmax")
    # masked entries are exactly zero
    mask = np.triu(np.ones((2048, 2048), dtype=bool), 1)
    assert np.all(got[:, mask] == 0)


def test_rmsnorm_vector_path_short_last_segment():
    # 16-byte segments, all but the last of one length: register path with the
    # direct segment lookup, but not the affine layout
    T, C = 40, 1032
    pt, pc = [0, 24, 40], [0, 512, 1024, 1032]
    x = synth.normal((T, C), 65, dtype="bf16")
    wv = synth.uniform((C,), 66, 0.5, 1.5, dtype="bf16")
    X, Wt = upload(x, "bf16", [pt, pc]), upload(wv, "bf16", [pc])
    Y = empty((T, C), "bf16", [pt, pc])
    ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=1e-6)
    ref = oracle.rmsnorm(synth.to_f64(x, "bf16"), synth.to_f64(wv, "bf16"), 1e-6)
    assert_close(values(Y), expected(ref, "bf16"), what="rmsnorm short last segment")


def test_rmsnorm_two_wavefronts_per_row_partial_task():
    # 8192-element bf16 rows in the block share's 512-blocks with bf16
    # weights: each row on two wavefronts; 1027 rows leave a last row block of
    # three rows, so its task has a wavefront pair with no row (it must meet
    # the halves' barrier and write nothing)
    T, C = 1027, 8192
    pt, pc = synth.splits(T, 512), synth.splits(C, 512)
    x = synth.normal((T, C), 67, dtype="bf16")
    wv = synth.uniform((C,), 68, 0.5, 1.5, dtype="bf16")
    X, Wt = upload(x, "bf16", [pt, pc]), upload(wv, "bf16", [pc])
    Y = empty((T, C), "bf16", [pt, pc])
    ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=1e-5)
    ref = oracle.rmsnorm(synth.to_f64(x, "bf16"), synth.to_f64(wv, "bf16"), 1e-5)
    got = values(Y)
    assert_close(got, expected(ref, "bf16"), what="rmsnorm, two wavefronts per row")
    assert_close(got[1024:], expected(ref[1024:], "bf16"), what="rmsnorm, partial last task")


def test_causal_softmax_two_heads_per_block():
    # equal blocks (affine layout), two heads per block: a group's rows run
    # over both heads, so the query position wraps at the query block's extent
    H, Q, K = 4, 96, 128
    ph, pq, pk = synth.splits(H, 2), [0, 48, 96], synth.splits(K, 32)
    s = synth.normal((H, Q, K), 72, 2.0, dtype="bf16")
    Sr = upload(s, "bf16", [ph, pq, pk])
    P = empty((H, Q, K), "bf16", [ph, pq, pk])
    ea.joinagg("hqk->hqk", ea.OP_SOFTMAX, ea.AGG_LSE, [Sr], P, causal=True)
    ref = oracle.softmax(synth.to_f64(s, "bf16"), True)
    got = values(P)
    assert_close(got, expected(ref, "bf16"), what="causal softmax, two heads per block")
    mask = np.triu(np.ones((Q, K), dtype=bool), 1)
    assert np.all(got[:, mask] == 0)


@pytest.mark.parametrize("causal", [False, True])
def test_softmax_ragged_and_f32(causal):
    rng = np.random.default_rng(9)
    H, Q, K = 3, 40, 40
    ph, pq, pk = synth.splits(H, 2), synth.random_splits(Q, 3, rng), synth.random_splits(K, 3, rng)
    s = synth.normal((H, Q, K), 71, 2.0, dtype="f32")
    Sr = upload(s, "f32", [ph, pq, pk])
    P = empty((H, Q, K), "f32", [ph, pq, pk])
    ea.joinagg("hqk->hqk", ea.OP_SOFTMAX, ea.AGG_LSE, [Sr], P, causal=causal)
    ref = oracle.softmax(synth.to_f64(s, "f32"), causal)
    assert_close(values(P), ref, rel_fro=1e-5, what="softmax ragged")


@pytest.mark.parametrize("T,C", [(1, 1), (1, 7), (5, 1), (1, 4096)])
def test_rmsnorm_degenerate_shapes(T, C):
    # one row and/or one column: with C = 1 every output is w / sqrt(1 + eps / x^2)
    x = synth.normal((T, C), 67, dtype="bf16")
    wv = synth.uniform((C,), 68, 0.5, 1.5, dtype="bf16")
    pt, pc = synth.whole(T), synth.whole(C)
    X, Wt = upload(x, "bf16", [pt, pc]), upload(wv, "bf16", [pc])
    Y = empty((T, C), "f32", [pt, pc])
    ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], Y, eps=1e-6)
    fx, fw = synth.to_f64(x, "bf16"), synth.to_f64(wv, "bf16")
    ref = oracle.rmsnorm(fx, fw, 1e-6)
    assert_close(values(Y), ref, rel_fro=1e-5, what=f"rmsnorm {T}x{C}")
    if C == 1:
        assert_close(values(Y), np.sign(fx) * fw / np.sqrt(1 + 1e-6 / fx ** 2), rel_fro=1e-5, what="C = 1")


@pytest.mark.parametrize("causal", [False, True])
def test_softmax_degenerate_shapes(causal):
    # one key per row gives exactly 1; a 1 x 1 causal block is its diagonal;
    # one query row over many key blocks sees only key 0 when causal
    for shape, parts in [((3, 5, 1), [synth.splits(3, 1), synth.whole(5), [0, 1]]),
                         ((1, 1, 1), [[0, 1], [0, 1], [0, 1]]),
                         ((1, 1, 300), [[0, 1], [0, 1], [0, 100, 200, 300]])]:
        s = synth.normal(shape, 73, 2.0, dtype="bf16")
        Sr = upload(s, "bf16", parts)
        P = empty(shape, "f32", parts)
        ea.joinagg("hqk->hqk", ea.OP_SOFTMAX, ea.AGG_LSE, [Sr], P, causal=causal)
        got = values(P)
        ref = oracle.softmax(synth.to_f64(s, "bf16"), causal)
        assert_close(got, ref, rel_fro=1e-5, what=f"softmax {shape}")
        if shape[2] == 1 or causal:
            assert np.all(got[..., 0] == 1.0) and np.all(got[..., 1:] == 0.0)
