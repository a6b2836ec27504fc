"""Work schedules and tile shapes of the direct-load block GEMM (one GPU's
share of 'tj,jk->tk' and SwiGLU, Section 3.2, Example "Matrix multiply,
decomposed").  With fewer output tiles than CUs a plan either splits each
tile's K steps evenly over a few workgroups, or shares all tiles' K steps out
in 256 equal runs, a run possibly finishing one tile and starting the next (a
tile cut into several runs is merged by the last to arrive); and a plain
product may take 256 x 128 tiles instead of 256 x 256 ones.  The plan's cost
model chooses; EA_GEMM_SCHEDULE and EA_GEMM_TILE_N force a choice when a plan
is built.  Integer-valued data make every summation order exact, so every
choice must give the same bits; N(0,1) data are compared with the oracle."""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_close, download, expected, upload
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu


def _run(schedule, spec, op, ins, out_shape, part, dtype="bf16", tile_n=None, residual=None):
    ea.plan_cache_clear()
    env = {"EA_GEMM_SCHEDULE": schedule}
    if tile_n is not None:
        env["EA_GEMM_TILE_N"] = str(tile_n)
    os.environ.update(env)
    try:
        Y = ea.Relation(out_shape, dtype, part)
        Y.data.fill_(0xFF)
        ea.joinagg(spec, op, ea.AGG_SUM, ins, Y, residual=residual)
        torch.cuda.synchronize()
    finally:
        for k in env:
            del os.environ[k]
        ea.plan_cache_clear()
    return Y


@pytest.mark.parametrize("kmajor", [False, True])
def test_balanced_and_even_schedules_agree_on_integer_data(kmajor):
    # 1024 x 4096 x 1536 in 512-blocks: 24 tiles of 256 x 256 and 128 K steps
    # each; balanced: 256 runs of 12 steps, most tiles cut into several runs and
    # many runs spanning two tiles
    T, J, K = 1024, 4096, 1536
    print(f"schedule test, kmajor={kmajor}", flush=True)
    x = synth.integers((T, J), 991, -2, 3, dtype="bf16")
    w = synth.integers((K, J) if kmajor else (J, K), 992, -2, 3, dtype="bf16")
    X = upload(x, "bf16", [synth.splits(T, 512), synth.splits(J, 512)])
    W = upload(w, "bf16", [synth.splits(K, 512), synth.splits(J, 512)] if kmajor else
               [synth.splits(J, 512), synth.splits(K, 512)])
    spec = "tj,kj->tk" if kmajor else "tj,jk->tk"
    py = [synth.splits(T, 512), synth.splits(K, 512)]
    Ye = _run("even", spec, ea.JOIN_MUL, [X, W], (T, K), py, "f32")
    Yb = _run("balanced", spec, ea.JOIN_MUL, [X, W], (T, K), py, "f32")
    assert torch.equal(Ye.bytes(), Yb.bytes())
    fx, fw = synth.to_f64(x, "bf16"), synth.to_f64(w, "bf16")
    ref = oracle.matmul(fx, fw.T.copy() if kmajor else fw)
    got = download(Yb).astype(np.float64)
    assert np.array_equal(got, ref)  # integer sums below 2^24: exact


def test_balanced_schedule_swiglu_and_ragged_blocks_match_the_oracle():
    # SwiGLU on the block share's FFN shapes cut to 512 tokens: 2 x 22 tiles of
    # 256 x 128 (the 2752-wide output ends in a 192-wide block), 256 K steps
    T, H, F = 512, 8192, 2752
    h = synth.normal((T, H), 993, dtype="bf16")
    wg = synth.normal((H, F), 994, 0.02, dtype="bf16")
    wu = synth.normal((H, F), 995, 0.02, dtype="bf16")
    pf = synth.splits(F, 512)
    Hh = upload(h, "bf16", [synth.splits(T, 512), synth.splits(H, 512)])
    Wg = upload(wg, "bf16", [synth.splits(H, 512), pf])
    Wu = upload(wu, "bf16", [synth.splits(H, 512), pf])
    py = [synth.splits(T, 512), pf]
    Yb = _run("balanced", "tj,jk,jk->tk", ea.OP_SWIGLU, [Hh, Wg, Wu], (T, F), py)
    Ye = _run("even", "tj,jk,jk->tk", ea.OP_SWIGLU, [Hh, Wg, Wu], (T, F), py)
    fh = synth.to_f64(h, "bf16")
    ref = oracle.silu_mul(oracle.matmul(fh, synth.to_f64(wg, "bf16")), oracle.matmul(fh, synth.to_f64(wu, "bf16")))
    for Y, name in ((Yb, "balanced"), (Ye, "even")):
        assert_close(synth.to_f64(download(Y), "bf16"), expected(ref, "bf16"), what=f"swiglu {name}")


@pytest.mark.parametrize("kmajor", [False, True])
def test_narrow_and_wide_tiles_agree_on_integer_data(kmajor):
    # 768 x 2048 x 1472 in 512-blocks (the last output block 448 wide, so
    # 256 x 128 tiles end half masked): wide and narrow tiles, each with the
    # even and the balanced schedule, give the same exact sums
    T, J, K = 768, 2048, 1472
    print(f"tile-width test, kmajor={kmajor}", flush=True)
    x = synth.integers((T, J), 996, -2, 3, dtype="bf16")
    w = synth.integers((K, J) if kmajor else (J, K), 997, -2, 3, dtype="bf16")
    pk = synth.splits(K, 512)
    X = upload(x, "bf16", [synth.splits(T, 512), synth.splits(J, 512)])
    W = upload(w, "bf16", [pk, synth.splits(J, 512)] if kmajor else [synth.splits(J, 512), pk])
    spec = "tj,kj->tk" if kmajor else "tj,jk->tk"
    py = [synth.splits(T, 512), pk]
    outs = [_run(sch, spec, ea.JOIN_MUL, [X, W], (T, K), py, "f32", tile_n=tn)
            for tn in (256, 128) for sch in ("even", "balanced")]
    for Y in outs[1:]:
        assert torch.equal(outs[0].bytes(), Y.bytes())
    fx, fw = synth.to_f64(x, "bf16"), synth.to_f64(w, "bf16")
    ref = oracle.matmul(fx, fw.T.copy() if kmajor else fw)
    assert np.array_equal(download(outs[1]).astype(np.float64), ref)


def test_narrow_tiles_with_residual_match_the_oracle():
    # the O projection's shape cut to 512 tokens, bf16 out with a residual:
    # 2 x 64 tiles of 256 x 128
    T, J, K = 512, 1024, 8192
    a = synth.normal((T, J), 998, dtype="bf16")
    w = synth.normal((J, K), 999, 0.02, dtype="bf16")
    r = synth.normal((T, K), 1000, dtype="bf16")
    py = [synth.splits(T, 512), synth.splits(K, 512)]
    A = upload(a, "bf16", [synth.splits(T, 512), synth.splits(J, 512)])
    W = upload(w, "bf16", [synth.splits(J, 512), synth.splits(K, 512)])
    R = upload(r, "bf16", py)
    Y = _run("even", "tj,jk->tk", ea.JOIN_MUL, [A, W], (T, K), py, "bf16", tile_n=128, residual=R)
    ref = oracle.matmul(synth.to_f64(a, "bf16"), synth.to_f64(w, "bf16")) + synth.to_f64(r, "bf16")
    assert_close(synth.to_f64(download(Y), "bf16"), expected(ref, "bf16"), what="narrow tiles + residual")


def _uneven_splits(n_blocks):
    # contracted block widths cycling 32, 64, 96, 32 (multiples of the
    # direct-load kernel's 32-deep K step)
    widths = [(32, 64, 96, 32)[i % 4] for i in range(n_blocks)]
    return [0] + list(np.cumsum(widths))


@pytest.mark.parametrize("schedule", ["even", "balanced"])
@pytest.mark.parametrize("n_blocks", [128, 129])
def test_most_tuples_per_key_and_uneven_k_blocks(schedule, n_blocks):
    # 128 contracted blocks per output key is the most the direct-load
    # kernel's tuple table holds (129 take the register-staged kernel); the
    # uneven widths make runs start inside a tuple.  Integer data: exact in
    # any summation order, so the bits equal the oracle's
    print(f"most tuples per key, {n_blocks} blocks, {schedule}", flush=True)
    pj = _uneven_splits(n_blocks)
    T, J, K = 512, int(pj[-1]), 256
    x = synth.integers((T, J), 995, -2, 3, dtype="bf16")
    w = synth.integers((J, K), 996, -2, 3, dtype="bf16")
    X = upload(x, "bf16", [synth.splits(T, 256), pj])
    W = upload(w, "bf16", [pj, [0, K]])
    py = [synth.splits(T, 256), [0, K]]
    Y = _run(schedule, "tj,jk->tk", ea.JOIN_MUL, [X, W], (T, K), py, "f32")
    exact = synth.to_f64(x, "bf16") @ synth.to_f64(w, "bf16")
    np.testing.assert_array_equal(download(Y), exact)
