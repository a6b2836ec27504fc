"""Work schedules of the direct-load block GEMM (one GPU's share of
'tj,jk->tk' and SwiGLU, Section 3.2, Example "Matrix multiply, decomposed").
With fewer output tiles than CUs a plan either splits each tile's K steps
evenly over a few workgroups, or shares all tiles' K steps out in 256 equal
runs, a run possibly finishing one tile and starting the next (a tile cut
into several runs is merged by the last to arrive).  The plan's cost model
chooses; EA_GEMM_SCHEDULE forces one when a plan is built.  Integer-valued
data make every summation order exact, so both schedules must give the same
bits; N(0,1) data are compared with the oracle."""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_close, download, expected, upload
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu


def _run(schedule, spec, op, ins, out_shape, part, dtype="bf16"):
    ea.plan_cache_clear()
    os.environ["EA_GEMM_SCHEDULE"] = schedule
    try:
        Y = ea.Relation(out_shape, dtype, part)
        Y.data.fill_(0xFF)
        ea.joinagg(spec, op, ea.AGG_SUM, ins, Y)
        torch.cuda.synchronize()
    finally:
        del os.environ["EA_GEMM_SCHEDULE"]
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
