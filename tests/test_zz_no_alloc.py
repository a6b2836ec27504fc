"""ea_joinagg_noalloc: a join-agg planned earlier, run with the library's
fixed per-device workspace array instead of a caller buffer (for callers that
cannot allocate).  Its output must equal ea_joinagg's bit for bit (the same
kernels and merge order) and the oracle's within the single-operator
tolerance, on two calls in a row with the second on a smaller input, for the
two split-key kernels (block GEMM, attention).  Collected last: it also runs
after every other GPU test has left the array as its last call did."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_close, download, expected, upload, values
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu


def _raw_noalloc(spec, join_op, agg_op, ins, out, **kw):
    """ea_joinagg_noalloc through the C ABI."""
    handles = (ctypes.c_void_p * len(ins))(*[r.handle.value for r in ins])
    prm, _ends = ea._params(**kw)
    return ea.lib().ea_joinagg_noalloc(spec.encode(), join_op, agg_op, len(ins), handles, out.handle,
                                       ctypes.byref(prm), ea._stream(None))


def _gemm_case(T, J, K, block, seed):
    x = synth.normal((T, J), seed, dtype="bf16")
    w = synth.normal((J, K), seed + 1, 0.02, dtype="bf16")
    X = upload(x, "bf16", [synth.splits(T, block), synth.splits(J, block)])
    W = upload(w, "bf16", [synth.splits(J, block), synth.splits(K, block)])
    py = [synth.splits(T, block), synth.splits(K, block)]
    return x, w, X, W, py


def test_noalloc_gemm_matches_joinagg_on_two_calls():
    # call 1: the block share's QKV projection, 2048 x 8192 x 3072 in 512-blocks
    # (96 tiles whose K steps are shared out over 256 workgroups: tens of MiB
    # of partials); call 2: a smaller split-key GEMM, 512 x 4096 x 512 in
    # 256-blocks
    spec = "tj,jk->tk"
    for (T, J, K, block, seed) in ((2048, 8192, 3072, 512, 961), (512, 4096, 512, 256, 963)):
        print(f"noalloc gemm {T}x{J}x{K}", flush=True)
        x, w, X, W, py = _gemm_case(T, J, K, block, seed)
        Yref = ea.Relation((T, K), "bf16", py)
        need = ea.joinagg_workspace(spec, ea.JOIN_MUL, ea.AGG_SUM, [X, W], Yref)
        assert ea.WS_COUNTER_BYTES < need <= (128 << 20)
        ea.joinagg(spec, ea.JOIN_MUL, ea.AGG_SUM, [X, W], Yref)
        Y = ea.Relation((T, K), "bf16", py)
        Y.data.fill_(0xFF)
        n_plans = ea.plan_cache_size()
        assert _raw_noalloc(spec, ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y) == 0
        torch.cuda.synchronize()
        assert ea.plan_cache_size() == n_plans  # no plan built by the call
        assert torch.equal(Y.bytes(), Yref.bytes())
        rows = np.array([0, 1, T // 2, T - 1])
        ref = oracle.matmul(synth.to_f64(x[rows], "bf16"), synth.to_f64(w, "bf16"))
        assert_close(synth.to_f64(download(Y)[rows], "bf16"), expected(ref, "bf16"), what=f"gemm {T}x{J}x{K}")


def test_noalloc_attention_matches_joinagg_on_two_calls():
    # call 1: the block share's causal attention (8 heads x 2048 tokens, key
    # splits of up to three parts); call 2: 2 heads x 1024 tokens
    spec = "bhqd,bhkd,bhkd->bhqd"
    scale = 1.0 / np.sqrt(128)
    for (H, S, seed) in ((8, 2048, 971), (2, 1024, 974)):
        print(f"noalloc attention {H} heads x {S}", flush=True)
        part = [[0, 1], synth.splits(H, 1), synth.splits(S, 128), [0, 128]]
        qkv = [synth.normal((1, H, S, 128), seed + i, dtype="bf16") for i in range(3)]
        Q, K, V = (upload(a, "bf16", part) for a in qkv)
        Oref = ea.Relation((1, H, S, 128), "bf16", part)
        ea.joinagg(spec, ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], Oref, scale=scale, causal=True)
        O = ea.Relation((1, H, S, 128), "bf16", part)
        O.data.fill_(0xFF)
        assert _raw_noalloc(spec, ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O, scale=scale, causal=True) == 0
        torch.cuda.synchronize()
        assert torch.equal(O.bytes(), Oref.bytes())
        ref = oracle.attention(*(synth.to_f64(a, "bf16") for a in qkv), True, scale)
        assert_close(values(O), expected(ref, "bf16"), what=f"attention {H}x{S}")


def test_noalloc_refuses_unplanned_and_oversized():
    # an unplanned configuration: EA_ERR_NOPLAN, nothing planned or run
    x, w, X, W, py = _gemm_case(640, 1280, 640, 320, 981)
    Y = ea.Relation((640, 640), "bf16", py)
    n_plans = ea.plan_cache_size()
    assert _raw_noalloc("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y) == -9
    assert ea.plan_cache_size() == n_plans
    # a plan whose workspace exceeds the 128 MiB array: EA_ERR_CAPACITY.  One
    # causal head of 131072 tokens in 128-blocks splits its long key runs over
    # up to 16 parts: thousands of 65 KiB partials
    S = 131072
    part = [[0, 1], [0, 1], synth.splits(S, 128), [0, 128]]
    Q, K, V, O = (ea.Relation((1, 1, S, 128), "bf16", part) for _ in range(4))
    need = ea.joinagg_workspace("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O,
                                scale=1.0 / np.sqrt(128), causal=True)
    assert need > (128 << 20)
    assert _raw_noalloc("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O,
                        scale=1.0 / np.sqrt(128), causal=True) == -4
