"""The caller-owned workspace of key-split join-aggs (include/ea.h,
"Workspace"): the block-share GEMM and attention configurations, whose output
tiles are split over several workgroups, run on two streams at once with two
workspaces and match the serial run bit for bit and the oracle; one workspace
serves a sequence of different configurations on one stream; a short or
missing workspace and an unplanned configuration are refused."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_close, download, expected, upload, values
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu

T, HID, WQKV = 2048, 8192, 3072


def _gemm_operands():
    # the block share's QKV projection: [2048, 8192] x [8192, 3072] in 512-blocks
    x = synth.normal((T, HID), 941, dtype="bf16")
    w = synth.normal((HID, WQKV), 942, 0.02, dtype="bf16")
    px = [synth.splits(T, 512), synth.splits(HID, 512)]
    pw = [synth.splits(HID, 512), synth.splits(WQKV, 512)]
    py = [synth.splits(T, 512), synth.splits(WQKV, 512)]
    return x, w, upload(x, "bf16", px), upload(w, "bf16", pw), py


def _attn_operands():
    # the block share's causal attention: 8 heads of 2048 tokens, 128-blocks
    part = [[0, 1], synth.splits(8, 1), synth.splits(T, 128), [0, 128]]
    q, k, v = (synth.normal((1, 8, T, 128), s, dtype="bf16") for s in (943, 944, 945))
    return (q, k, v), [upload(a, "bf16", part) for a in (q, k, v)], part


def _gemm(X, W, Y, **kw):
    ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y, **kw)


def _attn(Q, K, V, O, **kw):
    ea.joinagg("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O, scale=1.0 / np.sqrt(128),
               causal=True, **kw)


def test_split_key_gemm_and_attention_on_two_streams():
    x, w, X, W, py = _gemm_operands()
    qkv, (Q, K, V), part = _attn_operands()
    need_g = ea.joinagg_workspace("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], ea.Relation((T, WQKV), "bf16", py))
    O0 = ea.Relation((1, 8, T, 128), "bf16", part)
    need_a = ea.joinagg_workspace("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O0,
                                  scale=1.0 / np.sqrt(128), causal=True)
    print(f"workspace bytes: gemm {need_g}, attention {need_a}", flush=True)
    # both configurations split keys, so both need more than the counter area
    assert need_g > ea.WS_COUNTER_BYTES and need_a > ea.WS_COUNTER_BYTES
    # serial reference on the current stream
    Y0 = ea.Relation((T, WQKV), "bf16", py)
    _gemm(X, W, Y0)
    _attn(Q, K, V, O0)
    torch.cuda.synchronize()
    # the same two configurations, each on two streams at once, each stream
    # with its own workspace (zeroed once)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    wss = [ea.new_workspace(max(need_g, need_a)) for _ in streams]
    outs = [(ea.Relation((T, WQKV), "bf16", py), ea.Relation((1, 8, T, 128), "bf16", part)) for _ in streams]
    torch.cuda.synchronize()
    for _ in range(3):
        for s, ws, (Y, O) in zip(streams, wss, outs):
            with torch.cuda.stream(s):
                _gemm(X, W, Y, stream=s, workspace=ws)
                _attn(Q, K, V, O, stream=s, workspace=ws)
    torch.cuda.synchronize()
    for Y, O in outs:
        assert torch.equal(Y.bytes(), Y0.bytes())
        assert torch.equal(O.bytes(), O0.bytes())
    # every call left the counter area zero
    for ws in wss:
        assert int(ws[:ea.WS_COUNTER_BYTES].count_nonzero()) == 0
    # and the results are the join-aggs' (oracle on sampled rows / whole heads)
    rows = np.array([0, 1, 255, 256, 511, 1024, 1535, 2047])
    ref = oracle.matmul(synth.to_f64(x[rows], "bf16"), synth.to_f64(w, "bf16"))
    assert_close(synth.to_f64(download(Y0)[rows], "bf16"), expected(ref, "bf16"), what="gemm")
    f = [synth.to_f64(a, "bf16") for a in qkv]
    ref = oracle.attention(f[0], f[1], f[2], True, 1.0 / np.sqrt(128))
    assert_close(values(O0), expected(ref, "bf16"), what="attention")


def test_one_workspace_across_configurations():
    """Split-key plans place their partials after the counter area, so a
    GEMM, an attention and the GEMM again can share one workspace."""
    x, w, X, W, py = _gemm_operands()
    _, (Q, K, V), part = _attn_operands()
    Y1, Y2 = ea.Relation((T, WQKV), "bf16", py), ea.Relation((T, WQKV), "bf16", py)
    O1, O2 = ea.Relation((1, 8, T, 128), "bf16", part), ea.Relation((1, 8, T, 128), "bf16", part)
    need = max(ea.joinagg_workspace("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y1),
               ea.joinagg_workspace("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O1,
                                    scale=1.0 / np.sqrt(128), causal=True))
    ws = ea.new_workspace(need)
    _gemm(X, W, Y1, workspace=ws)
    _attn(Q, K, V, O1, workspace=ws)
    _gemm(X, W, Y2, workspace=ws)
    _attn(Q, K, V, O2, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(Y1.bytes(), Y2.bytes())
    assert torch.equal(O1.bytes(), O2.bytes())
    assert int(ws[:ea.WS_COUNTER_BYTES].count_nonzero()) == 0


def _raw(spec, join_op, agg_op, ins, out, ws_ptr, ws_bytes, **kw):
    handles = (ctypes.c_void_p * len(ins))(*[r.handle.value for r in ins])
    prm, _ends = ea._params(**kw)
    return ea.lib().ea_joinagg(spec.encode(), join_op, agg_op, len(ins), handles, out.handle, ctypes.byref(prm),
                               ws_ptr, ws_bytes, ea._stream(None))


def test_workspace_errors_and_unplanned_configurations():
    _, _, X, W, py = _gemm_operands()
    Y = ea.Relation((T, WQKV), "bf16", py)
    need = ea.joinagg_workspace("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y)
    ws = ea.new_workspace(need)
    p = ctypes.c_void_p(ws.data_ptr())
    assert _raw("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y, p, need - 1) == -4      # short: EA_ERR_CAPACITY
    assert _raw("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y, None, 0) == -1          # missing: EA_ERR_ARG
    assert _raw("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y, ctypes.c_void_p(ws.data_ptr() + 16),
                need) == -1                                                               # misaligned
    assert _raw("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], Y, p, need) == 0
    # a configuration never planned: EA_ERR_NOPLAN, and nothing was enqueued
    pz = [synth.splits(T, 384), synth.splits(WQKV, 384)]
    Xz = ea.Relation((T, HID), "bf16", [pz[0], synth.splits(HID, 384)])
    Wz = ea.Relation((HID, WQKV), "bf16", [synth.splits(HID, 384), pz[1]])
    Yz = ea.Relation((T, WQKV), "bf16", pz)
    assert _raw("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [Xz, Wz], Yz, p, need) == -9
    src = ea.Relation((64, 64), "bf16", [synth.splits(64, 16), synth.splits(64, 32)])
    dst = ea.Relation((64, 64), "bf16", [synth.splits(64, 32), synth.splits(64, 16)])
    assert ea.lib().ea_repartition(src.handle, dst.handle, None) == -9
    ea.repartition_plan(src, dst)
    assert ea.lib().ea_repartition(src.handle, dst.handle, None) == 0
    torch.cuda.synchronize()
