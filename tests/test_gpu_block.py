"""GPU parity of the composite: one GPU's share of a LLaMA-shaped block run as
a chain of join-aggs and repartitions.

Every arrow is checked on its own: each join-agg's output against the oracle
run on the GPU's own upstream relations (so no rounding cascade enters) at
the single-operator tolerance, and each repartition bit for bit.  The whole
chain is then checked end to end against the oracle's chain with bf16
rounding at the same relation boundaries, at CHAIN_REL_FRO (see helpers)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import CHAIN_REL_FRO, assert_close, download, values
from paper_2609_03905_amd.block import LlamaBlockShare

pytestmark = pytest.mark.gpu

_W = ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")


def _raw(rel):
    torch.cuda.synchronize()
    return rel.bytes().cpu().numpy()


def _stagewise(blk, w, rows=None):
    """Each stage of the chain against the oracle on the GPU's upstream
    relations: join-aggs at the single-operator tolerance (bf16 outputs
    against the RNE of the oracle), repartitions bit for bit.  rows: check
    the row-wise stages at these token rows only (attention at those query
    rows, over all the keys they see)."""
    r = oracle.rne_bf16
    f = {k: synth.to_f64(w[k], "bf16") for k in _W}
    heads, hkv, dh, eps = blk.heads, blk.heads_kv, blk.d_head, blk.eps
    hd, kvd, T = heads * dh, hkv * dh, blk.t
    sel = (lambda a: a) if rows is None else (lambda a: a[rows])

    def gv(name):
        rel = getattr(blk, name)
        return values(rel) if rows is None else synth.to_f64(download(rel)[rows], rel.dtype)

    h1 = gv("h1")
    assert_close(h1, r(oracle.rmsnorm(sel(f["x"]), f["n1"], eps)), what="stage rmsnorm1")
    qkv_all = values(blk.qkv)
    qkv = sel(qkv_all)
    assert_close(qkv, r(oracle.matmul(h1, f["wqkv"])), what="stage qkv_gemm")
    # repartition to per-head blocks: the same bytes under the new partition
    want = oracle.repartition(_raw(blk.qkv), blk.qkv.partition, blk.qkv_heads.partition, np.uint16)
    assert np.array_equal(_raw(blk.qkv_heads), want), "stage repart_heads not bit-exact"
    # attention on the GPU's q, k, v
    q = qkv_all[:, :hd].reshape(T, heads, dh).transpose(1, 0, 2)
    k = qkv_all[:, hd:hd + kvd].reshape(T, hkv, dh).transpose(1, 0, 2)
    v = qkv_all[:, hd + kvd:hd + 2 * kvd].reshape(T, hkv, dh).transpose(1, 0, 2)
    if rows is None:
        o = oracle.attention_ex(q[None], k[None], v[None], True, blk.scale, seq_ends=blk.seq_ends)[0]
        o = o.transpose(1, 0, 2).reshape(T, hd)
    else:
        o = oracle.attention_rows(q, k, v, rows, blk.scale, seq_ends=blk.seq_ends).reshape(len(rows), hd)
    attn = gv("attn")
    # the attention output as stored per head, and its repartition to 512-blocks
    want = oracle.repartition(_raw(blk.o_cols), blk.o_cols.partition, blk.attn.partition, np.uint16)
    assert np.array_equal(_raw(blk.attn), want), "stage repart_cols not bit-exact"
    assert_close(attn, r(o), what="stage attention")
    x2 = gv("x2")
    assert_close(x2, r(oracle.add(sel(f["x"]), oracle.matmul(attn, f["wo"]))), what="stage o_gemm_residual")
    h2 = gv("h2")
    assert_close(h2, r(oracle.rmsnorm(x2, f["n2"], eps)), what="stage rmsnorm2")
    a = gv("a")
    assert_close(a, r(oracle.silu_mul(oracle.matmul(h2, f["wg"]), oracle.matmul(h2, f["wu"]))), what="stage swiglu")
    assert_close(gv("y"), r(oracle.add(x2, oracle.matmul(a, f["wd"]))), what="stage down_gemm_residual")


def _device(w):
    return {k: torch.from_numpy(w[k].view(np.int16)).cuda() for k in ("x", "n1", "n2", "wqkv", "wo", "wg", "wu", "wd")}


def _oracle(w, rows=None):
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    x = f["x"] if rows is None else f["x"][:rows]
    return oracle.llama_block(x, f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"], f["n2"],
                              heads=w["heads"], d_head=w["d_head"], eps=w["eps"])


def _run(w):
    blk = LlamaBlockShare(w["t"], w["hidden"], w["heads"], w["d_head"], w["ffn"], block=w["block"], eps=w["eps"])
    blk.load(_device(w))
    blk.forward()
    torch.cuda.synchronize()
    return blk


def test_block_small_all_boundaries():
    w = synth.llama_block(t=256, hidden=512, heads=2, d_head=128, ffn=344, block=128)
    blk = _run(w)
    _stagewise(blk, w)
    ref = _oracle(w)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(values(getattr(blk, name)), ref[name], rel_fro=CHAIN_REL_FRO, what=name)


def test_block_well_conditioned_chain_strict():
    """Small weights keep the softmax flat and the SwiGLU product small, so
    rounding flips do not cascade: the whole chain meets 1e-3."""
    w = synth.llama_block(t=256, hidden=512, heads=2, d_head=128, ffn=344, block=128)
    for k in ("wqkv", "wo", "wg", "wu", "wd"):
        w[k] = synth.store(synth.to_f64(w[k], "bf16") * 0.1, "bf16")
    blk = _run(w)
    ref = _oracle(w)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(values(getattr(blk, name)), ref[name], what=name)


def test_block_full_size():
    w = synth.llama_block()
    blk = _run(w)
    _stagewise(blk, w)
    ref = _oracle(w)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(values(getattr(blk, name)), ref[name], rel_fro=CHAIN_REL_FRO, what=name)
    # a second forward pass reproduces the same bytes (fixed aggregation order)
    y1 = blk.y.bytes().clone()
    blk.forward()
    torch.cuda.synchronize()
    assert torch.equal(y1, blk.y.bytes())


def _run_w1(w):
    blk = LlamaBlockShare(w["t"], w["hidden"], w["heads"], w["d_head"], w["ffn"], block=w["block"], eps=w["eps"],
                          heads_kv=w["heads_kv"], seq_ends=w["seq_ends"])
    blk.load(_device(w))
    blk.forward()
    torch.cuda.synchronize()
    return blk


def _oracle_w1(w):
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    return oracle.llama_block(f["x"], f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"], f["n2"],
                              heads=w["heads"], d_head=w["d_head"], eps=w["eps"], heads_kv=w["heads_kv"],
                              seq_ends=w["seq_ends"])


def test_w1_block_small_grouped_heads_packed_sequences():
    # 4 query heads over 2 key/value heads, three packed sequences of 128, 256
    # and 128 tokens, ragged FFN blocks: every boundary relation
    w = synth.w1_block(t=512, hidden=512, heads=4, heads_kv=2, ffn=344, block=128, seq_len=128)
    w["seq_ends"] = [128, 384, 512]
    blk = _run_w1(w)
    _stagewise(blk, w)
    ref = _oracle_w1(w)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(values(getattr(blk, name)), ref[name], rel_fro=CHAIN_REL_FRO, what=name)


def test_w1_block_share_full_size():
    # the benchmarked share of the paper's block: d 4096, 4 of 32 query heads
    # over 1 of 8 key/value heads, FFN 1792 of 14336, eight packed 1K sequences
    w = synth.w1_block()
    blk = _run_w1(w)
    _stagewise(blk, w)
    ref = _oracle_w1(w)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(values(getattr(blk, name)), ref[name], rel_fro=CHAIN_REL_FRO, what=name)


# ---- the other W1 token workloads: single 1K, 8K and 128K sequences, and
# 128 packed 1K sequences (4 of 32 query heads over 1 of 8 key/value heads,
# FFN 1792 of 14336, d 4096)

_W1_INPUTS = {}


def _w1(t, seq_ends):
    if t not in _W1_INPUTS:
        _W1_INPUTS.clear()
        _W1_INPUTS[t] = synth.w1_block(t=t)
    w = dict(_W1_INPUTS[t])
    w["seq_ends"] = list(seq_ends)
    return w


def _rows_f64(rel, rows):
    return synth.to_f64(download(rel)[rows], rel.dtype)


def _check_w1_rows(w, rows):
    blk = _run_w1(w)
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    ref = oracle.llama_block_rows(f["x"], f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"], f["n2"],
                                  heads=w["heads"], d_head=w["d_head"], eps=w["eps"], rows=rows,
                                  heads_kv=w["heads_kv"], seq_ends=w["seq_ends"])
    rows = np.unique(np.asarray(rows))
    _stagewise(blk, w, rows=rows)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(_rows_f64(getattr(blk, name), rows), ref[name], rel_fro=CHAIN_REL_FRO, what=name)
    return blk


def test_w1_block_single_1k_sequence():
    w = _w1(1024, [1024])
    blk = _run_w1(w)
    _stagewise(blk, w)
    ref = _oracle_w1(w)
    for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
        assert_close(values(getattr(blk, name)), ref[name], rel_fro=CHAIN_REL_FRO, what=name)


def _sample_rows(t, seed, extra):
    rng = np.random.default_rng(seed)
    return sorted(set(extra) | set(rng.integers(0, t, 24).tolist()))


def test_w1_block_single_8k_sequence_sampled_rows():
    print("w1 8K single sequence", flush=True)
    _check_w1_rows(_w1(8192, [8192]), _sample_rows(8192, 81, [0, 1, 127, 128, 511, 512, 4095, 8190, 8191]))


def test_w1_block_single_128k_sequence_sampled_rows():
    # 131072 tokens: activations of 1 GiB per [T, 4096] relation; rows late in
    # the sequence attend over up to 128K keys (1024 key blocks per query tile)
    print("w1 128K single sequence", flush=True)
    t = 131072
    _check_w1_rows(_w1(t, [t]), _sample_rows(t, 128, [0, 511, 512, 65535, 65536, t - 129, t - 128, t - 1]))


def test_w1_block_128_packed_1k_sequences_sampled_sequences():
    # 128 packed 1K sequences: rows of a sequence equal the block run on that
    # sequence alone, so three whole sequences are checked against the oracle
    print("w1 128 x 1K packed sequences", flush=True)
    t = 131072
    w = _w1(t, range(1024, t + 1, 1024))
    blk = _run_w1(w)
    _stagewise(blk, w, rows=np.concatenate([np.arange(j * 1024, (j + 1) * 1024, 7) for j in (0, 77, 127)]))
    f = {k: synth.to_f64(w[k], "bf16") for k in ("n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    for j in (0, 77, 127):
        rows = np.arange(j * 1024, (j + 1) * 1024)
        x = synth.to_f64(w["x"][rows], "bf16")
        ref = oracle.llama_block(x, f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"], f["n2"],
                                 heads=w["heads"], d_head=w["d_head"], eps=w["eps"], heads_kv=w["heads_kv"],
                                 seq_ends=[1024])
        for name in ("h1", "qkv", "attn", "x2", "h2", "a", "y"):
            assert_close(_rows_f64(getattr(blk, name), rows), ref[name], rel_fro=CHAIN_REL_FRO,
                         what=f"sequence {j} {name}")
