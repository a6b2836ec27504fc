"""Output store policy: EA_STORE_STREAM writes the same bytes as
EA_STORE_CACHED.  RMSNorm, softmax and repartition stream their outputs
(non-temporal stores); the block GEMM (residual and SwiGLU epilogues, split
keys) and attention accept the policy and store plainly."""
import numpy as np
import pytest
import torch

import synth
from helpers import empty, upload
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu


def _same_bytes(make_out, run):
    a, b = make_out(), make_out()
    run(a, ea.STORE_CACHED)
    run(b, ea.STORE_STREAM)
    torch.cuda.synchronize()
    assert torch.equal(a.bytes(), b.bytes())


def test_stream_store_gemm_residual_and_split_keys():
    # 4 tiles of 256 x 256 over 2048-deep K: the keys are split over several
    # workgroups, whose last arriver stores
    T, J, K = 512, 2048, 512
    p = [synth.splits(T, 256), synth.splits(J, 512)]
    x = synth.normal((T, J), 81, dtype="bf16")
    w = synth.normal((J, K), 82, 0.05, dtype="bf16")
    r = synth.normal((T, K), 83, dtype="bf16")
    X, W = upload(x, "bf16", p), upload(w, "bf16", [synth.splits(J, 512), synth.splits(K, 256)])
    pout = [synth.splits(T, 256), synth.splits(K, 256)]
    R = upload(r, "bf16", pout)
    _same_bytes(lambda: empty((T, K), "bf16", pout),
                lambda y, st: ea.joinagg("tj,jk->tk", ea.JOIN_MUL, ea.AGG_SUM, [X, W], y, residual=R, store=st))


def test_stream_store_swiglu():
    T, H, F = 256, 512, 256
    pt, ph, pf = synth.splits(T, 128), synth.splits(H, 128), synth.splits(F, 128)
    x = synth.normal((T, H), 84, dtype="bf16")
    wg = synth.normal((H, F), 85, 0.05, dtype="bf16")
    wu = synth.normal((H, F), 86, 0.05, dtype="bf16")
    X, G, U = upload(x, "bf16", [pt, ph]), upload(wg, "bf16", [ph, pf]), upload(wu, "bf16", [ph, pf])
    _same_bytes(lambda: empty((T, F), "bf16", [pt, pf]),
                lambda y, st: ea.joinagg("tj,jk,jk->tk", ea.OP_SWIGLU, ea.AGG_SUM, [X, G, U], y, store=st))


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_stream_store_attention(out_dtype):
    B, H, S, D = 1, 2, 512, 128
    pq = [synth.splits(B, 1), synth.splits(H, 1), synth.splits(S, 128), synth.whole(D)]
    q, k, v = (synth.normal((B, H, S, D), 87 + i, dtype="bf16") for i in range(3))
    Q, K, V = upload(q, "bf16", pq), upload(k, "bf16", pq), upload(v, "bf16", pq)
    _same_bytes(lambda: empty((B, H, S, D), out_dtype, pq),
                lambda o, st: ea.joinagg("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], o,
                                         scale=1.0 / np.sqrt(D), causal=True, store=st))


def test_stream_store_rows():
    T, C = 64, 2048
    px = [synth.whole(T), synth.splits(C, 512)]
    x = synth.normal((T, C), 90, dtype="bf16")
    wv = synth.uniform((C,), 91, 0.5, 1.5, dtype="bf16")
    X, Wt = upload(x, "bf16", px), upload(wv, "bf16", [synth.splits(C, 512)])
    _same_bytes(lambda: empty((T, C), "bf16", px),
                lambda y, st: ea.joinagg("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [X, Wt], y, eps=1e-6, store=st))
    ps = [synth.splits(2, 1), synth.whole(256), synth.splits(256, 64)]
    s = synth.normal((2, 256, 256), 92, dtype="bf16")
    S = upload(s, "bf16", ps)
    _same_bytes(lambda: empty((2, 256, 256), "f32", ps),
                lambda p, st: ea.joinagg("hqk->hqk", ea.OP_SOFTMAX, ea.AGG_LSE, [S], p, causal=True, store=st))


def test_stream_store_repartition():
    rng = np.random.default_rng(93)
    shape = (96, 200)
    p1 = [synth.random_splits(n, 3, rng) for n in shape]
    p2 = [synth.random_splits(n, 4, rng) for n in shape]
    x = synth.normal(shape, 94, dtype="bf16")
    X = upload(x, "bf16", p1)
    _same_bytes(lambda: empty(shape, "bf16", p2), lambda d, st: ea.repartition(X, d, store=st))
