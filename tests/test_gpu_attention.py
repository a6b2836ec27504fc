"""GPU parity of the causal attention join-agg (key-blocked online-softmax
aggregation) against the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_close, empty, expected, upload, values
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu

SPEC = "bhqd,bhkd,bhkd->bhqd"


def _run(q, k, v, pq, pk, scale, causal, out_dtype="bf16"):
    Q, K, V = upload(q, "bf16", pq), upload(k, "bf16", pk), upload(v, "bf16", pk)
    O = empty(q.shape, out_dtype, pq)
    ea.joinagg(SPEC, ea.OP_ATTENTION, ea.AGG_LSE, [Q, K, V], O, scale=scale, causal=causal)
    return O


def test_attention_full_size_causal():
    w = synth.attention()
    O = _run(w["q"], w["k"], w["v"], w["pq"], w["pk"], w["scale"], True)
    ref = oracle.attention(*(synth.to_f64(w[n], "bf16") for n in "qkv"), True, w["scale"])
    assert_close(values(O), expected(ref, "bf16"), what="causal attention C4")


def test_attention_f32_output_and_determinism():
    B, H, S = 1, 2, 1024
    q, k, v = (synth.normal((B, H, S, 128), 410 + i, dtype="bf16") for i in range(3))
    p = [[0, 1], synth.splits(H, 1), synth.splits(S, 128), [0, 128]]
    scale = 1.0 / np.sqrt(128)
    O = _run(q, k, v, p, p, scale, True, "f32")
    ref = oracle.attention(*(synth.to_f64(a, "bf16") for a in (q, k, v)), True, scale)
    assert_close(values(O), ref, rel_fro=1e-3, what="attention f32 out")
    O2 = _run(q, k, v, p, p, scale, True, "f32")
    torch.cuda.synchronize()
    assert torch.equal(O.bytes(), O2.bytes())


def test_attention_split_tiles_two_and_three_parts_deterministic():
    # 24 key blocks of 128: query tiles past the 8th split their keys over two
    # and three work units, merged by the last one to arrive; the merge must
    # give the same bits whichever unit that is
    B, H, S = 1, 1, 3072
    q, k, v = (synth.normal((B, H, S, 128), 430 + i, dtype="bf16") for i in range(3))
    p = [[0, 1], [0, 1], synth.splits(S, 128), [0, 128]]
    scale = 1.0 / np.sqrt(128)
    ref = oracle.attention(*(synth.to_f64(a, "bf16") for a in (q, k, v)), True, scale)
    O = _run(q, k, v, p, p, scale, True, "f32")
    assert_close(values(O), ref, rel_fro=1e-3, what="attention, split tiles")
    for _ in range(3):
        O2 = _run(q, k, v, p, p, scale, True, "f32")
        torch.cuda.synchronize()
        assert torch.equal(O.bytes(), O2.bytes())


@pytest.mark.parametrize("qb,kb", [(256, 128), (128, 256), (512, 512), (128, 1024)])
def test_attention_block_size_invariance(qb, kb):
    B, H, S = 1, 2, 1024
    q, k, v = (synth.normal((B, H, S, 128), 420 + i, dtype="bf16") for i in range(3))
    pq = [[0, 1], synth.splits(H, 1), synth.splits(S, qb), [0, 128]]
    pk = [[0, 1], synth.splits(H, 1), synth.splits(S, kb), [0, 128]]
    scale = 1.0 / np.sqrt(128)
    ref = oracle.attention(*(synth.to_f64(a, "bf16") for a in (q, k, v)), True, scale)
    O = _run(q, k, v, pq, pk, scale, True, "f32")
    assert_close(values(O), ref, rel_fro=1e-3, what=f"q blocks {qb}, k blocks {kb}")


def test_attention_non_causal():
    B, H, S = 2, 1, 512
    q, k, v = (synth.normal((B, H, S, 128), 430 + i, dtype="bf16") for i in range(3))
    p = [synth.splits(B, 1), [0, 1], synth.splits(S, 128), [0, 128]]
    scale = 0.05
    O = _run(q, k, v, p, p, scale, False, "f32")
    ref = oracle.attention(*(synth.to_f64(a, "bf16") for a in (q, k, v)), False, scale)
    assert_close(values(O), ref, rel_fro=1e-3, what="non-causal attention")


def test_attention_closed_forms():
    B, H, S = 1, 1, 512
    p = [[0, 1], [0, 1], synth.splits(S, 128), [0, 128]]
    q = synth.normal((B, H, S, 128), 440, dtype="bf16")
    k = synth.normal((B, H, S, 128), 441, dtype="bf16")
    # identical value rows give that row back
    vrow = synth.normal((128,), 442, dtype="bf16")
    v = np.ascontiguousarray(np.broadcast_to(vrow, (B, H, S, 128)))
    O = _run(q, k, v, p, p, 0.1, True, "f32")
    assert_close(values(O), np.broadcast_to(synth.to_f64(vrow, "bf16"), (B, H, S, 128)), rel_fro=1e-3,
                 what="equal value rows")
    # zero keys: the causal prefix mean of the values; the first query sees only key 0
    v = synth.normal((B, H, S, 128), 443, dtype="bf16")
    kz = synth.store(np.zeros((B, H, S, 128)), "bf16")
    O = _run(q, kz, v, p, p, 0.1, True, "f32")
    fv = synth.to_f64(v, "bf16")
    prefix_mean = np.cumsum(fv, axis=2) / np.arange(1, S + 1)[None, None, :, None]
    got = values(O)
    assert_close(got, prefix_mean, rel_fro=1e-3, what="zero keys")
    np.testing.assert_allclose(got[0, 0, 0], fv[0, 0, 0], rtol=1e-3, atol=1e-3)


def test_attention_single_block_and_first_query():
    # one query and one key block of 128 per head (a single work unit, no merge);
    # causal: query 0 sees only key 0, so its output is value row 0 exactly
    B, H, S = 1, 3, 128
    q, k, v = (synth.normal((B, H, S, 128), 450 + i, dtype="bf16") for i in range(3))
    p = [[0, 1], synth.splits(H, 1), [0, 128], [0, 128]]
    scale = 1.0 / np.sqrt(128)
    for causal in (True, False):
        O = _run(q, k, v, p, p, scale, causal, "f32")
        ref = oracle.attention(*(synth.to_f64(a, "bf16") for a in (q, k, v)), causal, scale)
        got = values(O)
        assert_close(got, ref, rel_fro=1e-3, what=f"single block, causal={causal}")
        if causal:
            assert np.array_equal(got[:, :, 0, :], synth.to_f64(v, "bf16")[:, :, 0, :])


def test_attention_long_sequence_units_at_the_key_block_cap():
    # one causal head of 131072 tokens in 128-blocks: query tile i has i + 1
    # key blocks (up to 1024).  The plan's cost model then takes units of 64
    # key blocks, the cap of a unit's key-block table: 8704 units in 34 waves
    # of 256 CUs, at cost 34 x (64 + 0.5 x 15) against 66 x (32 + 0.5 x 31)
    # for 32, and tiles past the 64th split over 2 to 16 parts.  The units are
    # sized from the GPU join's group offsets.  Sampled query rows (tile and
    # unit boundaries among them) against the oracle evaluated at those rows.
    print("attention: one head of 131072 tokens", flush=True)
    S = 131072
    q, k, v = (synth.normal((1, 1, S, 128), 470 + i, dtype="bf16") for i in range(3))
    p = [[0, 1], [0, 1], synth.splits(S, 128), [0, 128]]
    scale = 1.0 / np.sqrt(128)
    O = _run(q, k, v, p, p, scale, True)
    rng = np.random.default_rng(471)
    rows = np.unique(np.concatenate([[0, 1, 127, 128, 8191, 8192, 8319, 65535, 65536, S - 129, S - 128, S - 1],
                                     rng.integers(0, S, 20)]))
    f = [synth.to_f64(a[0], "bf16") for a in (q, k, v)]
    ref = oracle.attention_rows(f[0], f[1], f[2], rows, scale)[:, 0]
    assert_close(values(O)[0, 0][rows], expected(ref, "bf16"), what="attention 128K, sampled rows")
