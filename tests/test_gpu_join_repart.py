"""GPU parity: the join enumerator and the repartition, bit-exact against the
oracle (Section 3.2 join; Section 5.3 overlay, decompose and recompose)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import download, empty, upload
from paper_2609_03905_amd import ea

pytestmark = pytest.mark.gpu


def _run_join(spec, join_op, shapes, dtypes, parts, group=None, causal=None, **kw):
    ins = [upload(synth.normal(s, 1, dtype=d), d, p) for s, d, p in zip(shapes[:-1], dtypes[:-1], parts[:-1])]
    out = ea.Relation(shapes[-1], dtypes[-1], parts[-1])
    tuples, goff = ea.join_tuples(spec, join_op, ins, out, causal=causal is not None, **kw)
    ref_t, ref_g = oracle.join(spec, parts, group=group, causal=causal)
    np.testing.assert_array_equal(tuples.cpu().numpy(), ref_t)
    np.testing.assert_array_equal(goff.cpu().numpy(), ref_g)
    return ref_t, ref_g


def test_join_matmul_fp32_4x4_blocks():
    p = [synth.splits(256, 64)] * 2
    t, g = _run_join("ij,jk->ik", ea.JOIN_MUL, [(256, 256)] * 3, ["f32"] * 3, [p, p, p])
    assert len(t) == 64 and len(g) == 17


def test_join_qkv_projection_blocks():
    w = synth.qkv_projection()
    t, g = _run_join("tj,jk->tk", ea.JOIN_MUL, [(4096, 4096), (4096, 1536), (4096, 1536)], ["bf16"] * 3,
                     [w["pX"], w["pW"], w["pY"]])
    assert len(t) == 192 and len(g) == 25


@pytest.mark.parametrize("seed", range(6))
def test_join_random_partitions(seed):
    rng = np.random.default_rng(seed)
    I, J, K, L = (int(v) for v in rng.integers(8, 60, 4))
    pi, pj, pk, pl = (synth.random_splits(n, int(rng.integers(1, 5)), rng) for n in (I, J, K, L))
    _run_join("ij,jk,kl->il", ea.JOIN_MUL, [(I, J), (J, K), (K, L), (I, L)], ["f32"] * 4,
              [[pi, pj], [pj, pk], [pk, pl], [pi, pl]])
    _run_join("ij->j", ea.JOIN_MUL, [(I, J), (J,)], ["f32"] * 2, [[pi, pj], [pj]])


def test_join_causal_attention_blocks():
    w = synth.attention()
    shp = (2, 4, 2048, 128)
    t, g = _run_join("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, [shp] * 4, ["bf16"] * 4, [w["pq"]] * 4,
                     causal=("q", "k"), scale=w["scale"])
    assert len(t) == 1088 and len(g) == 129


def test_join_rmsnorm_and_softmax_groups():
    px = [synth.splits(64, 32), synth.splits(256, 64)]
    _run_join("tc,c->tc", ea.OP_RMSNORM, [(64, 256), (256,), (64, 256)], ["bf16"] * 3, [px, [px[1]], px],
              group="t")
    # causal softmax keeps every key block: masked entries are stored zeros
    ps = [synth.splits(2, 1), synth.splits(256, 128), synth.splits(256, 64)]
    ins = [upload(synth.normal((2, 256, 256), 1, dtype="bf16"), "bf16", ps)]
    out = ea.Relation((2, 256, 256), "bf16", ps)
    tuples, goff = ea.join_tuples("hqk->hqk", ea.OP_SOFTMAX, ins, out, causal=True)
    ref_t, ref_g = oracle.join("hqk->hqk", [ps, ps], group="hq")
    np.testing.assert_array_equal(tuples.cpu().numpy(), ref_t)
    np.testing.assert_array_equal(goff.cpu().numpy(), ref_g)


# ---------------------------------------------------------------------------
# repartition
# ---------------------------------------------------------------------------
def _block_bytes(raw, partition, es):
    """Concatenated bytes of every block (padding between blocks excluded)."""
    offs, _ = oracle.layout(partition, es)
    sizes = [int(np.prod([s[c + 1] - s[c] for s, c in zip(partition, coords)])) * es
             for coords in np.ndindex(*[len(s) - 1 for s in partition])]
    return b"".join(raw[o:o + n].tobytes() for o, n in zip(offs, sizes))


def _check_repart(x, dtype, p1, p2):
    src = upload(x, dtype, p1)
    dst = empty(x.shape, dtype, p2)  # filled with 0xFF: unwritten bytes would show
    ea.repartition(src, dst)
    torch.cuda.synchronize()
    want = oracle.repartition(oracle.pack(x, p1), p1, p2, x.dtype)
    es = x.dtype.itemsize
    assert _block_bytes(dst.bytes().cpu().numpy(), p2, es) == _block_bytes(want, p2, es)


@pytest.mark.parametrize("seed", range(8))
def test_repartition_random_bitexact(seed):
    rng = np.random.default_rng(1000 + seed)
    rank = int(rng.integers(1, 5))
    shape = tuple(int(rng.integers(1, 40)) for _ in range(rank))
    dtype = ["f32", "bf16"][seed % 2]
    p1 = [synth.random_splits(n, int(rng.integers(1, 5)), rng) for n in shape]
    p2 = [synth.random_splits(n, int(rng.integers(1, 5)), rng) for n in shape]
    x = synth.normal(shape, seed, dtype=dtype)
    _check_repart(x, dtype, p1, p2)
    _check_repart(x, dtype, p2, p1)


def test_repartition_preamble_example():
    x = synth.normal((256, 256), 5, dtype="bf16")
    _check_repart(x, "bf16", [[0, 128, 256], [0, 256]], [[0, 64, 128, 192, 256], [0, 256]])


def test_repartition_qkv_output_to_heads_full_size():
    w = synth.qkv_projection()
    y = synth.normal((4096, 1536), 7, dtype="bf16")
    _check_repart(y, "bf16", w["pY"], w["pHead"])
    _check_repart(y, "bf16", w["pHead"], w["pY"])


def test_repartition_large_relation_bitexact():
    """A 64 MiB relation: the library cuts relations of at least 64 MiB into
    16 KiB tasks (smaller ones into 8 KiB tasks).  Ragged blocks both ways."""
    x = synth.normal((8192, 4096), 11, dtype="bf16")
    p1 = [synth.splits(8192, 1000), synth.splits(4096, 512)]
    p2 = [synth.splits(8192, 128), synth.splits(4096, 1536)]
    _check_repart(x, "bf16", p1, p2)
    _check_repart(x, "bf16", p2, p1)


def test_repartition_round_trip_and_single_block():
    x = synth.normal((300, 200), 9, dtype="f32")
    p1 = [synth.splits(300, 64), synth.splits(200, 48)]
    p2 = [[0, 300], [0, 200]]
    a = upload(x, "f32", p1)
    b = empty(x.shape, "f32", p2)
    c = empty(x.shape, "f32", p1)
    ea.repartition(a, b)
    ea.repartition(b, c)
    np.testing.assert_array_equal(download(b), x)
    assert _block_bytes(c.bytes().cpu().numpy(), p1, 4) == _block_bytes(a.bytes().cpu().numpy(), p1, 4)
