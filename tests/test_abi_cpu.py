"""Host-side tests of the C ABI (no GPU needed).

libea must load without a GPU, export every function include/ea.h declares,
agree with the oracle's independently written block layout, compute the
overlay of the paper's preamble example, and reject every invalid request
with the documented error code before touching HIP.
"""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import oracle
import synth

ea = pytest.importorskip("paper_2609_03905_amd")
from paper_2609_03905_amd import ea as eamod  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

FAKE = 1 << 20  # a 256-byte aligned address that host-side validation never dereferences


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "ea.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(ea_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert len(names) >= 14
    L = ctypes.CDLL(eamod.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_version_and_dtype_sizes():
    assert ea.version() == 1
    L = ea.lib()
    assert [L.ea_dtype_size(d) for d in (ea.F32, ea.BF16, ea.F16)] == [4, 2, 2]
    assert L.ea_dtype_size(7) == -2


@pytest.mark.parametrize("seed", range(8))
def test_layout_matches_oracle_layout(seed):
    rng = np.random.default_rng(seed)
    rank = int(rng.integers(1, 5))
    shape = [int(rng.integers(1, 50)) for _ in range(rank)]
    part = [synth.random_splits(n, int(rng.integers(1, 5)), rng) for n in shape]
    for dtype in ("f32", "bf16"):
        offs, nbytes = oracle.layout(part, eamod.ELEM_SIZE[dtype])
        assert ea.layout_nbytes(shape, dtype, part) == nbytes
        r = ea.Relation(shape, dtype, part, allocate=False)
        assert r.num_blocks() == len(offs)
        for b in range(len(offs)):
            lo, hi, off = r.block(b)
            assert off == offs[b]
            olo, ohi = _bounds(part, b)
            assert (lo, hi) == (olo, ohi)


def _bounds(partition, b):
    nb = [len(s) - 1 for s in partition]
    c = np.unravel_index(b, nb)
    return [s[i] for s, i in zip(partition, c)], [s[i + 1] for s, i in zip(partition, c)]


def test_overlay_of_the_preamble_example():
    g = json.load(open(os.path.join(GOLDEN, "preamble_overlay_example.json")))
    n, m = g["shape"]
    ov = ea.overlay([g["producer_rows"], [0, m]], [g["consumer_rows"], [0, m]])
    assert ov[0] == g["overlay_rows"]
    n_atoms = (len(ov[0]) - 1) * (len(ov[1]) - 1)
    assert n_atoms == g["n_atoms"]
    # every producer block is a disjoint union of atoms
    for lo, hi in zip(g["producer_rows"][:-1], g["producer_rows"][1:]):
        inside = [a for a in zip(ov[0][:-1], ov[0][1:]) if lo <= a[0] and a[1] <= hi]
        assert len(inside) == g["atoms_per_producer_block"]
        assert inside[0][0] == lo and inside[-1][1] == hi


# ---------------------------------------------------------------------------
# error codes
# ---------------------------------------------------------------------------
def _code(fn):
    with pytest.raises(ea.EAError) as e:
        fn()
    return e.value.code


def test_relation_errors():
    assert _code(lambda: ea.Relation([4, 4], "bf16", [[0, 2, 5], [0, 4]], allocate=False)) == -3
    assert _code(lambda: ea.Relation([4, 4], "bf16", [[0, 2, 2, 4], [0, 4]], allocate=False)) == -3
    assert _code(lambda: ea.Relation([4, 4], "bf16", [[1, 4], [0, 4]], allocate=False)) == -3
    assert _code(lambda: ea.Relation([0], "bf16", [[0, 0]], allocate=False)) == -1
    L = ea.lib()
    h = ctypes.c_void_p()
    shape = (ctypes.c_int64 * 9)(*([2] * 9))
    nb = (ctypes.c_int32 * 9)(*([1] * 9))
    sp = (ctypes.c_int64 * 18)(*([0, 2] * 9))
    assert L.ea_relation_create(9, shape, 1, nb, sp, None, 0, ctypes.byref(h)) == -1
    assert L.ea_relation_create(2, shape, 9, nb, sp, None, 0, ctypes.byref(h)) == -2
    # capacity below the layout, and a misaligned base
    assert L.ea_relation_create(2, shape, 1, nb, sp, ctypes.c_void_p(FAKE), 4, ctypes.byref(h)) == -4
    assert L.ea_relation_create(2, shape, 1, nb, sp, ctypes.c_void_p(FAKE + 2), 64, ctypes.byref(h)) == -1
    assert L.ea_relation_create(2, shape, 1, nb, sp, ctypes.c_void_p(FAKE), 64, ctypes.byref(h)) == 0
    assert L.ea_relation_destroy(h) == 0
    assert L.ea_relation_destroy(None) == 0


def _fake(shape, dtype, part):
    """A relation over a fake device address (validation never dereferences it)."""
    r = ea.Relation(shape, dtype, part, allocate=False)
    assert ea.lib().ea_relation_set_data(r.handle, ctypes.c_void_p(FAKE), r.nbytes) == 0
    return r


def _raw_joinagg(spec, join_op, agg_op, ins, out):
    """ea_joinagg through the C ABI with no workspace: validation of a run
    (data present, arguments) precedes the plan lookup."""
    handles = (ctypes.c_void_p * len(ins))(*[r.handle.value for r in ins])
    prm, _ = eamod._params()
    return ea.lib().ea_joinagg(spec.encode(), join_op, agg_op, len(ins), handles, out.handle, ctypes.byref(prm),
                               None, 0, None)


def test_joinagg_validation_errors():
    p64 = synth.splits(256, 64)
    A = _fake([256, 256], "bf16", [p64, p64])
    B = _fake([256, 256], "bf16", [p64, p64])
    C = _fake([256, 256], "f32", [p64, p64])
    Bj = _fake([256, 256], "bf16", [synth.splits(256, 128), p64])
    Cbad = _fake([256, 256], "f32", [synth.splits(256, 128), p64])
    J = lambda *a, **k: (lambda: ea.joinagg(*a, **k))
    assert _code(J("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, Bj], C)) == -6     # j split differently
    assert _code(J("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], Cbad)) == -6   # output not induced
    assert _code(J("ij,jk-ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)) == -5       # no arrow
    assert _code(J("ij,jk->iz", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)) == -5      # output letter in no input
    assert _code(J("ij,jk,kl->il", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)) == -5   # arity
    assert _code(J("iij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)) == -5     # repeated letter
    assert _code(J("ijk,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C)) == -5     # rank mismatch
    assert _code(J("ij,jk->ik", ea.JOIN_MUL, ea.AGG_NONE, [A, B], C)) == -5     # NONE with contraction
    assert _code(J("ij,jk->ik", 42, ea.AGG_SUM, [A, B], C)) == -1               # unknown join op
    assert _code(J("ij,jk->ik", ea.JOIN_MUL, ea.AGG_LSE, [A, B], C)) == -1      # LSE on an einsum
    nodata = ea.Relation([256, 256], "bf16", [p64, p64], allocate=False)
    assert _raw_joinagg("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, nodata], C) == -1
    assert _raw_joinagg("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], nodata) == -1
    res_bad = _fake([256, 256], "f32", [synth.splits(256, 128), p64])
    assert _code(J("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [A, B], C, residual=res_bad)) == -1


def test_fused_op_validation_errors():
    x = _fake([64, 256], "bf16", [[0, 64], synth.splits(256, 64)])
    w = _fake([256], "bf16", [synth.splits(256, 64)])
    w_bad = _fake([256], "bf16", [synth.splits(256, 128)])
    y = _fake([64, 256], "bf16", [[0, 64], synth.splits(256, 64)])
    J = lambda *a, **k: (lambda: ea.joinagg(*a, **k))
    assert _code(J("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [x, w_bad], y, eps=1e-6)) == -6
    assert _code(J("tc,c->tc", ea.OP_RMSNORM, ea.AGG_MAX, [x, w], y, eps=1e-6)) == -1
    assert _code(J("tc,t->tc", ea.OP_RMSNORM, ea.AGG_SUM, [x, w], y, eps=1e-6)) == -5
    assert _code(J("tc->tc", ea.OP_SOFTMAX, ea.AGG_SUM, [x], y)) == -1
    s1 = _fake([256], "bf16", [synth.splits(256, 64)])
    assert _code(J("k->k", ea.OP_SOFTMAX, ea.AGG_LSE, [s1], s1, causal=True)) == -5
    part = [[0, 1], [0, 1], synth.splits(256, 128), [0, 64]]
    q = _fake([1, 1, 256, 64], "bf16", part)
    assert _code(J("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [q, q, q], q, scale=0.1)) == -7
    part = [[0, 1], [0, 1], synth.splits(256, 64), [0, 128]]
    q = _fake([1, 1, 256, 128], "bf16", part)
    assert _code(J("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [q, q, q], q, scale=0.1)) == -7
    part = [[0, 1], [0, 1], synth.splits(256, 128), [0, 128]]
    q = _fake([1, 1, 256, 128], "bf16", part)
    assert _code(J("bhqd,bhkd,bhqd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [q, q, q], q, scale=0.1)) == -5
    for bad in (0.0, -0.5, float("inf")):
        assert _code(J("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [q, q, q], q, scale=bad)) == -1
    qf = _fake([1, 1, 256, 128], "f32", part)
    assert _code(J("bhqd,bhkd,bhkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [qf, q, q], q, scale=0.1)) == -2
    a = _fake([64, 256], "bf16", [[0, 64], synth.splits(256, 64)])
    wt = _fake([256, 100], "bf16", [synth.splits(256, 64), [0, 100]])
    o = _fake([64, 100], "bf16", [[0, 64], [0, 100]])
    assert _code(J("tj,jk,jk->tk", ea.OP_SWIGLU, ea.AGG_MAX, [a, wt, wt], o)) == -1
    assert _code(J("tj,jk,jk->tj", ea.OP_SWIGLU, ea.AGG_SUM, [a, wt, wt], o)) == -5
    # output store policy: only EA_STORE_CACHED (0) and EA_STORE_STREAM (1)
    for bad in (-1, 2, 7):
        assert _code(J("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [x, w], y, eps=1e-6, store=bad)) == -1


def test_repartition_validation_errors():
    a = _fake([64, 64], "bf16", [[0, 64], [0, 64]])
    b = _fake([64, 32], "bf16", [[0, 64], [0, 32]])
    c = _fake([64, 64], "f32", [[0, 64], [0, 64]])
    d = ea.Relation([64, 64], "bf16", [[0, 32, 64], [0, 64]], allocate=False)
    assert ea.lib().ea_relation_set_data(d.handle, ctypes.c_void_p(FAKE + 4096), d.nbytes) == 0
    assert _code(lambda: ea.repartition(a, b)) == -1       # shape differs
    assert _code(lambda: ea.repartition(a, c)) == -1       # dtype differs
    L = ea.lib()
    assert L.ea_repartition_plan(a.handle, b.handle, None) == -1  # planning validates too
    assert L.ea_repartition(a.handle, a.handle, None) == -1       # memory overlaps
    nodata = ea.Relation([64, 64], "bf16", [[0, 64], [0, 64]], allocate=False)
    assert L.ea_repartition(nodata.handle, d.handle, None) == -1
    for bad in (-1, 2):
        assert L.ea_repartition_ex(a.handle, d.handle, bad, None) == -1


def test_grouped_query_and_packed_sequence_validation_errors():
    J = lambda *a, **k: (lambda: ea.joinagg(*a, **k))
    pq = [[0, 1], synth.splits(8, 1), synth.splits(512, 128), [0, 128]]
    pk = [[0, 1], synth.splits(2, 1), synth.splits(512, 128), [0, 128]]
    q = _fake([1, 8, 512, 128], "bf16", pq)
    kv = _fake([1, 2, 512, 128], "bf16", pk)
    GQA = "bhqd,bgkd,bgkd->bhqd"
    # negative group size; the parameters on another operator
    assert _code(J(GQA, ea.OP_ATTENTION, ea.AGG_LSE, [q, kv, kv], q, scale=0.1, gqa_group=-2)) == -1
    x = _fake([64, 256], "bf16", [[0, 64], synth.splits(256, 64)])
    w = _fake([256], "bf16", [synth.splits(256, 64)])
    assert _code(J("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [x, w], x, eps=1e-6, gqa_group=4)) == -1
    assert _code(J("tc,c->tc", ea.OP_RMSNORM, ea.AGG_SUM, [x, w], x, eps=1e-6, seq_ends=[64])) == -1
    # 8 query heads are not 3 x 2; a separate K/V head letter without a group
    assert _code(J(GQA, ea.OP_ATTENTION, ea.AGG_LSE, [q, kv, kv], q, scale=0.1, gqa_group=3)) == -5
    assert _code(J(GQA, ea.OP_ATTENTION, ea.AGG_LSE, [q, kv, kv], q, scale=0.1)) == -5
    # K and V name different head letters
    assert _code(J("bhqd,bgkd,bfkd->bhqd", ea.OP_ATTENTION, ea.AGG_LSE, [q, kv, kv], q, scale=0.1,
                   gqa_group=4)) == -5
    # key/value heads in blocks of two
    kv2 = _fake([1, 2, 512, 128], "bf16", [[0, 1], [0, 2], synth.splits(512, 128), [0, 128]])
    assert _code(J(GQA, ea.OP_ATTENTION, ea.AGG_LSE, [q, kv2, kv2], q, scale=0.1, gqa_group=4)) == -7
    # packed sequences: out of order, past the extent, last not the extent,
    # an end inside a block
    p1 = [[0, 1], [0, 1], synth.splits(512, 128), [0, 128]]
    a = _fake([1, 1, 512, 128], "bf16", p1)
    MHA = "bhqd,bhkd,bhkd->bhqd"
    for ends, code in (([256, 128, 512], -1), ([256, 640], -1), ([128, 256], -1), ([192, 512], -7)):
        assert _code(J(MHA, ea.OP_ATTENTION, ea.AGG_LSE, [a, a, a], a, scale=0.1, causal=True,
                       seq_ends=ends)) == code, ends
