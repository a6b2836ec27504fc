"""The logical plan (Section 4) consumed by the hot path: the join-agg
specs chosen for a computation give the block partitions of its relations;
an input of an operator whose spec needs another tiling than its producer
delivered is repartitioned first (the cost the plan charged); the result
matches the oracle."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, empty, upload, values
from paper_2609_03905_amd import ea
from paper_2609_03905_amd import logical as lg

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("p", [4, 8, 27])
def test_planned_chain_runs_on_its_partitions(p):
    # chain C scaled down (10240 x 12288 x 32768 x 2048 / 64): M1 (M2 M3)
    dims = [d // 64 for d in synth.CHAINS["C"][0]]
    mats, d = synth.chain_matrices(synth.CHAINS["C"][0], 800, div=64)
    ops = [lg.LogicalOp("jk,kl->jl", dict(j=d[1], k=d[2], l=d[3]), [None, None]),
           lg.LogicalOp("ij,jl->il", dict(i=d[0], j=d[1], l=d[3]), [None, 0])]
    counts, cost = lg.plan(ops, p)
    p23 = lg.partitions(ops[0], counts[0])
    p1 = lg.partitions(ops[1], counts[1])
    M2, M3 = upload(mats[1], "bf16", p23[0]), upload(mats[2], "bf16", p23[1])
    P = empty((d[1], d[3]), "bf16", p23[2])
    ea.joinagg(ops[0].spec, ea.JOIN_MUL, ea.AGG_SUM, [M2, M3], P)
    if p1[1] != p23[2]:  # the second operator's spec needs another tiling of P
        P2 = empty((d[1], d[3]), "bf16", p1[1])
        ea.repartition(P, P2)
        P = P2
    M1 = upload(mats[0], "bf16", p1[0])
    Y = empty((d[0], d[3]), "bf16", p1[2])
    ea.joinagg(ops[1].spec, ea.JOIN_MUL, ea.AGG_SUM, [M1, P], Y)
    f = [synth.to_f64(m, "bf16") for m in mats]
    ref = oracle.rne_bf16(oracle.matmul(f[0], oracle.rne_bf16(oracle.matmul(f[1], f[2]))))
    assert_close(values(P), oracle.rne_bf16(oracle.matmul(f[1], f[2])), what=f"planned chain M2 M3, p={p}")
    assert_close(values(Y), oracle.rne_bf16(oracle.matmul(f[0], values(P))), what=f"planned chain M1 P, p={p}")
    assert_close(values(Y), ref, what=f"planned chain, p={p}")
    # the tuples of each join-agg are the spec's p function specifications
    assert int(np.prod(list(counts[0].values()))) == p
    t, _ = ea.join_tuples(ops[0].spec, ea.JOIN_MUL, [M2, M3], empty((d[1], d[3]), "bf16", p23[2]))
    assert len(t) == p
