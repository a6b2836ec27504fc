"""Logical optimization (Section 4) on the CPU: the oracle's cost function
against the paper's closed form for the 3D matrix multiply (Section 4.4),
and the native planner (ea_logical_plan) against the oracle's exhaustive
search over every combination of join-agg specs."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2609_03905_amd import ea
from paper_2609_03905_amd import logical as lg


@pytest.mark.parametrize("p", [8, 27, 64])
def test_oracle_3d_matmul_closed_form(p):
    # every spec of an N x N x N matmul decomposes i, j, k into a, b, c
    # intervals with abc = p; its cost is (a + b + c - 1) N^2, least exactly
    # at a = b = c = p^(1/3)
    N = 24
    ext = dict(i=N, j=N, k=N)
    specs = oracle.logical_specs("ij,jk->ik", ext, p)
    assert len(specs) == sum(1 for a in range(1, p + 1) for b in range(1, p + 1)
                             if p % (a * b) == 0 and p // (a * b) <= N and a <= N and b <= N)
    q = round(p ** (1 / 3))
    costs = {}
    for c in specs:
        cost = oracle.logical_spec_cost("ij,jk->ik", ext, c, [None, None])
        assert cost == (c["i"] + c["j"] + c["k"] - 1) * N * N
        costs[(c["i"], c["j"], c["k"])] = cost
    best = min(costs.values())
    assert [k for k, v in costs.items() if v == best] == [(q, q, q)]
    assert best == (3 * q - 1) * N * N


@pytest.mark.parametrize("p", [8, 27, 64])
def test_planner_3d_matmul(p):
    N = 24
    counts, cost = lg.plan([lg.LogicalOp("ij,jk->ik", dict(i=N, j=N, k=N), [None, None])], p)
    q = round(p ** (1 / 3))
    assert counts == [dict(i=q, j=q, k=q)] and cost == (3 * q - 1) * N * N


def _random_graph(rng, n_ops, shared=False):
    """Operators over letters of random small extents: matmuls, elementwise
    adds and row sums, each consuming earlier outputs (once, or more than once
    when shared) or computation inputs."""
    ops = []
    shapes = []  # output shape of each op
    users = [0] * n_ops
    for i in range(n_ops):
        kind = rng.integers(0, 3)
        cands = [j for j in range(i) if shared or users[j] == 0]
        src = int(rng.choice(cands)) if cands and rng.random() < 0.8 else None
        e = lambda: int(rng.integers(2, 9))
        if src is None:
            m, n = e(), e()
        else:
            m, n = shapes[src]
        if kind == 0:  # matmul
            k = e()
            ops.append(("ij,jk->ik", dict(i=m, j=n, k=k), [src, None], None))
            shapes.append((m, k))
        elif kind == 1:  # elementwise add
            ops.append(("ij,ij->ij", dict(i=m, j=n), [src, None], None))
            shapes.append((m, n))
        else:  # row sum, then a matmul keeps the graph two-dimensional
            k = e()
            ops.append(("ij,jk->ik", dict(i=m, j=n, k=k), [src, None], "ik"))
            shapes.append((m, k))
        if src is not None:
            users[src] += 1
    return ops


def _lops(ops):
    return [lg.LogicalOp(s, ext, ins, sh) for s, ext, ins, sh in ops]


@pytest.mark.parametrize("seed", range(12))
def test_planner_is_optimal_on_trees(seed):
    rng = np.random.default_rng(seed)
    ops = _random_graph(rng, int(rng.integers(1, 5)))
    p = int(rng.choice([2, 4, 6, 8]))
    try:
        counts, cost = lg.plan(_lops(ops), p)
    except ea.EAError as err:  # some operator cannot split into p pieces
        assert err.code == -7
        assert any(not oracle.logical_specs(s, ext, p, sh) for s, ext, _, sh in ops)
        return
    assert oracle.logical_plan_cost(ops, counts) == cost
    assert cost == oracle.logical_min_cost(ops, p)
    for (s, ext, _, sh), c in zip(ops, counts):
        assert int(np.prod(list(c.values()))) == p
        assert all(c[l] <= ext[l] for l in c) and (sh is None or all(c[l] == 1 for l in c if l not in sh))


@pytest.mark.parametrize("seed", range(6))
def test_planner_on_shared_tensors(seed):
    # outputs consumed twice cut the graph into trees (Section 4.5): the plan
    # is valid, its reported cost is its cost, and it is no better than the
    # exhaustive optimum
    rng = np.random.default_rng(100 + seed)
    ops = _random_graph(rng, 4, shared=True)
    try:
        counts, cost = lg.plan(_lops(ops), 4)
    except ea.EAError as err:
        assert err.code == -7
        return
    assert oracle.logical_plan_cost(ops, counts) == cost
    assert cost >= oracle.logical_min_cost(ops, 4)


def test_planner_chain_takes_the_repartition_into_account():
    # a thin second product: splitting k for the first operator forces a
    # repartition before the second; the plan weighs it against the join
    ops = [("ij,jk->ik", dict(i=8, j=8, k=8), [None, None], None),
           ("ik,kl->il", dict(i=8, k=8, l=2), [0, None], None)]
    counts, cost = lg.plan(_lops(ops), 4)
    assert cost == oracle.logical_min_cost(ops, 4) == oracle.logical_plan_cost(ops, counts)


def test_planner_errors():
    ok = lg.LogicalOp("ij,jk->ik", dict(i=4, j=4, k=4), [None, None])
    with pytest.raises(ea.EAError) as e:
        lg.plan([ok], 0)
    assert e.value.code == -1
    with pytest.raises(ea.EAError) as e:  # producer index not below the consumer's
        lg.plan([lg.LogicalOp("ij,jk->ik", dict(i=4, j=4, k=4), [0, None])], 2)
    assert e.value.code == -1
    with pytest.raises(ea.EAError) as e:  # producer output 4 x 4 into a 4 x 5 input
        lg.plan([ok, lg.LogicalOp("ij,jk->ik", dict(i=4, j=5, k=3), [0, None])], 2)
    assert e.value.code == -5
    with pytest.raises(ea.EAError) as e:  # 7 pieces of extents 4
        lg.plan([ok], 7)
    assert e.value.code == -7
    with pytest.raises(ea.EAError) as e:  # shardable letter not in the spec
        lg.plan([lg.LogicalOp("ij,jk->ik", dict(i=4, j=4, k=4), [None, None], "iz")], 2)
    assert e.value.code == -5


def test_near_equal_partitions():
    assert lg.near_equal_splits(10, 3) == [0, 3, 6, 10]
    op = lg.LogicalOp("ij,jk->ik", dict(i=10, j=4, k=6), [None, None])
    assert lg.partitions(op, dict(i=2, j=1, k=3)) == [[[0, 5, 10], [0, 4]], [[0, 4], [0, 2, 4, 6]],
                                                      [[0, 5, 10], [0, 2, 4, 6]]]
