"""GPU parity of the matrix chains (Section 6, chains A-E) run as chained
block-GEMM join-aggs.

Every product is checked on its own: the GPU's stored product against the
oracle's product of the GPU's own stored operands (rounded to bf16 as the
chain stores it), at the single-operator tolerance.  Whole chains are then
checked against the oracle's chain with bf16 rounding at every relation
boundary, at the single-operator tolerance, except the two deep chains whose
rounding flips compound past it even for an independent fp32 implementation
(helpers.CHAIN_END_TO_END)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import CHAIN_END_TO_END, assert_close, upload, values
from paper_2609_03905_amd import chain

pytestmark = pytest.mark.gpu


def _oracle_tree(tree, mats):
    """fp64 product of a subtree, rounded to bf16 as each stored product is."""
    if isinstance(tree, int):
        return synth.to_f64(mats[tree], "bf16")
    return oracle.rne_bf16(oracle.matmul(_oracle_tree(tree[0], mats), _oracle_tree(tree[1], mats)))


def _uploaded_chain(dims, tree, mats, block):
    ch = chain.MatrixChain(dims, tree, block=block)
    for i, m in enumerate(mats):
        ch.mats[i] = ch.rel[i] = upload(m, "bf16", ch.mats[i].partition)
    return ch


@pytest.mark.parametrize("name", sorted(synth.CHAINS))
def test_chain_scaled_down_parity(name):
    # every dim divided by 64 (necks of 16 and 24), 32-blocks: the same trees
    dims, tree = synth.CHAINS[name]
    mats, d = synth.chain_matrices(dims, 600 + 20 * "ABCDE".index(name), div=64)
    ch = _uploaded_chain(d, tree, mats, 32)
    out = ch.run()
    for node, left, right in chain.products(tree):
        ref = oracle.rne_bf16(oracle.matmul(values(ch.rel[left]), values(ch.rel[right])))
        assert_close(values(ch.rel[node]), ref, what=f"chain {name} / 64, product {node}")
    assert_close(values(out), _oracle_tree(tree, mats), rel_fro=CHAIN_END_TO_END[name], what=f"chain {name} / 64")


def test_chain_c_full_size_sampled_columns():
    # M1 (M2 M3), 10240 x 12288 x 32768 x 2048 in 512-blocks.  Rounding is
    # elementwise, so column j of the result is RNE(M1 RNE(M2 M3[:, j])):
    # the oracle computes sampled columns from matrix-vector products
    dims, tree = synth.CHAINS["C"]
    mats, d = synth.chain_matrices(dims, 700)
    ch = _uploaded_chain(d, tree, mats, 512)
    out = ch.run()
    cols = [0, 1, 511, 512, 1023, 1500, 2046, 2047]
    f = [synth.to_f64(m, "bf16") for m in mats]
    p = oracle.rne_bf16(oracle.matmul(f[1], np.ascontiguousarray(f[2][:, cols])))
    ref = oracle.rne_bf16(oracle.matmul(f[0], p))
    assert_close(values(out)[:, cols], ref, what="chain C, sampled columns")
    # each product on the GPU's own operands: M2 M3 at sampled columns, then
    # M1 times the GPU's stored M2 M3 at the same columns
    p_gpu = values(ch.rel[(1, 2)])
    assert_close(p_gpu[:, cols], p, what="chain C, product M2 M3")
    ref2 = oracle.rne_bf16(oracle.matmul(f[0], np.ascontiguousarray(p_gpu[:, cols])))
    assert_close(values(out)[:, cols], ref2, what="chain C, product M1 (M2 M3)")
