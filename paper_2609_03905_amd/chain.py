"""Matrix chains as chained block-GEMM join-aggs: the paper's second workload
family (Section 6), five chains A-E with fixed parenthesizations (their dims
and trees are workload definitions, kept with the input recipe).

A chain M_1 ... M_n and its parenthesization (a binary tree over the
matrices) run one 'ij,jk->ik' join-agg per inner node, children first.  Every
product is stored as a bf16 relation (the tree's relation boundaries), in
square blocks.  Matrix i is [dims[i], dims[i + 1]].  This module only
sequences calls: every product runs in libea's block-GEMM kernels.
"""
from __future__ import annotations

import torch

from . import ea

def _splits(n: int, b: int):
    return list(range(0, n, b)) + [n]


def span(tree):
    """(first, last) matrix index of a subtree."""
    if isinstance(tree, int):
        return tree, tree
    return span(tree[0])[0], span(tree[1])[1]


def products(tree):
    """The inner nodes in evaluation order (children first), each as
    (node, left, right)."""
    if isinstance(tree, int):
        return []
    return products(tree[0]) + products(tree[1]) + [(tree, tree[0], tree[1])]


def flops(dims, tree) -> float:
    total = 0.0
    for _, l, r in products(tree):
        a, b = span(l), span(r)
        total += 2.0 * dims[a[0]] * dims[a[1] + 1] * dims[b[1] + 1]
    return total


class MatrixChain:
    """Relations of a chain's matrices (filled by the caller) and of every
    product; run() evaluates the tree."""

    def __init__(self, dims, tree, block: int = 512, device="cuda"):
        self.dims, self.tree, self.block = list(dims), tree, block
        part = lambda i, j: [_splits(self.dims[i], block), _splits(self.dims[j], block)]
        n = len(self.dims) - 1
        self.mats = [ea.Relation((self.dims[i], self.dims[i + 1]), "bf16", part(i, i + 1), device=device)
                     for i in range(n)]
        self.rel = {i: self.mats[i] for i in range(n)}
        for node, _, _ in products(tree):
            a, b = span(node)
            self.rel[node] = ea.Relation((self.dims[a], self.dims[b + 1]), "bf16", part(a, b + 1), device=device)
        self.out = self.rel[tree]

    def load(self, i: int, dense) -> None:
        """Fill matrix i from a contiguous [d_i, d_(i+1)] bf16 device tensor
        (re-blocked by libea's repartition)."""
        raw = dense.contiguous().view(torch.uint8).reshape(-1)
        src = ea.Relation(tuple(dense.shape), "bf16", ea.whole_partition(dense.shape), data=raw)
        ea.repartition(src, self.mats[i])

    def run(self, stream=None):
        for node, l, r in products(self.tree):
            ea.joinagg("ij,jk->ik", ea.JOIN_MUL, ea.AGG_SUM, [self.rel[l], self.rel[r]], self.rel[node],
                       stream=stream)
        return self.out
