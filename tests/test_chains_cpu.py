"""The matrix-chain workloads (Section 6, chains A-E) against what the paper
states about them: each multiply averages about 8192^3 scalar multiplies, and
the fixed parenthesizations are the optimal ones of the classical
matrix-chain dynamic program (for A and B bushy, for C right-associated).
Checks the dims read from the text, which are not printed as a table."""
import pytest

import synth
from paper_2609_03905_amd import chain


def _dp_min_multiplies(d):
    n = len(d) - 1
    m = [[0] * n for _ in range(n)]
    for L in range(2, n + 1):
        for i in range(n - L + 1):
            j = i + L - 1
            m[i][j] = min(m[i][k] + m[k + 1][j] + d[i] * d[k + 1] * d[j + 1] for k in range(i, j))
    return m[0][n - 1]


@pytest.mark.parametrize("name", sorted(synth.CHAINS))
def test_chain_matches_the_papers_description(name):
    dims, tree = synth.CHAINS[name]
    n = len(dims) - 1
    assert chain.span(tree) == (0, n - 1)
    prods = chain.products(tree)
    assert len(prods) == n - 1
    mults = chain.flops(dims, tree) / 2
    assert 0.95 <= mults / len(prods) / 8192 ** 3 <= 1.05
    assert mults == _dp_min_multiplies(dims)


def test_chain_shapes_of_the_text():
    assert len(synth.CHAINS["A"][0]) - 1 == 9 and len(synth.CHAINS["B"][0]) - 1 == 5
    assert synth.CHAINS["C"] == ([10240, 12288, 32768, 2048], (0, (1, 2)))
    assert len(synth.CHAINS["D"][0]) - 1 == 9 and len(synth.CHAINS["E"][0]) - 1 == 13
    # chain C's optimal order is right-associated; A and B's are bushy (a product
    # of two products at the root)
    assert isinstance(synth.CHAINS["A"][1][0], tuple) and isinstance(synth.CHAINS["A"][1][1], tuple)
    assert isinstance(synth.CHAINS["B"][1][0], tuple) and isinstance(synth.CHAINS["B"][1][1], tuple)
