"""Where the end-to-end chain tolerance comes from (CPU only).

The block chain stores a bf16 relation at every arrow, and the oracle rounds
at the same arrows.  A correct implementation that accumulates in fp32 still
differs from the fp64 oracle: now and then an upstream value lands on the
other side of a bf16 rounding boundary, and the softmax and the SwiGLU
product amplify such one-ulp flips downstream.  This test measures that
effect with an implementation independent of both the oracle and the GPU
path -- torch library routines in fp32 on the CPU, rounded to bf16 at the
same boundaries -- on the full-size inputs of the LLaMA-65B-shape block
share, and pins the GPU tests' end-to-end tolerance (helpers.CHAIN_REL_FRO)
to between 1.25x and 2.5x the error it shows.  Each stage alone stays within
the single-operator tolerance, which the GPU tests hold every arrow to.

The matrix chains (Section 6, every dim divided by 64) are measured the same
way: products in fp32, rounded to bf16 at every boundary.  Where two values
differ by d their bf16 roundings differ by about sqrt(ulp * d), so deep chains
compound flips too; the test pins which chains stay under REL_FRO / 3 (held to
REL_FRO end to end on the GPU) and that CHAIN_REL_FRO covers the others."""
import numpy as np
import torch
import torch.nn.functional as F

import oracle
import synth
from helpers import CHAIN_END_TO_END, CHAIN_REL_FRO, REL_FRO


def _rel_fro(got, ref):
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))


def _torch_fp32_chain(w, heads, d_head, eps):
    b = lambda t: t.to(torch.bfloat16).to(torch.float32)  # the bf16 store at an arrow (RNE)
    t32 = {k: torch.from_numpy(synth.to_f64(w[k], "bf16").astype(np.float32)) for k in
           ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    x = t32["x"]
    T, C = x.shape
    hd = heads * d_head
    h1 = b(F.rms_norm(x, (C,), weight=t32["n1"], eps=eps))
    qkv = b(h1 @ t32["wqkv"])
    q, k, v = (qkv[:, i * hd:(i + 1) * hd].reshape(T, heads, d_head).transpose(0, 1).contiguous() for i in range(3))
    o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True, scale=1.0 / d_head ** 0.5)[0]
    attn = b(o.transpose(0, 1).reshape(T, hd))
    x2 = b(x + attn @ t32["wo"])
    h2 = b(F.rms_norm(x2, (C,), weight=t32["n2"], eps=eps))
    a = b(F.silu(h2 @ t32["wg"]) * (h2 @ t32["wu"]))
    y = b(x2 + a @ t32["wd"])
    out = dict(h1=h1, qkv=qkv, attn=attn, x2=x2, h2=h2, a=a, y=y)
    return {k: v.double().numpy() for k, v in out.items()}


def test_end_to_end_chain_tolerance_from_an_independent_fp32_chain():
    w = synth.llama_block()  # 2048 tokens, hidden 8192, 8 heads of 128, FFN 2752
    f = {k: synth.to_f64(w[k], "bf16") for k in ("x", "n1", "wqkv", "wo", "wg", "wu", "wd", "n2")}
    ref = oracle.llama_block(f["x"], f["n1"], f["wqkv"], f["wo"], f["wg"], f["wu"], f["wd"], f["n2"], heads=8,
                             d_head=128, eps=1e-6)
    got = _torch_fp32_chain(w, 8, 128, 1e-6)
    errs = {k: _rel_fro(got[k], ref[k]) for k in ref}
    print("fp32 torch chain vs fp64 oracle chain:", {k: f"{e:.3e}" for k, e in errs.items()})
    # the first arrows are single operators on exact inputs: within REL_FRO
    assert errs["h1"] < REL_FRO and errs["qkv"] < REL_FRO
    # downstream the flips accumulate: the chain's end misses REL_FRO even for
    # this correct implementation, so end to end REL_FRO cannot be the bar
    worst = max(errs.values())
    assert errs["y"] > REL_FRO or worst > REL_FRO
    # the tolerance the GPU chain is held to, derived from this figure
    assert 1.25 * worst <= CHAIN_REL_FRO <= 2.5 * worst, (worst, CHAIN_REL_FRO)


def _oracle_tree(tree, mats):
    if isinstance(tree, int):
        return synth.to_f64(mats[tree], "bf16")
    return oracle.rne_bf16(oracle.matmul(_oracle_tree(tree[0], mats), _oracle_tree(tree[1], mats)))


def _torch_tree(tree, mats):
    if isinstance(tree, int):
        return torch.from_numpy(synth.to_f64(mats[tree], "bf16").astype(np.float32))
    return (_torch_tree(tree[0], mats) @ _torch_tree(tree[1], mats)).to(torch.bfloat16).float()


def test_matrix_chain_end_to_end_tolerances():
    worst = 0.0
    for name in sorted(synth.CHAINS):
        dims, tree = synth.CHAINS[name]
        mats, _ = synth.chain_matrices(dims, 600 + 20 * "ABCDE".index(name), div=64)  # the GPU test's inputs
        err = _rel_fro(_torch_tree(tree, mats).double().numpy(), _oracle_tree(tree, mats))
        print(f"chain {name} / 64: fp32 torch chain vs fp64 oracle chain {err:.3e}")
        if CHAIN_END_TO_END[name] == REL_FRO:
            assert err <= REL_FRO / 3, name
        else:
            assert CHAIN_END_TO_END[name] == CHAIN_REL_FRO and err > REL_FRO / 3, name
            worst = max(worst, err)
    assert 1.25 * worst <= CHAIN_REL_FRO <= 2.5 * worst, (worst, CHAIN_REL_FRO)
