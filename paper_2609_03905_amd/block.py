"""One GPU's share of a pre-norm LLaMA-shaped transformer block, run as a
chain of join-aggs and repartitions through libea.

    h1  = RMSNorm(x; n1)              'tc,c->tc'        SUM of squares over c blocks
    qkv = h1 W_qkv                    'tj,jk->tk'       SUM over j blocks (matrix cores)
          repartition qkv: 512x512 blocks -> per-head [T, 128] blocks
    o   = CausalAttn(q, k, v)         'bhqd,bhkd,bhkd->bhqd'  online-softmax over key blocks
          repartition o (per-head) -> 512x512 blocks
    x2  = x + o W_o                   'tj,jk->tk' + residual epilogue
    h2  = RMSNorm(x2; n2)
    a   = SiLU(h2 W_g) * (h2 W_u)     'tj,jk,jk->tk'    fused SwiGLU epilogue
    y   = x2 + a W_d                  'tj,jk->tk' + residual epilogue

Every arrow stores a bf16 relation.  The columns of qkv are [Q heads | K
heads | V heads], 128 each; with grouped-query attention there are fewer K
and V heads than Q heads (query head h reads key/value head h / group), and
packed sequences restrict attention to each query's own sequence.  After the first repartition the qkv relation has
one row block and 128-wide column blocks, so head h of Q, K or V is one
contiguous [T, 128] block; Q, K and V are then viewed, without a copy, as
[1, heads, T, 128] relations with 128-row blocks (the same bytes).  The
attention output is viewed back as [T, heads*128] with 128-wide column blocks
before the second repartition.  This module only sequences calls: every step
runs in libea's kernels.
"""
from __future__ import annotations

import torch

from . import ea


def _splits(n: int, b: int):
    return list(range(0, n, b)) + [n]


class LlamaBlockShare:
    def __init__(self, t: int, hidden: int, heads: int, d_head: int, ffn: int, block: int = 512,
                 eps: float = 1e-6, device="cuda", heads_kv: int | None = None, seq_ends=None):
        assert d_head == 128, "the attention join-agg takes head dim 128"
        heads_kv = heads if heads_kv is None else heads_kv
        assert heads % heads_kv == 0, "query heads must be a multiple of key/value heads"
        self.t, self.hidden, self.heads, self.d_head, self.ffn = t, hidden, heads, d_head, ffn
        self.heads_kv, self.seq_ends = heads_kv, None if seq_ends is None else [int(e) for e in seq_ends]
        self.eps = eps
        self.scale = 1.0 / d_head ** 0.5
        hd = heads * d_head
        self.hd = hd
        wqkv = (heads + 2 * heads_kv) * d_head  # [Q heads | K heads | V heads]
        pt, ph = _splits(t, block), _splits(hidden, block)
        pf, phd, pqkv = _splits(ffn, block), _splits(hd, block), _splits(wqkv, block)
        R = lambda shape, part: ea.Relation(shape, "bf16", part, device=device)
        # parameters (filled by load())
        self.n1 = R((hidden,), [ph])
        self.n2 = R((hidden,), [ph])
        self.wqkv = R((hidden, wqkv), [ph, pqkv])
        self.wo = R((hd, hidden), [phd, ph])
        self.wg = R((hidden, ffn), [ph, pf])
        self.wu = R((hidden, ffn), [ph, pf])
        self.wd = R((ffn, hidden), [pf, ph])
        # activations
        self.x = R((t, hidden), [pt, ph])
        self.h1 = R((t, hidden), [pt, ph])
        self.qkv = R((t, wqkv), [pt, pqkv])
        self.qkv_heads = R((t, wqkv), [[0, t], _splits(wqkv, d_head)])
        head_part = [[0, 1], _splits(heads, 1), _splits(t, 128), [0, d_head]]
        kv_part = [[0, 1], _splits(heads_kv, 1), _splits(t, 128), [0, d_head]]
        head_bytes = heads * t * d_head * 2
        kv_bytes = heads_kv * t * d_head * 2
        self.q = self.qkv_heads.view(0, (1, heads, t, d_head), "bf16", head_part)
        self.k = self.qkv_heads.view(head_bytes, (1, heads_kv, t, d_head), "bf16", kv_part)
        self.v = self.qkv_heads.view(head_bytes + kv_bytes, (1, heads_kv, t, d_head), "bf16", kv_part)
        self.o = R((1, heads, t, d_head), head_part)
        self.o_cols = self.o.view(0, (t, hd), "bf16", [[0, t], _splits(hd, d_head)])
        self.attn = R((t, hd), [pt, phd])
        self.x2 = R((t, hidden), [pt, ph])
        self.h2 = R((t, hidden), [pt, ph])
        self.a = R((t, ffn), [pt, pf])
        self.y = R((t, hidden), [pt, ph])

    def load(self, dense: dict, stream=None):
        """Copy dense bf16 tensors (uint16/int16 storage on the device) into
        the block-partitioned parameter and input relations (re-blocked by
        the library's repartition)."""
        for name in ("x", "n1", "n2", "wqkv", "wo", "wg", "wu", "wd"):
            rel = getattr(self, name)
            src = ea.Relation(rel.shape, "bf16", ea.whole_partition(rel.shape),
                              data=dense[name].contiguous().view(torch.uint8).reshape(-1))
            ea.repartition(src, rel, stream)

    # each stage is one library call; the list is what a step runs
    def stages(self):
        J, S = ea.joinagg, ea.AGG_SUM
        group = self.heads // self.heads_kv if self.heads_kv < self.heads else 0
        attn_spec = "bhqd,bgkd,bgkd->bhqd" if group else "bhqd,bhkd,bhkd->bhqd"
        return [
            ("rmsnorm1", lambda: J("tc,c->tc", ea.OP_RMSNORM, S, [self.x, self.n1], self.h1, eps=self.eps)),
            ("qkv_gemm", lambda: J("tj,jk->tk", ea.JOIN_MUL, S, [self.h1, self.wqkv], self.qkv)),
            ("repart_heads", lambda: ea.repartition(self.qkv, self.qkv_heads)),
            ("attention", lambda: J(attn_spec, ea.OP_ATTENTION, ea.AGG_LSE, [self.q, self.k, self.v], self.o,
                                    scale=self.scale, causal=True, gqa_group=group, seq_ends=self.seq_ends)),
            ("repart_cols", lambda: ea.repartition(self.o_cols, self.attn)),
            ("o_gemm_residual", lambda: J("tj,jk->tk", ea.JOIN_MUL, S, [self.attn, self.wo], self.x2,
                                          residual=self.x)),
            ("rmsnorm2", lambda: J("tc,c->tc", ea.OP_RMSNORM, S, [self.x2, self.n2], self.h2, eps=self.eps)),
            ("swiglu_gemm", lambda: J("tj,jk,jk->tk", ea.OP_SWIGLU, S, [self.h2, self.wg, self.wu], self.a)),
            ("down_gemm_residual", lambda: J("tj,jk->tk", ea.JOIN_MUL, S, [self.a, self.wd], self.y,
                                             residual=self.x2)),
        ]

    def forward(self):
        for _, fn in self.stages():
            fn()
        return self.y

    # algorithmic work of each stage (FLOPs for contractions, bytes for the
    # memory-bound stages: read + write of the tensors they must touch)
    def work(self):
        T, Hd, hd, F = self.t, self.hidden, self.hd, self.ffn
        wqkv = (self.heads + 2 * self.heads_kv) * self.d_head
        ends = self.seq_ends or [T]
        lens = [e - s for s, e in zip([0] + ends[:-1], ends)]
        causal_pairs = self.heads * sum(n * (n + 1) // 2 for n in lens)
        return {
            "rmsnorm1": dict(bytes=2 * T * Hd * 2 + Hd * 2),
            "qkv_gemm": dict(flops=2 * T * Hd * wqkv),
            "repart_heads": dict(bytes=2 * T * wqkv * 2),
            "attention": dict(flops=4 * self.d_head * causal_pairs),
            "repart_cols": dict(bytes=2 * T * hd * 2),
            "o_gemm_residual": dict(flops=2 * T * hd * Hd),
            "rmsnorm2": dict(bytes=2 * T * Hd * 2 + Hd * 2),
            "swiglu_gemm": dict(flops=2 * 2 * T * Hd * F),
            "down_gemm_residual": dict(flops=2 * T * F * Hd),
        }
