"""Drop-in attention layers on the HIP kernels: a multi-head self-attention
module and a pre-norm Transformer block whose attention is the
memory-efficient one (the paper's Section 5 uses it as the attention of a
Transformer trained end to end; only the O(n) lse is kept for the backward).

The projections, normalisations and the MLP are ordinary torch layers; the
attention itself, forward and backward, runs in ``libmea.so``.  Head
dimensions 64 and 128 are supported, in float32, float16 or bfloat16.
"""
from __future__ import annotations

import torch
from torch import nn

from .attention import attention_packed


class MultiheadAttention(nn.Module):
    """Self-attention over ``x`` of shape ``[B, n, embed_dim]``.

    One fused input projection gives Q, K and V as a packed
    ``[B, n, 3, H, d]`` tensor that the kernels read in place (strided views,
    ``num_heads`` heads of ``embed_dim // num_heads`` features); the output
    ``[B, n, H, d]`` is the heads' concatenation, projected back.  ``causal``
    masks key j for query i when j > i; ``kv_len`` (int32 ``[B]`` on the GPU,
    optional) masks the padded positions j >= kv_len[b] of each sequence.
    """

    def __init__(self, embed_dim: int, num_heads: int, causal: bool = False, bias: bool = True,
                 device=None, dtype=None):
        super().__init__()
        if embed_dim % num_heads != 0:
            raise ValueError("embed_dim must be a multiple of num_heads")
        self.head_dim = embed_dim // num_heads
        if self.head_dim not in (64, 128):
            raise ValueError("head dimension must be 64 or 128, got %d" % self.head_dim)
        self.embed_dim, self.num_heads, self.causal = embed_dim, num_heads, causal
        kw = {"device": device, "dtype": dtype}
        self.qkv = nn.Linear(embed_dim, 3 * embed_dim, bias=bias, **kw)
        self.out = nn.Linear(embed_dim, embed_dim, bias=bias, **kw)

    def forward(self, x: torch.Tensor, kv_len: torch.Tensor | None = None) -> torch.Tensor:
        B, n, E = x.shape
        if E != self.embed_dim:
            raise ValueError("expected embed_dim %d, got %d" % (self.embed_dim, E))
        qkv = self.qkv(x).view(B, n, 3, self.num_heads, self.head_dim)
        # [B, n, H, d], no copies either way
        o = attention_packed(qkv, causal=self.causal, kv_len=kv_len)
        return self.out(o.reshape(B, n, E))


class TransformerBlock(nn.Module):
    """Pre-norm block: ``x + attn(norm(x))`` then ``x + mlp(norm(x))``, the MLP
    ``mlp_ratio`` times wider than the model with a GELU."""

    def __init__(self, embed_dim: int, num_heads: int, causal: bool = True, mlp_ratio: int = 4,
                 device=None, dtype=None):
        super().__init__()
        kw = {"device": device, "dtype": dtype}
        self.norm1 = nn.LayerNorm(embed_dim, **kw)
        self.attn = MultiheadAttention(embed_dim, num_heads, causal=causal, **kw)
        self.norm2 = nn.LayerNorm(embed_dim, **kw)
        self.mlp = nn.Sequential(nn.Linear(embed_dim, mlp_ratio * embed_dim, **kw), nn.GELU(),
                                 nn.Linear(mlp_ratio * embed_dim, embed_dim, **kw))

    def forward(self, x: torch.Tensor, kv_len: torch.Tensor | None = None) -> torch.Tensor:
        x = x + self.attn(self.norm1(x), kv_len)
        return x + self.mlp(self.norm2(x))


class TransformerLM(nn.Module):
    """Token embedding, learned positions, ``depth`` causal blocks, final norm
    and a tied output projection: the smallest model that exercises the
    attention's forward and backward inside a training step."""

    def __init__(self, vocab: int, embed_dim: int, num_heads: int, depth: int, max_len: int,
                 device=None, dtype=None):
        super().__init__()
        kw = {"device": device, "dtype": dtype}
        self.tok = nn.Embedding(vocab, embed_dim, **kw)
        self.pos = nn.Parameter(torch.zeros(max_len, embed_dim, **kw))
        self.blocks = nn.ModuleList(TransformerBlock(embed_dim, num_heads, causal=True, **kw)
                                    for _ in range(depth))
        self.norm = nn.LayerNorm(embed_dim, **kw)
        nn.init.normal_(self.tok.weight, std=0.02)

    def forward(self, tokens: torch.Tensor) -> torch.Tensor:
        n = tokens.shape[1]
        x = self.tok(tokens) + self.pos[:n]
        for blk in self.blocks:
            x = blk(x)
        return self.norm(x) @ self.tok.weight.t()
