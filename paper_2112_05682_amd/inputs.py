"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module draws random numbers and casts them; it holds none of the
attention arithmetic, so both the HIP path and the float64 oracle can be fed
from it without sharing any computation.

Recipe (the paper measures on i.i.d. standard-normal inputs, Section 5.1):
Q, K, V and the upstream gradient dO are drawn i.i.d. N(0, std^2) in float32
from ``torch.Generator`` seeded 0, 1, 2, 3 (Q, K, V, dO) unless other seeds are
given; Q and K may be multiplied by ``qk_mult`` (the large-logit stress case)
before the cast to the working dtype (round-to-nearest-even).  Everything is
generated on the CPU, so a given seed gives the same tensors on any machine.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

DTYPES = {"fp32": torch.float32, "fp16": torch.float16, "bf16": torch.bfloat16}


@dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic attention problem."""

    name: str
    batch: int
    heads: int
    n_q: int
    n_k: int
    d: int
    dtype: str
    causal: bool = False
    std: float = 1.0
    qk_mult: float = 1.0
    backward: bool = True


# Self-attention workloads at the sizes of the paper's sweep (one head at
# n = 2^8 .. 2^20, d = 64, Section 5.1) and multi-head / causal / long-key
# variants.
WORKLOADS = {
    w.name: w
    for w in (
        Workload("selfattn_fp32_b1h1_n256_d64", 1, 1, 256, 256, 64, "fp32"),
        Workload("selfattn_bf16_b1h8_n4096_d64", 1, 8, 4096, 4096, 64, "bf16", backward=False),
        Workload("selfattn_bf16_b1h8_n4096_d64_qk30", 1, 8, 4096, 4096, 64, "bf16",
                 qk_mult=30.0, backward=False),
        Workload("selfattn_bf16_b1h16_n16384_d64", 1, 16, 16384, 16384, 64, "bf16"),
        Workload("causal_bf16_b4h32_n8192_d128", 4, 32, 8192, 8192, 128, "bf16",
                 causal=True, std=0.5),
        Workload("longkv_bf16_b1h1_nq16384_nk1048576_d64", 1, 1, 16384, 1 << 20, 64, "bf16",
                 backward=False),
        # Decode-shaped: one query per (batch, head) against a long key
        # sequence (the paper's single-query setting, Section 2), and a group
        # of 16 queries.
        Workload("decode_bf16_b8h16_nq1_nk65536_d64", 8, 16, 1, 65536, 64, "bf16", backward=False),
        Workload("decode_bf16_b8h16_nq16_nk65536_d64", 8, 16, 16, 65536, 64, "bf16",
                 backward=False),
    )
}


def normal(shape, seed: int, std: float = 1.0, mult: float = 1.0,
           dtype: torch.dtype = torch.bfloat16) -> torch.Tensor:
    """i.i.d. N(0, std^2) float32 draw from ``seed``, times ``mult``, cast to dtype."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    x = torch.randn(tuple(shape), generator=g, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if mult != 1.0:
        x.mul_(mult)
    return x.to(dtype)


def attention_inputs(batch: int, heads: int, n_q: int, n_k: int, d: int,
                     dtype: str | torch.dtype = "bf16", std: float = 1.0,
                     qk_mult: float = 1.0, seeds=(0, 1, 2, 3), with_grad: bool = True,
                     d_v: int | None = None):
    """Q, K, V (and dO) as CPU tensors of layout [B, H, n, features]: q and k
    with d features, v and dO with d_v (default d)."""
    dt = DTYPES[dtype] if isinstance(dtype, str) else dtype
    d_v = d if d_v is None else d_v
    q = normal((batch, heads, n_q, d), seeds[0], std, qk_mult, dt)
    k = normal((batch, heads, n_k, d), seeds[1], std, qk_mult, dt)
    v = normal((batch, heads, n_k, d_v), seeds[2], std, 1.0, dt)
    out = {"q": q, "k": k, "v": v}
    if with_grad:
        out["do"] = normal((batch, heads, n_q, d_v), seeds[3], 1.0, 1.0, dt)
    return out


def workload_inputs(w: Workload, seeds=(0, 1, 2, 3), with_grad: bool | None = None):
    return attention_inputs(w.batch, w.heads, w.n_q, w.n_k, w.d, w.dtype, w.std, w.qk_mult,
                            seeds, w.backward if with_grad is None else with_grad)
