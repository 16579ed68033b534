"""Seeded synthetic inputs for PHSA workloads.

This module only draws random tensors; it holds none of the method's
arithmetic.  The GPU library, the tests, the benchmark and the CPU reference
all take their inputs from here, so both sides of every comparison see the
same bits.

Recipe: a CPU ``torch.Generator`` seeded with ``seed`` draws, in this order,
Q, K, V (and dO when asked) as float32 standard normals, then the
punctuation mask.  Floating tensors are then cast (round-to-nearest-even) to
the workload's dtype.  The mask is either Bernoulli(p) per token or a
"sentence-like" pattern: punctuation at cumulative geometric gaps with the
given mean (support >= 1), which has the same average density as
Bernoulli(1 / mean) but ends runs at sentence-like spacing.

The workloads mirror the shapes of the paper's long-context setting
(Qwen3-0.6B-like heads: 16 query heads, 8 KV heads, head dim 128; 32k tokens;
a 14-block budget of 64-token blocks, i.e. 896 active tokens = 97.3%
sparsity at 32k).  The paper's own evaluation suites (NIAH, LongBench) need
weights and data; these synthetic tensors stand in for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    seqlen_q: int
    seqlen_k: int
    n_heads_q: int
    n_heads_kv: int
    head_dim: int
    block_size: int
    top_k: int          # free picks, forced init/local blocks not counted
    n_init_blocks: int
    window: int         # local window in tokens (multiple of block_size)
    dtype: str          # "bf16" | "fp32"
    punct: str = "bernoulli"   # "bernoulli" | "geometric"
    punct_p: float = 0.08
    gap_mean: float = 12.0
    q_scale: float = 1.0
    lam: float = 0.5
    backward: bool = False

    @property
    def ksel(self) -> int:
        return self.n_init_blocks + self.window // self.block_size + 1 + self.top_k

    @property
    def n_blocks(self) -> int:
        return self.seqlen_k // self.block_size

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads.  "top-k" in the workload descriptions counts the forced
# init block and the diagonal (local) block, so the free pick count is two less.
WORKLOADS: Dict[str, Workload] = {
    "tiny_fp32": Workload("tiny_fp32", 1, 1024, 1024, 2, 1, 64, 64, 2, 1, 0, "fp32",
                          punct="bernoulli", punct_p=0.1),
    "prefill_8k": Workload("prefill_8k", 1, 8192, 8192, 16, 8, 128, 64, 14, 1, 0, "bf16",
                           punct="geometric", gap_mean=12.0, q_scale=1.0 / math.sqrt(128.0)),
    "prefill_32k": Workload("prefill_32k", 1, 32768, 32768, 16, 8, 128, 64, 12, 1, 0, "bf16"),
    "decode_32k": Workload("decode_32k", 64, 1, 32768, 16, 8, 128, 64, 12, 1, 0, "bf16"),
    "train_32k": Workload("train_32k", 4, 32768, 32768, 16, 8, 128, 64, 12, 1, 0, "bf16", backward=True),
    # the paper's own 32k training setting (Section 4.1, model configuration, and
    # Top-K = 16 in Section 4.2): 16-token blocks, 128 init tokens (8 blocks), a
    # 512-token local window (32 blocks + the query's own) and 16 free picks:
    # 57 blocks = 912 tokens per query
    "train_32k_paper": Workload("train_32k_paper", 4, 32768, 32768, 16, 8, 128, 16, 16, 8, 512, "bf16",
                                backward=True),
}


def _mask(wl: Workload, gen: torch.Generator) -> torch.Tensor:
    B, L = wl.batch, wl.seqlen_k
    if wl.punct == "bernoulli":
        return (torch.rand(B, L, generator=gen) < wl.punct_p).to(torch.uint8)
    if wl.punct == "geometric":
        p = 1.0 / wl.gap_mean
        n = int(L * p * 2 + 64)
        u = torch.rand(B, n, generator=gen, dtype=torch.float64).clamp_min(1e-300)
        gaps = torch.floor(torch.log(u) / math.log1p(-p)).to(torch.int64) + 1
        pos = torch.cumsum(gaps, dim=1) - 1
        out = torch.zeros(B, L, dtype=torch.uint8)
        for b in range(B):
            pb = pos[b][pos[b] < L]
            out[b, pb] = 1
        return out
    raise ValueError(wl.punct)


def make_inputs(wl: Workload, seed: int = 0, with_grad_out: Optional[bool] = None) -> Dict[str, torch.Tensor]:
    """Host tensors Q [B,Lq,Hq,d], K,V [B,Lk,Hkv,d], (dO [B,Lq,Hq,d]), punct uint8 [B,Lk]."""
    if with_grad_out is None:
        with_grad_out = wl.backward
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    B, Lq, Lk, Hq, Hkv, d = wl.batch, wl.seqlen_q, wl.seqlen_k, wl.n_heads_q, wl.n_heads_kv, wl.head_dim
    q = torch.randn(B, Lq, Hq, d, generator=gen)
    if wl.q_scale != 1.0:
        q = q * wl.q_scale
    k = torch.randn(B, Lk, Hkv, d, generator=gen)
    v = torch.randn(B, Lk, Hkv, d, generator=gen)
    out = {"q": q.to(wl.torch_dtype), "k": k.to(wl.torch_dtype), "v": v.to(wl.torch_dtype)}
    del q, k, v
    if with_grad_out:
        out["do"] = torch.randn(B, Lq, Hq, d, generator=gen).to(wl.torch_dtype)
    out["punct"] = _mask(wl, gen)
    return out
