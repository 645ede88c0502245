"""Seeded synthetic inputs shared by the HIP path's callers and the oracle's.

This module draws random numbers and builds layouts; it contains none of the
attention arithmetic.  Both the parity tests and the benchmark take their
inputs from here, so the oracle and the GPU see the same bf16 values.

Recipe: a CPU ``torch.Generator`` seeded per workload draws Q, K and V in
that order, each as ``[S][H][d]`` float32 N(0, 1), then rounds to bf16 with
round-to-nearest-even (torch's conversion).  Block tables are the identity,
or a seeded random permutation of the physical blocks.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    h_q: int
    h_kv: int
    head_dim: int
    seq_len: int
    num_chunks: int
    chunking: str           # "uniform" or "balanced"
    block_size: int
    seed: int
    permuted: bool = False  # block table: identity or seeded permutation
    perm_seed: int = 0
    align: int = 128        # boundary alignment of the balanced plan
    note: str = ""

    @property
    def scale(self) -> float:
        return float(torch.tensor(1.0 / self.head_dim ** 0.5, dtype=torch.float32))


# The five workloads: a small one the oracle finishes in seconds, and long-context
# prefill shapes of Llama-3-8B (32 q heads, 8 kv heads, d 128) and Llama-3-70B
# (64 q heads, 8 kv heads, d 128) attention layers.
WORKLOADS = {
    "small_d64": Workload("small_d64", 8, 8, 64, 1024, 4, "uniform", 256, seed=0,
                          note="1 layer, 8q=8kv heads, d64, S=1024 in 4x256"),
    "llama8b_32k_uniform": Workload("llama8b_32k_uniform", 32, 8, 128, 32768, 16, "uniform", 256,
                                    seed=1, note="Llama-3-8B attention, S=32768 in 16x2048"),
    "llama8b_128k_balanced": Workload("llama8b_128k_balanced", 32, 8, 128, 131072, 16, "balanced",
                                      256, seed=2,
                                      note="Llama-3-8B attention, S=131072 in 16 latency-balanced chunks"),
    "llama70b_64k_uniform": Workload("llama70b_64k_uniform", 64, 8, 128, 65536, 32, "uniform", 256,
                                     seed=3, note="Llama-3-70B attention, S=65536 in 32x2048, split-KV"),
    "llama8b_128k_paged": Workload("llama8b_128k_paged", 32, 8, 128, 131072, 32, "uniform", 256,
                                   seed=4, permuted=True, perm_seed=104,
                                   note="Llama-3-8B attention, S=131072 in 32x4096, 256-token blocks at "
                                        "permuted positions"),
}


def make_qkv(seed: int, seq_len: int, h_q: int, h_kv: int, head_dim: int):
    """Q [S][Hq][d], K [S][Hkv][d], V [S][Hkv][d] as CPU bf16 tensors."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    q = torch.randn((seq_len, h_q, head_dim), generator=g, dtype=torch.float32).to(torch.bfloat16)
    k = torch.randn((seq_len, h_kv, head_dim), generator=g, dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn((seq_len, h_kv, head_dim), generator=g, dtype=torch.float32).to(torch.bfloat16)
    return q, k, v


def make_kv_long(seed: int, n_tokens: int, h_kv: int, head_dim: int, piece: int = 65536):
    """K, V [n][Hkv][d] CPU bf16 for very long sequences, drawn N(0, 1) piece by
    piece (each piece from its own seeded generator) to bound host memory."""
    k = torch.empty((n_tokens, h_kv, head_dim), dtype=torch.bfloat16)
    v = torch.empty((n_tokens, h_kv, head_dim), dtype=torch.bfloat16)
    for i, start in enumerate(range(0, n_tokens, piece)):
        n = min(piece, n_tokens - start)
        g = torch.Generator(device="cpu")
        g.manual_seed(seed * 100003 + i)
        k[start:start + n] = torch.randn((n, h_kv, head_dim), generator=g, dtype=torch.float32).to(torch.bfloat16)
        v[start:start + n] = torch.randn((n, h_kv, head_dim), generator=g, dtype=torch.float32).to(torch.bfloat16)
    return k, v


def prefixes(lengths) -> List[int]:
    """P_c of every chunk: the number of tokens before it."""
    out, acc = [], 0
    for n in lengths:
        out.append(acc)
        acc += n
    return out


def identity_table(num_blocks: int) -> torch.Tensor:
    return torch.arange(num_blocks, dtype=torch.int32)


def permuted_table(num_blocks: int, seed: int, pool_blocks: Optional[int] = None) -> torch.Tensor:
    """Logical block i -> a distinct physical block, drawn from ``pool_blocks``."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    pool_blocks = num_blocks if pool_blocks is None else pool_blocks
    return torch.randperm(pool_blocks, generator=g)[:num_blocks].to(torch.int32)


def sample_rows(chunk_len: int, seed: int, n_random: int = 3) -> List[int]:
    """Chunk-local rows checked on large workloads: edges, middle and a few random."""
    fixed = {0, 1, chunk_len // 2, chunk_len - 2, chunk_len - 1}
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    extra = torch.randint(0, chunk_len, (n_random,), generator=g).tolist()
    return sorted(r for r in fixed.union(extra) if 0 <= r < chunk_len)


def bf16_bits(t: torch.Tensor):
    """A bf16 CPU tensor's bit patterns as a numpy uint16 array (no copy of values)."""
    import numpy as np
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)
