"""Per-chunk cost of a whole transformer layer: Eq. (1)'s two terms.

Eq. (1) of the paper splits a chunk's stage latency into attention, which
grows with c_i (p_i + c_i), and the dense projections and feed-forward
network, which grow with c_i alone.  This module runs one decoder layer per
chunk on one GPU to measure both terms:

    qkv  = x Wqkv                 [c, H] x [H, (Hq + 2 Hkv) d]   (library GEMM)
    K, V -> block store           mocap_kv_append
    o    = attention(q, store)    mocap_chunk_attn
    y    = x + o Wo               [c, Hq d] x [Hq d, H]          (library GEMM)
    z    = y + (silu(y Wg) * y Wu) Wd                            (library GEMMs)

The GEMMs are plain library GEMMs (torch.matmul, which runs hipBLASLt on
ROCm) with seeded random bf16 weights; the attention and the KV store are
this library's kernels.  Normalisation layers are omitted: they are
elementwise and add nothing to either term's shape.  Used to measure, not
part of libmocap_attn's hot path.
"""
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import torch

from . import binding
from .prefill import ChunkedPrefill


@dataclass(frozen=True)
class LayerShape:
    name: str
    hidden: int
    h_q: int
    h_kv: int
    head_dim: int
    ffn: int


# Decoder layer shapes of the published Llama-3 8B and 70B models.
SHAPES: Dict[str, LayerShape] = {
    "llama8b": LayerShape("llama8b", 4096, 32, 8, 128, 14336),
    "llama70b": LayerShape("llama70b", 8192, 64, 8, 128, 28672),
}


class ChunkedLayer:
    """One decoder layer applied chunk by chunk to one sequence."""

    def __init__(self, shape: LayerShape, lengths: Sequence[int], seed: int = 0, block_size: int = 256,
                 num_splits: int = 0, device="cuda"):
        self.shape = shape
        self.attn = ChunkedPrefill(shape.h_q, shape.h_kv, shape.head_dim, lengths, block_size=block_size,
                                   num_splits=num_splits, device=device)
        g = torch.Generator(device="cpu")
        g.manual_seed(seed)
        H, d = shape.hidden, shape.head_dim
        qkv_out = (shape.h_q + 2 * shape.h_kv) * d

        def weight(n_in, n_out):
            w = torch.randn((n_in, n_out), generator=g, dtype=torch.float32) * n_in ** -0.5
            return w.to(torch.bfloat16).to(device)

        self.w_qkv = weight(H, qkv_out)
        self.w_o = weight(shape.h_q * d, H)
        self.w_gu = weight(H, 2 * shape.ffn)
        self.w_d = weight(shape.ffn, H)

    @property
    def lengths(self) -> List[int]:
        return self.attn.lengths

    @property
    def prefixes(self) -> List[int]:
        return self.attn.prefixes

    def project_qkv(self, x: torch.Tensor):
        """q [S][Hq][d], k/v [S][Hkv][d] (contiguous) from x [S][H]."""
        s = self.shape
        qkv = x @ self.w_qkv
        nq, nk = s.h_q * s.head_dim, s.h_kv * s.head_dim
        q = qkv[:, :nq].reshape(-1, s.h_q, s.head_dim).contiguous()
        k = qkv[:, nq:nq + nk].reshape(-1, s.h_kv, s.head_dim).contiguous()
        v = qkv[:, nq + nk:].reshape(-1, s.h_kv, s.head_dim).contiguous()
        return q, k, v

    def run(self, x: torch.Tensor, scale: float, stream=None, events: Optional[list] = None) -> torch.Tensor:
        """All chunks in order; x is bf16 [S][H] on the device.  events, if
        given, is a list of (start, after_qkv, after_attention, end) event
        quadruples, one per chunk."""
        s = self.shape
        out = torch.empty_like(x)
        for c, (p, n) in enumerate(zip(self.prefixes, self.lengths)):
            xc = x[p:p + n]
            if events is not None:
                events[c][0].record(stream)
            q, k, v = self.project_qkv(xc)
            if events is not None:
                events[c][1].record(stream)
            # The chunk's K/V sit at positions [p, p + n) of the store.
            binding.mocap_kv_append(self.attn.store, self.attn.table, p, k, v, stream)
            binding.mocap_chunk_attn(self.attn.store, self.attn.table, q, p, scale, self.attn.o[p:p + n],
                                     self.attn.lse(c), self.attn.workspace, self.attn.num_splits, stream)
            if events is not None:
                events[c][2].record(stream)
            y = xc + self.attn.o[p:p + n].reshape(n, s.h_q * s.head_dim) @ self.w_o
            gu = y @ self.w_gu
            h = torch.nn.functional.silu(gu[:, :s.ffn]) * gu[:, s.ffn:]
            out[p:p + n] = y + h @ self.w_d
            if events is not None:
                events[c][3].record(stream)
        return out
