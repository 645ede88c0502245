"""Chunked prefill of one sequence on one GPU stream.

Models one pipeline stage of the paper's chunked pipeline (Section 2.2)
processing the whole chunk sequence: for every chunk c, append its keys and
values to the block store, then run its attention over the prefix and
itself.  All work happens in the library's kernels; this class only owns the
device buffers (through torch) and issues the calls in order.

With `remote=(begin, end)` the keys/values of positions [begin, end) are also
written to a second store, as the KV a debtor stage spills to its paired
creditor under memory-balanced KV reallocation (Section 4.1), and every later
chunk reads that range from the second store (mocap_chunk_attn_two_store).
"""
from typing import List, Optional, Sequence, Tuple

import torch

from . import binding


class ChunkedPrefill:
    def __init__(self, h_q: int, h_kv: int, head_dim: int, lengths: Sequence[int],
                 block_size: int = 256, table: Optional[torch.Tensor] = None,
                 pool_blocks: Optional[int] = None, num_splits: int = 0, device="cuda",
                 pool_fill: Optional[float] = None, remote: Optional[Tuple[int, int]] = None,
                 remote_table: Optional[torch.Tensor] = None):
        self.h_q, self.h_kv, self.head_dim = h_q, h_kv, head_dim
        self.lengths = [int(n) for n in lengths]
        self.prefixes = binding.mocap_chunk_prefixes(self.lengths)
        self.seq_len = (self.prefixes[-1] + self.lengths[-1]) if self.lengths else 0
        self.block_size = block_size
        n_logical = (self.seq_len + block_size - 1) // block_size
        if table is None:
            table = torch.arange(n_logical, dtype=torch.int32)
        if table.numel() < n_logical:
            raise ValueError("block table shorter than the sequence")
        pool_blocks = pool_blocks if pool_blocks is not None else int(table.max().item()) + 1
        self.table = table.to(device=device, dtype=torch.int32).contiguous()
        self.store = binding.KvStore(pool_blocks, block_size, h_kv, head_dim, device=device, fill=pool_fill)
        self.remote = None
        self.remote_store = None
        if remote is not None and remote[0] != remote[1]:
            begin, end = int(remote[0]), int(remote[1])
            if not (0 <= begin <= end <= self.seq_len) or begin % 64 or end % 64:
                raise ValueError("remote range must be whole 64-key tiles inside the sequence")
            if any(begin < p < end and p % 64 for p in self.prefixes):
                raise ValueError("a chunk boundary inside the remote range must be a multiple of 64")
            self.remote = (begin, end)
            n_remote = (end + block_size - 1) // block_size
            if remote_table is None:
                remote_table = torch.arange(n_remote, dtype=torch.int32)
            if remote_table.numel() < n_remote:
                raise ValueError("remote block table shorter than the remote range")
            self.remote_table = remote_table.to(device=device, dtype=torch.int32).contiguous()
            self.remote_store = binding.KvStore(int(remote_table.max().item()) + 1, block_size, h_kv, head_dim,
                                                device=device, fill=pool_fill)
        self.num_splits = num_splits
        self.splits: List[int] = []
        ws_bytes = 0
        for p, n in zip(self.prefixes, self.lengths):
            rb, re = self.remote_range(p)
            r, b = binding.mocap_chunk_attn_two_store_workspace_size(p, n, h_q, h_kv, head_dim, rb, re, num_splits)
            self.splits.append(r)
            ws_bytes = max(ws_bytes, b)
        self.workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=device)
        self.o = torch.empty((self.seq_len, h_q, head_dim), dtype=torch.bfloat16, device=device)
        # One fp32 [h_q][L_c] region per chunk, each starting on a 16-byte boundary.
        self._lse_off = []
        off = 0
        for n in self.lengths:
            self._lse_off.append(off)
            off += (h_q * n + 3) // 4 * 4
        self._lse_flat = torch.empty(max(off, 4), dtype=torch.float32, device=device)

    def lse(self, c: int) -> torch.Tensor:
        n = self.lengths[c]
        return self._lse_flat[self._lse_off[c]:self._lse_off[c] + self.h_q * n].view(self.h_q, n)

    def remote_range(self, prefix_len: int) -> Tuple[int, int]:
        """The part of [0, prefix_len) held by the second store (empty if none)."""
        if self.remote is None:
            return 0, 0
        return min(self.remote[0], prefix_len), min(self.remote[1], prefix_len)

    def append(self, c: int, k: torch.Tensor, v: torch.Tensor, stream=None):
        """Store chunk c's keys/values.  They always go to the first store (the
        chunk's own attention reads them there); with a remote range, the part
        inside it is also written to the second store, where every later chunk
        reads it (the first store's copy is not read again)."""
        p, n = self.prefixes[c], self.lengths[c]
        binding.mocap_kv_append(self.store, self.table, p, k[p:p + n], v[p:p + n], stream)
        if self.remote is not None:
            lo, hi = max(p, self.remote[0]), min(p + n, self.remote[1])
            if lo < hi:
                binding.mocap_kv_append(self.remote_store, self.remote_table, lo, k[lo:hi], v[lo:hi], stream)

    def attend(self, c: int, q: torch.Tensor, scale: float, stream=None):
        p, n = self.prefixes[c], self.lengths[c]
        rb, re = self.remote_range(p)
        if rb < re:
            binding.mocap_chunk_attn_two_store(self.store, self.table, self.remote_store, self.remote_table, rb, re,
                                               q[p:p + n], p, scale, self.o[p:p + n], self.lse(c),
                                               self.workspace, self.num_splits, stream)
        else:
            binding.mocap_chunk_attn(self.store, self.table, q[p:p + n], p, scale, self.o[p:p + n],
                                     self.lse(c), self.workspace, self.num_splits, stream)

    def run(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: float, stream=None,
            events: Optional[list] = None):
        """All chunks in order.  q [S][Hq][d], k/v [S][Hkv][d] bf16 on the device.

        events, if given, is a list of (start, after_append, end) event triples,
        one per chunk, recorded around each chunk's calls.
        """
        for c in range(len(self.lengths)):
            if events is not None:
                events[c][0].record(stream)
            self.append(c, k, v, stream)
            if events is not None:
                events[c][1].record(stream)
            self.attend(c, q, scale, stream)
            if events is not None:
                events[c][2].record(stream)
        return self.o
