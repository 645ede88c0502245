"""ctypes binding of libmocap_attn (argument marshalling only).

Each function carries the name of the C entry point it wraps and does no
arithmetic of its own: it checks tensor dtypes, devices, shapes and
contiguity, passes raw pointers, and turns a non-zero status into
``MocapError``.  The library must have been built (``build.py``); if it is
missing this module raises instead of falling back to anything else.
"""
import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmocap_attn.so")

MOCAP_OK = 0
MOCAP_ERR_INVALID_ARG = 1
MOCAP_ERR_UNSUPPORTED = 2
MOCAP_ERR_WORKSPACE = 3
MOCAP_ERR_HIP = 4

# MOCAP_NOALLOC_SCRATCH_BYTES: the static device scratch of mocap_chunk_attn_noalloc.
NOALLOC_SCRATCH_BYTES = 128 << 20

# Every entry point the header declares.
EXPORTED = (
    "mocap_kv_append",
    "mocap_chunk_attn_workspace_size",
    "mocap_chunk_attn",
    "mocap_chunk_attn_noalloc",
    "mocap_chunk_attn_two_store",
    "mocap_chunk_attn_two_store_workspace_size",
    "mocap_chunk_plan",
    "mocap_chunk_prefixes",
    "mocap_lbcp_plan",
    "mocap_lbcp_plan_table",
    "mocap_lbcp_refine",
    "mocap_lbcp_evaluate",
    "mocap_lbcp_refine_e2e",
    "mocap_status_string",
    "mocap_check_block_table",
)


class mocap_lbcp_serving(ctypes.Structure):
    _fields_ = [
        ("fixed_cost", ctypes.c_double),
        ("kv_bytes_per_token", ctypes.c_double),
        ("stage_capacity", ctypes.c_double),
        ("pairing", ctypes.c_int32),
        ("max_batch", ctypes.c_int32),
        ("requests", ctypes.c_int32),
    ]


class MocapError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {mocap_status_string(status)} ({status})")


class mocap_kv_store(ctypes.Structure):
    _fields_ = [
        ("k_pool", ctypes.c_void_p),
        ("v_pool", ctypes.c_void_p),
        ("num_blocks", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("h_kv", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
    ]


_lib = None

# Debug option: check the block-table entries every call will use (a host copy,
# so each call synchronises) before calling the library.
_check_tables = os.environ.get("MOCAP_CHECK_TABLES", "0") == "1"


def set_table_checks(enabled: bool) -> None:
    """Turn the host-side block-table check of every call on or off."""
    global _check_tables
    _check_tables = bool(enabled)


def load_library():
    """Load libmocap_attn.so from the package directory (no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2606_22968_amd.build` "
            "(or __graft_entry__.build()) before using the HIP path")
    lib = ctypes.CDLL(LIB_PATH)
    st = ctypes.c_int
    lib.mocap_status_string.restype = ctypes.c_char_p
    lib.mocap_status_string.argtypes = [st]
    lib.mocap_kv_append.restype = st
    lib.mocap_kv_append.argtypes = [
        ctypes.POINTER(mocap_kv_store), ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.mocap_chunk_attn_workspace_size.restype = st
    lib.mocap_chunk_attn_workspace_size.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_size_t)]
    lib.mocap_chunk_attn.restype = st
    lib.mocap_chunk_attn.argtypes = [
        ctypes.POINTER(mocap_kv_store), ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
        ctypes.c_int32, ctypes.c_void_p]
    lib.mocap_chunk_attn_noalloc.restype = st
    lib.mocap_chunk_attn_noalloc.argtypes = [
        ctypes.POINTER(mocap_kv_store), ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
    lib.mocap_chunk_attn_two_store.restype = st
    lib.mocap_chunk_attn_two_store.argtypes = [
        ctypes.POINTER(mocap_kv_store), ctypes.c_void_p, ctypes.c_int32,
        ctypes.POINTER(mocap_kv_store), ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
        ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
        ctypes.c_int32, ctypes.c_void_p]
    lib.mocap_chunk_attn_two_store_workspace_size.restype = st
    lib.mocap_chunk_attn_two_store_workspace_size.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
        ctypes.c_int64, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_size_t)]
    lib.mocap_lbcp_plan.restype = st
    lib.mocap_lbcp_plan.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
        ctypes.c_double, ctypes.c_double, ctypes.POINTER(ctypes.c_int32),
        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    lib.mocap_lbcp_plan_table.restype = st
    lib.mocap_lbcp_plan_table.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
        ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    lib.mocap_lbcp_refine.restype = st
    lib.mocap_lbcp_refine.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
        ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int32, ctypes.c_uint64,
        ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)]
    lib.mocap_lbcp_evaluate.restype = st
    lib.mocap_lbcp_evaluate.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
        ctypes.POINTER(mocap_lbcp_serving), ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    lib.mocap_lbcp_refine_e2e.restype = st
    lib.mocap_lbcp_refine_e2e.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
        ctypes.POINTER(mocap_lbcp_serving), ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int32,
        ctypes.c_uint64, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    lib.mocap_check_block_table.restype = st
    lib.mocap_check_block_table.argtypes = [
        ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
        ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
    lib.mocap_chunk_plan.restype = st
    lib.mocap_chunk_plan.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
        ctypes.POINTER(ctypes.c_int32)]
    lib.mocap_chunk_prefixes.restype = st
    lib.mocap_chunk_prefixes.argtypes = [
        ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)]
    _lib = lib
    return lib


def mocap_status_string(status: int) -> str:
    return load_library().mocap_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != MOCAP_OK:
        raise MocapError(status, where)


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _require(t: torch.Tensor, dtype, name: str, ndim: Optional[int] = None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {tuple(t.shape)}")


class KvStore:
    """Caller-owned block pools (torch device memory) plus the C descriptor.

    k_pool: bf16 [num_blocks][h_kv][block_size][head_dim]
    v_pool: bf16 [num_blocks][h_kv][head_dim][block_size]
    """

    def __init__(self, num_blocks: int, block_size: int, h_kv: int, head_dim: int,
                 device="cuda", fill: Optional[float] = None):
        self.num_blocks, self.block_size, self.h_kv, self.head_dim = num_blocks, block_size, h_kv, head_dim
        self.k_pool = torch.empty((num_blocks, h_kv, block_size, head_dim), dtype=torch.bfloat16, device=device)
        self.v_pool = torch.empty((num_blocks, h_kv, head_dim, block_size), dtype=torch.bfloat16, device=device)
        if fill is not None:
            self.k_pool.fill_(fill)
            self.v_pool.fill_(fill)

    def descriptor(self) -> mocap_kv_store:
        return mocap_kv_store(self.k_pool.data_ptr(), self.v_pool.data_ptr(), self.num_blocks,
                              self.block_size, self.h_kv, self.head_dim)


def mocap_check_block_table(block_table, first_pos: int, end_pos: int, block_size: int, num_blocks: int) -> None:
    """Checks the entries positions [first_pos, end_pos) use (a host copy of
    the table is taken if it lives on the GPU); raises MocapError, with
    .bad_index, if one is out of range or repeats a physical block."""
    t = block_table.detach().to("cpu", torch.int32).contiguous() if isinstance(block_table, torch.Tensor) \
        else torch.tensor(list(block_table), dtype=torch.int32)
    bad = ctypes.c_int32(-1)
    st = load_library().mocap_check_block_table(
        ctypes.cast(t.data_ptr(), ctypes.POINTER(ctypes.c_int32)), t.numel(), int(first_pos), int(end_pos),
        int(block_size), int(num_blocks), ctypes.byref(bad))
    if st != MOCAP_OK:
        err = MocapError(st, f"mocap_check_block_table (logical block {bad.value})")
        err.bad_index = bad.value
        raise err


def _maybe_check(store: "KvStore", block_table: torch.Tensor, first: int, end: int) -> None:
    if _check_tables and end > first:
        mocap_check_block_table(block_table, first, end, store.block_size, store.num_blocks)


def mocap_kv_append(store: KvStore, block_table: torch.Tensor, start_pos: int,
                    k_chunk: torch.Tensor, v_chunk: torch.Tensor, stream=None) -> None:
    _require(block_table, torch.int32, "block_table", 1)
    _require(k_chunk, torch.bfloat16, "k_chunk", 3)
    _require(v_chunk, torch.bfloat16, "v_chunk", 3)
    if k_chunk.shape != v_chunk.shape or tuple(k_chunk.shape[1:]) != (store.h_kv, store.head_dim):
        raise ValueError("k_chunk/v_chunk must be [chunk_len][h_kv][head_dim] of the store")
    _maybe_check(store, block_table, int(start_pos), int(start_pos) + k_chunk.shape[0])
    desc = store.descriptor()
    _check(load_library().mocap_kv_append(
        ctypes.byref(desc), block_table.data_ptr(), block_table.numel(), int(start_pos),
        k_chunk.shape[0], k_chunk.data_ptr(), v_chunk.data_ptr(), _stream_handle(stream)),
        "mocap_kv_append")


def mocap_chunk_attn_workspace_size(prefix_len: int, chunk_len: int, h_q: int, h_kv: int,
                                    head_dim: int, num_splits: int = 0) -> Tuple[int, int]:
    """Returns (number of KV ranges, workspace bytes)."""
    splits = ctypes.c_int32(0)
    nbytes = ctypes.c_size_t(0)
    _check(load_library().mocap_chunk_attn_workspace_size(
        int(prefix_len), int(chunk_len), int(h_q), int(h_kv), int(head_dim), int(num_splits),
        ctypes.byref(splits), ctypes.byref(nbytes)), "mocap_chunk_attn_workspace_size")
    return splits.value, nbytes.value


def mocap_chunk_attn(store: KvStore, block_table: torch.Tensor, q: torch.Tensor, prefix_len: int,
                     scale: float, o: torch.Tensor, lse: torch.Tensor,
                     workspace: Optional[torch.Tensor] = None, num_splits: int = 0,
                     stream=None) -> None:
    """q, o: bf16 [chunk_len][h_q][head_dim]; lse: fp32 [h_q][chunk_len]."""
    _require(block_table, torch.int32, "block_table", 1)
    _require(q, torch.bfloat16, "q", 3)
    _require(o, torch.bfloat16, "o", 3)
    _require(lse, torch.float32, "lse", 2)
    chunk_len, h_q, head_dim = q.shape
    if o.shape != q.shape or tuple(lse.shape) != (h_q, chunk_len):
        raise ValueError("o must match q and lse must be [h_q][chunk_len]")
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        _require(workspace, workspace.dtype, "workspace")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    _maybe_check(store, block_table, 0, int(prefix_len) + chunk_len)
    desc = store.descriptor()
    _check(load_library().mocap_chunk_attn(
        ctypes.byref(desc), block_table.data_ptr(), block_table.numel(), q.data_ptr(),
        int(prefix_len), chunk_len, h_q, store.h_kv, head_dim, float(scale), o.data_ptr(),
        lse.data_ptr(), ws_ptr, ws_bytes, int(num_splits), _stream_handle(stream)),
        "mocap_chunk_attn")


def mocap_chunk_attn_noalloc(store: KvStore, block_table: torch.Tensor, q: torch.Tensor, prefix_len: int,
                             scale: float, o: torch.Tensor, lse: torch.Tensor, num_splits: int = 0,
                             stream=None) -> None:
    """mocap_chunk_attn with the split partials in the library's static device scratch."""
    _require(block_table, torch.int32, "block_table", 1)
    _require(q, torch.bfloat16, "q", 3)
    _require(o, torch.bfloat16, "o", 3)
    _require(lse, torch.float32, "lse", 2)
    chunk_len, h_q, head_dim = q.shape
    if o.shape != q.shape or tuple(lse.shape) != (h_q, chunk_len):
        raise ValueError("o must match q and lse must be [h_q][chunk_len]")
    _maybe_check(store, block_table, 0, int(prefix_len) + chunk_len)
    desc = store.descriptor()
    _check(load_library().mocap_chunk_attn_noalloc(
        ctypes.byref(desc), block_table.data_ptr(), block_table.numel(), q.data_ptr(),
        int(prefix_len), chunk_len, h_q, store.h_kv, head_dim, float(scale), o.data_ptr(),
        lse.data_ptr(), int(num_splits), _stream_handle(stream)),
        "mocap_chunk_attn_noalloc")


def mocap_chunk_attn_two_store_workspace_size(prefix_len: int, chunk_len: int, h_q: int, h_kv: int,
                                              head_dim: int, remote_begin: int, remote_end: int,
                                              num_splits: int = 0) -> Tuple[int, int]:
    """Returns (number of KV ranges, workspace bytes)."""
    splits = ctypes.c_int32(0)
    nbytes = ctypes.c_size_t(0)
    _check(load_library().mocap_chunk_attn_two_store_workspace_size(
        int(prefix_len), int(chunk_len), int(h_q), int(h_kv), int(head_dim), int(remote_begin),
        int(remote_end), int(num_splits), ctypes.byref(splits), ctypes.byref(nbytes)),
        "mocap_chunk_attn_two_store_workspace_size")
    return splits.value, nbytes.value


def mocap_chunk_attn_two_store(store: KvStore, block_table: torch.Tensor, remote: Optional[KvStore],
                               remote_table: Optional[torch.Tensor], remote_begin: int, remote_end: int,
                               q: torch.Tensor, prefix_len: int, scale: float, o: torch.Tensor,
                               lse: torch.Tensor, workspace: Optional[torch.Tensor] = None,
                               num_splits: int = 0, stream=None) -> None:
    """As mocap_chunk_attn, with keys [remote_begin, remote_end) read from `remote`."""
    _require(block_table, torch.int32, "block_table", 1)
    _require(q, torch.bfloat16, "q", 3)
    _require(o, torch.bfloat16, "o", 3)
    _require(lse, torch.float32, "lse", 2)
    chunk_len, h_q, head_dim = q.shape
    if o.shape != q.shape or tuple(lse.shape) != (h_q, chunk_len):
        raise ValueError("o must match q and lse must be [h_q][chunk_len]")
    r_desc, r_table, r_n = None, None, 0
    if remote is not None:
        _require(remote_table, torch.int32, "remote_table", 1)
        r_desc = ctypes.byref(remote.descriptor())
        r_table, r_n = remote_table.data_ptr(), remote_table.numel()
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        _require(workspace, workspace.dtype, "workspace")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    if int(remote_end) > int(remote_begin) and remote is not None:
        _maybe_check(store, block_table, 0, int(remote_begin))
        _maybe_check(store, block_table, int(remote_end), int(prefix_len) + chunk_len)
        _maybe_check(remote, remote_table, int(remote_begin), int(remote_end))
    else:
        _maybe_check(store, block_table, 0, int(prefix_len) + chunk_len)
    desc = store.descriptor()
    _check(load_library().mocap_chunk_attn_two_store(
        ctypes.byref(desc), block_table.data_ptr(), block_table.numel(), r_desc, r_table, r_n,
        int(remote_begin), int(remote_end), q.data_ptr(), int(prefix_len), chunk_len, h_q, store.h_kv,
        head_dim, float(scale), o.data_ptr(), lse.data_ptr(), ws_ptr, ws_bytes, int(num_splits),
        _stream_handle(stream)), "mocap_chunk_attn_two_store")


def mocap_chunk_plan(seq_len: int, num_chunks: int, align: int = 128, balanced: bool = False) -> List[int]:
    out = (ctypes.c_int32 * num_chunks)()
    _check(load_library().mocap_chunk_plan(int(seq_len), int(num_chunks), int(align), int(bool(balanced)), out),
           "mocap_chunk_plan")
    return list(out)


def mocap_chunk_prefixes(lengths: Sequence[int]) -> List[int]:
    n = len(lengths)
    ln = (ctypes.c_int32 * max(n, 1))(*[int(x) for x in lengths])
    out = (ctypes.c_int64 * max(n, 1))()
    _check(load_library().mocap_chunk_prefixes(ln, n, out), "mocap_chunk_prefixes")
    return list(out)[:n]


def mocap_lbcp_plan(seq_len: int, num_chunks: int, num_stages: int, align: int, cost_pair: float,
                    cost_token: float = 0.0, cost_chunk: float = 0.0):
    """Returns (lengths, t_max, t_sum) of the dynamic-programming plan."""
    out = (ctypes.c_int32 * num_chunks)()
    t_max = ctypes.c_double(0.0)
    t_sum = ctypes.c_double(0.0)
    _check(load_library().mocap_lbcp_plan(int(seq_len), int(num_chunks), int(num_stages), int(align),
                                          float(cost_pair), float(cost_token), float(cost_chunk), out,
                                          ctypes.byref(t_max), ctypes.byref(t_sum)), "mocap_lbcp_plan")
    return list(out), t_max.value, t_sum.value


def _cost_table(chunk_cost, units: int):
    """A float64 [U][U] table as a ctypes pointer (the array must stay alive)."""
    import numpy as np
    arr = np.ascontiguousarray(chunk_cost, dtype=np.float64)
    if arr.shape != (units, units):
        raise ValueError(f"chunk_cost must be [{units}][{units}]")
    return arr, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def mocap_lbcp_plan_table(seq_len: int, num_chunks: int, num_stages: int, align: int, chunk_cost):
    """Returns (lengths, t_max, t_sum); chunk_cost[k - 1][s] in align units."""
    arr, ptr = _cost_table(chunk_cost, seq_len // align)
    out = (ctypes.c_int32 * num_chunks)()
    t_max = ctypes.c_double(0.0)
    t_sum = ctypes.c_double(0.0)
    _check(load_library().mocap_lbcp_plan_table(int(seq_len), int(num_chunks), int(num_stages), int(align), ptr,
                                                out, ctypes.byref(t_max), ctypes.byref(t_sum)),
           "mocap_lbcp_plan_table")
    return list(out), t_max.value, t_sum.value


def mocap_lbcp_refine(seq_len: int, num_chunks: int, num_stages: int, align: int, chunk_cost,
                      lengths: Sequence[int], temp0: float, temp_min: float, alpha: float, rounds: int,
                      seed: int):
    """Returns (lengths, latency) of the best partition the annealing found."""
    arr, ptr = _cost_table(chunk_cost, seq_len // align)
    io = (ctypes.c_int32 * num_chunks)(*[int(x) for x in lengths])
    lat = ctypes.c_double(0.0)
    _check(load_library().mocap_lbcp_refine(int(seq_len), int(num_chunks), int(num_stages), int(align), ptr,
                                            float(temp0), float(temp_min), float(alpha), int(rounds),
                                            int(seed) & 0xFFFFFFFFFFFFFFFF, io, ctypes.byref(lat)),
           "mocap_lbcp_refine")
    return list(io), lat.value


def _serving(fixed_cost: float, kv_bytes_per_token: float, stage_capacity: float, pairing: bool,
             max_batch: int, requests: int) -> mocap_lbcp_serving:
    return mocap_lbcp_serving(float(fixed_cost), float(kv_bytes_per_token), float(stage_capacity),
                              1 if pairing else 0, int(max_batch), int(requests))


def mocap_lbcp_evaluate(seq_len: int, num_chunks: int, num_stages: int, align: int, chunk_cost,
                        lengths: Sequence[int], fixed_cost: float, kv_bytes_per_token: float,
                        stage_capacity: float, pairing: bool, max_batch: int, requests: int):
    """Returns (B', T'_pre, T') of a partition under the serving model."""
    arr, ptr = _cost_table(chunk_cost, seq_len // align)
    sv = _serving(fixed_cost, kv_bytes_per_token, stage_capacity, pairing, max_batch, requests)
    ln = (ctypes.c_int32 * num_chunks)(*[int(x) for x in lengths])
    b, pre, t = ctypes.c_int32(0), ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(load_library().mocap_lbcp_evaluate(int(seq_len), int(num_chunks), int(num_stages), int(align), ptr,
                                              ctypes.byref(sv), ln, ctypes.byref(b), ctypes.byref(pre),
                                              ctypes.byref(t)), "mocap_lbcp_evaluate")
    return b.value, pre.value, t.value


def mocap_lbcp_refine_e2e(seq_len: int, num_chunks: int, num_stages: int, align: int, chunk_cost,
                          lengths: Sequence[int], fixed_cost: float, kv_bytes_per_token: float,
                          stage_capacity: float, pairing: bool, max_batch: int, requests: int,
                          temp0: float, temp_min: float, alpha: float, rounds: int, seed: int):
    """Returns (lengths, B', T'_pre, T') of the best partition the annealing found."""
    arr, ptr = _cost_table(chunk_cost, seq_len // align)
    sv = _serving(fixed_cost, kv_bytes_per_token, stage_capacity, pairing, max_batch, requests)
    io = (ctypes.c_int32 * num_chunks)(*[int(x) for x in lengths])
    b, pre, t = ctypes.c_int32(0), ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(load_library().mocap_lbcp_refine_e2e(
        int(seq_len), int(num_chunks), int(num_stages), int(align), ptr, ctypes.byref(sv), float(temp0),
        float(temp_min), float(alpha), int(rounds), int(seed) & 0xFFFFFFFFFFFFFFFF, io, ctypes.byref(b),
        ctypes.byref(pre), ctypes.byref(t)), "mocap_lbcp_refine_e2e")
    return list(io), b.value, pre.value, t.value
