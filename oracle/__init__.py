"""fp64 CPU oracle for chunked causal prefill attention -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or calls anything here, and this
package imports nothing from the product.

Contents
  chunk_attn       fp64 attention of one chunk against its prefix (C, OpenMP),
                   the plain definition: Section 2.2 of the paper (each chunk
                   attends to all earlier chunks' keys/values) with the causal
                   prefix/chunk split priced by Eq. (1), Section 3.2.
  bruteforce       a structurally different numpy routine: the whole S x S
                   masked score matrix of a monolithic causal prefill.
  plan             chunk plans (uniform, latency-balanced) and FLOP accounting.
  merge            log-sum-exp merge of attention over disjoint key sets.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = _build.LIB
    if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
        _build.build()
    lib = ctypes.CDLL(path)
    lib.oracle_chunk_attn.restype = ctypes.c_int
    lib.oracle_chunk_attn.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
        ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_double, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_int,
    ]
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_max_threads.argtypes = []
    _lib = lib
    return lib


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def _as_input(x):
    """Accept fp64 arrays, or bf16 bit patterns as uint16 arrays."""
    x = np.ascontiguousarray(x)
    if x.dtype == np.float64:
        return x, 0
    if x.dtype == np.uint16:
        return x, 1
    raise TypeError(f"oracle inputs must be float64 or uint16 (bf16 bits), got {x.dtype}")


def chunk_attn(q, k, v, prefix_len, scale, rows=None, threads=0):
    """fp64 attention of one chunk (plain definition).

    q: [L][Hq][d]; k, v: [>= P+L][Hkv][d] logical (contiguous) keys/values;
    all three either float64 or uint16 bf16 bit patterns (same kind).
    rows: chunk-local query rows to evaluate (default: all L rows).
    Returns (o [n_rows][Hq][d] float64, lse [Hq][n_rows] float64, natural log).
    """
    lib = _load()
    q, qb = _as_input(q)
    k, kb = _as_input(k)
    v, vb = _as_input(v)
    if not (qb == kb == vb):
        raise TypeError("q, k and v must share one input kind")
    L, h_q, d = q.shape
    _, h_kv, dk = k.shape
    if dk != d or v.shape[1:] != k.shape[1:]:
        raise ValueError("shape mismatch between q, k and v")
    if k.shape[0] < prefix_len + L or v.shape[0] < prefix_len + L:
        raise ValueError("k/v shorter than prefix_len + chunk_len")
    if rows is None:
        rows = np.arange(L, dtype=np.int64)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    n = rows.shape[0]
    o = np.empty((n, h_q, d), dtype=np.float64)
    lse = np.empty((h_q, n), dtype=np.float64)
    rc = lib.oracle_chunk_attn(
        q.ctypes.data, k.ctypes.data, v.ctypes.data, qb, int(prefix_len), int(L),
        int(h_q), int(h_kv), int(d), float(scale), rows.ctypes.data, int(n),
        o.ctypes.data, lse.ctypes.data, int(threads))
    if rc != 0:
        raise ValueError(f"oracle_chunk_attn failed with code {rc}")
    return o, lse
