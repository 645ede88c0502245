"""The C ABI on the host: exported symbols, status strings and validation.

Every malformed call must be rejected on the host before anything is
enqueued, so these checks run without a GPU: the pointers passed are fake
(but aligned) addresses that the library must never touch.
"""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mocap_attn.h")

FAKE = 0x10000  # aligned, never dereferenced
MIS = FAKE + 2  # misaligned


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mocap_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(mocap_lib):
    lib = mocap_lib.load_library()
    names = declared_functions()
    assert set(names) == set(mocap_lib.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(mocap_lib):
    assert mocap_lib.mocap_status_string(0) == "MOCAP_OK"
    assert mocap_lib.mocap_status_string(3) == "MOCAP_ERR_WORKSPACE"
    assert mocap_lib.mocap_status_string(99) == "MOCAP_ERR_UNKNOWN"


def store(mocap_lib, num_blocks=64, block_size=256, h_kv=8, head_dim=128, k=FAKE, v=FAKE):
    return mocap_lib.mocap_kv_store(k, v, num_blocks, block_size, h_kv, head_dim)


def attn(mocap_lib, kv=None, table=FAKE, n_table=64, q=FAKE, P=1024, L=256, h_q=32, h_kv=8, d=128,
         scale=0.088, o=FAKE, lse=FAKE, ws=None, ws_bytes=0, splits=1):
    lib = mocap_lib.load_library()
    kv = store(mocap_lib) if kv is None else kv
    ref = ctypes.byref(kv) if kv != "null" else None
    return lib.mocap_chunk_attn(ref, table, n_table, q, P, L, h_q, h_kv, d, scale, o, lse, ws, ws_bytes,
                                splits, None)


def append(mocap_lib, kv=None, table=FAKE, n_table=64, P=0, L=256, k=FAKE, v=FAKE):
    lib = mocap_lib.load_library()
    kv = store(mocap_lib) if kv is None else kv
    ref = ctypes.byref(kv) if kv != "null" else None
    return lib.mocap_kv_append(ref, table, n_table, P, L, k, v, None)


INVALID, UNSUPPORTED, WORKSPACE = 1, 2, 3


@pytest.mark.parametrize("kwargs,expect", [
    (dict(kv="null"), INVALID),
    (dict(h_q=30), INVALID),                    # not a multiple of h_kv
    (dict(h_kv=4, h_q=32), INVALID),            # differs from the store
    (dict(d=64), INVALID),                      # differs from the store
    (dict(scale=0.0), INVALID),
    (dict(scale=-0.1), INVALID),
    (dict(scale=math.nan), INVALID),
    (dict(scale=math.inf), INVALID),
    (dict(P=-1), INVALID),
    (dict(L=-5), INVALID),
    (dict(n_table=4), INVALID),                 # needs 5 blocks for 1280 positions
    (dict(P=(1 << 31) - 200, n_table=1 << 30), INVALID),   # beyond 32-bit positions
    (dict(q=0), INVALID),
    (dict(o=0), INVALID),
    (dict(lse=0), INVALID),
    (dict(table=0), INVALID),
    (dict(q=MIS), INVALID),
    (dict(o=MIS), INVALID),
    (dict(lse=FAKE + 4), INVALID),
    (dict(splits=-1), INVALID),
    (dict(splits=3), WORKSPACE),                # forced split without workspace
    (dict(splits=3, ws=FAKE, ws_bytes=1024), WORKSPACE),
    (dict(splits=3, ws=MIS, ws_bytes=1 << 30), WORKSPACE),
])
def test_chunk_attn_rejects(mocap_lib, kwargs, expect):
    assert attn(mocap_lib, **kwargs) == expect


@pytest.mark.parametrize("store_kwargs,expect", [
    (dict(head_dim=96), UNSUPPORTED),
    (dict(block_size=100), UNSUPPORTED),
    (dict(block_size=32), UNSUPPORTED),
    (dict(block_size=0), INVALID),
    (dict(num_blocks=0), INVALID),
    (dict(h_kv=0), INVALID),
])
def test_store_rejected(mocap_lib, store_kwargs, expect):
    kv = store(mocap_lib, **store_kwargs)
    h_kv = store_kwargs.get("h_kv", 8) or 8
    d = store_kwargs.get("head_dim", 128)
    assert attn(mocap_lib, kv=kv, h_kv=h_kv, d=d) == expect
    assert append(mocap_lib, kv=kv) == expect


def test_zero_length_chunk_is_a_noop(mocap_lib):
    # Valid sizes with chunk_len 0 return OK without touching anything, even
    # with null tensor pointers.
    assert attn(mocap_lib, L=0, q=0, o=0, lse=0) == 0
    assert append(mocap_lib, L=0, k=0, v=0) == 0


@pytest.mark.parametrize("kwargs,expect", [
    (dict(kv="null"), INVALID),
    (dict(P=-1), INVALID),
    (dict(L=-1), INVALID),
    (dict(n_table=0), INVALID),
    (dict(P=16300, L=200, n_table=64), INVALID),   # runs past the table
    (dict(k=0), INVALID),
    (dict(v=MIS), INVALID),
    (dict(table=MIS), INVALID),
])
def test_kv_append_rejects(mocap_lib, kwargs, expect):
    assert append(mocap_lib, **kwargs) == expect


def test_workspace_size_forced_splits(mocap_lib):
    ws = mocap_lib.mocap_chunk_attn_workspace_size
    # P = 4096 (64 tiles), L = 256, 32 heads, d 128, 5 ranges requested.
    r, b = ws(4096, 256, 32, 8, 128, 5)
    rows = 5 * 32 * 256
    assert r == 5
    assert b == rows * 128 * 4 + rows * 4
    assert ws(4096, 256, 32, 8, 128, 1) == (1, 0)
    assert ws(64, 256, 32, 8, 128, 5)[0] == 2    # one prefix tile: at most one prefix range
    assert ws(0, 256, 32, 8, 128, 5) == (1, 0)   # no prefix: nothing to split
    assert ws(100, 0, 32, 8, 128, 0) == (1, 0)
    with pytest.raises(mocap_lib.MocapError):
        ws(4096, 256, 32, 8, 96, 1)
    with pytest.raises(mocap_lib.MocapError):
        ws(4096, 256, 30, 8, 128, 1)


def attn2(mocap_lib, kv=None, table=FAKE, n_table=64, rkv=None, rtable=FAKE, n_rtable=64, rb=0, re=512,
          q=FAKE, P=1024, L=256, h_q=32, h_kv=8, d=128, scale=0.088, o=FAKE, lse=FAKE, ws=None, ws_bytes=0,
          splits=2):
    lib = mocap_lib.load_library()
    kv = store(mocap_lib) if kv is None else kv
    rkv = store(mocap_lib) if rkv is None else rkv
    rref = ctypes.byref(rkv) if rkv != "null" else None
    return lib.mocap_chunk_attn_two_store(ctypes.byref(kv), table, n_table, rref, rtable, n_rtable, rb, re, q,
                                          P, L, h_q, h_kv, d, scale, o, lse, ws, ws_bytes, splits, None)


@pytest.mark.parametrize("kwargs,expect", [
    (dict(rb=-64), INVALID),
    (dict(rb=512, re=256), INVALID),               # begin after end
    (dict(re=1088), INVALID),                      # beyond the prefix
    (dict(re=500), INVALID),                       # not a whole tile
    (dict(rb=32), INVALID),
    (dict(rkv="null"), INVALID),
    (dict(rtable=0), INVALID),
    (dict(rtable=MIS), INVALID),
    (dict(n_rtable=1), INVALID),                   # 512 positions need 2 blocks
    (dict(rkv="h_kv"), INVALID),
    (dict(rkv="block"), INVALID),
    (dict(rkv="dim"), INVALID),
    (dict(scale=0.0), INVALID),
    (dict(n_table=4), INVALID),
    (dict(splits=3), WORKSPACE),                   # a split plan without workspace
])
def test_two_store_rejects(mocap_lib, kwargs, expect):
    variants = {"h_kv": dict(h_kv=4), "block": dict(block_size=128), "dim": dict(head_dim=64)}
    if kwargs.get("rkv") in variants:
        kwargs = dict(kwargs, rkv=store(mocap_lib, **variants[kwargs["rkv"]]))
    assert attn2(mocap_lib, **kwargs) == expect


def test_two_store_empty_remote_range_is_single_store(mocap_lib):
    # remote arguments unused: the same status as mocap_chunk_attn
    assert attn2(mocap_lib, rkv="null", rtable=0, n_rtable=0, rb=256, re=256, splits=3) == WORKSPACE
    assert attn2(mocap_lib, rkv="null", rtable=0, n_rtable=0, rb=0, re=0, L=0, q=0, o=0, lse=0) == 0


def test_two_store_workspace_size(mocap_lib):
    ws2 = mocap_lib.mocap_chunk_attn_two_store_workspace_size
    ws = mocap_lib.mocap_chunk_attn_workspace_size
    # The store is chosen per tile, so the plan is the single-store plan.
    for rb, re in [(1024, 2048), (0, 2048), (2048, 4096), (0, 4096), (1024, 1024), (64, 128)]:
        for splits in (1, 2, 5, 500):
            assert ws2(4096, 256, 32, 8, 128, rb, re, splits) == ws(4096, 256, 32, 8, 128, splits)
    assert ws2(4096, 0, 32, 8, 128, 0, 1024, 0) == (1, 0)
    for bad in [(4096, 256, 32, 8, 128, 0, 4097, 0), (4096, 256, 32, 8, 128, 64, 0, 0),
                (4096, 256, 32, 8, 128, 10, 64, 0)]:
        with pytest.raises(mocap_lib.MocapError):
            ws2(*bad)


def noalloc(mocap_lib, kv=None, table=FAKE, n_table=64, q=FAKE, P=1024, L=256, h_q=32, h_kv=8, d=128,
            scale=0.088, o=FAKE, lse=FAKE, splits=1):
    lib = mocap_lib.load_library()
    kv = store(mocap_lib) if kv is None else kv
    ref = ctypes.byref(kv) if kv != "null" else None
    return lib.mocap_chunk_attn_noalloc(ref, table, n_table, q, P, L, h_q, h_kv, d, scale, o, lse, splits, None)


SCRATCH_BYTES = 128 << 20  # MOCAP_NOALLOC_SCRATCH_BYTES


def test_noalloc_scratch_size_matches_header():
    text = open(HEADER).read()
    assert "#define MOCAP_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)" in text


@pytest.mark.parametrize("kwargs,expect", [
    (dict(kv="null"), INVALID),
    (dict(h_q=30), INVALID),
    (dict(scale=math.nan), INVALID),
    (dict(P=-1), INVALID),
    (dict(n_table=4), INVALID),
    (dict(q=MIS), INVALID),
    (dict(lse=0), INVALID),
    (dict(splits=-1), INVALID),
    # A forced split whose partials exceed the scratch: P = 1M keys cut into
    # 16 ranges + 1, L = 2048 rows of 32 heads at d 128 (~285 MB of partials).
    (dict(P=1 << 20, L=2048, n_table=(1 << 20) // 256 + 8, splits=17), WORKSPACE),
])
def test_noalloc_rejects(mocap_lib, kwargs, expect):
    assert noalloc(mocap_lib, **kwargs) == expect


def test_noalloc_forced_split_just_over_the_scratch(mocap_lib):
    # Forced 8-range plans of L rows x 32 heads at d 128 around the cap: every
    # plan whose workspace (as mocap_chunk_attn_workspace_size reports it)
    # exceeds MOCAP_NOALLOC_SCRATCH_BYTES is rejected with WORKSPACE before
    # anything is launched.  (Plans that fit would launch, so they are left to
    # the GPU test.)
    ws = mocap_lib.mocap_chunk_attn_workspace_size
    sizes = {L: ws(1 << 16, L, 32, 8, 128, 8)[1] for L in (1000, 1100, 1200, 1300)}
    assert min(sizes.values()) <= SCRATCH_BYTES < max(sizes.values())
    for L, b in sizes.items():
        if b > SCRATCH_BYTES:
            assert noalloc(mocap_lib, P=1 << 16, L=L, n_table=((1 << 16) + L) // 256 + 1, splits=8) == WORKSPACE


def test_noalloc_zero_length_chunk_is_a_noop(mocap_lib):
    assert noalloc(mocap_lib, L=0, q=0, o=0, lse=0) == 0
