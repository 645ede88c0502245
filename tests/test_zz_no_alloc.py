"""The allocation-free entry point against the workspace entry point.

mocap_chunk_attn_noalloc keeps its split partials in the library's static
device scratch instead of a caller workspace.  Called through the C ABI on
the same inputs and plan, it must give the same bits as mocap_chunk_attn,
call after call: the scratch keeps the previous call's contents, so the
second call of each sequence is smaller than the first.
"""
import pytest
import torch

from helpers import say
from paper_2606_22968_amd import binding, synth

pytestmark = pytest.mark.gpu


def _setup(P, L, h_q, h_kv, d, seed, bs=256):
    S = P + L
    q, k, v = synth.make_qkv(seed, S, h_q, h_kv, d)
    nb = -(-S // bs)
    store = binding.KvStore(nb + 2, bs, h_kv, d, device="cuda", fill=float("nan"))
    table = synth.permuted_table(nb, seed + 1, pool_blocks=nb + 2).cuda()
    binding.mocap_kv_append(store, table, 0, k.cuda(), v.cuda())
    return store, table, q[P:].cuda().contiguous()


def _pair(store, table, q, P, scale, splits):
    L, h_q, d = q.shape
    n_ranges, ws_bytes = binding.mocap_chunk_attn_workspace_size(P, L, h_q, store.h_kv, d, splits)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda") if ws_bytes else None
    o_ref = torch.full_like(q, float("nan"))
    lse_ref = torch.full((h_q, L), float("nan"), dtype=torch.float32, device="cuda")
    binding.mocap_chunk_attn(store, table, q, P, scale, o_ref, lse_ref, workspace=ws, num_splits=splits)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((h_q, L), float("nan"), dtype=torch.float32, device="cuda")
    binding.mocap_chunk_attn_noalloc(store, table, q, P, scale, o, lse, num_splits=splits)
    torch.cuda.synchronize()
    return n_ranges, ws_bytes, o_ref, lse_ref, o, lse


# (first call, second call): (P, L, h_q, h_kv, d, num_splits, seed)
SEQUENCES = [
    ((3000, 700, 8, 2, 128, 5, 11), (500, 130, 8, 2, 128, 3, 12)),
    ((4096, 512, 32, 8, 128, 7, 13), (1024, 65, 32, 8, 128, 2, 14)),
    ((2500, 300, 16, 16, 64, 4, 15), (640, 1, 16, 16, 64, 3, 16)),
    ((65536, 256, 32, 8, 128, 0, 17), (16384, 128, 32, 8, 128, 0, 18)),  # automatic plans
]


@pytest.mark.parametrize("seq", range(len(SEQUENCES)))
def test_noalloc_equals_workspace_call(gpu, seq):
    for call, (P, L, h_q, h_kv, d, splits, seed) in enumerate(SEQUENCES[seq]):
        say(f"[case] noalloc sequence {seq} call {call}: P={P} L={L} h_q={h_q} h_kv={h_kv} d={d} splits={splits}")
        store, table, q = _setup(P, L, h_q, h_kv, d, seed)
        n_ranges, ws_bytes, o_ref, lse_ref, o, lse = _pair(store, table, q, P, d ** -0.5, splits)
        say(f"[case]   ranges {n_ranges}, partials {ws_bytes} bytes")
        assert n_ranges > 1 and 0 < ws_bytes <= binding.NOALLOC_SCRATCH_BYTES
        assert torch.isfinite(o_ref.float()).all() and torch.isfinite(lse_ref).all()
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(lse.view(torch.int32), lse_ref.view(torch.int32))


def test_noalloc_unsplit_and_too_large(gpu):
    store, table, q = _setup(0, 300, 8, 2, 128, 21)
    n_ranges, ws_bytes, o_ref, lse_ref, o, lse = _pair(store, table, q, 0, 128 ** -0.5, 0)
    assert n_ranges == 1 and ws_bytes == 0
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), lse_ref.view(torch.int32))
    # A forced plan whose partials do not fit the scratch is refused and
    # writes nothing.
    store, table, q = _setup(1 << 16, 2048, 32, 8, 128, 22)
    _, ws_bytes = binding.mocap_chunk_attn_workspace_size(1 << 16, 2048, 32, 8, 128, 9)
    assert ws_bytes > binding.NOALLOC_SCRATCH_BYTES
    o = torch.full_like(q, float("nan"))
    lse = torch.full((32, 2048), float("nan"), dtype=torch.float32, device="cuda")
    with pytest.raises(binding.MocapError) as err:
        binding.mocap_chunk_attn_noalloc(store, table, q, 1 << 16, 128 ** -0.5, o, lse, num_splits=9)
    assert err.value.status == binding.MOCAP_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(o.float()).all() and torch.isnan(lse).all()
