"""mocap_kv_append: the block-table gather must return exactly the bytes
appended, wherever the table puts the blocks, and touch nothing else."""
import pytest
import torch

from helpers import say
from paper_2606_22968_amd import binding, synth

pytestmark = pytest.mark.gpu


def gather(store, table, seq_len):
    """Read positions [0, seq_len) back through the table (test-side indexing)."""
    pos = torch.arange(seq_len, device=store.k_pool.device)
    blk = table.long()[pos // store.block_size]
    slot = pos % store.block_size
    k = store.k_pool[blk, :, slot, :]                        # [S][Hkv][D]
    v = store.v_pool.permute(0, 3, 1, 2)[blk, slot, :, :]    # [S][Hkv][D]
    return k, v


@pytest.mark.parametrize("permuted", [False, True])
@pytest.mark.parametrize("h_kv,d,bs,lengths", [
    (8, 128, 256, [2048, 2048, 1024]),
    (2, 64, 64, [13, 100, 1, 129, 64, 77]),
    (4, 128, 128, [5, 300, 211]),
    (2, 64, 64, [32, 96, 160, 7, 25]),          # 32-aligned starts inside 64-slot blocks
    (8, 128, 256, [2080, 32, 2016, 33]),
])
def test_gather_is_bit_exact(gpu, permuted, h_kv, d, bs, lengths):
    say(f"[case] append h_kv={h_kv} d={d} bs={bs} permuted={permuted}")
    S = sum(lengths)
    n_blocks = (S + bs - 1) // bs
    pool_blocks = 2 * n_blocks + 1
    table = (synth.permuted_table(n_blocks, 7, pool_blocks) if permuted else synth.identity_table(n_blocks)).cuda()
    store = binding.KvStore(pool_blocks, bs, h_kv, d, fill=float("nan"))
    k_before = store.k_pool.view(torch.int16).clone()
    v_before = store.v_pool.view(torch.int16).clone()
    _, k, v = synth.make_qkv(50 + h_kv, S, 1, h_kv, d)
    k, v = k.cuda(), v.cuda()
    p = 0
    for n in lengths:
        binding.mocap_kv_append(store, table, p, k[p:p + n], v[p:p + n])
        p += n
    torch.cuda.synchronize()
    gk, gv = gather(store, table, S)
    assert torch.equal(gk.view(torch.int16), k.view(torch.int16))
    assert torch.equal(gv.view(torch.int16), v.view(torch.int16))
    # Every slot not addressed by a position keeps its old bits.
    touched = torch.zeros(pool_blocks, bs, dtype=torch.bool, device="cuda")
    pos = torch.arange(S, device="cuda")
    touched[table.long()[pos // bs], pos % bs] = True
    ku = ~touched[:, None, :, None].expand_as(store.k_pool)
    vu = ~touched[:, None, None, :].expand_as(store.v_pool)
    assert torch.equal(store.k_pool.view(torch.int16)[ku], k_before[ku])
    assert torch.equal(store.v_pool.view(torch.int16)[vu], v_before[vu])


def test_empty_append_changes_nothing(gpu):
    store = binding.KvStore(2, 64, 1, 64, fill=1.0)
    table = synth.identity_table(2).cuda()
    before = store.k_pool.clone()
    empty = torch.empty((0, 1, 64), dtype=torch.bfloat16, device="cuda")
    binding.mocap_kv_append(store, table, 10, empty, empty)
    torch.cuda.synchronize()
    assert torch.equal(store.k_pool, before)
