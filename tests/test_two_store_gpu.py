"""Two-store attention (mocap_chunk_attn_two_store): prefix keys of one range
held by a second store, as a debtor stage's KV split into a remote and a
local portion under memory-balanced KV reallocation (Section 4.1).  Checked
against the oracle and, bit for bit, against the single-store path."""
import pytest
import torch

from helpers import check_chunks, say, workload_inputs
from paper_2606_22968_amd import binding, synth
from paper_2606_22968_amd.prefill import ChunkedPrefill

pytestmark = pytest.mark.gpu

NAN = float("nan")


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _poison_first_store(r, lo, hi):
    """NaN into the first store's slots of positions [lo, hi), so any read of
    them there would show in the output."""
    bs = r.block_size
    for pos in range(lo, hi, 64):  # 64-position pieces never cross a block (bs is a multiple of 64)
        blk = int(r.table[pos // bs].item())
        s0 = pos % bs
        r.store.k_pool[blk, :, s0:s0 + 64, :] = NAN
        r.store.v_pool[blk, :, :, s0:s0 + 64] = NAN


def _run(q, k, v, lengths, scale, **kw):
    """Chunk by chunk; with a remote range, the first store's copy of spilled
    positions is poisoned as soon as the chunk that produced them is done."""
    h_q, h_kv, d = q.shape[1], k.shape[1], q.shape[2]
    r = ChunkedPrefill(h_q, h_kv, d, lengths, **kw)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    for c, (p, n) in enumerate(zip(r.prefixes, r.lengths)):
        r.append(c, kd, vd)
        r.attend(c, qd, scale)
        if r.remote is not None:
            lo, hi = max(p, r.remote[0]), min(p + n, r.remote[1])
            if lo < hi:
                _poison_first_store(r, lo, hi)
    torch.cuda.synchronize()
    return r


@pytest.mark.parametrize("remote", [(512, 1536), (0, 1152), (1152, 2560), (0, 2560), (64, 128)])
@pytest.mark.parametrize("splits", [0, 1, 6])
def test_two_store_matches_oracle_all_rows(gpu, oracle_lib, remote, splits):
    lengths = [512, 640, 384, 1024, 77]
    h_q, h_kv, d = 8, 2, 128
    say(f"[case] two-store remote={remote} splits={splits} lengths={lengths}")
    q, k, v = synth.make_qkv(70, sum(lengths), h_q, h_kv, d)
    r = _run(q, k, v, lengths, 0.088, block_size=128, remote=remote, num_splits=splits, pool_fill=NAN)
    check_chunks(oracle_lib, r, q, k, v, 0.088, label=f"two-store {remote} splits={splits}")


def test_two_store_d64_permuted_tables(gpu, oracle_lib):
    lengths = [256, 320, 448, 200]
    h_q, h_kv, d = 16, 2, 64
    S = sum(lengths)
    say(f"[case] two-store d64, permuted tables, lengths={lengths}")
    q, k, v = synth.make_qkv(71, S, h_q, h_kv, d)
    n_blocks = (S + 63) // 64
    r = _run(q, k, v, lengths, 0.125, block_size=64, table=synth.permuted_table(n_blocks, 72, 2 * n_blocks),
             pool_blocks=2 * n_blocks, remote=(256, 1024),
             remote_table=synth.permuted_table(16, 73, 40), num_splits=0, pool_fill=NAN)
    check_chunks(oracle_lib, r, q, k, v, 0.125, label="two-store d64 permuted")


@pytest.mark.parametrize("remote", [(0, 2048), (1024, 3072), (64, 4096), (2048, 2112)])
@pytest.mark.parametrize("splits", [1, 3, 0])
def test_two_store_equals_single_store_bitwise(gpu, remote, splits):
    # The store is chosen per 64-key tile and the split plan is the
    # single-store plan, so the results equal the single-store run bit for
    # bit wherever the remote range's edges fall.
    lengths = [4096, 512, 700]
    say(f"[case] two-store vs single store, remote={remote} splits={splits}")
    q, k, v = synth.make_qkv(74, sum(lengths), 32, 8, 128)
    single = _run(q, k, v, lengths, 0.088, num_splits=splits)
    two = _run(q, k, v, lengths, 0.088, num_splits=splits, remote=remote, pool_fill=NAN)
    assert single.splits == two.splits
    assert torch.equal(_bits(single.o), _bits(two.o))
    for c in range(len(lengths)):
        assert torch.equal(_bits(single.lse(c)), _bits(two.lse(c)))


def test_empty_remote_range_is_single_store_bitwise(gpu):
    lengths = [1024, 1024, 333]
    say("[case] empty remote range")
    q, k, v = synth.make_qkv(75, sum(lengths), 32, 8, 128)
    single = _run(q, k, v, lengths, 0.088, num_splits=0)
    p, n = single.prefixes[2], single.lengths[2]
    o = torch.empty_like(single.o[p:p + n])
    lse = torch.empty_like(single.lse(2))
    qd = q.cuda()
    binding.mocap_chunk_attn_two_store(single.store, single.table, None, None, 1024, 1024, qd[p:p + n], p, 0.088,
                                       o, lse, single.workspace, 0)
    torch.cuda.synchronize()
    assert torch.equal(_bits(single.o[p:p + n]), _bits(o))
    assert torch.equal(_bits(single.lse(2)), _bits(lse))


def test_two_store_full_size_half_remote(gpu, oracle_lib):
    # 131072 tokens of the 8B shape in 32 chunks of 4096, the first half of the
    # sequence's KV held by the second store (a debtor that spilled half).
    w = synth.WORKLOADS["llama8b_128k_paged"]
    say(f"[case] {w.name} with KV [0, 65536) in a second store")
    q, k, v = workload_inputs(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, 1)
    n_blocks = w.seq_len // w.block_size
    two = _run(q, k, v, lengths, w.scale, table=synth.permuted_table(n_blocks, w.perm_seed),
               remote=(0, 65536), remote_table=synth.permuted_table(256, 105, 256))
    check_chunks(oracle_lib, two, q, k, v, w.scale,
                 rows_of=lambda c, n: synth.sample_rows(n, 900 + c, n_random=3),
                 label="128k half remote (sampled rows)")
    o_two = two.o.clone()
    del two
    single = _run(q, k, v, lengths, w.scale, table=synth.permuted_table(n_blocks, w.perm_seed))
    e = (single.o.double() - o_two.double()).abs()
    say(f"[compare] two-store vs single: O max {e.max().item():.3e} mean {e.mean().item():.3e}")
    assert e.max().item() <= 2e-2 and e.mean().item() <= 2e-3


def _random_two_store(index):
    """Seeded random two-store case: chunk lengths in whole tiles (the last
    one ragged), a tile-aligned remote range, random heads, head_dim, block
    size, tables and split count."""
    import random
    rng = random.Random(7000 + index)
    h_kv = rng.choice([1, 2, 4])
    h_q = h_kv * rng.choice([1, 2, 4])
    d = rng.choice([64, 128])
    block_size = rng.choice([64, 128, 192, 256])
    lengths = [64 * rng.randint(1, 10) for _ in range(rng.randint(2, 5))] + [rng.randint(1, 200)]
    tiles = sum(lengths[:-1]) // 64
    b = rng.randint(0, tiles - 1)
    e = rng.randint(b + 1, tiles)
    splits = rng.choice([0, 0, 1, 3])
    permuted = rng.random() < 0.5
    return h_q, h_kv, d, block_size, lengths, (64 * b, 64 * e), splits, permuted


@pytest.mark.parametrize("index", range(12))
def test_two_store_random_configs_all_rows(gpu, oracle_lib, index):
    h_q, h_kv, d, block_size, lengths, remote, splits, permuted = _random_two_store(index)
    S = sum(lengths)
    say(f"[case] two-store random #{index}: h_q={h_q} h_kv={h_kv} d={d} bs={block_size} lengths={lengths} "
        f"remote={remote} splits={splits} permuted={permuted}")
    q, k, v = synth.make_qkv(600 + index, S, h_q, h_kv, d)
    kw = dict(block_size=block_size, remote=remote, num_splits=splits, pool_fill=NAN)
    if permuted:
        n_blocks = -(-S // block_size)
        n_remote = -(-remote[1] // block_size)
        kw.update(table=synth.permuted_table(n_blocks, 80 + index, n_blocks + 3), pool_blocks=n_blocks + 3,
                  remote_table=synth.permuted_table(n_remote, 90 + index, n_remote + 2))
    scale = d ** -0.5
    r = _run(q, k, v, lengths, scale, **kw)
    check_chunks(oracle_lib, r, q, k, v, scale, label=f"two-store random #{index}")
