"""GPU parity: the HIP path against the fp64 oracle on the same seeded bf16
inputs.  Small shapes are compared on every output; the full-size workloads
on a seeded sample of rows (every chunk x every head x 8 rows), in the launch
configuration the benchmark times (automatic split planning)."""
import pytest
import torch

from helpers import check_chunks, run_gpu, say, workload_inputs
from paper_2606_22968_amd import binding, synth

pytestmark = pytest.mark.gpu


def test_small_d64_workload_all_rows(gpu, oracle_lib):
    w = synth.WORKLOADS["small_d64"]
    say(f"[case] {w.name}")
    q, k, v = workload_inputs(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, 1, balanced=False)
    runner = run_gpu(q, k, v, lengths, w.scale, block_size=w.block_size)
    check_chunks(oracle_lib, runner, q, k, v, w.scale, label=w.name)


@pytest.mark.parametrize("h_q,h_kv,d,lengths", [
    (32, 8, 128, [512, 512, 512, 512]),      # Llama-3-8B heads, short sequence
    (64, 8, 128, [256, 256, 256, 256]),      # Llama-3-70B heads, short sequence
])
def test_reduced_model_shapes_all_rows(gpu, oracle_lib, h_q, h_kv, d, lengths):
    say(f"[case] reduced h_q={h_q} h_kv={h_kv} d={d} lengths={lengths}")
    q, k, v = synth.make_qkv(20 + h_q, sum(lengths), h_q, h_kv, d)
    scale = d ** -0.5
    runner = run_gpu(q, k, v, lengths, scale)
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"reduced {h_q}/{h_kv}/{d}")


@pytest.mark.parametrize("h_q,h_kv,d", [(8, 8, 64), (8, 4, 128), (8, 2, 128), (16, 2, 64), (12, 4, 128),
                                        (32, 1, 128), (64, 1, 64), (6, 3, 128)])
def test_ragged_chunks_all_rows(gpu, oracle_lib, h_q, h_kv, d):
    # Chunk and prefix lengths that are not multiples of the 64-key tile, a
    # store of 64-position blocks, and NaN in every unwritten pool slot.
    lengths = [1, 7, 100, 129, 13, 255, 64, 3]
    say(f"[case] ragged h_q={h_q} h_kv={h_kv} d={d}")
    q, k, v = synth.make_qkv(30 + h_q + d, sum(lengths), h_q, h_kv, d)
    scale = 0.11
    runner = run_gpu(q, k, v, lengths, scale, block_size=64, pool_fill=float("nan"))
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"ragged {h_q}/{h_kv}/{d}")


@pytest.mark.parametrize("block_size,h_q,h_kv,d,splits", [(192, 8, 2, 128, 0), (320, 8, 4, 64, 3),
                                                          (448, 16, 4, 128, 2), (64 * 25, 4, 1, 128, 0)])
def test_block_sizes_not_powers_of_two(gpu, oracle_lib, block_size, h_q, h_kv, d, splits):
    # The kernel finds a position's block by multiply-and-shift division; a
    # permuted table and NaN in unwritten slots catch a wrong block or slot.
    lengths = [700, 129, 1000, 5, 64]
    say(f"[case] block_size={block_size} h_q={h_q} h_kv={h_kv} d={d} splits={splits}")
    q, k, v = synth.make_qkv(60 + block_size, sum(lengths), h_q, h_kv, d)
    n_blocks = -(-sum(lengths) // block_size)
    table = synth.permuted_table(n_blocks, 7 + block_size, pool_blocks=n_blocks + 3)
    scale = d ** -0.5
    runner = run_gpu(q, k, v, lengths, scale, block_size=block_size, table=table, pool_blocks=n_blocks + 3,
                     num_splits=splits, pool_fill=float("nan"))
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"block_size={block_size}")


@pytest.mark.parametrize("splits", [1, 2, 3, 7, 0])
def test_forced_splits(gpu, oracle_lib, splits):
    lengths = [1500, 37, 600, 1]
    say(f"[case] forced splits={splits}")
    q, k, v = synth.make_qkv(40, sum(lengths), 16, 4, 128)
    scale = 128 ** -0.5
    runner = run_gpu(q, k, v, lengths, scale, block_size=128, num_splits=splits)
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"splits={splits} plan={runner.splits}")


def _workload_plan(w):
    return binding.mocap_chunk_plan(w.seq_len, w.num_chunks, w.align, balanced=(w.chunking == "balanced"))


@pytest.mark.parametrize("name", ["llama8b_32k_uniform", "llama8b_128k_balanced", "llama70b_64k_uniform",
                                  "llama8b_128k_paged"])
def test_full_size_workload_sampled_rows(gpu, oracle_lib, name):
    w = synth.WORKLOADS[name]
    say(f"[case] {name}: generating inputs")
    q, k, v = workload_inputs(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    lengths = _workload_plan(w)
    n_blocks = w.seq_len // w.block_size
    table = synth.permuted_table(n_blocks, w.perm_seed) if w.permuted else None
    say(f"[case] {name}: GPU run, {len(lengths)} chunks")
    runner = run_gpu(q, k, v, lengths, w.scale, block_size=w.block_size, table=table)
    say(f"[case] {name}: splits per chunk {runner.splits}")
    check_chunks(oracle_lib, runner, q, k, v, w.scale,
                 rows_of=lambda c, n: synth.sample_rows(n, 1000 * w.seed + c), label=name)


@pytest.mark.parametrize("target", ["prefix", "diagonal"])
def test_score_far_above_first_block_reruns(gpu, oracle_lib, target):
    # One late key is 8 * q for every query of the last chunk, so its score
    # is ~90 natural-log units (~130 binary orders) above anything in the
    # first key block: the kernel's reference exponent overflows and the
    # kernel raises that row's reference exponent mid-range and rescales what
    # it has accumulated.  The output must still match the oracle.
    lengths = [1024, 256]
    S = sum(lengths)
    say(f"[case] overflow rescale, big key in the {target}")
    q, k, v = synth.make_qkv(70, S, 8, 2, 128)
    j = 900 if target == "prefix" else 1024 + 5
    qf = q.float()
    for h_kv in range(2):
        k[j, h_kv] = (8.0 * qf[1024 + 200, h_kv * 4]).to(torch.bfloat16)
    scale = 128 ** -0.5
    runner = run_gpu(q, k, v, lengths, scale)
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"overflow rescale ({target})")


@pytest.mark.parametrize("splits", [0, 1, 3])
@pytest.mark.parametrize("d", [64, 128])
def test_score_growing_over_several_blocks(gpu, oracle_lib, splits, d):
    # For one query row per KV head, three keys in different key blocks score
    # ~4, 8 and 12 times |q|^2 * scale: each one more than 60 binary orders
    # above the one before, so the row's reference exponent is raised three
    # times (the last time inside the chunk's own, masked, diagonal blocks),
    # across split ranges when the prefix is split.  Other rows of the group
    # see those keys at ordinary scores.
    lengths = [700, 300, 260]
    S = sum(lengths)
    h_q, h_kv = 8, 2
    g = h_q // h_kv
    say(f"[case] growing scores d={d} splits={splits}")
    q, k, v = synth.make_qkv(73 + d, S, h_q, h_kv, d)
    qf = q.float()
    row = 1000 + 200                      # a row of the last chunk
    mult = 128.0 / d                      # the same score scale at d = 64
    for h in range(h_kv):
        for pos, c in ((150, 4.0), (820, 8.0), (1000 + 70, 12.0)):
            k[pos + h, h] = (c * mult * qf[row + h, h * g]).to(torch.bfloat16)
    scale = d ** -0.5
    runner = run_gpu(q, k, v, lengths, scale, block_size=64, num_splits=splits)
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"growing scores d={d} splits={splits}")


def _random_config(index):
    """Seeded random shape: heads, head_dim, block size, chunk lengths, table
    and split count drawn independently (at most ~2500 tokens, 32 query heads)."""
    import random
    rng = random.Random(9000 + index)
    h_kv = rng.choice([1, 2, 4, 8])
    g = rng.choice([1, 2, 3, 4, 8])
    while h_kv * g > 32:
        g //= 2
    d = rng.choice([64, 128])
    block_size = rng.choice([64, 128, 192, 256, 320])
    lengths = [rng.choice([1, rng.randint(2, 63), rng.randint(64, 700)]) for _ in range(rng.randint(1, 6))]
    permuted = rng.random() < 0.5
    splits = rng.choice([0, 0, 1, 2, 3, 5])
    return h_kv * g, h_kv, d, block_size, lengths, permuted, splits


@pytest.mark.parametrize("index", range(24))
def test_random_configs_all_rows(gpu, oracle_lib, index):
    h_q, h_kv, d, block_size, lengths, permuted, splits = _random_config(index)
    say(f"[case] random #{index}: h_q={h_q} h_kv={h_kv} d={d} bs={block_size} lengths={lengths} "
        f"permuted={permuted} splits={splits}")
    q, k, v = synth.make_qkv(500 + index, sum(lengths), h_q, h_kv, d)
    n_blocks = -(-sum(lengths) // block_size)
    table = synth.permuted_table(n_blocks, 77 + index, pool_blocks=n_blocks + 2) if permuted else None
    scale = 0.7 * d ** -0.5
    runner = run_gpu(q, k, v, lengths, scale, block_size=block_size, table=table,
                     pool_blocks=(n_blocks + 2) if permuted else None, num_splits=splits, pool_fill=float("nan"))
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"random #{index}")
