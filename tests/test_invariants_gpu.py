"""Whole-output properties of the HIP path that hold at any size:
paged == contiguous bit for bit, run-to-run determinism, every output
written, split-KV on vs off, and latency-balanced vs uniform chunking of the
same 131072-token inputs."""
import numpy as np
import pytest
import torch

from helpers import O_MAX_ABS, O_MEAN_ABS, LSE_MAX_ABS, run_gpu, say, workload_inputs
from paper_2606_22968_amd import binding, synth
from paper_2606_22968_amd.prefill import ChunkedPrefill

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _all_lse(r):
    return torch.cat([r.lse(c).flatten() for c in range(len(r.lengths))])


def assert_bitwise_equal(a, b, label):
    assert torch.equal(_bits(a.o), _bits(b.o)), f"{label}: O differs"
    assert torch.equal(_bits(_all_lse(a)), _bits(_all_lse(b))), f"{label}: LSE differs"


def assert_close(a, b, label):
    e = (a.o.double() - b.o.double()).abs()
    le = (_all_lse(a).double() - _all_lse(b).double()).abs()
    say(f"[compare] {label}: O max {e.max().item():.3e} mean {e.mean().item():.3e} LSE max {le.max().item():.3e}")
    assert e.max().item() <= O_MAX_ABS and e.mean().item() <= O_MEAN_ABS and le.max().item() <= LSE_MAX_ABS


@pytest.mark.parametrize("splits", [1, 3, 0])
def test_paged_equals_contiguous_bitwise(gpu, splits):
    say(f"[case] paged vs contiguous, splits={splits}")
    lengths = [1024] * 6 + [300, 700]
    S = sum(lengths)
    q, k, v = synth.make_qkv(60, S, 32, 8, 128)
    n_blocks = (S + 255) // 256
    contiguous = run_gpu(q, k, v, lengths, 0.09, num_splits=splits)
    paged = run_gpu(q, k, v, lengths, 0.09, table=synth.permuted_table(n_blocks, 61, 2 * n_blocks),
                    pool_blocks=2 * n_blocks, num_splits=splits, pool_fill=float("nan"))
    assert_bitwise_equal(contiguous, paged, f"splits={splits}")


def test_paged_workload_equals_contiguous_bitwise(gpu):
    w = synth.WORKLOADS["llama8b_128k_paged"]
    say(f"[case] {w.name}: permuted vs identity table")
    q, k, v = workload_inputs(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, 1)
    n_blocks = w.seq_len // w.block_size
    paged = run_gpu(q, k, v, lengths, w.scale, table=synth.permuted_table(n_blocks, w.perm_seed))
    o_paged, lse_paged = paged.o.clone(), _all_lse(paged).clone()
    del paged
    # Same sequence in a larger pool: 768 blocks, the 256 unused ones all NaN.
    contiguous = run_gpu(q, k, v, lengths, w.scale, pool_blocks=768, pool_fill=float("nan"))
    assert torch.equal(_bits(contiguous.o), _bits(o_paged))
    assert torch.equal(_bits(_all_lse(contiguous)), _bits(lse_paged))


def test_deterministic_and_fully_written(gpu):
    say("[case] determinism + NaN-poisoned outputs")
    lengths = [640, 640, 1000, 33]
    S = sum(lengths)
    q, k, v = synth.make_qkv(62, S, 32, 8, 128)
    runs = []
    for _ in range(2):
        r = ChunkedPrefill(32, 8, 128, lengths, num_splits=0, pool_fill=float("nan"))
        r.o.fill_(float("nan"))
        r._lse_flat.fill_(float("nan"))
        r.workspace.fill_(255)
        run_gpu(q, k, v, lengths, 0.09, runner=r)
        assert torch.isfinite(r.o.float()).all()
        assert torch.isfinite(_all_lse(r)).all()
        runs.append(r)
    assert_bitwise_equal(runs[0], runs[1], "run 1 vs run 2")


def test_split_on_vs_off_70b_workload(gpu):
    w = synth.WORKLOADS["llama70b_64k_uniform"]
    say(f"[case] {w.name}: split auto vs off vs 5")
    q, k, v = workload_inputs(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, 1)
    off = run_gpu(q, k, v, lengths, w.scale, num_splits=1)
    o_off = off.o.clone()
    lse_off = _all_lse(off).clone()
    del off
    for splits in (0, 5):
        on = run_gpu(q, k, v, lengths, w.scale, num_splits=splits)
        e = (on.o.double() - o_off.double()).abs()
        le = (_all_lse(on).double() - lse_off.double()).abs()
        say(f"[compare] split {splits} (plan {on.splits[-1]}) vs off: O max {e.max().item():.3e} "
            f"LSE max {le.max().item():.3e}")
        assert e.max().item() <= O_MAX_ABS and e.mean().item() <= O_MEAN_ABS
        assert le.max().item() <= LSE_MAX_ABS
        del on


def test_balanced_equals_uniform_chunking(gpu):
    w = synth.WORKLOADS["llama8b_128k_balanced"]
    say(f"[case] {w.name}: balanced vs uniform chunking of the same inputs")
    q, k, v = workload_inputs(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    bal = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, w.align, balanced=True)
    uni = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, 1)
    a = run_gpu(q, k, v, bal, w.scale)
    o_a = a.o.clone()
    del a
    b = run_gpu(q, k, v, uni, w.scale)
    e = (b.o.double() - o_a.double()).abs()
    say(f"[compare] balanced vs uniform: O max {e.max().item():.3e} mean {e.mean().item():.3e}")
    assert e.max().item() <= O_MAX_ABS and e.mean().item() <= O_MEAN_ABS


def test_zero_length_chunk_leaves_outputs(gpu):
    store = binding.KvStore(4, 64, 2, 128)
    table = synth.identity_table(4).cuda()
    q = torch.empty((0, 8, 128), dtype=torch.bfloat16, device="cuda")
    o = torch.empty_like(q)
    lse = torch.empty((8, 0), dtype=torch.float32, device="cuda")
    binding.mocap_chunk_attn(store, table, q, 100, 0.1, o, lse)
    torch.cuda.synchronize()
