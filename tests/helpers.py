"""Shared pieces of the GPU parity tests: run the HIP path, run the oracle on
the same seeded bf16 inputs, and measure the error."""
import functools
import sys

import numpy as np
import torch

from paper_2606_22968_amd import synth
from paper_2606_22968_amd.prefill import ChunkedPrefill

# Parity bar for O (bf16 in, fp32 accumulate): max-abs and mean-abs error
# against the fp64 oracle.
O_MAX_ABS = 2e-2
O_MEAN_ABS = 2e-3
# LSE bar (no bar is stated for it): max-abs 1e-3 in natural-log units.  The
# kernel takes the log-sum-exp from fp32 sums of the unrounded exponentials
# (fp32 exp2 and accumulation: relative errors of order 1e-6 on ordinary rows);
# the bf16 rounding of the probabilities only enters O, whose normaliser sums
# the same rounded values that feed P*V.
LSE_MAX_ABS = 1e-3


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=3)
def workload_inputs(seed, seq_len, h_q, h_kv, head_dim):
    return synth.make_qkv(seed, seq_len, h_q, h_kv, head_dim)


def run_gpu(q, k, v, lengths, scale, block_size=256, table=None, pool_blocks=None, num_splits=0,
            pool_fill=None, runner=None):
    """Full chunk sequence on the GPU; returns the runner (outputs on device)."""
    h_q, h_kv, d = q.shape[1], k.shape[1], q.shape[2]
    if runner is None:
        runner = ChunkedPrefill(h_q, h_kv, d, lengths, block_size=block_size, table=table,
                                pool_blocks=pool_blocks, num_splits=num_splits, pool_fill=pool_fill)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    runner.run(qd, kd, vd, scale)
    torch.cuda.synchronize()
    return runner


def oracle_chunk(oracle, q, k, v, prefix, length, scale, rows=None):
    qb = synth.bf16_bits(q[prefix:prefix + length])
    kb = synth.bf16_bits(k[:prefix + length])
    vb = synth.bf16_bits(v[:prefix + length])
    return oracle.chunk_attn(qb, kb, vb, prefix, scale, rows=rows)


def errors(gpu_o, gpu_lse, ref_o, ref_lse):
    """gpu_o bf16 [n][Hq][d], gpu_lse fp32 [Hq][n] (CPU tensors); refs fp64."""
    e = np.abs(gpu_o.double().numpy() - ref_o)
    le = np.abs(gpu_lse.double().numpy() - ref_lse)
    return float(e.max()), float(e.mean()), float(le.max())


def check_chunks(oracle, runner, q, k, v, scale, rows_of=None, label=""):
    """Compare every chunk of a run with the oracle (all rows, or rows_of(c, L))."""
    worst = [0.0, 0.0, 0.0]
    total_abs, total_n = 0.0, 0
    for c, (p, n) in enumerate(zip(runner.prefixes, runner.lengths)):
        rows = None if rows_of is None else rows_of(c, n)
        ref_o, ref_lse = oracle_chunk(oracle, q, k, v, p, n, scale, rows=rows)
        o = runner.o[p:p + n].cpu()
        lse = runner.lse(c).cpu()
        if rows is not None:
            o, lse = o[rows], lse[:, rows]
        mx, mean, lmx = errors(o, lse, ref_o, ref_lse)
        assert np.isfinite(mx) and np.isfinite(lmx), f"{label} chunk {c}: non-finite output"
        worst[0] = max(worst[0], mx)
        worst[2] = max(worst[2], lmx)
        total_abs += mean * ref_o.size
        total_n += ref_o.size
    worst[1] = total_abs / max(total_n, 1)
    say(f"[parity] {label}: O max-abs {worst[0]:.3e} mean-abs {worst[1]:.3e} LSE max-abs {worst[2]:.3e}")
    assert worst[0] <= O_MAX_ABS, f"{label}: O max-abs {worst[0]}"
    assert worst[1] <= O_MEAN_ABS, f"{label}: O mean-abs {worst[1]}"
    assert worst[2] <= LSE_MAX_ABS, f"{label}: LSE max-abs {worst[2]}"
    return worst
