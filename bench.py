"""Benchmark: chunked causal prefill attention on one MI355X.

One step = one pass of the whole hot path over one sequence: for every chunk
(in order) append its K/V to the block store, then run its attention over
the prefix and itself (split-KV and merge when the planner asks for them).
Inputs are seeded synthetic bf16 tensors already resident in HBM.

Prints ONE JSON line:
  value      causal TFLOP/s of the whole step (algorithmic FLOPs over visible
             (query, key) pairs: 4 * d * Hq * S (S + 1) / 2, divided by the
             step's wall time)
  roofline   the attention kernel's algorithmic FLOPs per launch over its
             average launch duration (HIP events on the launch stream), against
             the bf16 dense MFMA peak
  cpu_baseline  the fp64 oracle on this host's cores over a bounded sample
             of the same workload (every chunk x every head x 64 rows, about ten
             seconds on 16 cores)

Usage: python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16: 256 CUs x 4096 FLOP/clk x 2.4 GHz
METRIC = "chunked-prefill attention causal TFLOP/s & % bf16 MFMA peak; per-chunk latency"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b_32k_uniform")
    ap.add_argument("--splits", type=int, default=0, help="0 = library's automatic split plan")
    ap.add_argument("--remote-fraction", type=float, default=0.0,
                    help="hold the KV of the first fraction of the sequence (whole blocks) in a second store, "
                         "as a debtor stage's remote portion, and read it with the two-store call")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=64, help="oracle rows per (chunk, head)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (a known-size "
                         "kernel for scaling a profiler's FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def recorded_traffic(workload):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, calibrated against a device copy), or
    None when there is none for this workload or the kernel source changed
    since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"chunk_attn_{workload.replace('_uniform', '')}_traffic.json")
    src = os.path.join(ROOT, "paper_2606_22968_amd", "csrc", "chunk_attn.hip")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    with open(src, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != rec.get("kernel_source_sha256"):
            return None
    return rec["avg_traffic_bytes_per_launch"]


def causal_pairs(lengths):
    total, p = 0, 0
    for n in lengths:
        total += n * p + n * (n + 1) // 2
        p += n
    return total


def cpu_baseline(w, q, k, v, lengths, rows_per_chunk):
    """Time the fp64 oracle on a bounded sample of the workload."""
    import oracle
    from paper_2606_22968_amd import synth

    qb, kb, vb = synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v)
    flops, p = 0, 0
    t0 = time.perf_counter()
    for c, n in enumerate(lengths):
        rows = synth.sample_rows(n, 1000 * w.seed + c, n_random=max(rows_per_chunk - 5, 0))
        oracle.chunk_attn(qb[p:p + n], kb, vb, p, w.scale, rows=rows)
        flops += sum(4 * w.head_dim * w.h_q * (p + r + 1) for r in rows)
        p += n
    dt = time.perf_counter() - t0
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.max_threads(),
        "kind": "oracle",
        "sample": (f"{w.name}: every chunk x all {w.h_q} heads x {rows_per_chunk} rows "
                   f"(edges, middle, seeded random); {flops / 1e9:.1f} GFLOP fp64 in {dt:.1f} s; "
                   f"host has {os.cpu_count()} logical CPUs"),
    }


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: this build has no multi-GPU path "
              "(--gpus N with N > 1 is not supported).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_22968_amd import binding, synth
    from paper_2606_22968_amd.prefill import ChunkedPrefill

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    w = synth.WORKLOADS[args.workload]
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, w.align, balanced=(w.chunking == "balanced"))
    q, k, v = synth.make_qkv(w.seed, w.seq_len, w.h_q, w.h_kv, w.head_dim)
    n_blocks = (w.seq_len + w.block_size - 1) // w.block_size
    table = synth.permuted_table(n_blocks, w.perm_seed) if w.permuted else None
    remote = None
    if args.remote_fraction > 0:
        end = int(args.remote_fraction * w.seq_len) // w.block_size * w.block_size
        # A chunk boundary inside the range must sit on a 64-key tile: move the end back to one.
        while any(0 < p < end and p % 64 for p in synth.prefixes(lengths)):
            end -= w.block_size
        remote = (0, max(end, 0))
    runner = ChunkedPrefill(w.h_q, w.h_kv, w.head_dim, lengths, block_size=w.block_size, table=table,
                            num_splits=args.splits, remote=remote)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    stream = torch.cuda.current_stream()
    print(f"[bench] {w.name}: {len(lengths)} chunks, splits per chunk {runner.splits}", file=sys.stderr,
          flush=True)

    for _ in range(args.warmup):
        runner.run(qd, kd, vd, w.scale)
    torch.cuda.synchronize()

    n_chunks = len(lengths)
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_chunks)]
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        runner.run(qd, kd, vd, w.scale, stream=stream, events=ev[s])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    ms_per_step = elapsed * 1e3 / args.steps
    pairs = causal_pairs(lengths)
    flops = 4 * w.head_dim * w.h_q * pairs
    value = flops / (ms_per_step * 1e-3) / 1e12

    chunk_us = [statistics.median(ev[s][c][0].elapsed_time(ev[s][c][2]) * 1e3 for s in range(args.steps))
                for c in range(n_chunks)]
    attn_ms = [[ev[s][c][1].elapsed_time(ev[s][c][2]) for c in range(n_chunks)] for s in range(args.steps)]
    append_ms = [[ev[s][c][0].elapsed_time(ev[s][c][1]) for c in range(n_chunks)] for s in range(args.steps)]
    attn_total_ms = statistics.median(sum(x) for x in attn_ms)
    append_total_ms = statistics.median(sum(x) for x in append_ms)
    # Roofline of the attention kernel: average algorithmic FLOPs per launch
    # over the average launch duration.
    achieved = flops / (attn_total_ms * 1e-3) / 1e12
    split_chunks = sum(1 for r in runner.splits if r > 1)

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "description": w.note,
            "h_q": w.h_q, "h_kv": w.h_kv, "head_dim": w.head_dim,
            "seq_len": w.seq_len, "chunks": n_chunks, "chunking": w.chunking,
            "block_size": w.block_size, "block_table": "permuted" if w.permuted else "identity",
            "split_plan": runner.splits,
            "remote_kv": list(runner.remote) if runner.remote else None,
            "parallelism": "single GPU",
        },
        "pct_of_bf16_peak": round(100.0 * value / MFMA_BF16_PEAK_TFLOPS, 2),
        "per_chunk_us": [round(x, 1) for x in chunk_us],
        "per_chunk_max_over_min": round(max(chunk_us) / min(chunk_us), 2),
        "attention_ms_per_step": round(attn_total_ms, 4),
        "append_ms_per_step": round(append_total_ms, 4),
        "causal_flops_per_step": flops,
        "roofline": {
            "bound": "mfma",
            "kernel": f"chunk_attn_kernel<{w.head_dim}, {'true' if runner.remote else 'false'}>",
            "achieved": round(achieved, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": recorded_traffic(w.name),
            "traffic_unit": "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE)",
            "launches_per_step": n_chunks,
            "includes_merge_launches": split_chunks > 0,
        },
    }
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on host cores", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, q, k, v, lengths, args.cpu_rows)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
