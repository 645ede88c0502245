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
  clock      the attention kernel's average graphics clock from the committed
             rocprofv3 counter profile of this workload (GRBM_GUI_ACTIVE cycles
             per XCD over each dispatch's duration), when that profile was
             taken on the current kernel source; and the kernel's fraction of
             the bf16 peak at that clock (256 CUs x 4096 FLOP per clock)
  cpu_baseline  the fp64 oracle on this host's cores: the 1024-token d64
             workload in full, then the parity row sample of the benchmark
             workload (every chunk x every head x 8 rows) and its last chunk
             in full; the measured fp64 rate, and the full workload's oracle
             time projected from it (about a minute of CPU work)

Usage: python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
       python bench.py --summarize-trace KERNEL_TRACE_CSV [--steps K] [--workload NAME]
           (summary of the attention launches of the timed steps in a
            rocprofv3 --kernel-trace run of this script)
       python bench.py --summarize-counters DIR --copy-calibration-mib M [--steps K] [--workload NAME]
           (summary of three rocprofv3 --pmc runs of this script with
            --copy-calibration-mib, written under DIR/fetch (FETCH_SIZE),
            DIR/write (WRITE_SIZE) and DIR/sq (GRBM_GUI_ACTIVE and SQ
            counters); writes profiles/chunk_attn_<workload>_counters.json)
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
FLOP_PER_CLOCK = 256 * 4096      # dense bf16 MFMA FLOP per clock over the whole chip
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
    ap.add_argument("--dominant-key", action="store_true",
                    help="plant, for every KV head, one key of the last chunk at 8x a later query of that "
                         "chunk, so that query's score sits ~130 binary orders above its first key block and "
                         "the kernel raises that row's reference exponent and rescales it (times the data-dependent slow path)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=8, help="oracle sample rows per (chunk, head)")
    ap.add_argument("--summarize-trace", default=None,
                    help="print a summary of a rocprofv3 kernel trace of this script and exit")
    ap.add_argument("--summarize-counters", default=None,
                    help="summarize rocprofv3 --pmc runs of this script (see usage) and exit")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (a known-size "
                         "kernel for scaling a profiler's FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def recorded_counters(workload):
    """Counter figures of the attention kernel from the committed rocprofv3
    summary of this workload (HBM bytes per launch from FETCH_SIZE and
    WRITE_SIZE scaled by a device-copy calibration; average clock from
    GRBM_GUI_ACTIVE), or None when there is none or the kernel source changed
    since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"chunk_attn_{workload}_counters.json")
    src = os.path.join(ROOT, "paper_2606_22968_amd", "csrc", "chunk_attn.hip")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    with open(src, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != rec.get("kernel_source_sha256"):
            return None
    return rec


def causal_pairs(lengths):
    total, p = 0, 0
    for n in lengths:
        total += n * p + n * (n + 1) // 2
        p += n
    return total


def cpu_baseline(w, q, k, v, lengths, rows_per_chunk):
    """Time the fp64 oracle: the small workload in full, then a row sample of
    the benchmark workload and its last chunk in full."""
    import oracle
    from paper_2606_22968_amd import synth

    def run_chunks(wl, qb, kb, vb, plan, rows_of):
        flops, p = 0, 0
        for c, n in enumerate(plan):
            rows = rows_of(c, n)
            oracle.chunk_attn(qb[p:p + n], kb[:p + n], vb[:p + n], p, wl.scale, rows=rows)
            rows = range(n) if rows is None else rows
            flops += sum(4 * wl.head_dim * wl.h_q * (p + r + 1) for r in rows)
            p += n
        return flops

    w0 = synth.WORKLOADS["small_d64"]
    q0, k0, v0 = synth.make_qkv(w0.seed, w0.seq_len, w0.h_q, w0.h_kv, w0.head_dim)
    plan0 = [w0.seq_len // w0.num_chunks] * w0.num_chunks
    t0 = time.perf_counter()
    f0 = run_chunks(w0, synth.bf16_bits(q0), synth.bf16_bits(k0), synth.bf16_bits(v0), plan0, lambda c, n: None)
    small_s = time.perf_counter() - t0

    qb, kb, vb = synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v)
    t0 = time.perf_counter()
    f_rows = run_chunks(w, qb, kb, vb, lengths, lambda c, n: synth.sample_rows(
        n, 1000 * w.seed + c, n_random=max(rows_per_chunk - 5, 0)))
    rows_s = time.perf_counter() - t0
    p_last, n_last = sum(lengths[:-1]), lengths[-1]
    t0 = time.perf_counter()
    oracle.chunk_attn(qb[p_last:], kb, vb, p_last, w.scale)
    last_s = time.perf_counter() - t0
    f_last = 4 * w.head_dim * w.h_q * (n_last * p_last + n_last * (n_last + 1) // 2)
    rate = (f_rows + f_last) / (rows_s + last_s)
    full = 4 * w.head_dim * w.h_q * causal_pairs(lengths)
    return {
        "value": rate / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.max_threads(),
        "kind": "oracle",
        "sample": (f"{w0.name} in full ({f0 / 1e9:.2f} GFLOP, {small_s:.2f} s); {w.name}: every chunk x "
                   f"{w.h_q} heads x {rows_per_chunk} rows ({f_rows / 1e9:.0f} GFLOP, {rows_s:.1f} s) and the "
                   f"last chunk in full ({f_last / 1e12:.3f} TFLOP, {last_s:.1f} s); fp64, "
                   f"{os.cpu_count()} logical CPUs"),
        "gflops_fp64": round(rate / 1e9, 2),
        "small_d64_full_s": round(small_s, 3),
        "last_chunk_full_s": round(last_s, 2),
        "projected_full_s": round(full / rate, 1),
        "projected": True,
    }


def summarize_trace(path, workload, steps):
    """Attention launches of the last `steps` steps of a rocprofv3 kernel trace
    (CSV) of this script: the timed passes, without the warm-up ones."""
    import csv
    from paper_2606_22968_amd import binding, synth
    w = synth.WORKLOADS[workload]
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, w.align, balanced=(w.chunking == "balanced"))
    rows = list(csv.DictReader(open(path)))
    attn = [r for r in rows if "chunk_attn_kernel" in r["Kernel_Name"]]
    n = steps * len(lengths)
    if len(attn) < n:
        raise SystemExit(f"{path}: {len(attn)} attention launches, fewer than {steps} steps x {len(lengths)}")
    timed = attn[-n:]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3 for r in timed]  # us
    per_chunk = [statistics.median(dur[s * len(lengths) + c] for s in range(steps)) for c in range(len(lengths))]
    flops = 4 * w.head_dim * w.h_q * causal_pairs(lengths)
    step_us = sum(dur) / steps
    achieved = flops / (step_us * 1e-6) / 1e12
    names = sorted({r["Kernel_Name"] for r in timed})
    print(f"kernel(s): {', '.join(names)}")
    print(f"timed steps: {steps} x {len(lengths)} launches (the last {n} attention launches of the trace)")
    print(f"average launch: {statistics.mean(dur):.1f} us; attention per step: {step_us / 1e3:.4f} ms")
    print(f"achieved: {achieved:.1f} TFLOP/s = {achieved / MFMA_BF16_PEAK_TFLOPS:.4f} of {MFMA_BF16_PEAK_TFLOPS}")
    print("per-chunk median us: " + ", ".join(f"{x:.1f}" for x in per_chunk))


XCDS = 8  # MI355X: GRBM_GUI_ACTIVE is reported summed over the 8 accelerator complex dies


def _counter_rows(path):
    """Rows of a rocprofv3 counter_collection.csv as (dispatch id, kernel,
    counter, value, start ns, end ns)."""
    import csv
    out = []
    with open(path) as f:
        for r in csv.DictReader(f):
            out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"]),
                        int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    return out


def _per_dispatch(rows, match):
    """{dispatch id: (kernel, {counter: value}, start, end)} for kernels whose name contains `match`."""
    d = {}
    for did, name, ctr, val, t0, t1 in rows:
        if match in name:
            d.setdefault(did, (name, {}, t0, t1))[1][ctr] = val
    return dict(sorted(d.items()))


def summarize_counters(root, workload, steps, calib_mib):
    """HBM bytes and average clock of the attention launches of the timed
    steps, from rocprofv3 --pmc runs of this script (one run per counter
    group, each with --copy-calibration-mib).  FETCH_SIZE and WRITE_SIZE are
    scaled so that the calibration copy (the largest device copy of the run)
    reads and writes its known size; the clock is the least-squares slope of
    GRBM_GUI_ACTIVE per die against each launch's duration, which removes the
    fixed per-dispatch part of the counter window."""
    import glob
    import hashlib
    from paper_2606_22968_amd import binding, synth
    w = synth.WORKLOADS[workload]
    lengths = binding.mocap_chunk_plan(w.seq_len, w.num_chunks, w.align, balanced=(w.chunking == "balanced"))
    n = steps * len(lengths)

    def load(sub):
        files = glob.glob(os.path.join(root, sub, "**", "*counter_collection.csv"), recursive=True)
        if len(files) != 1:
            raise SystemExit(f"{root}/{sub}: expected one counter_collection.csv, found {len(files)}")
        rows = _counter_rows(files[0])
        attn = list(_per_dispatch(rows, "chunk_attn_kernel").values())
        if len(attn) < n:
            raise SystemExit(f"{files[0]}: {len(attn)} attention launches, fewer than {steps} x {len(lengths)}")
        copies = list(_per_dispatch(rows, "copyBuffer").values())
        append = list(_per_dispatch(rows, "kv_append_kernel").values())
        return attn[-n:], copies, append[-n:]

    calib_bytes = None
    scales, per_launch = {}, {}
    for sub, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        attn, copies, append = load(sub)
        # The calibration copy (the run's largest device copy) reads and
        # writes calib_mib MiB.
        big = max(copies, key=lambda c: c[1].get(ctr, 0.0))
        kib = big[1][ctr]
        calib_bytes = calib_mib * 2**20
        scales[ctr] = calib_bytes / (kib * 1024)
        per_launch[ctr] = statistics.mean(a[1][ctr] for a in attn) * 1024 * scales[ctr]
        per_launch["append_" + ctr] = statistics.mean(a[1][ctr] for a in append) * 1024 * scales[ctr]
    attn, _, append = load("sq")
    dur = [(a[3] - a[2]) for a in attn]  # ns
    cyc = [a[1]["GRBM_GUI_ACTIVE"] / XCDS for a in attn]
    md, mc = statistics.mean(dur), statistics.mean(cyc)
    slope = sum((d - md) * (c - mc) for d, c in zip(dur, cyc)) / sum((d - md) ** 2 for d in dur)
    intercept = mc - slope * md
    sums = {}
    for a in attn:
        for k, v in a[1].items():
            sums[k] = sums.get(k, 0.0) + v
    app = {}
    for a in append:
        for k, v in a[1].items():
            app[k] = app.get(k, 0.0) + v
    src = os.path.join(ROOT, "paper_2606_22968_amd", "csrc", "chunk_attn.hip")
    with open(src, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    rec = {
        "kernel": attn[0][0],
        "workload": workload,
        "kernel_source_sha256": sha,
        "launches": n,
        "calibration_copy_bytes": calib_bytes,
        "fetch_scale": scales["FETCH_SIZE"],
        "write_scale": scales["WRITE_SIZE"],
        "avg_fetch_bytes_per_launch": per_launch["FETCH_SIZE"],
        "avg_write_bytes_per_launch": per_launch["WRITE_SIZE"],
        "avg_traffic_bytes_per_launch": per_launch["FETCH_SIZE"] + per_launch["WRITE_SIZE"],
        "avg_clock_ghz": round(slope, 4),
        "clock_fit_intercept_cycles": round(intercept, 1),
        "sq_totals": sums,
        "kv_append": {
            "kernel": append[0][0] if append else None,
            "avg_fetch_bytes_per_launch": per_launch["append_FETCH_SIZE"],
            "avg_write_bytes_per_launch": per_launch["append_WRITE_SIZE"],
            "sq_totals": app,
        },
    }
    out = os.path.join(ROOT, "profiles", f"chunk_attn_{workload}_counters.json")
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    mfma = sums.get("SQ_INSTS_MFMA", 0.0)
    busy_cycles = sum(cyc)
    print(f"kernel: {rec['kernel']} ({n} launches of the timed step(s)); source sha256 {sha[:16]}")
    print(f"calibration copy {calib_bytes / 2**20:.0f} MiB: FETCH_SIZE x {scales['FETCH_SIZE']:.4f}, "
          f"WRITE_SIZE x {scales['WRITE_SIZE']:.4f}")
    print(f"HBM bytes per launch: fetched {per_launch['FETCH_SIZE']:.4e}, written {per_launch['WRITE_SIZE']:.4e}, "
          f"total {rec['avg_traffic_bytes_per_launch']:.4e}")
    print(f"clock: {slope:.3f} GHz (slope of GRBM_GUI_ACTIVE / {XCDS} over duration; "
          f"intercept {intercept:.0f} cycles per launch)")
    for k in sorted(sums):
        extra = f"  ({sums[k] / mfma:.2f} per MFMA)" if mfma and k.startswith("SQ_INSTS") else ""
        print(f"  {k}: {sums[k]:.4e}{extra}")
    if "SQ_VALU_MFMA_BUSY_CYCLES" in sums and busy_cycles > 0:
        # 4 SIMDs x 32 CUs per die: MFMA-busy cycles per SIMD over the die's active cycles.
        print(f"MFMA unit busy: {sums['SQ_VALU_MFMA_BUSY_CYCLES'] / (busy_cycles * 1024):.3f} of active cycles")
    if append:
        print(f"kv_append ({len(append)} launches): fetched {per_launch['append_FETCH_SIZE']:.4e}, written "
              f"{per_launch['append_WRITE_SIZE']:.4e} bytes per launch; "
              + ", ".join(f"{k} {v:.4e}" for k, v in sorted(app.items())))
    print(f"wrote {os.path.relpath(out, ROOT)}")


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.workload, args.steps)
        return
    if args.summarize_counters:
        if args.copy_calibration_mib <= 0:
            raise SystemExit("--summarize-counters needs the --copy-calibration-mib of the profiled runs")
        summarize_counters(args.summarize_counters, args.workload, args.steps, args.copy_calibration_mib)
        return
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
    planted = None
    if args.dominant_key:
        p_last = synth.prefixes(lengths)[-1]
        key, row = p_last + 5, p_last + min(200, lengths[-1] - 1)
        g = w.h_q // w.h_kv
        for h in range(w.h_kv):
            k[key, h] = (8.0 * q[row, h * g].float()).to(torch.bfloat16)
        planted = {"key": key, "query_row": row}
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
    counters = recorded_counters(w.name)
    clk = None
    if counters and counters.get("avg_clock_ghz"):
        peak_at_clock = FLOP_PER_CLOCK * counters["avg_clock_ghz"] * 1e9 / 1e12
        clk = {"ghz": counters["avg_clock_ghz"], "peak_tflops_at_clock": round(peak_at_clock, 1),
               "frac_at_clock": round(achieved / peak_at_clock, 4),
               "source": f"profiles/chunk_attn_{w.name}_counters.json (rocprofv3 GRBM_GUI_ACTIVE)"}

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
            "dominant_key": planted,
            "parallelism": "single GPU",
        },
        "pct_of_bf16_peak": round(100.0 * value / MFMA_BF16_PEAK_TFLOPS, 2),
        "clock": clk,
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
            "traffic": counters.get("avg_traffic_bytes_per_launch") if counters else None,
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
