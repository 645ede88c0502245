"""Latency-balanced chunk partitioning, first stage, driven by measured latency.

The paper's LBCP (Section 4.2, Alg. 1) starts from a dynamic program whose
EvaluateChunk(k, s) returns the compute latency of a chunk of k tokens
starting at s.  Here that latency is the measured time of this library's
per-chunk calls (mocap_kv_append followed by mocap_chunk_attn) on the current
GPU, summarised by the model of Eq. (1):

    t(c, p) = cost_pair * (c p + c (c + 1) / 2) + cost_token * c + cost_chunk

(visible (query, key) pairs, tokens, and a fixed per-chunk cost), fitted by
non-negative least squares in relative error.  The dynamic program itself
runs in the library (mocap_lbcp_plan).

Run as a module to measure, fit, plan and compare against the closed-form
balanced plan:

    python -m paper_2606_22968_amd.lbcp --workload llama8b_128k_balanced --stages 16

With --layer, EvaluateChunk is the latency of a whole decoder layer per chunk
(projections and feed-forward network included, layer.py), so both terms of
Eq. (1) enter the model.

With --stage2 the command also measures a (length, prefix) grid, builds a
chunk-cost table and runs the second stage of Alg. 1 (mocap_lbcp_refine, the
single-request refinement); --e2e adds the serving model of the second stage
(mocap_lbcp_refine_e2e: the feasible batch under per-stage KV capacity, with
and without the cross-half pairing of Section 4.1, and the end-to-end
latency of a queue of requests) for several capacities.
"""
import argparse
import json
import random
import statistics
import sys
from dataclasses import dataclass
from typing import List, Sequence, Tuple

from . import binding


@dataclass(frozen=True)
class LatencyModel:
    cost_pair: float   # microseconds per visible (query, key) pair
    cost_token: float  # microseconds per chunk token
    cost_chunk: float  # microseconds per chunk
    rms_rel_err: float  # of the fit over its samples

    def __call__(self, c: int, p: int) -> float:
        return self.cost_pair * (c * p + c * (c + 1) / 2.0) + self.cost_token * c + self.cost_chunk


def visible_pairs(c: int, p: int) -> int:
    return c * p + c * (c + 1) // 2


def fit(samples: Sequence[Tuple[int, int, float]]) -> LatencyModel:
    """Non-negative least squares of (c, p, microseconds) samples, each row
    weighted by 1 / latency so that short and long chunks count alike."""
    import numpy as np
    from scipy.optimize import nnls

    if len(samples) < 3:
        raise ValueError("need at least three latency samples")
    a = np.array([[visible_pairs(c, p), c, 1.0] for c, p, _ in samples], dtype=np.float64)
    y = np.array([t for _, _, t in samples], dtype=np.float64)
    if not np.all(y > 0):
        raise ValueError("latencies must be positive")
    w = 1.0 / y
    col = a.max(axis=0)  # column scaling keeps the solve well conditioned
    x, _ = nnls(a * w[:, None] / col, y * w)
    x = x / col
    rel = (a @ x - y) / y
    return LatencyModel(float(x[0]), float(x[1]), float(x[2]), float(np.sqrt(np.mean(rel ** 2))))


def plan(seq_len: int, num_chunks: int, num_stages: int, align: int, model: LatencyModel):
    """Alg. 1's dynamic program under the model; returns (lengths, t_max, t_sum)."""
    return binding.mocap_lbcp_plan(seq_len, num_chunks, num_stages, align, model.cost_pair,
                                   model.cost_token, model.cost_chunk)


def probe_plans(seq_len: int, num_chunks: int, align: int, seed: int = 0, n_random: int = 4) -> List[List[int]]:
    """Chunk plans whose chunks cover a wide range of (length, prefix): the
    uniform and closed-form balanced plans plus seeded random compositions."""
    plans = [binding.mocap_chunk_plan(seq_len, num_chunks, align, balanced=False),
             binding.mocap_chunk_plan(seq_len, num_chunks, align, balanced=True)]
    rng = random.Random(seed)
    units = seq_len // align
    for _ in range(n_random):
        cuts = sorted(rng.sample(range(1, units), num_chunks - 1))
        bounds = [0] + cuts + [units]
        plans.append([(b - a) * align for a, b in zip(bounds[:-1], bounds[1:])])
    return plans


def measure(h_q: int, h_kv: int, head_dim: int, plans: Sequence[Sequence[int]], scale: float,
            block_size: int = 256, reps: int = 3, seed: int = 0, num_splits: int = 0):
    """Median per-chunk latency (microseconds, append + attention, HIP events
    on the launch stream) of every chunk of every plan.  Returns
    [(plan_index, chunk_len, prefix_len, microseconds)]."""
    import torch

    from . import synth
    from .prefill import ChunkedPrefill

    seq_len = sum(plans[0])
    if any(sum(p) != seq_len for p in plans):
        raise ValueError("every plan must cover the same sequence")
    q, k, v = (t.cuda() for t in synth.make_qkv(seed, seq_len, h_q, h_kv, head_dim))
    stream = torch.cuda.current_stream()
    out = []
    for i, lengths in enumerate(plans):
        runner = ChunkedPrefill(h_q, h_kv, head_dim, lengths, block_size=block_size, num_splits=num_splits)
        runner.run(q, k, v, scale, stream=stream)  # warm-up
        ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in lengths] for _ in range(reps)]
        for r in range(reps):
            runner.run(q, k, v, scale, stream=stream, events=ev[r])
        torch.cuda.synchronize()
        for c, (n, p) in enumerate(zip(runner.lengths, runner.prefixes)):
            us = statistics.median(ev[r][c][0].elapsed_time(ev[r][c][2]) * 1e3 for r in range(reps))
            out.append((i, n, p, us))
        del runner
    return out


def measure_layer(shape, plans: Sequence[Sequence[int]], reps: int = 3, seed: int = 0, block_size: int = 256):
    """As measure(), for a whole decoder layer per chunk (layer.ChunkedLayer):
    returns [(plan_index, chunk_len, prefix_len, total_us, attention_us, gemm_us)],
    attention_us covering mocap_kv_append + mocap_chunk_attn and gemm_us the
    projections and the feed-forward network."""
    import torch

    from .layer import ChunkedLayer

    seq_len = sum(plans[0])
    if any(sum(p) != seq_len for p in plans):
        raise ValueError("every plan must cover the same sequence")
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    x = torch.randn((seq_len, shape.hidden), generator=g, dtype=torch.float32).to(torch.bfloat16).cuda()
    scale = shape.head_dim ** -0.5
    stream = torch.cuda.current_stream()
    out = []
    for i, lengths in enumerate(plans):
        layer = ChunkedLayer(shape, lengths, seed=seed, block_size=block_size)
        layer.run(x, scale, stream=stream)  # warm-up
        ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in lengths] for _ in range(reps)]
        for r in range(reps):
            layer.run(x, scale, stream=stream, events=ev[r])
        torch.cuda.synchronize()
        for c, (n, p) in enumerate(zip(layer.lengths, layer.prefixes)):
            def med(a, b):
                return statistics.median(ev[r][c][a].elapsed_time(ev[r][c][b]) * 1e3 for r in range(reps))
            total, attn = med(0, 3), med(1, 2)
            out.append((i, n, p, total, attn, total - attn))
        del layer
    return out


def measure_grid(shape, seq_len: int, c_grid: Sequence[int], p_fracs: Sequence[float], align: int,
                 reps: int = 3, seed: int = 0, block_size: int = 256, attn=None):
    """Latency (microseconds) of single chunks at chosen (length, prefix)
    points, every chunk run against one store holding the whole sequence:
    for each c in c_grid, prefixes round(f (S - c)) to multiples of align for
    f in p_fracs.  shape: a layer.LayerShape (whole decoder layer per chunk)
    or None with attn = (h_q, h_kv, head_dim, scale) (append + attention).
    Returns {(c, p): us}."""
    import torch

    from . import synth
    from .layer import ChunkedLayer
    from .prefill import ChunkedPrefill

    stream = torch.cuda.current_stream()
    if shape is not None:
        g = torch.Generator(device="cpu")
        g.manual_seed(seed)
        x = torch.randn((seq_len, shape.hidden), generator=g, dtype=torch.float32).to(torch.bfloat16).cuda()
        runner = ChunkedLayer(shape, [seq_len], seed=seed, block_size=block_size)
        scale = shape.head_dim ** -0.5
        runner.run(x, scale, stream=stream)  # fills the whole store once

        def one(c, p):
            xc = x[p:p + c]
            q, k, v = runner.project_qkv(xc)
            binding.mocap_kv_append(runner.attn.store, runner.attn.table, p, k, v, stream)
            o = torch.empty((c, shape.h_q, shape.head_dim), dtype=torch.bfloat16, device="cuda")
            lse = torch.empty((shape.h_q, c), dtype=torch.float32, device="cuda")
            binding.mocap_chunk_attn(runner.attn.store, runner.attn.table, q, p, scale, o, lse,
                                     ws_for(p, c, shape.h_q, shape.h_kv, shape.head_dim), 0, stream)
            y = xc + o.reshape(c, -1) @ runner.w_o
            gu = y @ runner.w_gu
            h = torch.nn.functional.silu(gu[:, :shape.ffn]) * gu[:, shape.ffn:]
            return y + h @ runner.w_d
    else:
        h_q, h_kv, d, scale = attn
        q, k, v = (t.cuda() for t in synth.make_qkv(seed, seq_len, h_q, h_kv, d))
        runner = ChunkedPrefill(h_q, h_kv, d, [seq_len], block_size=block_size)
        runner.run(q, k, v, scale, stream=stream)

        def one(c, p):
            binding.mocap_kv_append(runner.store, runner.table, p, k[p:p + c], v[p:p + c], stream)
            o = torch.empty((c, h_q, d), dtype=torch.bfloat16, device="cuda")
            lse = torch.empty((h_q, c), dtype=torch.float32, device="cuda")
            binding.mocap_chunk_attn(runner.store, runner.table, q[p:p + c], p, scale, o, lse,
                                     ws_for(p, c, h_q, h_kv, d), 0, stream)
            return o

    workspaces = {}

    def ws_for(p, c, h_q, h_kv, d):
        _, nbytes = binding.mocap_chunk_attn_workspace_size(p, c, h_q, h_kv, d, 0)
        if nbytes not in workspaces:
            workspaces[nbytes] = torch.empty(max(nbytes, 16), dtype=torch.uint8, device="cuda")
        return workspaces[nbytes]

    out = {}
    for c in c_grid:
        for f in p_fracs:
            p = int(round(f * (seq_len - c) / align)) * align
            if (c, p) in out:
                continue
            one(c, p)  # warm-up
            times = []
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                one(c, p)
                e1.record(stream)
                e1.synchronize()
                times.append(e0.elapsed_time(e1) * 1e3)
            out[(c, p)] = statistics.median(times)
    return out


def cost_table(grid, model: LatencyModel, seq_len: int, align: int):
    """Chunk-cost table [k - 1][s] (align units) for mocap_lbcp_plan_table:
    the fitted model times a measured correction, interpolated linearly in
    chunk length between grid lengths and, for each grid length, linearly in
    the prefix fraction p / (S - c)."""
    import numpy as np

    U = seq_len // align
    lengths = sorted({c for c, _ in grid})
    corr = {}
    for c in lengths:
        pts = sorted((p / max(seq_len - c, 1), t / model(c, p)) for (cc, p), t in grid.items() if cc == c)
        corr[c] = ([x for x, _ in pts], [y for _, y in pts])

    def factor(c, p):
        frac = p / max(seq_len - c, 1)
        if c <= lengths[0]:
            lo = hi = lengths[0]
        elif c >= lengths[-1]:
            lo = hi = lengths[-1]
        else:
            hi = next(x for x in lengths if x >= c)
            lo = max(x for x in lengths if x <= c)
        f_lo = float(np.interp(frac, *corr[lo]))
        f_hi = float(np.interp(frac, *corr[hi]))
        if hi == lo:
            return f_lo
        w = (c - lo) / (hi - lo)
        return f_lo * (1 - w) + f_hi * w

    table = np.zeros((U, U), dtype=np.float64)
    for k in range(1, U + 1):
        c = k * align
        for s in range(U - k + 1):
            p = s * align
            table[k - 1, s] = model(c, p) * factor(c, p)
    return table


def serving_study(table, start, model, seq_len, num_chunks, num_stages, align, h_kv, head_dim,
                  layers_per_stage, requests, max_batch, capacities, seed):
    """The table's plan against the annealed plan under the serving model
    (mocap_lbcp_evaluate / mocap_lbcp_refine_e2e), per capacity and pairing.
    A stage runs layers_per_stage layers: its chunk cost is that many times
    the table's, its fixed per-chunk cost that many times the fitted
    per-chunk constant, and a request token holds 2 h_kv d bf16 values per
    layer on it."""
    stage_table = table * layers_per_stage
    e = model.cost_chunk * layers_per_stage
    kv = float(layers_per_stage * 2 * h_kv * head_dim * 2)
    one = seq_len * kv
    out = []
    for cap_units in capacities:
        for pairing in (False, True):
            args = (seq_len, num_chunks, num_stages, align, stage_table)
            model_args = dict(fixed_cost=e, kv_bytes_per_token=kv, stage_capacity=cap_units * one,
                              pairing=pairing, max_batch=max_batch, requests=requests)
            b0, pre0, t0 = binding.mocap_lbcp_evaluate(*args, start, **model_args)
            temp0 = 0.05 * t0 if t0 < float("inf") else 1e3
            lengths, b1, pre1, t1 = binding.mocap_lbcp_refine_e2e(*args, start, **model_args, temp0=temp0,
                                                                   temp_min=2e-3 * temp0, alpha=0.9, rounds=30,
                                                                   seed=seed)
            out.append({"capacity_requests": cap_units, "pairing": pairing,
                        "dp": {"batch": b0, "t_pre_us": round(pre0, 1), "e2e_us": round(t0, 1)},
                        "annealed": {"batch": b1, "t_pre_us": round(pre1, 1), "e2e_us": round(t1, 1),
                                     "lengths": lengths, "left_dp_plan": list(lengths) != list(start)}})
            print(f"[lbcp] e2e capacity {cap_units} pairing {pairing}: B {b0} -> {b1}, "
                  f"T {t0 / 1e3:.1f} -> {t1 / 1e3:.1f} ms", file=sys.stderr, flush=True)
    return {"requests": requests, "layers_per_stage": layers_per_stage, "fixed_cost_us": round(e, 1),
            "kv_bytes_per_token_per_stage": kv, "max_batch": max_batch, "runs": out}


def _objective(latencies: Sequence[float], num_stages: int) -> float:
    return sum(latencies) + (num_stages - 1) * max(latencies)


def main(argv=None):
    from . import synth
    from .layer import SHAPES

    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="llama8b_128k_balanced")
    ap.add_argument("--layer", choices=sorted(SHAPES), default=None,
                    help="time a whole decoder layer per chunk (projections, attention, feed-forward) "
                         "instead of the attention calls alone")
    ap.add_argument("--seq-len", type=int, default=0, help="0 = the workload's sequence length")
    ap.add_argument("--stages", type=int, default=16, help="pipeline stages N of the objective")
    ap.add_argument("--chunks", type=int, default=0, help="0 = the workload's chunk count")
    ap.add_argument("--align", type=int, default=0, help="0 = the workload's alignment")
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--random-plans", type=int, default=4)
    ap.add_argument("--stage2", action="store_true",
                    help="also build a measured chunk-cost table over a (length, prefix) grid, run the "
                         "table-driven dynamic program and the simulated-annealing refinement, and "
                         "measure their plans")
    ap.add_argument("--e2e", action="store_true",
                    help="with --stage2: also refine the table's plan under the serving model "
                         "(feasible batch under per-stage KV capacity, with and without cross-half pairing, "
                         "and the workload's end-to-end latency) for several capacities")
    ap.add_argument("--layers-per-stage", type=int, default=2,
                    help="decoder layers per pipeline stage: scales the table, the fixed per-chunk cost and "
                         "the KV bytes per token of a stage")
    ap.add_argument("--requests", type=int, default=64, help="requests queued for the end-to-end latency")
    ap.add_argument("--max-batch", type=int, default=16)
    ap.add_argument("--capacities", default="2.5,4,5.5,7",
                    help="per-stage KV capacities, in units of one request's KV on a stage")
    args = ap.parse_args(argv)

    w = synth.WORKLOADS[args.workload]
    seq_len = args.seq_len or w.seq_len
    m = args.chunks or w.num_chunks
    align = args.align or w.align
    probes = probe_plans(seq_len, m, align, seed=w.seed, n_random=args.random_plans)
    shape = SHAPES[args.layer] if args.layer else None
    what = f"{shape.name} decoder layer" if shape else f"{w.name} attention"

    def timed(plans):
        if shape is None:
            return [(i, c, p, t, t, 0.0) for i, c, p, t in
                    measure(w.h_q, w.h_kv, w.head_dim, plans, w.scale, w.block_size, args.reps, w.seed)]
        return measure_layer(shape, plans, args.reps, w.seed, w.block_size)

    print(f"[lbcp] measuring {len(probes)} probe plans of {what}, S={seq_len}", file=sys.stderr, flush=True)
    samples = timed(probes)
    model = fit([(c, p, t) for _, c, p, t, _, _ in samples])
    dp_lengths, t_max, t_sum = plan(seq_len, m, args.stages, align, model)
    closed = probes[1]
    plans = [closed, dp_lengths]
    stage2 = None
    if args.stage2:
        c_grid = [c for c in (128, 256, 384, 512, 768, 1024, 1536, 2048, 3072, 4096, 6144, 8192, 12288, 16384,
                              24576, 32768, 49152, 65536) if c % align == 0 and c <= seq_len - (m - 1) * align]
        print(f"[lbcp] measuring a {len(c_grid)} x 6 (length, prefix) grid", file=sys.stderr, flush=True)
        attn = None if shape else (w.h_q, w.h_kv, w.head_dim, w.scale)
        grid = measure_grid(shape, seq_len, c_grid, (0.0, 0.125, 0.25, 0.5, 0.75, 1.0), align, args.reps,
                            w.seed, w.block_size, attn=attn)
        table = cost_table(grid, model, seq_len, align)
        table_lengths, tt_max, tt_sum = binding.mocap_lbcp_plan_table(seq_len, m, args.stages, align, table)
        t0 = tt_sum + (args.stages - 1) * tt_max
        sa_lengths, sa_lat = binding.mocap_lbcp_refine(seq_len, m, args.stages, align, table, table_lengths,
                                                       temp0=0.01 * t0, temp_min=1e-5 * t0, alpha=0.95,
                                                       rounds=50, seed=w.seed)
        stage2 = {"grid_points": len(grid), "table_dp_model_us": round(t0, 1),
                  "refined_model_us": round(sa_lat, 1)}
        plans += [table_lengths, sa_lengths]
        if args.e2e:
            stage2["e2e"] = serving_study(table, table_lengths, model, seq_len, m, args.stages, align,
                                          w.h_kv, w.head_dim, args.layers_per_stage, args.requests,
                                          args.max_batch, [float(x) for x in args.capacities.split(",")],
                                          w.seed)
    print("[lbcp] measuring the candidate plans", file=sys.stderr, flush=True)
    final = timed(plans)

    def summary(i, lengths):
        rows = [x for x in final if x[0] == i]
        lat = [x[3] for x in rows]
        return {"lengths": list(lengths), "chunk_us": [round(t, 1) for t in lat],
                "attention_us": [round(x[4], 1) for x in rows], "gemm_us": [round(x[5], 1) for x in rows],
                "max_over_min": round(max(lat) / min(lat), 3),
                "objective_us": round(_objective(lat, args.stages), 1)}

    report = {
        "workload": what, "seq_len": seq_len, "stages": args.stages, "chunks": m, "align": align,
        "model_us": {"cost_pair": model.cost_pair, "cost_token": model.cost_token,
                     "cost_chunk": model.cost_chunk, "rms_rel_err": round(model.rms_rel_err, 4),
                     "samples": len(samples)},
        "closed_form": summary(0, closed),
        "dp": dict(summary(1, dp_lengths), model_t_max_us=round(t_max, 1), model_t_sum_us=round(t_sum, 1)),
    }
    if stage2 is not None:
        report["stage2"] = dict(stage2, table_dp=summary(2, plans[2]), refined=summary(3, plans[3]))
    print(json.dumps(report), flush=True)
    return report


if __name__ == "__main__":
    main()
