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
    print("[lbcp] measuring the closed-form and dynamic-programming plans", file=sys.stderr, flush=True)
    final = timed([closed, dp_lengths])

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
    print(json.dumps(report), flush=True)
    return report


if __name__ == "__main__":
    main()
