"""Chunk plans and work accounting -- TEST INFRASTRUCTURE.

Eq. (1) of the paper (Section 3.2) prices chunk i of length c_i behind a
prefix p_i = c_1 + ... + c_{i-1} as T_attn ~ c_i (p_i + c_i).  The
latency-balanced workload used here equalises the causal attention work of
each chunk, L_c (P_c + L_c / 2): the exact count of visible (query, key)
pairs of a chunk is L_c P_c + L_c (L_c + 1) / 2.  Because the cumulative
work up to boundary x is x^2 / 2, equal work per chunk puts boundary c of M
at x_c = S sqrt(c / M); each boundary is then rounded to the nearest multiple
of the alignment.

This module computes plans the plain way (fp64 square root, then rounding),
independently of the library's integer planner, so tests can compare the two.
"""
import math


def uniform_plan(seq_len, num_chunks):
    """Boundaries floor(c S / M): equal lengths when M divides S."""
    bounds = [(c * seq_len) // num_chunks for c in range(num_chunks + 1)]
    return [bounds[c + 1] - bounds[c] for c in range(num_chunks)]


def balanced_plan(seq_len, num_chunks, align):
    """Equal causal work per chunk; boundaries on multiples of ``align``."""
    if seq_len % align != 0:
        raise ValueError("seq_len must be a multiple of align")
    bounds = [0]
    for c in range(1, num_chunks):
        x = seq_len * math.sqrt(c / num_chunks)
        units = x / align
        frac = units - math.floor(units)
        if abs(frac - 0.5) < 1e-9:
            raise ValueError(f"boundary {c} is a rounding tie; plan is ambiguous")
        bounds.append(int(math.floor(units + 0.5)) * align)
    bounds.append(seq_len)
    lengths = [bounds[c + 1] - bounds[c] for c in range(num_chunks)]
    if min(lengths) <= 0:
        raise ValueError("plan has an empty chunk")
    return lengths


def prefixes(lengths):
    """P_c = sum of lengths before chunk c."""
    out, acc = [], 0
    for n in lengths:
        out.append(acc)
        acc += n
    return out


def visible_pairs(chunk_len, prefix_len):
    """Causally visible (query, key) pairs of one chunk: L P + L (L + 1) / 2."""
    return chunk_len * prefix_len + chunk_len * (chunk_len + 1) // 2


def balance_cost(chunk_len, prefix_len):
    """The balancing criterion of the latency-balanced workload: L (P + L / 2)."""
    return chunk_len * (prefix_len + chunk_len / 2.0)


def causal_flops(lengths, h_q, head_dim):
    """Algorithmic FLOPs of QK^T and PV over visible pairs: 4 d Hq pairs."""
    pairs = sum(visible_pairs(n, p) for n, p in zip(lengths, prefixes(lengths)))
    return 4 * head_dim * h_q * pairs
