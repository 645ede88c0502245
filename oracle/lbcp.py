"""LBCP stage 1 -- TEST INFRASTRUCTURE.

The first stage of the paper's latency-balanced chunk partitioning (Section
4.2, Alg. 1, the dynamic-programming initialisation), written from the
algorithm's description in its own order and notation: chunk index m runs
from M down to 1, start position s from S-1 down to 0, candidate length k
from 1 to S-s-(M-m); EvaluateChunk(k, s) gives t, which is combined with the
suffix state (m+1, s+k) into t'_max and t'_sum; the candidate with the
smallest t'_sum + (N-1) t'_max is recorded in ss[m][s].  Positions are in
units of `align` tokens.  The suffix boundary, left implicit by the paper,
is t = 0 at (M+1, S) and infeasible elsewhere.

Plain Python loops: for small S/align only.  Also a brute-force search over
all compositions, for pinning the dynamic program where it is exact.
"""
import itertools
import math


def chunk_cost(c, p, cost_pair, cost_token, cost_chunk):
    """EvaluateChunk: visible-pair term of Eq. (1) plus per-token and per-chunk terms."""
    return cost_pair * (c * p + c * (c + 1) / 2.0) + cost_token * c + cost_chunk


def lbcp_dp(S, M, N, align, cost_pair=0.0, cost_token=0.0, cost_chunk=0.0, evaluate=None):
    """Returns (lengths, t_max, t_sum).

    evaluate(c, p), when given, replaces the linear latency model: the cost of
    a chunk of c tokens behind p tokens (any deterministic function)."""
    if evaluate is None:
        def evaluate(c, p):
            return chunk_cost(c, p, cost_pair, cost_token, cost_chunk)
    U = S // align
    inf = math.inf
    t_max = [[inf] * (U + 1) for _ in range(M + 2)]
    t_sum = [[inf] * (U + 1) for _ in range(M + 2)]
    ss = [[0] * (U + 1) for _ in range(M + 2)]
    t_max[M + 1][U] = 0.0
    t_sum[M + 1][U] = 0.0
    for m in range(M, 0, -1):
        for s in range(U - 1, -1, -1):
            best = inf  # objective of the candidate recorded so far at (m, s)
            for k in range(1, U - s - (M - m) + 1):
                if t_sum[m + 1][s + k] == inf:
                    continue
                t = evaluate(k * align, s * align)  # EvaluateChunk(k, s)
                t_max_new = max(t_max[m + 1][s + k], t)
                t_sum_new = t_sum[m + 1][s + k] + t
                objective = t_sum_new + (N - 1) * t_max_new
                if objective < best:
                    best = objective
                    t_max[m][s] = t_max_new
                    t_sum[m][s] = t_sum_new
                    ss[m][s] = k
    lengths, s = [], 0
    for m in range(1, M + 1):
        k = ss[m][s]
        lengths.append(k * align)
        s += k
    return lengths, t_max[1][0], t_sum[1][0]


def plan_costs(lengths, evaluate):
    out, p = [], 0
    for c in lengths:
        out.append(evaluate(c, p))
        p += c
    return out


def brute_force(S, M, align, objective, evaluate):
    """Best plan over every composition of S/align into M positive parts."""
    U = S // align
    best = None
    for cuts in itertools.combinations(range(1, U), M - 1):
        bounds = (0,) + cuts + (U,)
        lengths = [(b - a) * align for a, b in zip(bounds[:-1], bounds[1:])]
        val = objective(plan_costs(lengths, evaluate))
        if best is None or val < best[0]:
            best = (val, lengths)
    return best
