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


# --- second stage: simulated annealing (Section 4.2, Alg. 1) --------------

class SplitMix64:
    """SplitMix64 (Steele, Lea and Flood, 2014), written from its definition:
    the state advances by 0x9E3779B97F4A7C15 and each output is that state
    through two xor-shift-multiply rounds and a final xor-shift."""
    MASK = (1 << 64) - 1

    def __init__(self, seed):
        self.x = seed & self.MASK

    def next(self):
        self.x = (self.x + 0x9E3779B97F4A7C15) & self.MASK
        z = self.x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & self.MASK
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & self.MASK
        return z ^ (z >> 31)

    def uniform(self):
        return (self.next() >> 11) * (1.0 / 9007199254740992.0)


def prefill_latency(lengths_units, N, evaluate_units):
    """Single-request pipeline latency of a partition: sum of chunk costs plus
    (N - 1) times the largest (EvaluatePrefill without the batch model)."""
    t_sum, t_max, s = 0.0, 0.0, 0
    for k in lengths_units:
        t = evaluate_units(k, s)
        t_sum += t
        t_max = max(t_max, t)
        s += k
    return t_sum + (N - 1) * t_max


def lbcp_refine(S, M, N, align, lengths, temp0, temp_min, alpha, rounds, seed, evaluate):
    """Alg. 1's second stage from an initial partition: while Temp > Temp_min,
    R times: ss' = Perturb(ss) (one inner boundary moved by one align unit,
    S and M preserved, moves that empty a chunk skipped); T' its latency;
    accept if T' < T or Rand(0, 1) < exp(-(T' - T) / Temp); keep the best;
    then Temp = alpha Temp.  evaluate(c, p) is in tokens.  Returns
    (lengths, latency)."""
    U = S // align
    ev = lambda k, s: evaluate(k * align, s * align)
    ss = [c // align for c in lengths]
    assert sum(ss) == U and all(k >= 1 for k in ss)
    rng = SplitMix64(seed)
    T = prefill_latency(ss, N, ev)
    best, T_best = list(ss), T
    temp = temp0
    while temp > temp_min:
        for _ in range(rounds):
            if M < 2:
                break
            j = 1 + rng.next() % (M - 1)            # boundary between chunks j-1 and j
            step = 1 if rng.next() & 1 else -1       # +1 moves it right
            cand = list(ss)
            cand[j - 1] += step
            cand[j] -= step
            if cand[j - 1] < 1 or cand[j] < 1:
                continue
            T_new = prefill_latency(cand, N, ev)
            u = rng.uniform()
            if T_new < T or u < math.exp(-(T_new - T) / temp):
                ss, T = cand, T_new
            if T < T_best:
                best, T_best = list(ss), T
        temp *= alpha
    return [k * align for k in best], T_best
