"""LBCP (Alg. 1, both stages) -- TEST INFRASTRUCTURE.

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


# --- second stage with batch and memory: EvaluatePrefill and EvaluateE2E ----
#
# Readings (the paper names these functions but its simulator is not given):
# * N identical stages run the same sequence of chunk operations; operation k
#   of a batch of n requests takes t_k(n) = t_k + (n - 1) * max(t_k - e, 0),
#   where t_k is the table's latency of that chunk for one request and e the
#   part of it a batch does not multiply (a fixed per-chunk cost).
# * Q requests wait at time 0 and are served in order, in batches of B (the
#   last one smaller); the batches follow each other through the pipeline.
# * A stage holds the KV of a batch's chunks from the start of each chunk on
#   that stage until the batch leaves the last stage (Section 3.1: earlier
#   stages hold their KV longer).  Without reallocation every stage's KV must
#   fit its own capacity at all times; with MBKR's fixed cross-half pairing
#   (Section 4.1) stage i and stage i + N/2 pool their capacity.
# * EvaluatePrefill returns B' (the largest feasible batch up to max_batch,
#   0 if none) and T'_pre, the prefill latency of one batch of B' requests;
#   EvaluateE2E returns the completion time of the last of the Q requests
#   served in batches of B' (the workload's end-to-end latency).

def batch_op_times(lengths_units, evaluate_units, n, e):
    """Latency of each chunk operation of one batch of n requests."""
    out, s = [], 0
    for k in lengths_units:
        t = evaluate_units(k, s)
        out.append(t + (n - 1) * max(t - e, 0.0))
        s += k
    return out


def schedule(lengths_units, evaluate_units, e, Q, B):
    """Operations of Q requests in batches of B: list of (batch, chunk, n, time)."""
    ops, b, left = [], 0, Q
    while left > 0:
        n = min(B, left)
        for j, t in enumerate(batch_op_times(lengths_units, evaluate_units, n, e)):
            ops.append((b, j, n, t))
        left -= n
        b += 1
    return ops


def completion_times(times, N):
    """C[s][k], s = 1..N: completion of operation k on stage s when every stage
    takes the same time for it and runs the operations in order.  Closed
    form of the flow-shop recurrence: sum of times up to k plus (s - 1)
    times their maximum."""
    C = [None] + [[0.0] * len(times) for _ in range(N)]
    acc, mx = 0.0, 0.0
    for k, t in enumerate(times):
        acc += t
        mx = max(mx, t)
        for s in range(1, N + 1):
            C[s][k] = acc + (s - 1) * mx
    return C


def flowshop_bruteforce(times, N):
    """The same completion times from the recurrence itself:
    C[s][k] = max(C[s-1][k], C[s][k-1]) + t_k."""
    C = [[0.0] * len(times) for _ in range(N + 1)]
    for k, t in enumerate(times):
        for s in range(1, N + 1):
            C[s][k] = max(C[s - 1][k], C[s][k - 1] if k else 0.0) + t
    return [None] + C[1:]


def peak_kv_tokens(lengths_units, align, ops, C, N, stages):
    """Largest number of KV tokens held together by `stages` (a set of stage
    numbers) over the schedule; a batch's tokens leave at the moment the
    batch completes on stage N, before anything starting at that moment."""
    done = {}
    for k, (b, j, n, t) in enumerate(ops):
        done[b] = C[N][k]
    events = []  # (time, kind, stage, batch, chunk, delta); kind 0 = leave, 1 = start
    for s in stages:
        for k, (b, j, n, t) in enumerate(ops):
            events.append((C[s][k] - t, 1, s, b, j, n * lengths_units[j] * align))
    for b, when in done.items():
        for s in stages:
            events.append((when, 0, s, b, -1, None))
    events.sort(key=lambda ev: ev[:5])
    held = {}  # (stage, batch) -> tokens
    cur = peak = 0
    for when, kind, s, b, j, delta in events:
        if kind == 0:
            cur -= held.pop((s, b), 0)
        else:
            held[(s, b)] = held.get((s, b), 0) + delta
            cur += delta
            peak = max(peak, cur)
    return peak


def feasible(lengths_units, align, evaluate_units, N, e, kv_bytes, capacity, pairing, Q, B):
    ops = schedule(lengths_units, evaluate_units, e, Q, B)
    C = completion_times([op[3] for op in ops], N)
    if pairing:
        groups = [({s, s + N // 2}, 2.0 * capacity) for s in range(1, N // 2 + 1)]
    else:
        groups = [({s}, capacity) for s in range(1, N + 1)]
    return all(peak_kv_tokens(lengths_units, align, ops, C, N, g) * kv_bytes <= cap for g, cap in groups)


def evaluate_prefill(lengths_units, align, evaluate_units, N, e, kv_bytes, capacity, pairing, max_batch, Q):
    """EvaluatePrefill: (B', T'_pre)."""
    best = 0
    for B in range(1, min(max_batch, Q) + 1):
        if feasible(lengths_units, align, evaluate_units, N, e, kv_bytes, capacity, pairing, Q, B):
            best = B
    if best == 0:
        return 0, math.inf
    times = batch_op_times(lengths_units, evaluate_units, best, e)
    return best, sum_then_max(times, N)


def sum_then_max(times, N):
    acc, mx = 0.0, 0.0
    for t in times:
        acc += t
        mx = max(mx, t)
    return acc + (N - 1) * mx


def evaluate_e2e(lengths_units, evaluate_units, N, e, Q, B):
    """EvaluateE2E: completion time of the last of the Q requests served in
    batches of B (the end-to-end latency of the workload; Q / T is its
    throughput)."""
    if B == 0:
        return math.inf
    ops = schedule(lengths_units, evaluate_units, e, Q, B)
    C = completion_times([op[3] for op in ops], N)
    return C[N][len(ops) - 1]


def lbcp_refine_e2e(S, M, N, align, lengths, temp0, temp_min, alpha, rounds, seed, evaluate,
                    e, kv_bytes, capacity, pairing, max_batch, Q):
    """Alg. 1's second stage under the serving model: each candidate ss' is
    scored by (B', T'_pre) = EvaluatePrefill(ss'), T' = EvaluateE2E(B',
    T'_pre) (the E2E latency uses the schedule of B' batches, of which T'_pre
    is the first batch's part); Perturb, acceptance and cooling as in
    lbcp_refine.  Returns (lengths, B, T_pre, T)."""
    U = S // align
    ev = lambda k, s: evaluate(k * align, s * align)
    ss = [c // align for c in lengths]
    assert sum(ss) == U and all(k >= 1 for k in ss)

    def score(x):
        B, T_pre = evaluate_prefill(x, align, ev, N, e, kv_bytes, capacity, pairing, max_batch, Q)
        return B, T_pre, evaluate_e2e(x, ev, N, e, Q, B)

    rng = SplitMix64(seed)
    B, T_pre, T = score(ss)
    best = (list(ss), B, T_pre, T)
    temp = temp0
    while temp > temp_min:
        for _ in range(rounds):
            if M < 2:
                break
            j = 1 + rng.next() % (M - 1)
            step = 1 if rng.next() & 1 else -1
            cand = list(ss)
            cand[j - 1] += step
            cand[j] -= step
            if cand[j - 1] < 1 or cand[j] < 1:
                continue
            B_new, T_pre_new, T_new = score(cand)
            u = rng.uniform()
            if T_new < T or (math.isfinite(T_new) and u < math.exp(-(T_new - T) / temp)):
                ss, B, T_pre, T = cand, B_new, T_pre_new, T_new
            if T < best[3]:
                best = (list(ss), B, T_pre, T)
        temp *= alpha
    return [k * align for k in best[0]], best[1], best[2], best[3]
