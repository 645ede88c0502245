"""LBCP's second stage under the serving model (Section 4.2, Alg. 1's
EvaluatePrefill / EvaluateE2E; Section 4.1's fixed cross-half pairing).

The oracle (oracle/lbcp.py) is pinned by brute force, a worked example and
invariants; the library's C implementation must then equal it bit for bit.
"""
import itertools
import math
import random

import pytest

from oracle import lbcp


def _table_eval(table, U):
    return lambda k, s: table[(k - 1) * U + s]


def _square(table, U):
    import numpy as np
    return np.asarray(table, dtype=np.float64).reshape(U, U)


def _random_table(U, rng, lo=1.0, hi=5.0):
    return [rng.uniform(lo, hi) for _ in range(U * U)]


@pytest.mark.parametrize("seed", range(6))
def test_completion_times_closed_form_equals_recurrence(seed):
    rng = random.Random(seed)
    times = [rng.uniform(0.1, 3.0) for _ in range(rng.randint(1, 12))]
    N = rng.randint(1, 5)
    a = lbcp.completion_times(times, N)
    b = lbcp.flowshop_bruteforce(times, N)
    for s in range(1, N + 1):
        for x, y in zip(a[s], b[s]):
            assert x == pytest.approx(y, rel=1e-12, abs=1e-12)


def _peak_by_definition(lengths_units, align, ops, C, N, stages):
    done = {}
    for k, (b, j, n, t) in enumerate(ops):
        done[b] = C[N][k]
    best = 0
    for s0 in stages:
        for k0, (_, _, _, t0) in enumerate(ops):
            tau = C[s0][k0] - t0
            occ = 0
            for s in stages:
                for k, (b, j, n, t) in enumerate(ops):
                    if C[s][k] - t <= tau and done[b] > tau:
                        occ += n * lengths_units[j] * align
            best = max(best, occ)
    return best


@pytest.mark.parametrize("seed", range(8))
def test_peak_kv_equals_definition(seed):
    rng = random.Random(100 + seed)
    U, M = rng.randint(3, 7), None
    M = rng.randint(1, U)
    cuts = sorted(rng.sample(range(1, U), M - 1))
    ss = [b - a for a, b in zip([0] + cuts, cuts + [U])]
    N = rng.choice([2, 4])
    table = _random_table(U, rng)
    ev = _table_eval(table, U)
    e = rng.uniform(0.0, 1.0)
    Q, B = rng.randint(1, 5), rng.randint(1, 3)
    ops = lbcp.schedule(ss, ev, e, Q, B)
    C = lbcp.completion_times([op[3] for op in ops], N)
    for stages in ([1], [N], list(range(1, N + 1)), [1, 1 + N // 2]):
        assert lbcp.peak_kv_tokens(ss, 128, ops, C, N, set(stages)) == \
            _peak_by_definition(ss, 128, ops, C, N, stages)


def test_worked_two_stage_example():
    # Two stages, two chunks of one token each costing 1 per request, e = 0,
    # two requests.  Batches of one: operations finish on stage 1 at 1, 2,
    # 3, 4 and on stage 2 at 2, 3, 4, 5, so request 1 leaves at 3 and request
    # 2 at 5 (the end-to-end latency).  Stage 1 holds 1, 2, then 3 tokens (request 2's first
    # chunk starts at 2, before request 1 leaves at 3); stage 2 peaks at 2;
    # the pair together peaks at 5 (at time 2).  One batch of two: both
    # chunks take 2, the batch leaves at 6 and each stage peaks at 4 (8
    # together).
    U = 2
    ev = _table_eval([1.0] * (U * U), U)
    ss = [1, 1]
    ops = lbcp.schedule(ss, ev, 0.0, 2, 1)
    C = lbcp.completion_times([op[3] for op in ops], 2)
    assert C[1] == [1.0, 2.0, 3.0, 4.0] and C[2] == [2.0, 3.0, 4.0, 5.0]
    assert lbcp.peak_kv_tokens(ss, 1, ops, C, 2, {1}) == 3
    assert lbcp.peak_kv_tokens(ss, 1, ops, C, 2, {2}) == 2
    assert lbcp.peak_kv_tokens(ss, 1, ops, C, 2, {1, 2}) == 5
    assert lbcp.evaluate_e2e(ss, ev, 2, 0.0, 2, 1) == 5.0
    assert lbcp.evaluate_e2e(ss, ev, 2, 0.0, 2, 2) == 6.0
    # Capacity 3 tokens per stage: a batch of two needs 4 -> B' = 1 either way.
    assert lbcp.evaluate_prefill(ss, 1, ev, 2, 0.0, 1.0, 3.0, False, 4, 2) == (1, 3.0)
    assert lbcp.evaluate_prefill(ss, 1, ev, 2, 0.0, 1.0, 3.0, True, 4, 2) == (1, 3.0)
    # Capacity 2.5: stage 1 alone cannot hold its 3 tokens, the pair's 5 fit
    # in 2 x 2.5 -- reallocation makes the schedule feasible.
    assert lbcp.evaluate_prefill(ss, 1, ev, 2, 0.0, 1.0, 2.5, False, 4, 2)[0] == 0
    assert lbcp.evaluate_prefill(ss, 1, ev, 2, 0.0, 1.0, 2.5, True, 4, 2) == (1, 3.0)
    assert lbcp.evaluate_e2e(ss, ev, 2, 0.0, 2, 0) == math.inf


@pytest.mark.parametrize("seed", range(5))
def test_single_batch_closed_forms(seed):
    rng = random.Random(200 + seed)
    U = rng.randint(2, 8)
    M = rng.randint(1, U)
    cuts = sorted(rng.sample(range(1, U), M - 1))
    ss = [b - a for a, b in zip([0] + cuts, cuts + [U])]
    N, B = rng.randint(1, 6), rng.randint(1, 4)
    table = _random_table(U, rng)
    ev = _table_eval(table, U)
    e = rng.uniform(0.0, 1.0)
    times = lbcp.batch_op_times(ss, ev, B, e)
    # one batch of B requests: T_pre = sum + (N - 1) max; E2E = T_pre
    assert lbcp.evaluate_e2e(ss, ev, N, e, B, B) == pytest.approx(sum(times) + (N - 1) * max(times))
    # each chunk of a batch costs B times its batch-proportional part plus e
    for t1, tb, k in zip(lbcp.batch_op_times(ss, ev, 1, e), times, ss):
        assert tb == pytest.approx(B * (t1 - e) + e) if t1 >= e else tb == pytest.approx(t1)
    # one batch holds all of its tokens on every stage until it leaves
    ops = lbcp.schedule(ss, ev, e, B, B)
    C = lbcp.completion_times([op[3] for op in ops], N)
    for s in range(1, N + 1):
        assert lbcp.peak_kv_tokens(ss, 64, ops, C, N, {s}) == B * U * 64
    # so a single batch of B fits exactly when B S kv <= capacity
    for cap in (B * U * 64 - 0.5, B * U * 64, rng.uniform(1.0, 5.0) * U * 64):
        assert lbcp.feasible(ss, 64, ev, N, e, 1.0, cap, False, B, B) == (B * U * 64 <= cap)


@pytest.mark.parametrize("seed", range(6))
def test_pairing_never_lowers_the_batch(seed):
    rng = random.Random(300 + seed)
    U = rng.randint(3, 8)
    M = rng.randint(2, min(U, 4))
    cuts = sorted(rng.sample(range(1, U), M - 1))
    ss = [b - a for a, b in zip([0] + cuts, cuts + [U])]
    N = rng.choice([2, 4, 6])
    table = _random_table(U, rng)
    ev = _table_eval(table, U)
    e, Q = rng.uniform(0.0, 1.0), rng.randint(2, 6)
    cap = rng.uniform(1.0, 4.0) * U * 64
    b0, _ = lbcp.evaluate_prefill(ss, 64, ev, N, e, 1.0, cap, False, 6, Q)
    b1, _ = lbcp.evaluate_prefill(ss, 64, ev, N, e, 1.0, cap, True, 6, Q)
    assert b1 >= b0


def _brute_force_e2e(U, M, N, ev, e, kv, cap, pairing, max_batch, Q):
    best = None
    for cuts in itertools.combinations(range(1, U), M - 1):
        ss = [b - a for a, b in zip((0,) + cuts, cuts + (U,))]
        B, _ = lbcp.evaluate_prefill(ss, 1, ev, N, e, kv, cap, pairing, max_batch, Q)
        T = lbcp.evaluate_e2e(ss, ev, N, e, Q, B)
        if best is None or T < best[0]:
            best = (T, ss)
    return best


@pytest.mark.parametrize("seed,cap", [(s, c) for s in range(3) for c in (16.0, 20.0)])
def test_annealing_reaches_brute_force_e2e_optimum(seed, cap):
    # Every partition is feasible at these capacities (B' is 1 or 2), so the
    # annealing can walk the whole space from a poor start.
    rng = random.Random(400 + seed)
    U, M, N, Q = 8, 3, 2, 3
    table = [rng.uniform(1.0, 4.0) * k for k in range(1, U + 1) for _ in range(U)]
    ev = _table_eval(table, U)
    e = 0.5
    T_best, ss_best = _brute_force_e2e(U, M, N, ev, e, 1.0, cap, True, 3, Q)
    assert math.isfinite(T_best)
    lengths, B, T_pre, T = lbcp.lbcp_refine_e2e(U, M, N, 1, [U - 2, 1, 1], 50.0, 1e-2, 0.9, 30, seed,
                                                lambda c, p: table[(c - 1) * U + p], e, 1.0, cap, True, 3, Q)
    assert T == pytest.approx(T_best, rel=1e-12)
    assert sum(lengths) == U and min(lengths) >= 1


def test_library_evaluate_equals_oracle(mocap_lib):
    for seed in range(10):
        rng = random.Random(500 + seed)
        align = rng.choice([1, 64, 128])
        U = rng.randint(2, 9)
        M = rng.randint(1, U)
        cuts = sorted(rng.sample(range(1, U), M - 1))
        ss = [b - a for a, b in zip([0] + cuts, cuts + [U])]
        N = rng.choice([1, 2, 3, 4, 8]) if seed % 2 else rng.choice([2, 4, 8])
        pairing = seed % 2 == 0
        table = _random_table(U, rng, 0.5, 3.0)
        ev = _table_eval(table, U)
        e = rng.uniform(0.0, 1.0)
        kv, Q, max_batch = rng.uniform(0.5, 2.0), rng.randint(1, 7), rng.randint(1, 6)
        cap = rng.uniform(0.5, 4.0) * U * align * kv
        B, T_pre = lbcp.evaluate_prefill(ss, align, ev, N, e, kv, cap, pairing, max_batch, Q)
        T = lbcp.evaluate_e2e(ss, ev, N, e, Q, B)
        got = mocap_lib.mocap_lbcp_evaluate(U * align, M, N, align, _square(table, U), [k * align for k in ss], e, kv, cap,
                                            pairing, max_batch, Q)
        assert got == (B, T_pre, T), (seed, got, (B, T_pre, T))


@pytest.mark.parametrize("seed", range(4))
def test_library_refine_e2e_equals_oracle(mocap_lib, seed):
    rng = random.Random(600 + seed)
    align = 64
    U, M, N = rng.randint(5, 9), rng.randint(2, 4), rng.choice([2, 4])
    table = [rng.uniform(0.5, 2.0) * k + rng.uniform(0.0, 0.1) * s for k in range(1, U + 1) for s in range(U)]
    e = rng.uniform(0.0, 0.4)
    kv, Q, max_batch = 1.0, rng.randint(2, 5), 4
    cap = rng.uniform(1.2, 3.0) * U * align
    start = [1] * (M - 1) + [U - M + 1]
    ev_tokens = lambda c, p: table[(c // align - 1) * U + p // align]
    want = lbcp.lbcp_refine_e2e(U * align, M, N, align, [k * align for k in start], 2.0, 1e-2, 0.8, 8, seed,
                                ev_tokens, e, kv, cap, True, max_batch, Q)
    got = mocap_lib.mocap_lbcp_refine_e2e(U * align, M, N, align, _square(table, U), [k * align for k in start], e, kv, cap,
                                          True, max_batch, Q, 2.0, 1e-2, 0.8, 8, seed)
    assert tuple(got) == (want[0], want[1], want[2], want[3])


def test_library_serving_model_rejections(mocap_lib):
    U, align = 4, 64
    table = _square([1.0] * (U * U), U)
    base = dict(fixed_cost=0.1, kv_bytes_per_token=1.0, stage_capacity=1e6, pairing=False, max_batch=4,
                requests=4)
    for bad in (dict(fixed_cost=-1.0), dict(kv_bytes_per_token=0.0), dict(stage_capacity=float("inf")),
                dict(max_batch=0), dict(requests=0), dict(requests=5000)):
        kw = dict(base, **bad)
        with pytest.raises(mocap_lib.MocapError):
            mocap_lib.mocap_lbcp_evaluate(U * align, 2, 4, align, table, [2 * align, 2 * align], **kw)
    with pytest.raises(mocap_lib.MocapError):  # pairing needs an even number of stages
        mocap_lib.mocap_lbcp_evaluate(U * align, 2, 3, align, table, [2 * align, 2 * align],
                                      **dict(base, pairing=True))
    with pytest.raises(mocap_lib.MocapError):  # not a partition of seq_len
        mocap_lib.mocap_lbcp_evaluate(U * align, 2, 4, align, table, [2 * align, align], **base)


@pytest.mark.parametrize("seed", range(5))
def test_e2e_is_the_last_completion_of_the_recurrence(seed):
    rng = random.Random(700 + seed)
    U = rng.randint(2, 7)
    M = rng.randint(1, U)
    cuts = sorted(rng.sample(range(1, U), M - 1))
    ss = [b - a for a, b in zip([0] + cuts, cuts + [U])]
    N, e, Q, B = rng.randint(1, 5), rng.uniform(0.0, 1.0), rng.randint(1, 7), rng.randint(1, 4)
    ev = _table_eval(_random_table(U, rng), U)
    times = [op[3] for op in lbcp.schedule(ss, ev, e, Q, B)]
    assert len(times) == M * -(-Q // B)
    assert lbcp.evaluate_e2e(ss, ev, N, e, Q, B) == pytest.approx(lbcp.flowshop_bruteforce(times, N)[N][-1],
                                                                  rel=1e-12)
