"""LBCP stage 1 (Section 4.2, Alg. 1): the oracle's dynamic program pinned to
brute force and closed forms, then the library's C implementation compared
with it exactly."""
import math
import random

import pytest

from oracle import lbcp
from oracle import plan as oplan


def linear(cost_pair, cost_token=0.0, cost_chunk=0.0):
    return lambda c, p: lbcp.chunk_cost(c, p, cost_pair, cost_token, cost_chunk)


# --- oracle pins ----------------------------------------------------------

@pytest.mark.parametrize("S,M,align", [(12, 3, 1), (16, 4, 2), (10, 1, 1), (9, 9, 1), (14, 5, 1)])
def test_sum_is_invariant_under_linear_model(S, M, align):
    # Every (query, key) pair of the causal square is visible in exactly one
    # chunk, so under the linear model the sum of chunk costs is
    # cost_pair * S (S + 1) / 2 + cost_token * S + M * cost_chunk for ANY plan.
    lengths, t_max, t_sum = lbcp.lbcp_dp(S, M, 4, align, 3.0, 5.0, 7.0)
    assert sum(lengths) == S and len(lengths) == M
    assert all(c > 0 and c % align == 0 for c in lengths)
    assert t_sum == 3.0 * S * (S + 1) / 2 + 5.0 * S + 7.0 * M


@pytest.mark.parametrize("S,M", [(12, 3), (13, 4), (10, 2), (15, 5), (11, 11)])
@pytest.mark.parametrize("N", [2, 4, 10 ** 9])
def test_min_max_equals_brute_force(S, M, N):
    # Integer coefficients keep every cost exact; with a plan-independent sum
    # the objective t_sum + (N - 1) t_max is minimised exactly by the smallest
    # attainable largest chunk cost, which brute force finds.
    ev = linear(2.0, 1.0, 3.0)
    _, t_max, t_sum = lbcp.lbcp_dp(S, M, N, 1, evaluate=ev)
    best_max, _ = lbcp.brute_force(S, M, 1, max, ev)
    assert t_max == best_max


@pytest.mark.parametrize("S,M", [(12, 3), (13, 4), (9, 2), (10, 5)])
def test_single_stage_is_min_sum_for_any_cost(S, M):
    # N = 1 makes the objective additive, where the dynamic program is exact:
    # a position-dependent, non-linear cost checks the suffix bookkeeping.
    def ev(c, p):
        return c * c * c + 7 * p + ((c * 31 + p * 17) % 11)
    _, _, t_sum = lbcp.lbcp_dp(S, M, 1, 1, evaluate=ev)
    best_sum, _ = lbcp.brute_force(S, M, 1, sum, ev)
    assert t_sum == best_sum


@pytest.mark.parametrize("S,M", [(12, 3), (11, 4), (10, 3)])
def test_huge_stage_count_is_min_max_for_any_cost(S, M):
    # For N large enough that any difference in the largest chunk cost
    # outweighs any difference in the sum, the chosen suffix at every state
    # has the smallest attainable maximum, so the plan's maximum is optimal.
    def ev(c, p):
        return c * c + 3 * p + ((c * 13 + p * 7) % 5)
    _, t_max, _ = lbcp.lbcp_dp(S, M, 10 ** 9, 1, evaluate=ev)
    best_max, _ = lbcp.brute_force(S, M, 1, max, ev)
    assert t_max == best_max


@pytest.mark.parametrize("N", [1, 3, 8])
def test_reported_costs_match_plan(N):
    ev = linear(0.5, 2.0, 1.0)
    lengths, t_max, t_sum = lbcp.lbcp_dp(64, 5, N, 4, evaluate=ev)
    costs = lbcp.plan_costs(lengths, ev)
    assert t_max == max(costs)
    assert t_sum == pytest.approx(sum(costs), rel=1e-15)


def test_token_only_cost_gives_uniform_plan():
    # With cost proportional to chunk length only, the smallest maximum is the
    # ceiling of S / M (in align units).
    lengths, t_max, _ = lbcp.lbcp_dp(40 * 8, 6, 4, 8, 0.0, 1.0, 0.0)
    assert t_max == math.ceil(40 / 6) * 8
    assert max(lengths) == math.ceil(40 / 6) * 8


def test_pair_cost_tracks_square_root_boundaries():
    # Under the pair cost alone the balanced chunks have boundaries near
    # S sqrt(c / M) (the continuous optimum of the balanced plan); the
    # discrete min-max plan's boundaries stay within a few align units.
    S, M, align = 2048, 8, 16
    lengths, _, _ = lbcp.lbcp_dp(S, M, 10 ** 6, align, 1.0)
    dp_bounds = oplan.prefixes(lengths)[1:]
    cont = [S * math.sqrt(c / M) for c in range(1, M + 1)]
    assert all(abs(a - b) <= 3 * align for a, b in zip(dp_bounds, cont))
    # and its maximum is no worse than the rounded closed-form plan's.
    closed = oplan.balanced_plan(S, M, align)
    ev = linear(1.0)
    assert max(lbcp.plan_costs(lengths, ev)) <= max(lbcp.plan_costs(closed, ev))


def test_oracle_catches_planted_index_error():
    # A suffix looked up one position off must disagree with brute force.
    def bad_dp(S, M, N):
        ev = linear(2.0, 1.0, 3.0)
        # Plant the mistake by evaluating chunks one token behind where they start.
        return lbcp.lbcp_dp(S, M, N, 1, evaluate=lambda c, p: ev(c, max(p - 1, 0)))
    _, t_max, _ = bad_dp(13, 4, 10 ** 9)
    best_max, _ = lbcp.brute_force(13, 4, 1, max, linear(2.0, 1.0, 3.0))
    assert t_max != best_max


# --- library == oracle ----------------------------------------------------

def test_library_matches_oracle_exactly(mocap_lib):
    from paper_2606_22968_amd import binding
    rng = random.Random(7)
    cases = [(2048, 8, 4, 64), (4096, 16, 4, 128), (1024, 5, 1, 32), (1536, 12, 16, 64), (640, 10, 2, 64)]
    for S, M, N, align in cases:
        for _ in range(3):
            cp, ct, cc = rng.uniform(0, 1e-3), rng.uniform(0, 1e-1), rng.uniform(0, 50)
            got = binding.mocap_lbcp_plan(S, M, N, align, cp, ct, cc)
            want = lbcp.lbcp_dp(S, M, N, align, cp, ct, cc)
            assert got[0] == want[0], (S, M, N, align)
            assert got[1] == want[1] and got[2] == want[2]


def test_library_validation(mocap_lib):
    from paper_2606_22968_amd import binding
    bad = [
        dict(seq_len=1000, num_chunks=4, num_stages=4, align=64),   # not a multiple of align
        dict(seq_len=256, num_chunks=5, num_stages=4, align=64),    # more chunks than units
        dict(seq_len=256, num_chunks=0, num_stages=4, align=64),
        dict(seq_len=256, num_chunks=2, num_stages=0, align=64),
        dict(seq_len=256, num_chunks=2, num_stages=1, align=0),
    ]
    for kw in bad:
        with pytest.raises(binding.MocapError) as e:
            binding.mocap_lbcp_plan(**kw, cost_pair=1.0)
        assert e.value.status == binding.MOCAP_ERR_INVALID_ARG
    for cp in (-1.0, math.inf, math.nan):
        with pytest.raises(binding.MocapError):
            binding.mocap_lbcp_plan(256, 2, 2, 64, cp)
    with pytest.raises(binding.MocapError) as e:
        binding.mocap_lbcp_plan(1 << 20, 64, 4, 1, 1.0)
    assert e.value.status == binding.MOCAP_ERR_UNSUPPORTED


# --- latency model fit and probe plans (host logic) ----------------------

def test_fit_recovers_known_model():
    from paper_2606_22968_amd import lbcp as plbcp
    true = (2.5e-6, 3e-3, 40.0)
    rng = random.Random(3)
    samples = []
    for _ in range(60):
        c = rng.randrange(128, 32768, 128)
        p = rng.randrange(0, 131072 - c + 1, 128)
        t = true[0] * plbcp.visible_pairs(c, p) + true[1] * c + true[2]
        samples.append((c, p, t * (1 + rng.uniform(-1e-3, 1e-3))))
    m = plbcp.fit(samples)
    assert m.cost_pair == pytest.approx(true[0], rel=1e-2)
    assert m.cost_token == pytest.approx(true[1], rel=0.2)
    assert m.cost_chunk == pytest.approx(true[2], rel=0.2)
    assert m.rms_rel_err < 2e-3
    assert m(4096, 8192) == pytest.approx(lbcp.chunk_cost(4096, 8192, *true), rel=1e-2)


def test_fit_keeps_coefficients_non_negative():
    from paper_2606_22968_amd import lbcp as plbcp
    # Latency that falls with chunk length would need a negative token cost.
    samples = [(c, 0, 100.0 - 0.001 * c + 1e-6 * c * c) for c in range(128, 8192, 512)]
    m = plbcp.fit(samples)
    assert min(m.cost_pair, m.cost_token, m.cost_chunk) >= 0.0


def test_probe_plans_are_valid(mocap_lib):
    from paper_2606_22968_amd import lbcp as plbcp
    plans = plbcp.probe_plans(131072, 16, 128, seed=2, n_random=5)
    assert len(plans) == 7
    for lengths in plans:
        assert len(lengths) == 16 and sum(lengths) == 131072
        assert all(c > 0 and c % 128 == 0 for c in lengths)


# --- stage 2: simulated annealing ----------------------------------------

def _table(units, seed):
    """A seeded non-linear, position-dependent cost table [k-1][s] (align units)."""
    rng = random.Random(seed)
    jitter = [[rng.uniform(0.0, 3.0) for _ in range(units)] for _ in range(units)]
    t = [[0.0] * units for _ in range(units)]
    for k in range(1, units + 1):
        for s in range(units - k + 1):
            t[k - 1][s] = k * k * 0.7 + k * s * 1.3 + 5.0 + jitter[k - 1][s]
    return t


def test_splitmix64_reference_outputs():
    # First outputs of SplitMix64 from seed 0, as published with the
    # generator's reference implementation.
    g = lbcp.SplitMix64(0)
    assert [g.next() for _ in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_refine_reaches_brute_force_optimum(seed):
    U, M, N = 14, 4, 6
    t = _table(U, seed)
    ev = lambda c, p: t[c - 1][p]
    start = [U - 3, 1, 1, 1]
    lengths, lat = lbcp.lbcp_refine(U, M, N, 1, start, 200.0, 0.05, 0.97, 40, seed, ev)
    best, _ = lbcp.brute_force(U, M, 1, lambda costs: sum(costs) + (N - 1) * max(costs), ev)
    assert lat == pytest.approx(best, rel=1e-12)
    assert lbcp.prefill_latency(lengths, N, lambda k, s: t[k - 1][s]) == lat


def test_refine_at_zero_temperature_is_a_local_optimum():
    # With a vanishing temperature only improvements are accepted: no single
    # one-unit boundary move improves the result.
    U, M, N = 20, 5, 8
    t = _table(U, 9)
    ev = lambda c, p: t[c - 1][p]
    lengths, lat = lbcp.lbcp_refine(U, M, N, 1, [4] * 5, 1e-300, 1e-301, 0.5, 4000, 17, ev)
    evu = lambda k, s: t[k - 1][s]
    for j in range(1, M):
        for step in (1, -1):
            cand = list(lengths)
            cand[j - 1] += step
            cand[j] -= step
            if min(cand) >= 1:
                assert lbcp.prefill_latency(cand, N, evu) >= lat


def test_refine_never_worse_than_its_start():
    U, M, N = 30, 6, 4
    t = _table(U, 4)
    ev = lambda c, p: t[c - 1][p]
    start = [5] * 6
    lengths, lat = lbcp.lbcp_refine(U, M, N, 1, start, 50.0, 1.0, 0.9, 10, 5, ev)
    assert sum(lengths) == U and min(lengths) >= 1
    assert lat <= lbcp.prefill_latency(start, N, lambda k, s: t[k - 1][s])


def test_library_table_dp_and_refine_match_oracle(mocap_lib):
    import numpy as np
    from paper_2606_22968_amd import binding
    for U, M, N, align, seed in [(24, 5, 4, 64, 1), (40, 8, 16, 128, 2), (17, 1, 3, 32, 3), (33, 11, 2, 16, 4)]:
        t = np.array(_table(U, seed))
        ev = lambda c, p: float(t[c // align - 1][p // align])
        got = binding.mocap_lbcp_plan_table(U * align, M, N, align, t)
        want = lbcp.lbcp_dp(U * align, M, N, align, evaluate=ev)
        assert got[0] == want[0] and got[1] == want[1] and got[2] == want[2]
        for sa_seed in (7, 8):
            got_r = binding.mocap_lbcp_refine(U * align, M, N, align, t, got[0], 30.0, 0.5, 0.9, 12, sa_seed)
            want_r = lbcp.lbcp_refine(U * align, M, N, align, got[0], 30.0, 0.5, 0.9, 12, sa_seed, ev)
            assert got_r[0] == want_r[0] and got_r[1] == want_r[1], (U, M, seed, sa_seed)


def test_refine_and_table_validation(mocap_lib):
    import numpy as np
    from paper_2606_22968_amd import binding
    t = np.ones((8, 8))
    with pytest.raises(binding.MocapError):
        binding.mocap_lbcp_refine(512, 2, 2, 64, t, [256, 255], 1.0, 0.1, 0.5, 1, 0)   # not aligned
    with pytest.raises(binding.MocapError):
        binding.mocap_lbcp_refine(512, 2, 2, 64, t, [256, 128], 1.0, 0.1, 0.5, 1, 0)   # wrong total
    with pytest.raises(binding.MocapError):
        binding.mocap_lbcp_refine(512, 2, 2, 64, t, [256, 256], 1.0, 0.1, 1.0, 1, 0)   # alpha >= 1
    with pytest.raises(binding.MocapError):
        binding.mocap_lbcp_refine(512, 2, 2, 64, t, [256, 256], 0.0, 0.1, 0.5, 1, 0)   # temp0 <= 0
    bad = t.copy()
    bad[0][3] = np.nan
    with pytest.raises(binding.MocapError):
        binding.mocap_lbcp_plan_table(512, 2, 2, 64, bad)
    bad[0][3] = 1.0
    bad[7][1] = np.nan   # k = 8, s = 1: never read (k + s > U), so accepted
    lengths, _, _ = binding.mocap_lbcp_plan_table(512, 2, 2, 64, bad)
    assert sum(lengths) == 512 and min(lengths) >= 64


def test_cost_table_interpolates_the_measured_correction():
    from paper_2606_22968_amd import lbcp as plbcp
    model = plbcp.LatencyModel(2e-6, 1e-2, 30.0, 0.0)
    S, align = 4096, 128
    c_grid = [128, 512, 2048, 4096 - 128]
    grid = {}
    for c in c_grid:
        for f in (0.0, 0.5, 1.0):
            p = int(round(f * (S - c) / align)) * align
            grid[(c, p)] = model(c, p) * (1.5 if c >= 2048 else 1.0)
    t = plbcp.cost_table(grid, model, S, align)
    U = S // align
    assert t.shape == (U, U)
    assert t[0, 5] == pytest.approx(model(128, 5 * 128))               # factor 1 at a grid length
    assert t[2048 // 128 - 1, 3] == pytest.approx(1.5 * model(2048, 3 * 128))
    k = 1280 // 128  # halfway between 512 and 2048: factor 1.25
    assert t[k - 1, 7] == pytest.approx(1.25 * model(1280, 7 * 128))
    assert t[U - 1, 0] > 0 and t[0, U - 1] > 0
