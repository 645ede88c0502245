"""Chunk plans and work accounting (host only).

The oracle's plans are pinned by the exact integer definition of "nearest
multiple of the alignment to S sqrt(c/M)", by the balance they are meant to
achieve, and by brute-force counting of visible pairs; the library's integer
planner (mocap_chunk_plan) must then agree with the oracle exactly.
"""
import os
import random

import pytest

from oracle import plan

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "balanced_plan_131072x16_align128.txt")


def _golden_lengths():
    with open(GOLDEN) as f:
        return [int(x) for x in [ln for ln in f if not ln.startswith("#")][0].split()]


def _is_nearest_multiple(bound, S, c, M, align):
    # k = bound/align is the integer nearest to u = (S/align) sqrt(c/M):
    # (2k-1)^2 M <= 4 A^2 c <= (2k+1)^2 M, with A = S/align.
    k, A = bound // align, S // align
    return bound % align == 0 and (2 * k - 1) ** 2 * M <= 4 * A * A * c <= (2 * k + 1) ** 2 * M


def test_balanced_plan_matches_definition():
    S, M, a = 131072, 16, 128
    lengths = plan.balanced_plan(S, M, a)
    assert lengths == _golden_lengths()
    assert sum(lengths) == S
    bounds = [sum(lengths[:c]) for c in range(1, M)]
    for c, b in enumerate(bounds, start=1):
        assert _is_nearest_multiple(b, S, c, M, a)
    assert all(x >= y for x, y in zip(lengths, lengths[1:]))  # later chunks are shorter
    costs = [plan.balance_cost(n, p) for n, p in zip(lengths, plan.prefixes(lengths))]
    assert max(costs) / min(costs) < 1.04
    # Uniform chunks of the same sequence are far from balanced (Eq. (1)).
    uni = plan.uniform_plan(S, M)
    ucost = [plan.balance_cost(n, p) for n, p in zip(uni, plan.prefixes(uni))]
    assert max(ucost) / min(ucost) == pytest.approx(31.0)


@pytest.mark.parametrize("S,M,a", [(8192, 4, 64), (65536, 32, 128), (12800, 10, 128), (4096, 3, 128)])
def test_balanced_plan_definition_other_sizes(S, M, a):
    lengths = plan.balanced_plan(S, M, a)
    assert sum(lengths) == S
    for c in range(1, M):
        assert _is_nearest_multiple(sum(lengths[:c]), S, c, M, a)


def test_uniform_plan():
    assert plan.uniform_plan(32768, 16) == [2048] * 16
    assert plan.uniform_plan(10, 3) == [3, 3, 4]


def test_visible_pairs_brute_force():
    for L, P in [(1, 0), (5, 0), (4, 3), (7, 11), (16, 1)]:
        count = sum(1 for i in range(L) for j in range(P + L) if j <= P + i)
        assert plan.visible_pairs(L, P) == count


def test_flops_independent_of_chunking():
    rng = random.Random(0)
    S = 5000
    for _ in range(20):
        cuts = sorted(rng.sample(range(1, S), rng.randint(1, 30)))
        b = [0] + cuts + [S]
        lengths = [y - x for x, y in zip(b[:-1], b[1:])]
        assert sum(plan.visible_pairs(n, p) for n, p in zip(lengths, plan.prefixes(lengths))) == S * (S + 1) // 2
    assert plan.causal_flops([2048] * 16, 32, 128) == 4 * 128 * 32 * 32768 * 32769 // 2


def test_library_planner_matches_oracle(mocap_lib):
    cases = [(131072, 16, 128), (32768, 16, 128), (8192, 4, 64), (65536, 32, 128), (12800, 10, 128),
             (4096, 3, 128), (1 << 20, 64, 256)]
    for S, M, a in cases:
        assert mocap_lib.mocap_chunk_plan(S, M, a, balanced=True) == plan.balanced_plan(S, M, a)
    for S, M in [(32768, 16), (10, 3), (1000, 7), (131072, 32)]:
        assert mocap_lib.mocap_chunk_plan(S, M, 1, balanced=False) == plan.uniform_plan(S, M)


def test_library_planner_rejects_bad_input(mocap_lib):
    with pytest.raises(mocap_lib.MocapError):
        mocap_lib.mocap_chunk_plan(1000, 4, 128, balanced=True)   # S not a multiple of align
    with pytest.raises(mocap_lib.MocapError):
        mocap_lib.mocap_chunk_plan(3, 5, 1, balanced=False)       # empty chunks
    with pytest.raises(mocap_lib.MocapError):
        mocap_lib.mocap_chunk_plan(256, 4, 128, balanced=True)    # rounding leaves a chunk empty


def test_oracle_prefixes_invariants():
    # P_0 = 0, P_{c+1} = P_c + L_c, and the last prefix plus its chunk is S.
    rng = random.Random(11)
    for _ in range(20):
        lengths = [rng.randint(0, 300) for _ in range(rng.randint(1, 40))]
        p = plan.prefixes(lengths)
        assert p[0] == 0
        assert all(p[c + 1] == p[c] + lengths[c] for c in range(len(lengths) - 1))
        assert p[-1] + lengths[-1] == sum(lengths)
        # P_c counts the tokens that belong to earlier chunks, one by one.
        owner = [c for c, n in enumerate(lengths) for _ in range(n)]
        assert p == [sum(1 for o in owner if o < c) for c in range(len(lengths))]


def test_library_prefixes_match_oracle(mocap_lib):
    rng = random.Random(12)
    cases = [[1], [0, 0, 3], plan.balanced_plan(131072, 16, 128), [2**31 - 1] * 5]
    cases += [[rng.randint(0, 100000) for _ in range(rng.randint(1, 64))] for _ in range(10)]
    for lengths in cases:
        assert mocap_lib.mocap_chunk_prefixes(lengths) == plan.prefixes(lengths)
    assert mocap_lib.mocap_chunk_prefixes([]) == []


def test_library_prefixes_reject(mocap_lib):
    with pytest.raises(mocap_lib.MocapError):
        mocap_lib.mocap_chunk_prefixes([5, -1, 3])
    lib = mocap_lib.load_library()
    out = (mocap_lib.ctypes.c_int64 * 2)()
    assert lib.mocap_chunk_prefixes(None, 2, out) == mocap_lib.MOCAP_ERR_INVALID_ARG
    assert lib.mocap_chunk_prefixes(None, -1, out) == mocap_lib.MOCAP_ERR_INVALID_ARG
