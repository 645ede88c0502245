"""Pins of the fp64 oracle against facts fixed by the mathematics.

The paper prints no attention values, so the oracle is pinned by:
  * a library routine on the special case it reduces to: one chunk (P = 0)
    is monolithic causal attention, checked against torch's fp64
    scaled_dot_product_attention with is_causal (square case only: its mask
    is top-left aligned) and GQA head grouping;
  * the chunking invariant of Section 2.2 (a chunk sees every earlier chunk's
    keys plus its own, causally): concatenated chunk outputs equal a
    structurally different brute-force S x S computation for any split;
  * closed forms: Q = 0 gives uniform weights (LSE = ln(t+1), O = running
    mean of V); a single key gives LSE = s_0 and O = V_0; an overwhelming
    score picks out one V row;
  * invariants: probabilities of a row sum to one and vanish above the
    diagonal (read out through one-hot V rows);
  * the log-sum-exp merge identity over disjoint key sets.
"""
import numpy as np
import pytest
import torch

from oracle import bruteforce, merge


def chunked(oracle, q, k, v, lengths, scale):
    outs, lses, p = [], [], 0
    for n in lengths:
        o, lse = oracle.chunk_attn(q[p:p + n], k, v, p, scale)
        outs.append(o)
        lses.append(lse)
        p += n
    return np.concatenate(outs, axis=0), np.concatenate(lses, axis=1)


def rand_qkv(rng, S, h_q, h_kv, d):
    return (rng.standard_normal((S, h_q, d)), rng.standard_normal((S, h_kv, d)),
            rng.standard_normal((S, h_kv, d)))


@pytest.mark.parametrize("h_q,h_kv", [(4, 4), (4, 2), (6, 2), (8, 1)])
def test_single_chunk_matches_torch_sdpa(oracle_lib, h_q, h_kv):
    rng = np.random.default_rng(10 + h_q * 3 + h_kv)
    S, d, scale = 37, 16, 0.3
    q, k, v = rand_qkv(rng, S, h_q, h_kv, d)
    o, _ = oracle_lib.chunk_attn(q, k, v, 0, scale)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2)[None], torch.from_numpy(k).permute(1, 0, 2)[None],
        torch.from_numpy(v).permute(1, 0, 2)[None], is_causal=True, scale=scale,
        enable_gqa=True)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("lengths", [[64], [1, 63], [10, 1, 1, 30, 22], [7] * 9 + [1], [33, 31]])
def test_chunked_equals_monolithic_bruteforce(oracle_lib, lengths):
    rng = np.random.default_rng(sum(lengths) + len(lengths))
    S = sum(lengths)
    q, k, v = rand_qkv(rng, S, 4, 2, 8)
    o, lse = chunked(oracle_lib, q, k, v, lengths, 0.45)
    o_ref, lse_ref = bruteforce.monolithic(q, k, v, 0.45)
    np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref, rtol=0, atol=1e-12)


def test_random_splits_equal_monolithic(oracle_lib):
    rng = np.random.default_rng(7)
    S = 96
    q, k, v = rand_qkv(rng, S, 2, 1, 12)
    o_ref, lse_ref = bruteforce.monolithic(q, k, v, 0.25)
    for _ in range(6):
        cuts = sorted(rng.choice(np.arange(1, S), size=rng.integers(1, 8), replace=False).tolist())
        bounds = [0] + cuts + [S]
        lengths = [b - a for a, b in zip(bounds[:-1], bounds[1:])]
        o, lse = chunked(oracle_lib, q, k, v, lengths, 0.25)
        np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, lse_ref, rtol=0, atol=1e-12)


def test_probabilities_via_one_hot_values(oracle_lib):
    # V row j = e_j makes O[i] the attention weights of row i: they must sum
    # to one and be exactly zero for every key after the query's position.
    rng = np.random.default_rng(3)
    S, P = 24, 9
    q = rng.standard_normal((S, 1, S)) * 0.4
    k = rng.standard_normal((S, 1, S))
    v = np.eye(S)[:, None, :]
    o, _ = oracle_lib.chunk_attn(q[P:], k, v, P, 0.7)
    w = o[:, 0, :]
    np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-13)
    for i in range(S - P):
        assert np.all(w[i, P + i + 1:] == 0.0)
        assert np.all(w[i, :P + i + 1] > 0.0)
    ref = bruteforce.probabilities(q, k, 0.7)[P:]
    np.testing.assert_allclose(w, ref, rtol=0, atol=1e-13)


def test_zero_queries_give_uniform_weights(oracle_lib):
    rng = np.random.default_rng(4)
    S, P = 40, 15
    q = np.zeros((S - P, 3, 6))
    k = rng.standard_normal((S, 3, 6))
    v = rng.standard_normal((S, 3, 6))
    o, lse = oracle_lib.chunk_attn(q, k, v, P, 1.3)
    t = P + np.arange(S - P)
    np.testing.assert_allclose(lse, np.broadcast_to(np.log(t + 1.0), lse.shape), rtol=0, atol=1e-13)
    running_mean = np.cumsum(v, axis=0) / np.arange(1, S + 1)[:, None, None]
    np.testing.assert_allclose(o, running_mean[P:], rtol=0, atol=1e-13)


def test_single_key(oracle_lib):
    rng = np.random.default_rng(5)
    q, k, v = rand_qkv(rng, 1, 2, 1, 16)
    o, lse = oracle_lib.chunk_attn(q, k, v, 0, 0.2)
    for h in range(2):
        assert lse[h, 0] == pytest.approx(0.2 * float(q[0, h] @ k[0, 0]), abs=1e-13)
        np.testing.assert_array_equal(o[0, h], v[0, 0])


def test_dominant_score_selects_value_row(oracle_lib):
    rng = np.random.default_rng(6)
    S, d = 50, 32
    k = rng.standard_normal((S, 1, d))
    v = rng.standard_normal((S, 1, d))
    targets = [0, 17, 33, 49]
    q = np.stack([50.0 * k[j, 0] for j in targets])[:, None, :]
    # chunk of 4 query rows at positions 46..49 (all targets are visible)
    o, _ = oracle_lib.chunk_attn(q, k, v, S - 4, 0.2)
    for r, j in enumerate(targets):
        np.testing.assert_allclose(o[r, 0], v[j, 0], rtol=0, atol=1e-9)


def test_gqa_grouping_is_contiguous(oracle_lib):
    rng = np.random.default_rng(8)
    S = 12
    q, k, v = rand_qkv(rng, S, 4, 2, 8)
    v[:, 1, :] = 0.0
    o, _ = oracle_lib.chunk_attn(q, k, v, 0, 0.5)
    assert np.all(o[:, 2:, :] == 0.0)
    assert np.all(np.abs(o[:, :2, :]).sum(axis=-1) > 0)


def test_bf16_bits_equal_widened_fp64(oracle_lib):
    g = torch.Generator().manual_seed(9)
    q, k, v = (torch.randn(s, generator=g).to(torch.bfloat16) for s in [(20, 4, 16), (50, 2, 16), (50, 2, 16)])
    bits = [t.view(torch.int16).numpy().view(np.uint16) for t in (q, k, v)]
    wide = [t.double().numpy() for t in (q, k, v)]
    o1, l1 = oracle_lib.chunk_attn(*bits, 30, 0.25)
    o2, l2 = oracle_lib.chunk_attn(*wide, 30, 0.25)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_row_subset_matches_full(oracle_lib):
    rng = np.random.default_rng(11)
    q, k, v = rand_qkv(rng, 70, 4, 4, 8)
    o, lse = oracle_lib.chunk_attn(q[30:], k, v, 30, 0.3)
    rows = [0, 5, 39, 17]
    o_s, lse_s = oracle_lib.chunk_attn(q[30:], k, v, 30, 0.3, rows=rows)
    np.testing.assert_array_equal(o_s, o[rows])
    np.testing.assert_array_equal(lse_s, lse[:, rows])


def test_merge_of_disjoint_ranges_equals_direct(oracle_lib):
    rng = np.random.default_rng(12)
    S, P = 80, 50
    q, k, v = rand_qkv(rng, S, 4, 2, 8)
    o_ref, lse_ref = oracle_lib.chunk_attn(q[P:], k, v, P, 0.4)
    for cuts in ([20], [3, 40], [10, 20, 30, 45]):
        bounds = [0] + cuts + [P, S]
        parts = [merge.range_attn(q[P:], k, v, P, 0.4, a, b) for a, b in zip(bounds[:-1], bounds[1:])]
        o, lse = merge.merge([p[1] for p in parts], [p[0] for p in parts])
        np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, lse_ref, rtol=0, atol=1e-12)


def test_merge_closed_form():
    o1 = np.full((1, 1, 2), 1.0)
    o2 = np.full((1, 1, 2), 3.0)
    lse1 = np.full((1, 1), 0.7)
    o, lse = merge.merge([lse1, lse1], [o1, o2])
    assert lse[0, 0] == pytest.approx(0.7 + np.log(2.0), abs=1e-15)
    np.testing.assert_allclose(o, 2.0, atol=1e-15)
    # a part with no mass (lse = -inf) does not contribute
    o, lse = merge.merge([lse1, np.full((1, 1), -np.inf)], [o1, o2])
    np.testing.assert_allclose(o, 1.0, atol=1e-15)
    assert lse[0, 0] == pytest.approx(0.7, abs=1e-15)
