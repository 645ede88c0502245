"""Monolithic causal prefill by brute force -- TEST INFRASTRUCTURE.

A deliberately different construction from ``oracle.chunk_attn``: no chunks,
no prefix bookkeeping, no per-row loops.  For every head the whole S x S
score matrix is formed, entries above the diagonal are set to -inf, and each
row is normalised.  Chunked prefill (Section 2.2 of the paper: a chunk sees
every earlier chunk's keys plus its own, causally) must reproduce exactly
this result for any chunk split, which is what the oracle tests check.
"""
import numpy as np


def monolithic(q, k, v, scale):
    """q [S][Hq][d], k/v [S][Hkv][d] float64 -> (o [S][Hq][d], lse [Hq][S])."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    S, h_q, d = q.shape
    h_kv = k.shape[1]
    group = h_q // h_kv
    above = np.triu(np.ones((S, S), dtype=bool), 1)
    o = np.empty((S, h_q, d))
    lse = np.empty((h_q, S))
    for h in range(h_q):
        kvh = h // group
        scores = scale * (q[:, h, :] @ k[:, kvh, :].T)
        scores[above] = -np.inf
        row_max = scores.max(axis=1, keepdims=True)
        w = np.exp(scores - row_max)
        z = w.sum(axis=1, keepdims=True)
        o[:, h, :] = (w / z) @ v[:, kvh, :]
        lse[h] = (row_max + np.log(z))[:, 0]
    return o, lse


def probabilities(q, k, scale, head=0, group=1):
    """Row-normalised causal attention weights of one head (S x S), for checks."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    S = q.shape[0]
    scores = scale * (q[:, head, :] @ k[:, head // group, :].T)
    scores[np.triu(np.ones((S, S), dtype=bool), 1)] = -np.inf
    w = np.exp(scores - scores.max(axis=1, keepdims=True))
    return w / w.sum(axis=1, keepdims=True)
