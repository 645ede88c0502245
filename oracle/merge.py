"""Attention over a key subset and the log-sum-exp merge -- TEST INFRASTRUCTURE.

The paper's memory-balanced reallocation (Section 4.1, runtime policy) lets a
debtor stage read its KV in two portions, a remote one and a local one.  The
attention of one query over the union of disjoint key sets equals the
combination of the per-set results weighted by their softmax mass:
    lse = log(sum_s exp(lse_s)),   o = sum_s exp(lse_s - lse) * o_s
where (o_s, lse_s) is ordinary attention restricted to set s.  These helpers
state that in fp64 so tests can pin the identity and check the HIP split path.
"""
import numpy as np


def range_attn(q, k, v, prefix_len, scale, key_lo, key_hi, rows=None):
    """fp64 attention of chunk rows over keys in [key_lo, key_hi) that are also
    causally visible (key <= prefix_len + row).

    q [L][Hq][d], k/v [>= key_hi][Hkv][d] float64.  Returns (o, lse) with
    o [n][Hq][d] and lse [Hq][n]; a row with no visible key in the range gets
    lse = -inf and o = 0.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    L, h_q, d = q.shape
    group = h_q // k.shape[1]
    rows = np.arange(L) if rows is None else np.asarray(rows)
    o = np.zeros((len(rows), h_q, d))
    lse = np.full((h_q, len(rows)), -np.inf)
    for n, i in enumerate(rows):
        hi = min(key_hi, prefix_len + int(i) + 1)
        if hi <= key_lo:
            continue
        for h in range(h_q):
            kvh = h // group
            s = scale * (k[key_lo:hi, kvh, :] @ q[i, h, :])
            m = s.max()
            w = np.exp(s - m)
            z = w.sum()
            o[n, h, :] = (w / z) @ v[key_lo:hi, kvh, :]
            lse[h, n] = m + np.log(z)
    return o, lse


def merge(lse_parts, o_parts):
    """Combine partial attention results over disjoint key sets.

    lse_parts [n_parts][Hq][n] and o_parts [n_parts][n][Hq][d] (float64).
    Parts with lse = -inf carry no mass.  Returns (o [n][Hq][d], lse [Hq][n]).
    """
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    o_parts = np.asarray(o_parts, dtype=np.float64)
    m = lse_parts.max(axis=0)
    lse = m + np.log(np.exp(lse_parts - m).sum(axis=0))
    w = np.exp(lse_parts - lse)                    # [n_parts][Hq][n]
    o = np.einsum("phn,pnhd->nhd", w, o_parts)
    return o, lse
