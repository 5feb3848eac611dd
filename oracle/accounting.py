"""Counting formulas: visible pairs, useful FLOPs, KV bytes.

* Sparsity is the fraction of streaming heads (Sec. 1 footnote); with G KV
  groups and target sparsity s the k = ceil((1 - s) G) lowest-rank groups are
  retrieval groups (Sec. 4 group-level classification; the source prints the
  product as "(1-s),G", read here as (1-s)*G).
* A streaming head stores s_sink + s_recent tokens, a retrieval head all T
  tokens (Sec. 5); resident KV bytes per layer are therefore
  D * 2 (K and V) * elt * (G_r * T + G_s * min(T, n_sink + window)).
  With 128 + 256 cache tokens this reproduces the KV-memory columns of the
  efficiency tables (Appendix "Additional Efficiency Results") and the 32K
  LongBench KV-memory table (Appendix "Details on Baseline Budgets").
"""
import math


def n_retrieval_groups(n_groups, sparsity):
    """k = ceil((1 - s) * G), computed exactly for s given in percent or as a
    float with at most a few decimals (avoids ceil(3.0000000004) = 4)."""
    return math.ceil(round((1.0 - sparsity) * n_groups, 9))


def visible_pairs_row(i, streaming, n_sink, window):
    """Number of keys visible to the query at position i."""
    if not streaming:
        return i + 1
    recent = min(i + 1, window)
    sink = min(n_sink, max(0, i + 1 - window))
    return recent + sink


def visible_pairs(t, streaming, n_sink, window):
    """Sum of visible_pairs_row over rows 0..t-1, in closed form."""
    if not streaming:
        return t * (t + 1) // 2
    # recent part: sum_{i<t} min(i+1, window)
    w = min(window, t)
    recent = w * (w + 1) // 2 + (t - w) * window
    # sink part: sum_{i<t} min(n_sink, max(0, i+1-window)); let u = i+1-window in 1..t-window
    m = max(0, t - window)
    if m <= n_sink:
        sink = m * (m + 1) // 2
    else:
        sink = n_sink * (n_sink + 1) // 2 + (m - n_sink) * n_sink
    return recent + sink


def prefill_flops(t, d, n_q_heads_retrieval, n_q_heads_streaming, n_sink, window, batch=1):
    """Useful prefill FLOPs: 4 D per visible (query, key) pair (2D for Q K^T,
    2D for P V); the exponentials are not counted."""
    pr = visible_pairs(t, False, n_sink, window)
    ps = visible_pairs(t, True, n_sink, window)
    return 4 * d * batch * (n_q_heads_retrieval * pr + n_q_heads_streaming * ps)


def kv_cache_bytes(n_layers, d, elt_bytes, g_ret, g_str, t, n_sink, window):
    """Resident KV-cache bytes for one sequence of length t."""
    return n_layers * d * 2 * elt_bytes * (g_ret * t + g_str * min(t, n_sink + window))


def decode_kv_bytes(lens, g_ret, g_str, d, elt_bytes, n_sink, window):
    """KV bytes one decode step must read: every retrieval token and every
    live ring slot, K and V."""
    tot = 0
    for n in lens:
        tot += (g_ret * n + g_str * min(n, n_sink + window)) * d * 2 * elt_bytes
    return tot
