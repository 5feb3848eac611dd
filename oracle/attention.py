"""Masked-softmax attention for retrieval and streaming heads, in float64.

Follows the paper's statement of the method:
  * attention is softmax(Q K^T / sqrt(d)) V with the softmax in full precision
    (Appendix "Additional Efficiency Results", measurement protocol);
  * retrieval heads attend to the whole causal prefix; streaming heads keep only
    the first s_sink "sink" tokens and the s_recent most recent tokens
    (Sec. 5 "Deploying LLMs With AoH", decode stage and chunked-prefill stage;
    Sec. 3 observation-2 footnote: 128 sink + 256 recent);
  * outputs of both head types are concatenated along the head axis in the
    original head order (Sec. 5, Eq. 8);
  * GQA: H query heads form G groups of H/G consecutive heads that share one
    KV head, and the streaming/retrieval label is per KV group
    (Appendix "GQA Extension", group-level classification and weight
    reordering).

Readings of points the paper leaves open:
  * the recent window includes the current token: key j is in the window of
    query i when i - j < window, so a streaming query sees at most
    n_sink + window keys, the size of the streaming cache;
  * sink and window may overlap for early rows; the visible set is their union;
  * the prefill mask for streaming heads is the per-token sink + band mask
    (the chunk-size-independent form, equal to decode), not the chunk-eviction
    mask of a particular chunk size K;
  * query head h uses KV group g = h // (Hq // Hkv);
  * scale is exactly 1/sqrt(D); Q and K arrive after any positional encoding.

Inputs are converted to float64 from the exact values handed to the GPU (the
bf16 bit patterns upcast), so a comparison measures kernel error only.
"""
import numpy as np


def group_of(h, n_q_heads, n_kv_heads):
    """KV group of query head h (GQA: contiguous blocks of Hq/Hkv heads)."""
    return h // (n_q_heads // n_kv_heads)


def visible_mask(q_pos, n_keys, streaming, n_sink, window, chunk=0):
    """Boolean [len(q_pos), n_keys]: key j is visible to the query at position i.

    Retrieval: j <= i.
    Streaming, per-token band (chunk = 0): j <= i and (j < n_sink or i - j < window).
    Streaming, chunk eviction (chunk = K >= 1; Sec. 5 chunked-prefill stage):
    the prompt is processed in chunks of K tokens and after each chunk the cache
    keeps only the sink tokens and the `window` most recent tokens, so a query
    of the chunk starting at c = (i // K) * K sees the sink, the `window`
    tokens before c, and its own chunk up to itself:
        j <= i and (j < n_sink or j >= c - window).
    """
    i = np.asarray(q_pos, dtype=np.int64)[:, None]
    j = np.arange(n_keys, dtype=np.int64)[None, :]
    mask = j <= i
    if streaming:
        if chunk:
            lo = (i // chunk) * chunk - window
            mask = mask & ((j < n_sink) | (j >= lo))
        else:
            mask = mask & ((j < n_sink) | (i - j < window))
    return mask


def attend_rows(q_rows, q_pos, k, v, streaming, n_sink, window, chunk=0):
    """Attention output for a set of query rows of one head.

    q_rows [R, D] at absolute positions q_pos [R]; k, v [T, D] hold the keys and
    values of positions 0..T-1 of the KV head this query head reads.
    Returns [R, D] float64.  Row i: sum over visible j of e^{s_ij - m_i} v_j
    divided by sum over visible j of e^{s_ij - m_i}, with s_ij = q_i . k_j / sqrt(D)
    and m_i the largest visible score.
    """
    q_rows = np.asarray(q_rows, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    d = q_rows.shape[-1]
    s = (q_rows @ k.T) / np.sqrt(d)
    mask = visible_mask(q_pos, k.shape[0], streaming, n_sink, window, chunk)
    if not mask.any(axis=1).all():
        raise ValueError("a query row has no visible key")
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    return (p @ v) / p.sum(axis=1, keepdims=True)


def attention_weights(q_rows, q_pos, k, streaming, n_sink, window):
    """The attention-probability matrix P [R, T] for one head (tiny inputs)."""
    q_rows = np.asarray(q_rows, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    s = (q_rows @ k.T) / np.sqrt(q_rows.shape[-1])
    mask = visible_mask(q_pos, k.shape[0], streaming, n_sink, window)
    s = np.where(mask, s, -np.inf)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    return p / p.sum(axis=1, keepdims=True)


def prefill(q, k, v, head_is_streaming, n_sink, window, rows=None, row_block=512, chunk=0):
    """Head-mixed causal prefill.

    q [B, T, Hq, D]; k, v [B, T, Hkv, D]; head_is_streaming [Hkv] (0/1).
    rows: optional sorted positions to evaluate (default: all T rows).
    chunk: 0 for the per-token band mask, K >= 1 for chunk eviction.
    Returns [B, len(rows), Hq, D] float64 in the original query-head order.
    """
    q = np.asarray(q)
    b_n, t_n, hq, d = q.shape
    hkv = k.shape[2]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    rows = np.arange(t_n) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((b_n, len(rows), hq, d), dtype=np.float64)
    for b in range(b_n):
        for h in range(hq):
            g = group_of(h, hq, hkv)
            kg = np.asarray(k[b, :, g, :], dtype=np.float64)
            vg = np.asarray(v[b, :, g, :], dtype=np.float64)
            for r0 in range(0, len(rows), row_block):
                pos = rows[r0:r0 + row_block]
                hi = int(pos.max()) + 1  # keys beyond the last row are never visible
                out[b, r0:r0 + len(pos), h, :] = attend_rows(
                    np.asarray(q[b, pos, h, :], dtype=np.float64), pos,
                    kg[:hi], vg[:hi], bool(head_is_streaming[g]), n_sink, window, chunk)
    return out


def decode(q, k_seq, v_seq, lens, head_is_streaming, n_sink, window):
    """One decode step per sequence, computed from the logical sequence.

    q [B, Hq, D] is the query of the token at position lens[b] - 1;
    k_seq, v_seq [B, Lmax, Hkv, D] hold every token appended so far (no cache,
    no eviction: the mask alone decides what a streaming head sees).
    Returns [B, Hq, D] float64.  This equals row lens[b]-1 of prefill() over
    tokens 0..lens[b]-1.
    """
    b_n, hq, d = q.shape
    hkv = k_seq.shape[2]
    out = np.empty((b_n, hq, d), dtype=np.float64)
    for b in range(b_n):
        p = int(lens[b]) - 1
        for g in range(hkv):
            kg = np.asarray(k_seq[b, :p + 1, g, :], dtype=np.float64)
            vg = np.asarray(v_seq[b, :p + 1, g, :], dtype=np.float64)
            for h in range(hq):
                if group_of(h, hq, hkv) != g:
                    continue
                out[b, h] = attend_rows(np.asarray(q[b, h][None, :], dtype=np.float64), [p], kg, vg,
                                        bool(head_is_streaming[g]), n_sink, window)[0]
    return out


def brute_force(q, k, v, head_is_streaming, n_sink, window, chunk=0):
    """Second, independent path for tiny inputs (T <= 64).

    Builds the dense visibility matrix with explicit Python loops from the
    rule "causal, and for streaming heads sink or recent", then applies the
    textbook softmax exp(s) / sum exp(s) without max-subtraction, one element
    at a time.  Shares nothing with prefill() but numpy's scalar exp.
    """
    b_n, t_n, hq, d = q.shape
    hkv = k.shape[2]
    gs = hq // hkv
    out = np.zeros((b_n, t_n, hq, d), dtype=np.float64)
    for b in range(b_n):
        for h in range(hq):
            g = h // gs
            stream = bool(head_is_streaming[g])
            for i in range(t_n):
                keep = []
                for j in range(t_n):
                    if j > i:
                        continue
                    if stream:
                        if chunk:
                            # the cache before i's chunk: sink + the window tokens before it
                            chunk_start = i - i % chunk
                            if not (j < n_sink or j >= chunk_start - window):
                                continue
                        elif not (j < n_sink or j >= i - window + 1):
                            continue
                    keep.append(j)
                w = []
                for j in keep:
                    s = 0.0
                    for e in range(d):
                        s += float(q[b, i, h, e]) * float(k[b, j, g, e])
                    w.append(np.exp(s / np.sqrt(d)))
                z = sum(w)
                for wj, j in zip(w, keep):
                    out[b, i, h, :] += (wj / z) * np.asarray(v[b, j, g, :], dtype=np.float64)
    return out
