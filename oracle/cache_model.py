"""Where each token's K/V lives in the two caches, and the expected cache image.

The paper keeps an O(T) cache for retrieval heads and, for streaming heads, only
the s_sink sink tokens and the s_recent most recent tokens
(Sec. 5, decode and chunked-prefill stages; Sec. 1 footnote on sparsity).
This module is the plain definition of the two caches of this library, written
from that description and from the documented cache layout of the C interface:

  paged cache (retrieval KV heads, rank r = position of the head among the
  retrieval KV heads in ascending KV-head id), pages of 16 tokens:
      token p of sequence b  ->  physical page block_table[b][p // 16],
                                 row p % 16 of that page
      K page: [num_pages][n_ret][16][D]   (token-major inside a page)
      V page: [num_pages][n_ret][D][16]   (dimension-major inside a page), or
              [num_pages][n_ret][16][D] for a cache with token-major V pages
              (the option meant for H2Share reuse layers)

  ring cache (streaming KV heads, rank s among the streaming KV heads),
  capacity C = n_sink + window slots, padded to a multiple of 16:
      slot(p) = p                               if p <  n_sink
              = n_sink + (p - n_sink) % window  otherwise
      K ring: [B][n_str][Cpad/16][16][D];  V ring: [B][n_str][Cpad/16][D][16]
      slot c -> block c // 16, row c % 16.

Reading of what the paper leaves open: after any sequence of appends, each
slot holds the token with the greatest position that maps to it (later tokens
overwrite earlier ones, as eviction of the oldest recent token implies).
"""
import numpy as np

PAGE = 16


def ring_capacity(n_sink, window):
    return n_sink + window


def ring_capacity_padded(n_sink, window):
    c = n_sink + window
    return (c + PAGE - 1) // PAGE * PAGE


def ring_slot(p, n_sink, window):
    """Slot of token position p in a streaming head's ring."""
    if p < n_sink:
        return p
    return n_sink + (p - n_sink) % window


def ring_tokens(length, n_sink, window):
    """Token position held by each slot after tokens 0..length-1 were appended.

    Plain replay: append tokens in order, each overwriting its slot.
    Returns int64 [n_sink + window], -1 for a slot never written.
    """
    held = np.full(n_sink + window, -1, dtype=np.int64)
    for p in range(length):
        held[ring_slot(p, n_sink, window)] = p
    return held


def split_heads(head_is_streaming):
    """Retrieval and streaming KV-head ids, each in ascending order."""
    ret = [g for g, s in enumerate(head_is_streaming) if not s]
    st = [g for g, s in enumerate(head_is_streaming) if s]
    return ret, st


def paged_read_token(k_pages, v_pages, block_table, b, r, p, v_token_major=False):
    """(K row, V row) of token p of sequence b, retrieval rank r, per the layout."""
    page = int(block_table[b][p // PAGE])
    row = p % PAGE
    v_row = v_pages[page, r, row, :] if v_token_major else v_pages[page, r, :, row]
    return k_pages[page, r, row, :], v_row


def ring_read_slot(k_ring, v_ring, b, s, slot):
    """(K row, V row) stored in a ring slot, per the layout."""
    blk, row = slot // PAGE, slot % PAGE
    return k_ring[b, s, blk, row, :], v_ring[b, s, blk, :, row]


def check_paged(k_pages, v_pages, block_table, k_seq, v_seq, lens, head_is_streaming, v_token_major=False):
    """Compare every stored token of every retrieval head with the logical
    sequence, bit for bit.  Returns the number of mismatching tokens."""
    ret, _ = split_heads(head_is_streaming)
    bad = 0
    for b in range(len(lens)):
        for r, g in enumerate(ret):
            for p in range(int(lens[b])):
                kr, vr = paged_read_token(k_pages, v_pages, block_table, b, r, p, v_token_major)
                if not (np.array_equal(kr, k_seq[b, p, g]) and np.array_equal(vr, v_seq[b, p, g])):
                    bad += 1
    return bad


def check_ring(k_ring, v_ring, k_seq, v_seq, lens, head_is_streaming, n_sink, window):
    """Compare every written ring slot of every streaming head with the token
    ring_tokens() says it holds, bit for bit.  Returns the mismatch count."""
    _, st = split_heads(head_is_streaming)
    bad = 0
    for b in range(len(lens)):
        held = ring_tokens(int(lens[b]), n_sink, window)
        for s, g in enumerate(st):
            for slot, p in enumerate(held):
                if p < 0:
                    continue
                kr, vr = ring_read_slot(k_ring, v_ring, b, s, slot)
                if not (np.array_equal(kr, k_seq[b, p, g]) and np.array_equal(vr, v_seq[b, p, g])):
                    bad += 1
    return bad


def gather_paged(k_pages, v_pages, block_table, b, r, length, v_token_major=False):
    """K [length, D] and V [length, D] of sequence b, retrieval rank r, read
    through the block table per the layout (vectorised form of
    paged_read_token over positions 0..length-1)."""
    p = np.arange(length)
    pages = np.asarray(block_table[b])[p // PAGE]
    rows = p % PAGE
    v_rows = v_pages[pages, r, rows, :] if v_token_major else v_pages[pages, r, :, rows]
    return k_pages[pages, r, rows, :], v_rows


def gather_ring(k_ring, v_ring, b, s, length, n_sink, window):
    """(token positions held, K rows, V rows) of a streaming head's ring after
    `length` appends, per the layout and ring_tokens()."""
    held = ring_tokens(length, n_sink, window)
    slots = np.nonzero(held >= 0)[0]
    blk, row = slots // PAGE, slots % PAGE
    return held[slots], k_ring[b, s, blk, row, :], v_ring[b, s, blk, :, row]
