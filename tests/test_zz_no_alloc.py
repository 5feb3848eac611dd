"""The decode step that allocates nothing (aoh_decode_step_noalloc), through
the C interface, against aoh_decode_step with a caller workspace: outputs and
both caches bit-identical, on two calls in a row, the second with a smaller
input (the static scratch area keeps the first call's contents)."""
import numpy as np
import pytest
import torch

import synth
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode_step, aoh_decode_step_noalloc,
                                  aoh_decode_workspace_bytes, aoh_kv_append)
from tests.helpers import bits

pytestmark = pytest.mark.gpu
DEV = "cuda"
BF = torch.bfloat16


def _setup(B, L, Hq, Hkv, D, mask, n_sink, window, seed):
    """Two identical cache pairs filled with L seeded tokens per sequence, the
    step's query and new token."""
    k = torch.from_numpy(synth.gaussian((B, L, Hkv, D), seed, "na-k")).to(BF).to(DEV)
    v = torch.from_numpy(synth.gaussian((B, L, Hkv, D), seed, "na-v")).to(BF).to(DEV)
    max_pages = (L + 1 + 15) // 16
    perm = synth.page_permutation(B * max_pages, seed, "na-pages")
    bt = torch.from_numpy(perm.reshape(B, max_pages).astype(np.int32))
    pairs = []
    for _ in range(2):
        full = PagedCache.allocate(B * max_pages, mask.count(0), D, BF, bt)
        ring = RingCache.allocate(B, mask.count(1), n_sink, window, D, BF)
        for c in (full, ring):
            c.k.fill_(float("nan"))
            c.v.fill_(float("nan"))
        aoh_kv_append(k, v, mask, torch.zeros(B, dtype=torch.int32, device=DEV), full, ring, n_sink, window)
        pairs.append((full, ring))
    q = torch.from_numpy(synth.gaussian((B, Hq, D), seed, "na-q")).to(BF).to(DEV)
    kn = torch.from_numpy(synth.gaussian((B, Hkv, D), seed, "na-kn")).to(BF).to(DEV)
    vn = torch.from_numpy(synth.gaussian((B, Hkv, D), seed, "na-vn")).to(BF).to(DEV)
    lens = torch.full((B,), L + 1, dtype=torch.int32, device=DEV)
    return pairs, q, kn, vn, lens, max_pages


def _compare(B, L, Hq, Hkv, D, mask, n_sink, window, seed):
    pairs, q, kn, vn, lens, max_pages = _setup(B, L, Hq, Hkv, D, mask, n_sink, window, seed)
    (f1, r1), (f2, r2) = pairs
    out_na = aoh_decode_step_noalloc(q, kn, vn, f1, r1, mask, lens, n_sink, window)
    ws = torch.empty(aoh_decode_workspace_bytes(B, Hq, D, max_pages, n_sink + window), dtype=torch.uint8, device=DEV)
    out_ws = aoh_decode_step(q, kn, vn, f2, r2, mask, lens, n_sink, window, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_na), bits(out_ws)), f"output differs {B, L, Hq, Hkv, D}"
    for a, b, name in ((f1.k, f2.k, "paged K"), (f1.v, f2.v, "paged V"), (r1.k, r2.k, "ring K"), (r1.v, r2.v, "ring V")):
        assert np.array_equal(bits(a), bits(b)), f"{name} differs {B, L, Hq, Hkv, D}"
    return out_na


def test_noalloc_step_matches_workspace_step_twice():
    # first call: batch 8 x 9000 tokens, Llama-3-8B-shaped heads (4 of 8 KV heads streaming)
    o1 = _compare(8, 9000, 32, 8, 128, [0, 1, 0, 1, 1, 0, 0, 1], 64, 1024, 31)
    # second call, smaller: batch 2 x 700 tokens, GQA 4, d_head 64
    o2 = _compare(2, 700, 8, 2, 64, [1, 0], 4, 100, 32)
    assert o1.shape != o2.shape
