"""Prefill that fills the caches (aoh_prefill_append) on the GPU.

For each case the caches start NaN-filled; the fused call must leave
* the attention output bit-identical to aoh_prefill / aoh_prefill_chunked,
* every cache slot bit-identical to what aoh_prefill + aoh_kv_append(start 0)
  leave in a second pair of NaN-filled caches (so no slot is written that the
  separate append would not write, and none is missed),
* and the stored tokens equal to the prompt per the oracle's cache model.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import cache_model as CM
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_kv_append, aoh_prefill, aoh_prefill_append,
                                  aoh_prefill_chunked)
from tests.helpers import bits, to_dtype

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _caches(B, T, mask, D, dtype, n_sink, window, seed, extra_pages=3):
    n_ret, n_str = mask.count(0), mask.count(1)
    max_pages = (T + 15) // 16 + 1
    perm = synth.page_permutation(B * max_pages + extra_pages, seed, "append-pages")[:B * max_pages]
    bt = torch.from_numpy(perm.reshape(B, max_pages).astype(np.int32))
    full = PagedCache.allocate(B * max_pages + extra_pages, n_ret, D, dtype, bt) if n_ret else None
    ring = RingCache.allocate(B, n_str, n_sink, window, D, dtype) if n_str else None
    for c in (full, ring):
        if c is not None:
            c.k.fill_(float("nan"))
            c.v.fill_(float("nan"))
    return full, ring


CASES = [
    # B, T, Hq, Hkv, D, mask, n_sink, window, chunk, dtype
    (2, 300, 8, 2, 128, [1, 0], 4, 100, 0, torch.bfloat16),     # ragged tail, partial last page
    (1, 1000, 14, 2, 128, [0, 1], 64, 128, 0, torch.bfloat16),  # GQA 7, several query blocks
    (1, 777, 4, 4, 64, [1, 0, 0, 1], 70, 33, 0, torch.bfloat16),  # d 64, sink over two tiles
    (1, 513, 8, 2, 128, [1, 0], 8, 64, 100, torch.bfloat16),    # chunk-eviction mask
    (3, 17, 4, 2, 128, [1, 0], 2, 8, 0, torch.bfloat16),        # one page + 1 token
    (1, 64, 4, 2, 128, [1, 1], 80, 32, 0, torch.bfloat16),      # sink longer than the prompt
    (1, 1, 4, 2, 128, [0, 1], 4, 16, 0, torch.bfloat16),        # single token
    (1, 2048, 8, 8, 128, [0] * 8, 64, 1024, 0, torch.bfloat16),  # all retrieval
    (1, 300, 4, 2, 64, [1, 0], 4, 100, 0, torch.float32),       # fp32: separate append launch
]


@pytest.mark.parametrize("B,T,Hq,Hkv,D,mask,n_sink,window,chunk,dtype", CASES)
def test_prefill_append_matches_separate_calls(B, T, Hq, Hkv, D, mask, n_sink, window, chunk, dtype):
    seed = T * 3 + Hq
    q = to_dtype(synth.gaussian((B, T, Hq, D), seed, "q"), dtype).to(DEV)
    k = to_dtype(synth.gaussian((B, T, Hkv, D), seed, "k"), dtype).to(DEV)
    v = to_dtype(synth.gaussian((B, T, Hkv, D), seed, "v"), dtype).to(DEV)
    f1, r1 = _caches(B, T, mask, D, dtype, n_sink, window, seed)
    f2, r2 = _caches(B, T, mask, D, dtype, n_sink, window, seed)
    out1 = aoh_prefill_append(q, k, v, mask, n_sink, window, f1, r1, chunk=chunk)
    out2 = aoh_prefill_chunked(q, k, v, mask, n_sink, window, chunk) if chunk else aoh_prefill(q, k, v, mask, n_sink, window)
    aoh_kv_append(k, v, mask, torch.zeros(B, dtype=torch.int32, device=DEV), f2, r2, n_sink, window)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out1), bits(out2)), "output differs from the plain prefill"
    for a, b_, name in ((f1, f2, "paged"), (r1, r2, "ring")):
        if a is None:
            continue
        assert np.array_equal(bits(a.k), bits(b_.k)), f"{name} K differs from the separate append"
        assert np.array_equal(bits(a.v), bits(b_.v)), f"{name} V differs from the separate append"
    kb, vb = bits(k), bits(v)
    lens = [T] * B
    if f1 is not None:
        assert CM.check_paged(bits(f1.k), bits(f1.v), f1.block_table.cpu().numpy(), kb, vb, lens, mask) == 0
    if r1 is not None:
        assert CM.check_ring(bits(r1.k), bits(r1.v), kb, vb, lens, mask, n_sink, window) == 0


def _check_caches_against_prompt(full, ring, k, v, mask, T, n_sink, window, what):
    """Every stored token of both caches equals the prompt, bit for bit, read
    through the oracle's placement model (vectorised readers)."""
    kb, vb = bits(k), bits(v)
    ret, st = CM.split_heads(mask)
    fk, fv, btn = bits(full.k), bits(full.v), full.block_table.cpu().numpy()
    for r, g in enumerate(ret):
        K, V = CM.gather_paged(fk, fv, btn, 0, r, T)
        assert np.array_equal(K, kb[0, :T, g]) and np.array_equal(V, vb[0, :T, g]), f"{what}: paged head {g}"
    rk, rv = bits(ring.k), bits(ring.v)
    for s, g in enumerate(st):
        pos, K, V = CM.gather_ring(rk, rv, 0, s, T, n_sink, window)
        assert np.array_equal(K, kb[0, pos, g]) and np.array_equal(V, vb[0, pos, g]), f"{what}: ring head {g}"
        assert len(pos) == min(T, n_sink + window), f"{what}: ring slots held"


def test_prefill_append_qwen_32k_one_launch():
    # The benchmark's prefill: Qwen2.5-7B-shaped layer, 32768 tokens, KV heads 1
    # and 3 streaming, both head types in one launch that also fills the caches.
    w = synth.qwen_prefill_inputs()
    q, k, v = (torch.from_numpy(w[n]).to(torch.bfloat16).to(DEV) for n in ("q", "k", "v"))
    del w
    mask, n_sink, window = [0, 1, 0, 1], 64, 1024
    T = q.shape[1]
    max_pages = (T + 1 + 15) // 16
    bt = torch.arange(max_pages, dtype=torch.int32)[None]
    full = PagedCache.allocate(max_pages, 2, 128, torch.bfloat16, bt)
    ring = RingCache.allocate(1, 2, n_sink, window, 128, torch.bfloat16)
    for c in (full, ring):
        c.k.fill_(float("nan"))
        c.v.fill_(float("nan"))
    out_a = aoh_prefill_append(q, k, v, mask, n_sink, window, full, ring)
    out_p = aoh_prefill(q, k, v, mask, n_sink, window)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_p)), "fused-append output differs from aoh_prefill"
    _check_caches_against_prompt(full, ring, k, v, mask, T, n_sink, window, "qwen 32k")
    # the page past the prompt (position T, the next decode token) is untouched
    assert torch.isnan(full.k[T // 16, :, T % 16:].float()).all()
    print("qwen 32k: fused-append output bit-identical, caches bit-exact")


def test_prefill_append_stack_layer_262144():
    # One layer of the 28-layer stack at its full length: two launches (one per
    # head type) that fill the caches as they go.
    c = synth.CONFIGS["qwen25_stack_256k"]
    T, n_sink, window = c["seq"], c["n_sink"], c["window"]
    w = synth.stack_layer_inputs(0)
    mask = w["mask"]
    q, k, v = (torch.from_numpy(w[n]).to(torch.bfloat16).to(DEV) for n in ("q", "k", "v"))
    del w
    max_pages = (T + 15) // 16
    perm = synth.page_permutation(max_pages, 77, "stack-append-pages")
    bt = torch.from_numpy(perm[None].astype(np.int32))
    full = PagedCache.allocate(max_pages, mask.count(0), 128, torch.bfloat16, bt)
    ring = RingCache.allocate(1, mask.count(1), n_sink, window, 128, torch.bfloat16)
    for cc in (full, ring):
        cc.k.fill_(float("nan"))
        cc.v.fill_(float("nan"))
    out_a = aoh_prefill_append(q, k, v, mask, n_sink, window, full, ring)
    torch.cuda.synchronize()
    out_a = out_a.cpu()
    out_p = aoh_prefill(q, k, v, mask, n_sink, window)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_p)), "fused-append output differs from aoh_prefill"
    del out_p, q
    _check_caches_against_prompt(full, ring, k, v, mask, T, n_sink, window, "stack layer 0, 262144")
    print("stack layer 262144: fused-append output bit-identical, caches bit-exact")
