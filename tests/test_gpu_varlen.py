"""Packed variable-length prefill (aoh_prefill_varlen) on the GPU.

Every sequence's rows must be bit-identical to aoh_prefill / aoh_prefill_chunked
on that sequence alone (same kernels, same tiles), the caches filled by the
packed call bit-identical to per-sequence fused appends, and sampled rows
within the bf16 bar of the oracle.  Includes empty sequences, a single token,
max_seqlen above every length, GQA 7, d 64 and fp32.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_prefill, aoh_prefill_append, aoh_prefill_chunked,
                                  aoh_prefill_varlen)
from tests.helpers import assert_parity, bits, f64, to_dtype

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _packed(lens, hq, hkv, d, dtype, seed):
    tot = int(sum(lens))
    q = to_dtype(synth.gaussian((max(tot, 1), hq, d), seed, "vl-q"), dtype)[:tot].to(DEV)
    k = to_dtype(synth.gaussian((max(tot, 1), hkv, d), seed, "vl-k"), dtype)[:tot].to(DEV)
    v = to_dtype(synth.gaussian((max(tot, 1), hkv, d), seed, "vl-v"), dtype)[:tot].to(DEV)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device=DEV)
    return q, k, v, cu


CASES = [
    # lens, hq, hkv, d, mask, n_sink, window, chunk, dtype
    ([1, 17, 300, 256, 1000, 513, 2048], 14, 2, 128, [0, 1], 64, 128, 0, torch.bfloat16),
    ([700, 0, 33, 1500], 8, 2, 128, [1, 0], 4, 100, 0, torch.bfloat16),      # an empty sequence
    ([400, 1200, 64], 4, 4, 64, [1, 0, 0, 1], 16, 50, 96, torch.bfloat16),  # d 64, chunk eviction
    ([130, 1, 77], 4, 2, 64, [0, 1], 4, 32, 0, torch.float32),               # fp32
]


@pytest.mark.parametrize("lens,hq,hkv,d,mask,n_sink,window,chunk,dtype", CASES)
def test_varlen_equals_per_sequence(lens, hq, hkv, d, mask, n_sink, window, chunk, dtype):
    q, k, v, cu = _packed(lens, hq, hkv, d, dtype, seed=len(lens) * 11 + d)
    out = aoh_prefill_varlen(q, k, v, cu, max(lens) + 37, mask, n_sink, window, chunk=chunk)
    torch.cuda.synchronize()
    off = 0
    for i, n in enumerate(lens):
        if n == 0:
            continue
        qs, ks, vs = (t[off:off + n][None].contiguous() for t in (q, k, v))
        ref = aoh_prefill_chunked(qs, ks, vs, mask, n_sink, window, chunk) if chunk else \
            aoh_prefill(qs, ks, vs, mask, n_sink, window)
        torch.cuda.synchronize()
        assert np.array_equal(bits(out[off:off + n]), bits(ref[0])), f"sequence {i} (len {n}) differs"
        if i < 2:
            want = OA.prefill(f64(qs), f64(ks), f64(vs), mask, n_sink, window, chunk=chunk)
            assert_parity(out[off:off + n][None], want, dtype, f"varlen sequence {i}")
        off += n


def test_varlen_fills_the_caches_like_per_sequence_appends():
    lens = [300, 17, 1025, 0, 640]
    hq, hkv, d, mask, n_sink, window = 8, 2, 128, [0, 1], 8, 64
    bf = torch.bfloat16
    q, k, v, cu = _packed(lens, hq, hkv, d, bf, seed=5)
    B = len(lens)
    max_pages = (max(lens) + 15) // 16 + 1
    perm = synth.page_permutation(B * max_pages, 5, "vl-pages")
    bt = torch.from_numpy(perm.reshape(B, max_pages).astype(np.int32))

    def caches():
        f = PagedCache.allocate(B * max_pages, mask.count(0), d, bf, bt)
        r = RingCache.allocate(B, mask.count(1), n_sink, window, d, bf)
        for c in (f, r):
            c.k.fill_(float("nan"))
            c.v.fill_(float("nan"))
        return f, r

    f1, r1 = caches()
    f2, r2 = caches()
    out = aoh_prefill_varlen(q, k, v, cu, max(lens), mask, n_sink, window, kv_full=f1, kv_ring=r1)
    off = 0
    for b, n in enumerate(lens):
        if n:
            fb = f2.rows(b, b + 1)
            rb = RingCache(r2.k[b:b + 1], r2.v[b:b + 1], r2.capacity)
            ref = aoh_prefill_append(q[off:off + n][None].contiguous(), k[off:off + n][None].contiguous(),
                                     v[off:off + n][None].contiguous(), mask, n_sink, window, fb, rb)
            torch.cuda.synchronize()
            assert np.array_equal(bits(out[off:off + n]), bits(ref[0]))
        off += n
    torch.cuda.synchronize()
    for a_, b_ in ((f1.k, f2.k), (f1.v, f2.v), (r1.k, r2.k), (r1.v, r2.v)):
        assert np.array_equal(bits(a_), bits(b_))


def test_varlen_sweep_workload_packed():
    # the 16-sequence variable-length workload (U[4096, 65536] tokens, 32 q / 8 KV
    # heads, needles) at 50% streaming, window 4096: one packed call against the
    # per-sequence calls, every row bit-identical
    c = synth.CONFIGS["varlen_sweep"]
    lens = synth.lengths_uniform(c["n_seq"], c["len_lo"], c["len_hi"], c["seed"])
    n_str = synth.n_streaming_for(c["hkv"], 50)
    mask = synth.choose_streaming(c["hkv"], n_str, c["seed"], "streaming", 50, 4096).tolist()
    bf = torch.bfloat16
    parts = [synth.sweep_sequence(b, int(lens[b])) for b in range(len(lens))]
    q = torch.cat([torch.from_numpy(p["q"][0]).to(bf) for p in parts]).to(DEV)
    k = torch.cat([torch.from_numpy(p["k"][0]).to(bf) for p in parts]).to(DEV)
    v = torch.cat([torch.from_numpy(p["v"][0]).to(bf) for p in parts]).to(DEV)
    del parts
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device=DEV)
    out = aoh_prefill_varlen(q, k, v, cu, int(lens.max()), mask, c["n_sink"], 4096)
    torch.cuda.synchronize()
    off = 0
    for i, n in enumerate(lens):
        n = int(n)
        ref = aoh_prefill(q[off:off + n][None], k[off:off + n][None], v[off:off + n][None], mask, c["n_sink"], 4096)
        torch.cuda.synchronize()
        assert np.array_equal(bits(out[off:off + n]), bits(ref[0])), f"sequence {i}"
        off += n
    print(f"packed sweep: {len(lens)} sequences, {off} tokens, bit-identical to per-sequence prefill")
