"""Parity at full workload sizes, in the launch configuration bench.py times.

* Qwen2.5-7B-shaped prefill, 32768 tokens, 28 query / 4 KV heads, KV heads 1
  and 3 streaming (n_sink 64, window 1024): sampled query rows (every mask
  boundary plus seeded random rows) for all heads against the oracle.
* Llama-3-8B-shaped decode, batch 8 x 131072-token contexts on shuffled
  16-token pages, 4 streaming KV heads, 64 steps: the first and last steps
  against the oracle's logical-sequence decode, and the whole paged cache and
  ring bit for bit against the oracle's placement model.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from oracle import cache_model as CM
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode_step, aoh_decode_workspace_bytes,
                                  aoh_kv_append, aoh_prefill)
from tests.helpers import assert_parity, bits, f64

pytestmark = pytest.mark.gpu
DEV = "cuda"
BF = torch.bfloat16


def test_qwen_prefill_32k_sampled_rows():
    w = synth.qwen_prefill_inputs()
    q, k, v = (torch.from_numpy(w[n]).to(BF) for n in ("q", "k", "v"))
    del w
    mask, n_sink, window = [0, 1, 0, 1], 64, 1024
    T = q.shape[1]
    out = aoh_prefill(q.to(DEV), k.to(DEV), v.to(DEV), mask, n_sink, window)
    torch.cuda.synchronize()
    boundary = [0, 1, 63, 64, 65, 127, 128, 1023, 1024, 1087, 1088, 1089, 2047, 2048, T - 129, T - 128, T - 1]
    rows = np.unique(np.concatenate([boundary, np.random.default_rng(2).integers(0, T, 24)]))
    want = OA.prefill(f64(q), f64(k), f64(v), mask, n_sink, window, rows=rows)
    got = out[:, torch.from_numpy(rows).to(DEV)]
    mx, mean = assert_parity(got, want, BF, "qwen 32k prefill")
    print(f"qwen 32k prefill: {len(rows)} rows x 28 heads, max abs {mx:.3e}, mean abs {mean:.3e}")


def test_llama_decode_b8_128k():
    steps = 64
    w = synth.llama_decode_inputs(steps)
    mask, n_sink, window = w["mask"], w["n_sink"], w["window"]
    B, Hkv, L0, D = w["k_ctx"].shape
    Hq = w["q_steps"].shape[2]
    n_ret, n_str = mask.count(0), mask.count(1)
    k_ctx = torch.from_numpy(w["k_ctx"]).to(BF)   # [B, Hkv, L0, D]
    v_ctx = torch.from_numpy(w["v_ctx"]).to(BF)
    q_steps = torch.from_numpy(w["q_steps"]).to(BF)
    kv_steps = torch.from_numpy(w["kv_steps"]).to(BF)
    max_pages = w["max_pages"]
    bt = torch.from_numpy(w["pages"].copy())
    del w
    full = PagedCache.allocate(B * max_pages, n_ret, D, BF, bt)
    ring = RingCache.allocate(B, n_str, n_sink, window, D, BF)
    for c in (full, ring):
        c.k.fill_(float("nan"))
        c.v.fill_(float("nan"))
    kd, vd = k_ctx.to(DEV), v_ctx.to(DEV)
    aoh_kv_append(kd.permute(0, 2, 1, 3), vd.permute(0, 2, 1, 3), mask, torch.zeros(B, dtype=torch.int32, device=DEV),
                  full, ring, n_sink, window)
    del kd, vd
    ws = torch.empty(aoh_decode_workspace_bytes(B, Hq, D, max_pages, n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=DEV)
    outs = {}
    for s in range(steps):
        # one fused step (store the token at L0 + s, decode), as the benchmark runs it
        lens = torch.full((B,), L0 + s + 1, dtype=torch.int32, device=DEV)
        out = aoh_decode_step(q_steps[s].to(DEV), kv_steps[s, 0, :, 0].to(DEV), kv_steps[s, 1, :, 0].to(DEV), full,
                              ring, mask, lens, n_sink, window, workspace=ws)
        if s in (0, steps - 1):
            outs[s] = out.cpu()
    torch.cuda.synchronize()

    # logical sequences: context, then the appended step tokens
    k_seq = torch.cat([k_ctx.permute(0, 2, 1, 3), kv_steps[:, 0, :, 0].permute(1, 0, 2, 3)], 1).float().numpy()
    v_seq = torch.cat([v_ctx.permute(0, 2, 1, 3), kv_steps[:, 1, :, 0].permute(1, 0, 2, 3)], 1).float().numpy()
    for s, out in outs.items():
        want = OA.decode(f64(q_steps[s]), k_seq, v_seq, [L0 + s + 1] * B, mask, n_sink, window)
        mx, mean = assert_parity(out, want, BF, f"llama decode step {s}")
        print(f"llama decode step {s}: max abs {mx:.3e}, mean abs {mean:.3e}")

    # caches, bit for bit
    L = L0 + steps
    kb = torch.from_numpy(k_seq).to(BF).view(torch.int16).numpy()
    vb = torch.from_numpy(v_seq).to(BF).view(torch.int16).numpy()
    fk, fv, btn = bits(full.k), bits(full.v), full.block_table.cpu().numpy()
    rk, rv = bits(ring.k), bits(ring.v)
    ret, st = CM.split_heads(mask)
    for b in range(B):
        for r, g in enumerate(ret):
            K, V = CM.gather_paged(fk, fv, btn, b, r, L)
            assert np.array_equal(K, kb[b, :L, g]) and np.array_equal(V, vb[b, :L, g]), (b, g)
        for si, g in enumerate(st):
            pos, K, V = CM.gather_ring(rk, rv, b, si, L, n_sink, window)
            assert np.array_equal(K, kb[b, pos, g]) and np.array_equal(V, vb[b, pos, g]), (b, g)
