"""Parity of the two remaining workloads at their full sizes.

* 28-layer stack of the Qwen2.5-7B attention shape (28 query / 4 KV heads,
  d_head 128, bf16), batch 1, 262144-token prefill then 128 decode steps; per
  layer a seeded 2 of 4 KV heads stream (n_sink 64, window 2048).  Every layer
  runs through prefill, bulk append and the 128 steps; three layers are checked
  against the oracle (sampled prefill rows incl. every mask boundary, the first
  and last decode step).  Resident KV bytes are measured on the allocated caches
  and compared with the all-retrieval cache of the same stack.
* Variable-length sweep: 16 sequences of U[4096, 65536] tokens, 32 query / 8 KV
  heads, 8 planted needles per sequence, streaming fraction 25/50/75% x window
  512/4096 (n_sink 64): prefill per sequence (sampled rows of two sequences per
  setting, including needle positions) and 32 batched decode steps (first and
  last step, all sequences and heads) against the oracle.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import accounting as ACC
from oracle import attention as OA
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode, aoh_decode_step, aoh_decode_workspace_bytes,
                                  aoh_kv_append, aoh_prefill)
from tests.helpers import assert_parity, f64


def f32(t):
    """float32 numpy copy (exact for bf16 values); the oracle upcasts per slice."""
    return t.float().cpu().numpy()

pytestmark = pytest.mark.gpu
DEV = "cuda"
BF = torch.bfloat16


def _rows(T, n_sink, window, extra, seed):
    b = [0, 1, n_sink - 1, n_sink, n_sink + 1, window - 1, window, window + 1, n_sink + window - 1,
         n_sink + window, n_sink + window + 1, 255, 256, T - 257, T - 256, T - 1]
    r = np.random.default_rng(seed).integers(0, T, 12)
    return np.unique(np.clip(np.concatenate([b, r, extra]), 0, T - 1)).astype(np.int64)


def test_qwen_stack_28_layers_256k():
    c = synth.CONFIGS["qwen25_stack_256k"]
    L, T, Hq, Hkv, D = c["layers"], c["seq"], c["hq"], c["hkv"], c["d"]
    n_sink, window, steps = c["n_sink"], c["window"], c["decode_steps"]
    check = {0, 13, L - 1}
    max_pages = (T + steps + 15) // 16
    bt = torch.arange(max_pages, dtype=torch.int32)[None]
    zero = torch.zeros(1, dtype=torch.int32, device=DEV)
    layers, host = [], {}
    resident = 0
    for l in range(L):
        w = synth.stack_layer_inputs(l)
        mask = w["mask"]
        q, k, v = (torch.from_numpy(w[n]).to(BF) for n in ("q", "k", "v"))
        del w
        qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
        out = aoh_prefill(qd, kd, vd, mask, n_sink, window)
        full = PagedCache.allocate(max_pages, mask.count(0), D, BF, bt)
        ring = RingCache.allocate(1, mask.count(1), n_sink, window, D, BF)
        aoh_kv_append(kd, vd, mask, zero, full, ring, n_sink, window)
        resident += (full.k.numel() + full.v.numel() + ring.k.numel() + ring.v.numel()) * 2
        if l in check:
            rows = _rows(T, n_sink, window, [], l)
            got = out[:, torch.from_numpy(rows).to(DEV)].cpu()
            want = OA.prefill(f32(q), f32(k), f32(v), mask, n_sink, window, rows=rows)
            mx, mean = assert_parity(got, want, BF, f"stack layer {l} prefill")
            print(f"layer {l}: prefill {len(rows)} rows x {Hq} heads max abs {mx:.3e} mean {mean:.3e}")
            host[l] = (k[0].float().numpy(), v[0].float().numpy())
        del q, k, v, qd, kd, vd, out
        layers.append((mask, full, ring))
        print(f"layer {l}: prefill + append done (streaming KV heads {[g for g in range(Hkv) if mask[g]]})", flush=True)
    torch.cuda.synchronize()

    # 128 decode steps through every layer
    ws = torch.empty(aoh_decode_workspace_bytes(1, Hq, D, max_pages, n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=DEV)
    dec_in = {l: tuple(torch.from_numpy(x).to(BF) for x in synth.stack_decode_inputs(l, steps)) for l in range(L)}
    kept = {}
    for s in range(steps):
        lens = torch.full((1,), T + s, dtype=torch.int32, device=DEV)
        for l, (mask, full, ring) in enumerate(layers):
            qs, kvs = dec_in[l]
            # one fused step per layer (store the token at T + s, decode), as the benchmark runs it
            o = aoh_decode_step(qs[s].to(DEV), kvs[s, 0, :, 0].to(DEV), kvs[s, 1, :, 0].to(DEV), full, ring, mask,
                                lens + 1, n_sink, window, workspace=ws)
            if l in check and s in (0, steps - 1):
                kept[(l, s)] = o.cpu()
        if s % 32 == 0:
            print(f"decode step {s} done", flush=True)
    torch.cuda.synchronize()
    for (l, s), o in kept.items():
        mask = layers[l][0]
        qs, kvs = dec_in[l]
        k_seq = np.concatenate([host[l][0], kvs[:, 0, 0, 0].float().numpy()], 0)[None]
        v_seq = np.concatenate([host[l][1], kvs[:, 1, 0, 0].float().numpy()], 0)[None]
        want = OA.decode(f64(qs[s]), k_seq, v_seq, [T + s + 1], mask, n_sink, window)
        mx, mean = assert_parity(o, want, BF, f"stack layer {l} decode step {s}")
        print(f"layer {l} step {s}: decode max abs {mx:.3e} mean {mean:.3e}")

    # resident KV: measured allocation vs all-retrieval, and vs the formula
    all_ret = L * Hkv * T * D * 2 * 2
    pad_tokens = max_pages * 16
    g_str = synth.CONFIGS["qwen25_stack_256k"]["n_streaming"]
    ring_slots = (n_sink + window + 15) // 16 * 16
    want_bytes = L * D * 2 * 2 * ((Hkv - g_str) * pad_tokens + g_str * ring_slots)
    assert resident == want_bytes
    formula = ACC.kv_cache_bytes(L, D, 2, Hkv - g_str, g_str, T, n_sink, window)
    print(f"resident KV {resident / 1e9:.3f} GB (formula at T: {formula / 1e9:.3f} GB) vs all-retrieval "
          f"{all_ret / 1e9:.3f} GB: {all_ret / resident:.2f}x smaller")
    assert resident < 0.51 * all_ret
    assert abs(all_ret / 1e9 - 15.032) < 5e-4  # the paper's Qwen2.5-7B full-attention KV at 256K


@pytest.fixture(scope="module")
def sweep_seqs():
    c = synth.CONFIGS["varlen_sweep"]
    lens0 = synth.lengths_uniform(c["n_seq"], c["len_lo"], c["len_hi"], c["seed"])
    seqs = []
    for b in range(c["n_seq"]):
        w = synth.sweep_sequence(b, int(lens0[b]))
        seqs.append({k: (torch.from_numpy(x).to(BF) if k != "needles" else x) for k, x in w.items()})
        del w
    return lens0, seqs


@pytest.mark.parametrize("sparsity", [25, 50, 75])
def test_varlen_sweep(sparsity, sweep_seqs):
    c = synth.CONFIGS["varlen_sweep"]
    n, Hq, Hkv, D, n_sink, steps, seed = c["n_seq"], c["hq"], c["hkv"], c["d"], c["n_sink"], c["decode_steps"], c["seed"]
    lens0, seqs = sweep_seqs
    q_steps = torch.from_numpy(synth.gaussian((steps, n, Hq, D), seed, "qsteps")).to(BF)
    kv_steps = torch.from_numpy(synth.gaussian((steps, 2, n, 1, Hkv, D), seed, "kvsteps")).to(BF)
    n_str = synth.n_streaming_for(Hkv, sparsity)
    max_pages = (int(lens0.max()) + steps + 15) // 16
    for window in c["windows"]:
        mask = synth.choose_streaming(Hkv, n_str, seed, "streaming", sparsity, window).tolist()
        perm = synth.page_permutation(n * max_pages, seed, f"pages-{sparsity}-{window}")
        bt = torch.from_numpy(perm.reshape(n, max_pages).copy())
        full = PagedCache.allocate(n * max_pages, Hkv - n_str, D, BF, bt) if n_str < Hkv else None
        ring = RingCache.allocate(n, n_str, n_sink, window, D, BF) if n_str else None
        lens = torch.zeros(n, dtype=torch.int32, device=DEV)
        for b, sq in enumerate(seqs):
            T = sq["q"].shape[1]
            qd, kd, vd = sq["q"].to(DEV), sq["k"].to(DEV), sq["v"].to(DEV)
            out = aoh_prefill(qd, kd, vd, mask, n_sink, window)
            f = full.rows(b, b + 1) if full else None
            r = RingCache(ring.k[b:b + 1], ring.v[b:b + 1], ring.capacity) if ring else None
            aoh_kv_append(kd, vd, mask, lens[b:b + 1], f, r, n_sink, window)
            lens[b:b + 1] += T
            if b < 2:
                rows = _rows(T, n_sink, window, sq["needles"].reshape(-1), b)
                got = out[:, torch.from_numpy(rows).to(DEV)].cpu()
                want = OA.prefill(f32(sq["q"]), f32(sq["k"]), f32(sq["v"]), mask, n_sink, window, rows=rows)
                mx, mean = assert_parity(got, want, BF, f"sweep s{sparsity} w{window} seq {b} prefill")
                print(f"s{sparsity} w{window} seq {b} (T {T}): prefill max abs {mx:.3e} mean {mean:.3e}", flush=True)
            del qd, kd, vd, out
        print(f"s{sparsity} w{window}: 16 prefills appended", flush=True)
        ws = torch.empty(aoh_decode_workspace_bytes(n, Hq, D, max_pages, n_sink + window) // 4 + 4,
                         dtype=torch.float32, device=DEV)
        kept = {}
        for s in range(steps):
            aoh_kv_append(kv_steps[s, 0].to(DEV), kv_steps[s, 1].to(DEV), mask, lens, full, ring, n_sink, window)
            lens += 1
            o = aoh_decode(q_steps[s].to(DEV), full, ring, mask, lens, n_sink, window, workspace=ws)
            if s in (0, steps - 1):
                kept[s] = o.cpu()
        torch.cuda.synchronize()
        for s, o in kept.items():
            for b, sq in enumerate(seqs):
                T = sq["k"].shape[1]
                k_seq = torch.cat([sq["k"][0], kv_steps[:s + 1, 0, b, 0]], 0).float().numpy()[None]
                v_seq = torch.cat([sq["v"][0], kv_steps[:s + 1, 1, b, 0]], 0).float().numpy()[None]
                want = OA.decode(f64(q_steps[s, b:b + 1]), k_seq, v_seq, [T + s + 1], mask, n_sink, window)
                assert_parity(o[b:b + 1], want, BF, f"sweep s{sparsity} w{window} seq {b} step {s}")
            print(f"s{sparsity} w{window} step {s}: decode parity ok for {n} sequences")
        del full, ring
