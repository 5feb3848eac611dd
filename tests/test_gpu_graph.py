"""Whole-step HIP-graph capture of a multi-layer decode step (the paper
captures its Qwen2.5-7B decode step in a CUDA graph, appendix efficiency
tables).  Every library call is capturable: grids depend on capacities only,
lengths are read on the device, nothing is allocated or cleared with memset.

The captured step (per layer: append one token, decode) is replayed several
times with eager work and synchronisations between replays; every replay must
match the same step run eagerly, bit for bit, and the caches must match."""
import numpy as np
import pytest
import torch

import synth
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode, aoh_decode_step, aoh_decode_workspace_bytes,
                                  aoh_kv_append)
from tests.helpers import bits

pytestmark = pytest.mark.gpu
DEV = "cuda"
BF = torch.bfloat16


def _stack(n_layers, B, Hq, Hkv, D, L0, n_sink, window, seed):
    layers = []
    max_pages = (L0 + 8 + 15) // 16
    for l in range(n_layers):
        mask = synth.choose_streaming(Hkv, Hkv // 2, seed, "graph-streaming", l).tolist()
        bt = torch.from_numpy(synth.page_permutation(B * max_pages, seed, f"graph-pages-{l}").reshape(B, max_pages).copy())
        full = PagedCache.allocate(B * max_pages, mask.count(0), D, BF, bt)
        ring = RingCache.allocate(B, mask.count(1), n_sink, window, D, BF)
        k = torch.from_numpy(synth.gaussian((B, L0, Hkv, D), seed, "graph-k", l)).to(BF).to(DEV)
        v = torch.from_numpy(synth.gaussian((B, L0, Hkv, D), seed, "graph-v", l)).to(BF).to(DEV)
        aoh_kv_append(k, v, mask, torch.zeros(B, dtype=torch.int32, device=DEV), full, ring, n_sink, window)
        layers.append((mask, full, ring))
    return layers, max_pages


@pytest.mark.parametrize("fused", [False, True])
def test_graph_replay_matches_eager(fused):
    n_layers, B, Hq, Hkv, D, L0, n_sink, window, seed = 4, 2, 8, 4, 128, 3000, 16, 256, 11
    layers, max_pages = _stack(n_layers, B, Hq, Hkv, D, L0, n_sink, window, seed)
    ws = torch.empty(aoh_decode_workspace_bytes(B, Hq, D, max_pages, n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=DEV)
    q = torch.from_numpy(synth.gaussian((n_layers, B, Hq, D), seed, "graph-q")).to(BF).to(DEV)
    kn = torch.from_numpy(synth.gaussian((n_layers, 2, B, 1, Hkv, D), seed, "graph-kn")).to(BF).to(DEV)
    lens_before = torch.full((B,), L0, dtype=torch.int32, device=DEV)
    lens_after = lens_before + 1
    outs = torch.empty((n_layers, B, Hq, D), dtype=BF, device=DEV)

    def step(fused=False):
        for l, (mask, full, ring) in enumerate(layers):
            if fused:
                aoh_decode_step(q[l], kn[l, 0, :, 0], kn[l, 1, :, 0], full, ring, mask, lens_after, n_sink, window,
                                out=outs[l], workspace=ws)
            else:
                aoh_kv_append(kn[l, 0], kn[l, 1], mask, lens_before, full, ring, n_sink, window)
                aoh_decode(q[l], full, ring, mask, lens_after, n_sink, window, out=outs[l], workspace=ws)

    # eager reference: the two-call step (appending the same token again is
    # idempotent); the captured step is the two-call or the fused one
    step()
    torch.cuda.synchronize()
    want = bits(outs)
    caches = [(bits(f.k), bits(f.v), bits(r.k), bits(r.v)) for _, f, r in layers]

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(fused)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(fused)
    for rep in range(4):
        outs.fill_(float("nan"))            # eager work between replays
        junk = torch.randn(1 << 20, device=DEV).sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(outs), want), f"replay {rep}"
        del junk
    for (mask, f, r), c in zip(layers, caches):
        assert np.array_equal(bits(f.k), c[0]) and np.array_equal(bits(f.v), c[1])
        assert np.array_equal(bits(r.k), c[2]) and np.array_equal(bits(r.v), c[3])
