"""Decode and cache parity on the GPU.

A run = a prompt appended in bulk per sequence, then single-token steps
(append, then decode).  The oracle keeps the logical sequence and never a
cache: its decode output is the prefill row of the last token.  Cache contents
are checked bit for bit against the oracle's placement model.  Caches start
filled with NaN so any read of a slot that was never written would show."""
import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from oracle import cache_model as CM
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode, aoh_decode_workspace_bytes,
                                  aoh_kv_append, aoh_prefill)
from tests.helpers import assert_parity, bits, f64, to_dtype

pytestmark = pytest.mark.gpu
DEV = "cuda"


class Run:
    def __init__(self, B, Hq, Hkv, D, mask, n_sink, window, prompt_lens, steps, dtype, seed,
                 spare_pages=3):
        self.B, self.Hq, self.Hkv, self.D = B, Hq, Hkv, D
        self.mask, self.n_sink, self.window, self.dtype = list(mask), n_sink, window, dtype
        self.prompt = np.asarray(prompt_lens, dtype=np.int64)
        self.steps = steps
        L = int(self.prompt.max()) + steps
        self.k_seq = to_dtype(synth.gaussian((B, L, Hkv, D), seed, "kseq"), dtype)
        self.v_seq = to_dtype(synth.gaussian((B, L, Hkv, D), seed, "vseq"), dtype)
        self.q_steps = to_dtype(synth.gaussian((steps, B, Hq, D), seed, "qstep"), dtype)
        n_ret = mask.count(0) if isinstance(mask, list) else int((np.asarray(mask) == 0).sum())
        n_str = Hkv - n_ret
        self.max_pages = (L + 15) // 16
        num_pages = B * self.max_pages + spare_pages
        perm = synth.page_permutation(num_pages, seed)[: B * self.max_pages]
        bt = torch.from_numpy(perm.reshape(B, self.max_pages).copy())
        self.full = PagedCache.allocate(num_pages, n_ret, D, dtype, bt) if n_ret else None
        self.ring = RingCache.allocate(B, n_str, n_sink, window, D, dtype) if n_str else None
        for c in (self.full, self.ring):
            if c is not None:
                c.k.fill_(float("nan"))
                c.v.fill_(float("nan"))
        self.lens = torch.zeros(B, dtype=torch.int32, device=DEV)
        ws = aoh_decode_workspace_bytes(B, Hq, D, self.max_pages, n_sink + window)
        self.ws = torch.empty(max(ws, 16) // 4 + 4, dtype=torch.float32, device=DEV)

    def _views(self, b):
        f = self.full.rows(b, b + 1) if self.full else None
        r = RingCache(self.ring.k[b:b + 1], self.ring.v[b:b + 1], self.ring.capacity) if self.ring else None
        return f, r

    def append_prompts(self):
        for b in range(self.B):
            n = int(self.prompt[b])
            f, r = self._views(b)
            kn = self.k_seq[b:b + 1, :n].to(DEV)
            vn = self.v_seq[b:b + 1, :n].to(DEV)
            aoh_kv_append(kn, vn, self.mask, self.lens[b:b + 1], f, r, self.n_sink, self.window)
            self.lens[b:b + 1] += n

    def step(self, s):
        pos = self.lens.cpu().numpy()
        kn = torch.stack([self.k_seq[b, int(pos[b])] for b in range(self.B)])[:, None].to(DEV)
        vn = torch.stack([self.v_seq[b, int(pos[b])] for b in range(self.B)])[:, None].to(DEV)
        aoh_kv_append(kn, vn, self.mask, self.lens, self.full, self.ring, self.n_sink, self.window)
        self.lens += 1
        q = self.q_steps[s].to(DEV)
        out = aoh_decode(q, self.full, self.ring, self.mask, self.lens, self.n_sink, self.window,
                         workspace=self.ws)
        torch.cuda.synchronize()
        return q, out

    def expected(self, q):
        lens = self.lens.cpu().numpy()
        return OA.decode(f64(q), f64(self.k_seq), f64(self.v_seq), lens, self.mask, self.n_sink, self.window)

    def check_caches(self):
        lens = self.lens.cpu().numpy()
        kb, vb = bits(self.k_seq), bits(self.v_seq)
        if self.full is not None:
            assert CM.check_paged(bits(self.full.k), bits(self.full.v), self.full.block_table.cpu().numpy(),
                                  kb, vb, lens, self.mask) == 0
        if self.ring is not None:
            assert CM.check_ring(bits(self.ring.k), bits(self.ring.v), kb, vb, lens, self.mask,
                                 self.n_sink, self.window) == 0


def test_tiny_fp32_prefill_then_decode():
    # 256-token prompt, then 16 decode steps appending seeded K/V
    cfg = synth.CONFIGS["tiny"]
    run = Run(1, 4, 2, 64, cfg["streaming"], cfg["n_sink"], cfg["window"], [256], 16, torch.float32,
              cfg["seed"])
    run.append_prompts()
    run.check_caches()
    for s in range(16):
        q, out = run.step(s)
        assert_parity(out, run.expected(q), torch.float32, f"tiny decode step {s}")
    run.check_caches()


DECODE_CASES = [
    # B, Hq, Hkv, D, mask, n_sink, window, prompt lens, steps
    (3, 8, 4, 128, [0, 1, 1, 0], 4, 40, [1, 17, 1000], 5),
    (2, 14, 2, 128, [1, 0], 64, 128, [300, 2049], 3),   # GQA 7
    (2, 8, 2, 64, [0, 1], 0, 1, [33, 64], 4),           # window 1, no sink
    (1, 32, 8, 128, [0, 1, 0, 1, 1, 0, 1, 0], 64, 1024, [5000], 3),
    (2, 4, 1, 128, [0], 4, 32, [31, 32], 34),           # all retrieval, page crossings
    (2, 4, 1, 128, [1], 4, 32, [31, 100], 40),          # all streaming, ring wrap
    # mixed lengths: the step's work space is split by its total length, so
    # the sequences take different numbers of split workgroups
    (16, 8, 2, 128, [0, 1], 16, 256,
     [1, 5000, 37, 900, 16, 17, 3000, 2, 64, 65, 1200, 4096, 8, 333, 2047, 60], 3),
    (64, 4, 1, 64, [0], 4, 32, [(37 * i) % 500 + 1 for i in range(64)], 2),       # largest work-space batch
    (24, 8, 4, 128, [1, 1, 1, 1], 8, 100, [(71 * i) % 400 + 1 for i in range(24)], 2),  # rings only
    (9, 16, 2, 64, [0, 0], 4, 32, [1, 2, 3, 17, 250, 900, 1, 4000, 33], 2),         # paged only, 1-token prompts
    (70, 4, 2, 64, [0, 1], 4, 32, [(53 * i) % 300 + 1 for i in range(70)], 2),   # beyond it: capacity plan
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("B,Hq,Hkv,D,mask,n_sink,window,prompt,steps", DECODE_CASES)
def test_decode_matches_oracle(B, Hq, Hkv, D, mask, n_sink, window, prompt, steps, dtype):
    run = Run(B, Hq, Hkv, D, mask, n_sink, window, prompt, steps, dtype, seed=B * 100 + Hq + steps)
    run.append_prompts()
    run.check_caches()
    for s in range(steps):
        q, out = run.step(s)
        assert_parity(out, run.expected(q), dtype, f"decode step {s}")
    run.check_caches()


def test_decode_equals_prefill_last_row():
    # decode at position p equals row p of prefill over the same tokens
    B, Hq, Hkv, D, T = 1, 8, 2, 128, 700
    mask, n_sink, window = [0, 1], 8, 64
    run = Run(B, Hq, Hkv, D, mask, n_sink, window, [T - 1], 1, torch.bfloat16, seed=21)
    run.append_prompts()
    q, out = run.step(0)
    qfull = torch.cat([to_dtype(synth.gaussian((B, T - 1, Hq, D), 1, "qpre"), torch.bfloat16), q.cpu()[:, None]], 1)
    pre = aoh_prefill(qfull.to(DEV), run.k_seq[:, :T].to(DEV), run.v_seq[:, :T].to(DEV), mask, n_sink, window,
                      out=torch.empty((B, T, Hq, D), dtype=torch.float32, device=DEV))
    dec = torch.empty((B, Hq, D), dtype=torch.float32, device=DEV)
    aoh_decode(q, run.full, run.ring, mask, run.lens, n_sink, window, out=dec, workspace=run.ws)
    torch.cuda.synchronize()
    assert np.abs(f64(dec) - f64(pre[:, -1])).max() < 1e-2


def test_zero_keys_decode_averages_positions():
    # K = 0 and V[p] = p mod 64: the decode output is the mean of the visible
    # values, which pins the page gather and the ring contents
    B, Hq, Hkv, D = 2, 4, 2, 128
    mask, n_sink, window = [0, 1], 5, 37
    run = Run(B, Hq, Hkv, D, mask, n_sink, window, [900, 77], 2, torch.bfloat16, seed=4)
    L = run.k_seq.shape[1]
    run.k_seq.zero_()
    run.v_seq.copy_(torch.from_numpy(np.broadcast_to((np.arange(L) % 64).astype(np.float32)[None, :, None, None],
                                                     run.v_seq.shape).copy()).to(torch.bfloat16))
    run.append_prompts()
    for s in range(2):
        q, _ = run.step(s)
        out = torch.empty((B, Hq, D), dtype=torch.float32, device=DEV)
        aoh_decode(q, run.full, run.ring, mask, run.lens, n_sink, window, out=out, workspace=run.ws)
        torch.cuda.synchronize()
        assert np.abs(f64(out) - run.expected(q)).max() < 1e-4
