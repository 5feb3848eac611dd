#!/usr/bin/env python3
"""Benchmark of AoH head-mixed attention on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Step = one pass of the whole hot path over the Qwen2.5-7B-shaped layer
(28 query heads, 4 KV heads of which 1 and 3 are streaming, d_head 128, bf16,
one 32768-token sequence, n_sink 64, window 1024):
  head scheduling -> one prefill launch holding the retrieval and the
  streaming work items, which also writes the prompt's K/V into the paged
  cache and the ring -> one decode step (store the next token, split-K
  decode, merge).
`value` is the useful prefill FLOPs of a step (4 D per visible query-key pair)
divided by the step time.  `roofline` is the step's prefill launch, timed by
HIP events around that launch on its stream, against the bf16 MFMA peak, with
the useful and the computed-tile FLOP counts.

A decode leg runs the Llama-3-8B-shaped batch (32 query heads, 8 KV heads of
which 4 streaming, batch 8, 131072-token contexts on a paged cache of shuffled
16-token pages, ring n_sink 64 + window 1024) for 64 single-token steps and
reports KV GB/s and tokens/s.  Both legs are also run all-retrieval with the
same kernels for the speedup.  A stack leg runs decode steps through the 28
layers of a 262144-token Qwen2.5-7B-shaped stack (eager and as one HIP graph)
and one layer's prefill, with the resident KV of the 28 layers; a sweep leg
runs the 16-sequence variable-length workload (packed prefill and 32 batched
decode steps per setting); a classifier leg times the offline head
classification of a 28-layer model.  Inputs are seeded synthetic data (synth)
and resident in HBM before timing.  The timed prefill steps follow at least W
untimed ones and at least 0.5 s of them: the GPU clock ramps up over the first
tens of milliseconds of sustained work, and the figure is the steady state.
One JSON line goes to stdout; progress goes to stderr.
"""
import argparse
import json
import os
import sys
import time

import numpy as np


def log(*a):
    print(*a, file=sys.stderr, flush=True)


PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
SETTLE_S = 0.5              # minimum untimed warm-up of the prefill step (clock ramp)
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E


def visible_pairs(t, streaming, n_sink, window):
    """Visible (query, key) pairs of a t-token causal prefill for one head."""
    if not streaming:
        return t * (t + 1) // 2
    w = min(window, t)
    recent = w * (w + 1) // 2 + (t - w) * window
    m = max(0, t - window)
    sink = m * (m + 1) // 2 if m <= n_sink else n_sink * (n_sink + 1) // 2 + (m - n_sink) * n_sink
    return recent + sink


def useful_prefill_flops(t, d, hq_ret, hq_str, n_sink, window):
    """4 D FLOPs (Q K^T and P V) per visible pair; masked work is not counted."""
    return 4 * d * (hq_ret * visible_pairs(t, False, n_sink, window) + hq_str * visible_pairs(t, True, n_sink, window))


def computed_tile_flops(t, d, hq_ret, hq_str, n_sink, window, rows=256, bn=64, chunk=0):
    """MFMA FLOPs the prefill kernel issues: 4 D per (row, key) pair of every
    rows x bn tile a workgroup of `rows` query rows visits (the causal
    diagonal and band-edge tiles count whole).  Retrieval blocks visit tiles
    0 .. last; streaming blocks the sink tiles plus the band from the first
    row's lowest visible key."""
    per_tile = 4 * d * rows * bn
    ret = st = 0
    for i0 in range(0, t, rows):
        last_tile = (min(i0 + rows, t) - 1) // bn
        ret += last_tile + 1
        lo = (i0 // chunk) * chunk - window if chunk else i0 - window + 1
        band_first = max(0, lo) // bn
        sink_tiles = min((n_sink + bn - 1) // bn, band_first)
        st += sink_tiles + (last_tile - band_first + 1)
    return per_tile * (hq_ret * ret + hq_str * st)


def decode_bytes(lens, g_ret, g_str, d, elt, n_sink, window):
    """KV bytes a decode step must read: all retrieval tokens, live ring slots."""
    return sum((g_ret * n + g_str * min(n, n_sink + window)) * d * 2 * elt for n in lens)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--decode-steps", type=int, default=64)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-all-retrieval", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-stack-decode", action="store_true")
    ap.add_argument("--no-classify", action="store_true")
    ap.add_argument("--no-varlen", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (for scaling HBM counters)")
    return ap.parse_args()


def copy_calibration():
    """A plain copy of known size: 1 GiB read + 1 GiB written per dispatch."""
    import torch
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("copy calibration: 5 x 1 GiB device-to-device copies done")


# HBM traffic per launch measured with rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE
# (KiB per dispatch), divided by the ratio those counters read for a plain
# 1 GiB copy (bench.py --copy-calibration).  Each figure carries the hash of
# the sources its kernel is built from: a change to them makes the figure
# stale and it is dropped.
PREFILL_SOURCES = ("prefill.hip", "aoh_device.h", "aoh_internal.h")
DECODE_SOURCES = ("decode.hip", "aoh_device.h", "aoh_internal.h")
TRAFFIC = {
    "fetch_factor": 524301.2 / 1048576.0,   # FETCH_SIZE of a 1 GiB copy / 1 GiB
    "write_factor": 1048576.0 / 1048576.0,  # WRITE_SIZE of a 1 GiB copy / 1 GiB
    "prefill_mixed": {"fetch_kib": 461597.2, "write_kib": 263393.8,
                      "sources": PREFILL_SOURCES, "source_hash": "154d329fa4c197b3"},
    "decode_ws": {"fetch_kib": 1081565.0, "write_kib": 1169.9,
                  "sources": DECODE_SOURCES, "source_hash": "21a01592fbd3549f"},
}


def kernel_source_hash(names, read=None):
    """Hash of the kernel sources a traffic figure was measured on: their code
    lines, with // comments and blank lines dropped (comments do not change
    the kernels)."""
    import hashlib
    import re
    root = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2608_06849_amd", "csrc")
    h = hashlib.sha256()
    for name in names:
        if read is None:
            with open(os.path.join(root, name), "rb") as f:
                text = f.read().decode()
        else:
            text = read(name)
        for line in text.splitlines():
            code = re.sub(r"//.*$", "", line).rstrip()
            if code.strip():
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def traffic_for(kernel):
    t = TRAFFIC.get(kernel) if TRAFFIC else None
    if t is None or t["source_hash"] != kernel_source_hash(t["sources"]):
        return None
    return round((t["fetch_kib"] / TRAFFIC["fetch_factor"] + t["write_kib"] / TRAFFIC["write_factor"]) * 1024)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the hot path is not sharded across GPUs", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return

    import torch

    import synth
    from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode, aoh_decode_step, aoh_decode_workspace_bytes,
                                      aoh_kv_append, aoh_prefill, aoh_prefill_append)
    from paper_2608_06849_amd import aoh as A

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    A.lib()  # fail loudly if the HIP library is not built
    dev = "cuda"
    bf = torch.bfloat16

    # ------------------------------------------------------------------ prefill step workload
    cfg = synth.CONFIGS["qwen25_prefill_32k"]
    T, Hq, Hkv, D, seed = cfg["seq"], cfg["hq"], cfg["hkv"], cfg["d"], cfg["seed"]
    mask, n_sink, window = cfg["streaming"], cfg["n_sink"], cfg["window"]
    gs = Hq // Hkv
    t0 = time.time()
    w = synth.qwen_prefill_inputs()
    q, k, v = (torch.from_numpy(w[n]).to(bf).to(dev) for n in ("q", "k", "v"))
    del w
    q_dec = torch.from_numpy(synth.gaussian((1, Hq, D), seed, "qdec")).to(bf).to(dev)
    kv_next = torch.from_numpy(synth.gaussian((2, 1, 1, Hkv, D), seed, "kvnext")).to(bf).to(dev)
    out = torch.empty_like(q)
    n_ret, n_str = mask.count(0), mask.count(1)
    max_pages = (T + 1 + 15) // 16
    bt = torch.arange(max_pages, dtype=torch.int32)[None]
    full = PagedCache.allocate(max_pages, n_ret, D, bf, bt)
    ring = RingCache.allocate(1, n_str, n_sink, window, D, bf)
    startT = torch.full((1,), T, dtype=torch.int32, device=dev)
    lensT1 = torch.full((1,), T + 1, dtype=torch.int32, device=dev)
    ws = torch.empty(aoh_decode_workspace_bytes(1, Hq, D, max_pages, n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=dev)
    dec_out = torch.empty_like(q_dec)
    torch.cuda.synchronize()
    log(f"prefill workload ready in {time.time() - t0:.1f}s")

    flops_step = useful_prefill_flops(T, D, gs * n_ret, gs * n_str, n_sink, window)
    flops_ret = useful_prefill_flops(T, D, gs * n_ret, 0, n_sink, window)
    flops_tiles = computed_tile_flops(T, D, gs * n_ret, gs * n_str, n_sink, window)

    def step(m=mask, f=full, r=ring, ev=None):
        if ev is not None:
            ev[0].record()
        aoh_prefill_append(q, k, v, m, n_sink, window, f, r, out=out)
        if ev is not None:
            ev[1].record()
        aoh_decode_step(q_dec, kv_next[0][:, 0], kv_next[1][:, 0], f, r, m, lensT1, n_sink, window, out=dec_out,
                        workspace=ws)
        if ev is not None:
            ev[2].record()

    # The GPU raises its clock over the first tens of milliseconds of sustained
    # work (~1.6 -> ~1.9-2.1 GHz under this load); untimed steps run until
    # at least SETTLE_S seconds have passed, and at least W of them.
    settle = 0
    t_settle = time.perf_counter()
    while settle < args.warmup or time.perf_counter() - t_settle < SETTLE_S:
        step()
        torch.cuda.synchronize()
        settle += 1
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t_start = time.perf_counter()
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(ev=evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    prefill_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    step_ms = float(np.mean([e[0].elapsed_time(e[2]) for e in evs]))
    log(f"step {step_ms:.3f} ms (prefill {prefill_ms:.3f} ms), wall {wall * 1e3 / args.steps:.3f} ms/step")

    # The retrieval items alone, as their own launch with the same grid (the
    # retrieval query heads and KV heads as their own tensors): context for
    # the one-launch figure.
    ret_q = torch.tensor([h for h in range(Hq) if mask[h // gs] == 0], device=dev)
    ret_kv = torch.tensor([g for g in range(Hkv) if mask[g] == 0], device=dev)
    q_r = q.index_select(2, ret_q).contiguous()
    k_r = k.index_select(2, ret_kv).contiguous()
    v_r = v.index_select(2, ret_kv).contiguous()
    o_r = torch.empty_like(q_r)
    mask_r = [0] * n_ret
    for _ in range(2):
        aoh_prefill(q_r, k_r, v_r, mask_r, n_sink, window, out=o_r)
    n_rep = max(3, args.steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(n_rep):
        aoh_prefill(q_r, k_r, v_r, mask_r, n_sink, window, out=o_r)
    e1.record()
    torch.cuda.synchronize()
    ret_ms = e0.elapsed_time(e1) / n_rep
    ret_tflops = flops_ret / (ret_ms * 1e-3) / 1e12
    log(f"retrieval prefill kernel {ret_ms:.3f} ms = {ret_tflops:.1f} TFLOP/s")
    del q_r, k_r, v_r, o_r

    # Same kernels, all heads retrieval.
    all_ret = None
    if not args.no_all_retrieval:
        mask_all = [0] * Hkv
        full_all = PagedCache.allocate(max_pages, Hkv, D, bf, bt)
        for _ in range(2):
            step(mask_all, full_all, None)
        evs_a = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(max(3, args.steps // 2))]
        torch.cuda.synchronize()
        for e in evs_a:
            step(mask_all, full_all, None, ev=e)
        torch.cuda.synchronize()
        all_ret = dict(step_ms=float(np.mean([e[0].elapsed_time(e[2]) for e in evs_a])),
                       prefill_ms=float(np.mean([e[0].elapsed_time(e[1]) for e in evs_a])))
        log(f"all-retrieval step {all_ret['step_ms']:.3f} ms (prefill {all_ret['prefill_ms']:.3f})")
        del full_all

    # ------------------------------------------------------------------ decode leg
    dec = None
    if not args.no_decode:
        dec = decode_leg(args, torch, synth, PagedCache, RingCache, aoh_decode, aoh_decode_workspace_bytes,
                         aoh_kv_append, decode_bytes)

    stack = None
    if not args.no_stack_decode:
        stack = stack_decode_leg(args, torch, synth, PagedCache, RingCache, aoh_decode, aoh_decode_workspace_bytes,
                                 aoh_kv_append, decode_bytes)
        stack["prefill"] = stack_prefill_leg(torch, synth, PagedCache, RingCache)

    cls = None
    if not args.no_classify:
        cls = classify_leg(args, torch, synth)
    vlen = None
    if not args.no_varlen:
        vlen = varlen_leg(args, torch, synth)

    # ------------------------------------------------------------------ CPU baseline (oracle)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(q, k, v, mask, n_sink, window, T, D, gs)

    value = flops_step / (step_ms * 1e-3) / 1e12
    result = {
        "metric": "prefill TFLOP/s + decode KV GB/s (frac of roofline), 50% streaming heads",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": settle,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1), K scaled by 0.5)",
        "config": {
            "workload": "Qwen2.5-7B-shaped attention layer: prefill 32768 tokens, 28 q heads / 4 KV heads "
                        "(KV heads 1,3 streaming), d_head 128, n_sink 64, window 1024; step = schedule + "
                        "prefill writing the caches (one launch for both head types) + 1 decode step",
            "global_batch": 1, "seq_len": T, "parallelism": "none (1 GPU)",
        },
        "prefill": {
            "ms": round(prefill_ms, 4),
            "useful_tflop": round(flops_step / 1e12, 4),
            "tflops": round(flops_step / (prefill_ms * 1e-3) / 1e12, 2),
            "frac_of_bf16_peak": round(flops_step / (prefill_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        },
        # The step's dominant kernel: its prefill launch (both head types in
        # one launch that also fills the caches), timed by the events around
        # that one launch on the stream it runs on, averaged over the timed steps.
        "roofline": {
            "kernel": f"prefill_pp_mixed_kernel<bf16 out, append> ({gs * n_ret} retrieval + {gs * n_str} streaming "
                      f"q heads x {T} rows, d_head 128)",
            "bound": "mfma", "achieved": round(flops_step / (prefill_ms * 1e-3) / 1e12, 2), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(flops_step / (prefill_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic_for("prefill_mixed"),
            "algorithmic_per_launch": f"{flops_step:.4e} FLOP (4 D per visible pair)",
            "avg_launch_ms": round(prefill_ms, 4),
            "computed_tile_per_launch": f"{flops_tiles:.4e} FLOP (4 D x 256 rows x 64 keys per visited tile)",
            "computed_tile_tflops": round(flops_tiles / (prefill_ms * 1e-3) / 1e12, 2),
            "computed_tile_frac": round(flops_tiles / (prefill_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "retrieval_launch_alone": {"ms": round(ret_ms, 4), "tflops": round(ret_tflops, 2),
                                       "frac": round(ret_tflops / PEAK_BF16_TFLOPS, 4)},
        },
        "all_retrieval": None if all_ret is None else {
            "step_ms": round(all_ret["step_ms"], 4), "prefill_ms": round(all_ret["prefill_ms"], 4),
            "speedup_step": round(all_ret["step_ms"] / step_ms, 3),
            "speedup_prefill": round(all_ret["prefill_ms"] / prefill_ms, 3),
        },
        "decode": dec,
        "stack_decode": stack,
        "classify": cls,
        "varlen_prefill": vlen,
        "cpu_baseline": cpu,
        "paper_context": "paper (hardware unstated, end-to-end model latency, bf16, batch 1): prefill/decode "
                         "latency reduction up to 41.4%/66.0% and 50.0% KV saving at 256K, 50% sparsity",
    }
    print(json.dumps(result), flush=True)


def decode_leg(args, torch, synth, PagedCache, RingCache, aoh_decode, aoh_decode_workspace_bytes, aoh_kv_append,
               decode_bytes):
    cfg = synth.CONFIGS["llama_decode_b8_128k"]
    B, Hq, Hkv, D, L0 = cfg["batch"], cfg["hq"], cfg["hkv"], cfg["d"], cfg["context"]
    n_sink, window, seed, steps = cfg["n_sink"], cfg["window"], cfg["seed"], args.decode_steps
    dev, bf = "cuda", torch.bfloat16
    t0 = time.time()
    w = synth.llama_decode_inputs(steps)
    mask = w["mask"]
    n_ret, n_str = mask.count(0), mask.count(1)
    max_pages = w["max_pages"]
    num_pages = B * max_pages
    bt = torch.from_numpy(w["pages"].copy())
    full = PagedCache.allocate(num_pages, n_ret, D, bf, bt)
    ring = RingCache.allocate(B, n_str, n_sink, window, D, bf)
    full_all = None if args.no_all_retrieval else PagedCache.allocate(num_pages, Hkv, D, bf, bt)
    zero = torch.zeros(B, dtype=torch.int32, device=dev)
    # context K/V, one (sequence, KV head) block at a time on the host -> [B, L0, Hkv, D] views
    kc = torch.from_numpy(w["k_ctx"]).to(bf).to(dev)
    vc = torch.from_numpy(w["v_ctx"]).to(bf).to(dev)
    k_ctx, v_ctx = kc.permute(0, 2, 1, 3), vc.permute(0, 2, 1, 3)
    aoh_kv_append(k_ctx, v_ctx, mask, zero, full, ring, n_sink, window)
    if full_all is not None:
        aoh_kv_append(k_ctx, v_ctx, [0] * Hkv, zero, full_all, None, n_sink, window)
    torch.cuda.synchronize()
    del kc, vc, k_ctx, v_ctx
    q_steps = torch.from_numpy(w["q_steps"]).to(bf).to(dev)
    kv_steps = torch.from_numpy(w["kv_steps"]).to(bf).to(dev)
    del w
    ws = torch.empty(aoh_decode_workspace_bytes(B, Hq, D, max_pages, n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=dev)
    out = torch.empty((B, Hq, D), dtype=bf, device=dev)
    lens_tab = [torch.full((B,), L0 + s, dtype=torch.int32, device=dev) for s in range(steps + 1)]
    log(f"decode workload ready in {time.time() - t0:.1f}s")

    from paper_2608_06849_amd import aoh_decode_step

    def run(m, f, r, fused=True):
        # warm up on the initial state (decode only, no append), then time all
        # steps: one fused call per step, or an append call then a decode call
        for _ in range(2):
            aoh_decode(q_steps[0], f, r, m, lens_tab[0], n_sink, window, out=out, workspace=ws)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for s in range(steps):
            if fused:
                aoh_decode_step(q_steps[s], kv_steps[s, 0, :, 0], kv_steps[s, 1, :, 0], f, r, m, lens_tab[s + 1],
                                n_sink, window, out=out, workspace=ws)
            else:
                aoh_kv_append(kv_steps[s, 0], kv_steps[s, 1], m, lens_tab[s], f, r, n_sink, window)
                aoh_decode(q_steps[s], f, r, m, lens_tab[s + 1], n_sink, window, out=out, workspace=ws)
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    ms_two = run(mask, full, ring, fused=False)
    ms = run(mask, full, ring)
    lens = [L0 + s + 1 for s in range(steps)]
    kv_bytes = np.mean([decode_bytes([n] * B, n_ret, n_str, D, 2, n_sink, window) for n in lens])
    gbps = kv_bytes / (ms * 1e-3) / 1e9
    # decode kernels alone (no append) for the roofline of the split pass + merge
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(20):
        aoh_decode(q_steps[-1], full, ring, mask, lens_tab[steps], n_sink, window, out=out, workspace=ws)
    ev[1].record()
    torch.cuda.synchronize()
    dec_ms = ev[0].elapsed_time(ev[1]) / 20
    b_last = decode_bytes([L0 + steps] * B, n_ret, n_str, D, 2, n_sink, window)
    res = {
        "workload": "Llama-3-8B-shaped decode: batch 8 x 131072-token contexts, 32 q heads / 8 KV heads "
                    f"(streaming KV heads {[g for g in range(Hkv) if mask[g]]}), d_head 128, bf16, paged 16-token "
                    "pages (shuffled), ring n_sink 64 + window 1024; step = append 1 token/seq + decode "
                    "(one aoh_decode_step call)",
        "steps": steps,
        "ms_per_step": round(ms, 4),
        "two_call_ms_per_step": round(ms_two, 4),
        "tokens_per_s": round(B / (ms * 1e-3), 1),
        "kv_gb_per_step": round(kv_bytes / 1e9, 4),
        "kv_gbps": round(gbps, 1),
        "frac_of_hbm_peak": round(gbps / PEAK_HBM_GBPS, 4),
        "resident_kv_gb": round((full.k.numel() + full.v.numel() + ring.k.numel() + ring.v.numel()) * 2 / 1e9, 4),
        "roofline": {
            "kernel": "decode_ws_kernel<128> (paged and ring items in one work-space split) + merge (one aoh_decode call)",
            "bound": "hbm", "achieved": round(b_last / (dec_ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(b_last / (dec_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "traffic": traffic_for("decode_ws"),
            "algorithmic_per_launch": f"{b_last:.4e} B", "avg_launch_ms": round(dec_ms, 4),
        },
    }
    log(f"decode {ms:.4f} ms/step ({ms_two:.4f} as two calls), {gbps:.0f} GB/s ({res['frac_of_hbm_peak']:.3f} of peak); "
        f"decode call alone {dec_ms:.4f} ms")
    res["h2share"] = h2share_decode(torch, q_steps[-1], full, ring, mask, lens_tab[steps], n_sink, window, B, Hq, D,
                                    max_pages, L0 + steps, dec_ms)
    if full_all is not None:
        ms_all = run([0] * Hkv, full_all, None)
        res["all_retrieval_ms_per_step"] = round(ms_all, 4)
        res["speedup_vs_all_retrieval"] = round(ms_all / ms, 3)
        res["resident_kv_gb_all_retrieval"] = round((full_all.k.numel() + full_all.v.numel()) * 2 / 1e9, 4)
        log(f"decode all-retrieval {ms_all:.4f} ms/step")
    return res


def h2share_decode(torch, q, full, ring, mask, lens, n_sink, window, B, Hq, D, max_pages, length, plain_ms,
                   top_k=2048, block=4):
    """H2Share decode on the same caches: an anchor step (decode + top-k
    selection) and a reuse step (retrieval groups attend to the anchor's
    top_k positions in their own cache; identity group mapping), each timed
    alone; a block of `block` layers costs one anchor and block-1 reuse steps.
    The reuse step is timed on token-major V pages (the layout of a reuse
    layer's cache; the same tokens, V transposed) and, for comparison, on the
    dimension-major pages the anchor reads."""
    from paper_2608_06849_amd import (aoh_decode_anchor, aoh_decode_anchor_workspace_bytes, aoh_decode_reuse,
                                      aoh_decode_reuse_workspace_bytes)
    n_ret, n_str = mask.count(0), mask.count(1)
    out = torch.empty_like(q)
    idx = torch.empty((B, n_ret, top_k), dtype=torch.int32, device="cuda")
    ws_a = torch.empty(aoh_decode_anchor_workspace_bytes(B, Hq, D, max_pages, n_sink + window), dtype=torch.uint8,
                       device="cuda")
    ws_r = torch.empty(aoh_decode_reuse_workspace_bytes(B, Hq, D, top_k, n_sink + window), dtype=torch.uint8,
                       device="cuda")
    mapping = [0] * len(mask)
    r = 0
    for g in range(len(mask)):
        if not mask[g]:
            mapping[g] = r
            r += 1

    def timed(fn, n=20):
        for _ in range(3):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(n):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    def graph_timed(fn, n=20, reps=5):
        """Per-call time of fn from one HIP graph of n calls replayed reps
        times (GPU time, without a host dispatch per call, which a ~20 us
        call cannot hide), and whether the last replay left the same outputs,
        bit for bit, as an eager call."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                fn()
        g.replay()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(reps):
            g.replay()
        ev[1].record()
        torch.cuda.synchronize()
        got, got_idx = out.clone(), idx.clone()
        fn()
        torch.cuda.synchronize()
        same = bool(torch.equal(got.view(torch.int16), out.view(torch.int16)) and torch.equal(got_idx, idx))
        del g
        return ev[0].elapsed_time(ev[1]) / (reps * n), same

    def anchor():
        aoh_decode_anchor(q, full, ring, mask, lens, n_sink, window, top_k, indices=idx, out=out, workspace=ws_a)

    # a reuse layer's own cache keeps token-major V pages (the layout its
    # scattered reads want): the same pages with V transposed
    from paper_2608_06849_amd import PagedCache
    full_tm = PagedCache(full.k, full.v.transpose(-1, -2).contiguous(), full.block_table, v_token_major=True)

    def reuse(f):
        return lambda: aoh_decode_reuse(q, f, ring, mask, lens, n_sink, window, idx, mapping, out=out, workspace=ws_r)

    anchor_eager_ms = timed(anchor)
    reuse_eager_ms = timed(reuse(full_tm))
    anchor_ms, ok_a = graph_timed(anchor)
    anchor()                                   # the reuse steps borrow this anchor's selection
    reuse_dm_ms, ok_dm = graph_timed(reuse(full))
    reuse_ms, ok_r = graph_timed(reuse(full_tm))
    del full_tm
    gs = Hq // len(mask)
    reuse_bytes = B * (n_ret * top_k + n_str * min(length, n_sink + window)) * D * 2 * 2
    per_layer = (anchor_ms + (block - 1) * reuse_ms) / block
    log(f"H2Share (graph-timed): anchor {anchor_ms:.4f} ms, reuse {reuse_ms:.4f} ms (top-{top_k}; {reuse_dm_ms:.4f} ms "
        f"with dimension-major V pages); block of {block}: {per_layer:.4f} ms/layer vs {plain_ms:.4f} plain; "
        f"eager calls: anchor {anchor_eager_ms:.4f} ms, reuse {reuse_eager_ms:.4f} ms; "
        f"graph replays equal eager: {ok_a and ok_dm and ok_r}")
    return {
        "top_k": top_k, "block": block, "timing": "per call from a HIP graph of 20 calls",
        "anchor_ms": round(anchor_ms, 4), "reuse_ms": round(reuse_ms, 4),
        "reuse_ms_v_dim_major": round(reuse_dm_ms, 4), "plain_ms": round(plain_ms, 4),
        "anchor_eager_ms": round(anchor_eager_ms, 4), "reuse_eager_ms": round(reuse_eager_ms, 4),
        "graph_replays_equal_eager": ok_a and ok_dm and ok_r,
        "anchor_overhead": round(anchor_ms / plain_ms, 3),
        "ms_per_layer_in_block": round(per_layer, 4),
        "speedup_per_layer_vs_plain": round(plain_ms / per_layer, 3),
        "reuse_useful_gb": round(reuse_bytes / 1e9, 5),
        "reuse_useful_gbps": round(reuse_bytes / (reuse_ms * 1e-3) / 1e9, 1),
        "group_size": gs,
    }


def stack_decode_leg(args, torch, synth, PagedCache, RingCache, aoh_decode, aoh_decode_workspace_bytes,
                     aoh_kv_append, decode_bytes):
    """Decode steps through all 28 layers of the Qwen2.5-7B-shaped stack at a
    262144-token context (batch 1, 2 of 4 KV heads streaming per layer,
    n_sink 64, window 2048), issued eagerly and as one captured HIP graph per
    step.  Cache contents do not change the timing; they are filled from
    torch's seeded device generator."""
    c = synth.CONFIGS["qwen25_stack_256k"]
    L, T, Hq, Hkv, D, n_sink, window = c["layers"], c["seq"], c["hq"], c["hkv"], c["d"], c["n_sink"], c["window"]
    steps = 16
    dev, bf = "cuda", torch.bfloat16
    gen = torch.Generator(device=dev)
    gen.manual_seed(c["seed"])
    max_pages = (T + 4 * steps + 16 + 15) // 16  # every run and replay below appends one token
    bt = torch.arange(max_pages, dtype=torch.int32)[None]
    layers = []
    for l in range(L):
        mask = synth.choose_streaming(Hkv, c["n_streaming"], c["seed"], "streaming", l).tolist()
        full = PagedCache.allocate(max_pages, mask.count(0), D, bf, bt)
        ring = RingCache.allocate(1, mask.count(1), n_sink, window, D, bf)
        for t in (full.k, full.v, ring.k, ring.v):
            t.normal_(generator=gen)
        layers.append((mask, full, ring))
    q = torch.randn((L, 1, Hq, D), device=dev, generator=gen).to(bf)
    kv = torch.randn((L, 2, 1, 1, Hkv, D), device=dev, generator=gen).to(bf)
    lens_before = torch.full((1,), T, dtype=torch.int32, device=dev)
    lens_after = lens_before + 1
    ws = torch.empty(aoh_decode_workspace_bytes(1, Hq, D, max_pages, n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=dev)
    outs = torch.empty((L, 1, Hq, D), dtype=bf, device=dev)

    from paper_2608_06849_amd import aoh_decode_step

    def one_step(fused=True):
        # the position advances once per step (one small device add, as a
        # serving loop does); the two-call form also moves the append position
        for l, (mask, full, ring) in enumerate(layers):
            if fused:
                aoh_decode_step(q[l], kv[l, 0, :, 0], kv[l, 1, :, 0], full, ring, mask, lens_after, n_sink, window,
                                out=outs[l], workspace=ws)
            else:
                aoh_kv_append(kv[l, 0], kv[l, 1], mask, lens_before, full, ring, n_sink, window)
                aoh_decode(q[l], full, ring, mask, lens_after, n_sink, window, out=outs[l], workspace=ws)
        lens_after.add_(1)
        if not fused:
            lens_before.add_(1)

    def timed(fn):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(steps):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    one_step()
    eager_ms = timed(one_step)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        one_step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        one_step()
    graph_ms = timed(g.replay)
    lens_before.copy_(lens_after - 1)
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2):
        one_step(fused=False)
    graph_two_ms = timed(g2.replay)
    by = L * decode_bytes([T + steps], Hkv - c["n_streaming"], c["n_streaming"], D, 2, n_sink, window)
    # resident KV of the 28 layers' caches at the 262144-token prompt length
    # (the allocations also hold the decode steps' pages), against every head
    # keeping all T tokens
    resident = sum((f.k.numel() + f.v.numel()) // max_pages * ((T + 15) // 16) + r.k.numel() + r.v.numel()
                   for _, f, r in layers) * 2
    resident_all = L * Hkv * T * D * 2 * 2
    res = {
        "workload": "decode step through 28 layers of the Qwen2.5-7B attention shape, batch 1, context 262144, "
                    "2 of 4 KV heads streaming per layer (n_sink 64, window 2048); per layer: append 1 token + decode "
                    "(one aoh_decode_step call)",
        "eager_ms_per_step": round(eager_ms, 4),
        "graph_ms_per_step": round(graph_ms, 4),
        "graph_two_call_ms_per_step": round(graph_two_ms, 4),
        "graph_speedup": round(eager_ms / graph_ms, 3),
        "kv_gb_per_step": round(by / 1e9, 4),
        "kv_gbps_graph": round(by / (graph_ms * 1e-3) / 1e9, 1),
        "frac_of_hbm_peak_graph": round(by / (graph_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "kv_gbps_eager": round(by / (eager_ms * 1e-3) / 1e9, 1),
        "frac_of_hbm_peak_eager": round(by / (eager_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "resident_kv_gb": round(resident / 1e9, 4),
        "resident_kv_gb_all_retrieval": round(resident_all / 1e9, 4),
        "resident_kv_saving": round(1 - resident / resident_all, 4),
    }
    log(f"stack decode: eager {eager_ms:.3f} ms/step, graph {graph_ms:.3f} ms/step ({graph_two_ms:.3f} as two calls), "
        f"{res['kv_gbps_graph']:.0f} GB/s with the graph")
    return res


def stack_prefill_leg(torch, synth, PagedCache, RingCache):
    """One layer of the 28-layer stack's 262144-token prefill (28 query / 4 KV
    heads, d_head 128, bf16, the layer-0 choice of 2 streaming KV heads, n_sink
    64, window 2048), filling the paged cache and the ring as in serving, timed
    over three calls; the same kernels with every head retrieval for
    comparison.  Inputs come from torch's seeded device generator (the cost
    does not depend on the values); the 28-layer figure is 28 x this layer."""
    from paper_2608_06849_amd import aoh_prefill_append
    c = synth.CONFIGS["qwen25_stack_256k"]
    L, T, Hq, Hkv, D, n_sink, window = c["layers"], c["seq"], c["hq"], c["hkv"], c["d"], c["n_sink"], c["window"]
    dev, bf = "cuda", torch.bfloat16
    gen = torch.Generator(device=dev)
    gen.manual_seed(c["seed"] + 1)
    mask = synth.choose_streaming(Hkv, c["n_streaming"], c["seed"], "streaming", 0).tolist()
    q = torch.randn((1, T, Hq, D), device=dev, generator=gen).to(bf)
    k = (0.5 * torch.randn((1, T, Hkv, D), device=dev, generator=gen)).to(bf)
    v = torch.randn((1, T, Hkv, D), device=dev, generator=gen).to(bf)
    out = torch.empty_like(q)
    max_pages = (T + 15) // 16
    bt = torch.arange(max_pages, dtype=torch.int32)[None]
    gs = Hq // Hkv

    def timed(m, n=3):
        full = PagedCache.allocate(max_pages, m.count(0), D, bf, bt)
        ring = RingCache.allocate(1, m.count(1), n_sink, window, D, bf) if m.count(1) else None
        aoh_prefill_append(q, k, v, m, n_sink, window, full, ring, out=out)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(n):
            aoh_prefill_append(q, k, v, m, n_sink, window, full, ring, out=out)
        ev[1].record()
        torch.cuda.synchronize()
        del full, ring
        return ev[0].elapsed_time(ev[1]) / n

    ms = timed(mask)
    ms_all = timed([0] * Hkv)
    fl = useful_prefill_flops(T, D, gs * mask.count(0), gs * mask.count(1), n_sink, window)
    fl_all = useful_prefill_flops(T, D, gs * Hkv, 0, n_sink, window)
    res = {
        "workload": "one layer of the 28-layer Qwen2.5-7B-shaped stack: 262144-token prefill filling the caches, "
                    f"28 q / 4 KV heads (streaming KV heads {[g for g in range(Hkv) if mask[g]]}), d_head 128, bf16, "
                    "n_sink 64, window 2048",
        "layer_ms": round(ms, 2),
        "useful_tflop": round(fl / 1e12, 2),
        "tflops": round(fl / (ms * 1e-3) / 1e12, 1),
        "frac_of_bf16_peak": round(fl / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "all_retrieval_layer_ms": round(ms_all, 2),
        "all_retrieval_tflops": round(fl_all / (ms_all * 1e-3) / 1e12, 1),
        "speedup_vs_all_retrieval": round(ms_all / ms, 3),
        "stack_prefill_s_extrapolated": round(L * ms / 1e3, 3),
    }
    log(f"stack prefill: {ms:.1f} ms per 262144-token layer ({res['tflops']:.0f} TFLOP/s useful), "
        f"all-retrieval {ms_all:.1f} ms; 28 layers ~{L * ms / 1e3:.2f} s (extrapolated)")
    return res


def varlen_leg(args, torch, synth):
    """The variable-length workload (16 sequences of U[4096, 65536] tokens, 32 q /
    8 KV heads, d_head 128, bf16, n_sink 64) as one packed prefill per setting
    (streaming fraction x window), against one prefill call per sequence."""
    from paper_2608_06849_amd import aoh_prefill, aoh_prefill_varlen
    c = synth.CONFIGS["varlen_sweep"]
    lens = synth.lengths_uniform(c["n_seq"], c["len_lo"], c["len_hi"], c["seed"])
    bf = torch.bfloat16
    t0 = time.time()
    parts = [synth.sweep_sequence(b, int(lens[b])) for b in range(len(lens))]
    q = torch.cat([torch.from_numpy(p["q"][0]).to(bf) for p in parts]).to("cuda")
    k = torch.cat([torch.from_numpy(p["k"][0]).to(bf) for p in parts]).to("cuda")
    v = torch.cat([torch.from_numpy(p["v"][0]).to(bf) for p in parts]).to("cuda")
    del parts
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda")
    out = torch.empty_like(q)
    offs = np.concatenate([[0], np.cumsum(lens)])
    hq, hkv, d, n_sink = c["hq"], c["hkv"], c["d"], c["n_sink"]
    gs = hq // hkv
    torch.cuda.synchronize()
    log(f"varlen workload ready in {time.time() - t0:.1f}s ({int(lens.sum())} tokens)")

    def timed(fn, n=3):
        fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(n):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    res = {"workload": f"{len(lens)} sequences of U[4096, 65536] tokens ({int(lens.sum())} total), 32 q / 8 KV heads, "
                       "d_head 128, bf16, n_sink 64; one packed prefill call", "settings": []}
    for sp in c["sparsity_pct"]:
        n_str = synth.n_streaming_for(hkv, sp)
        for window in c["windows"]:
            mask = synth.choose_streaming(hkv, n_str, c["seed"], "streaming", sp, window).tolist()
            fl = sum(useful_prefill_flops(int(n), d, gs * (hkv - n_str), gs * n_str, n_sink, window) for n in lens)
            ms = timed(lambda: aoh_prefill_varlen(q, k, v, cu, int(lens.max()), mask, n_sink, window, out=out))
            entry = {"streaming_pct": sp, "window": window, "ms": round(ms, 3),
                     "useful_tflop": round(fl / 1e12, 3), "tflops": round(fl / (ms * 1e-3) / 1e12, 1)}
            entry["decode"] = varlen_decode(torch, q, k, v, cu, lens, mask, n_sink, window, hq, hkv, d,
                                            c["decode_steps"])
            if sp == 50 and window == 4096:
                def per_seq():
                    for b in range(len(lens)):
                        sl = slice(int(offs[b]), int(offs[b + 1]))
                        aoh_prefill(q[sl][None], k[sl][None], v[sl][None], mask, n_sink, window, out=out[sl][None])
                entry["per_sequence_calls_ms"] = round(timed(per_seq), 3)
            res["settings"].append(entry)
            log(f"varlen {sp}% w{window}: {ms:.2f} ms, {entry['tflops']} TFLOP/s; decode "
                f"{entry['decode']['ms_per_step']:.4f} ms/step, {entry['decode']['kv_gbps']:.0f} GB/s")
    del q, k, v, out
    return res


def varlen_decode(torch, q, k, v, cu, lens, mask, n_sink, window, hq, hkv, d, steps):
    """The sweep's decode: the packed prefill fills a paged cache and a ring
    for the 16 sequences, then `steps` batched single-token steps (one
    aoh_decode_step call each: store the token, decode) are timed."""
    from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode_step, aoh_decode_workspace_bytes,
                                      aoh_prefill_varlen)
    B, bf, dev = len(lens), torch.bfloat16, "cuda"
    n_ret, n_str = mask.count(0), mask.count(1)
    max_pages = (int(lens.max()) + steps + 15) // 16
    bt = torch.arange(B * max_pages, dtype=torch.int32).reshape(B, max_pages)
    full = PagedCache.allocate(B * max_pages, n_ret, d, bf, bt) if n_ret else None
    ring = RingCache.allocate(B, n_str, n_sink, window, d, bf) if n_str else None
    out = torch.empty_like(q)
    aoh_prefill_varlen(q, k, v, cu, int(lens.max()), mask, n_sink, window, kv_full=full, kv_ring=ring, out=out)
    gen = torch.Generator(device=dev)
    gen.manual_seed(4321)
    qs = torch.randn((steps, B, hq, d), device=dev, generator=gen).to(bf)
    kvs = torch.randn((steps, 2, B, hkv, d), device=dev, generator=gen).to(bf)
    lens_dev = [torch.tensor(lens + s + 1, dtype=torch.int32, device=dev) for s in range(steps)]
    ws = torch.empty(aoh_decode_workspace_bytes(B, hq, d, max_pages, n_sink + window), dtype=torch.uint8, device=dev)
    o = torch.empty((B, hq, d), dtype=bf, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(3):  # warm-up: stores step 0's token, which step 0 stores again
        aoh_decode_step(qs[0], kvs[0, 0], kvs[0, 1], full, ring, mask, lens_dev[0], n_sink, window, out=o,
                        workspace=ws)
    torch.cuda.synchronize()
    ev[0].record()
    for s in range(steps):
        aoh_decode_step(qs[s], kvs[s, 0], kvs[s, 1], full, ring, mask, lens_dev[s], n_sink, window, out=o,
                        workspace=ws)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    by = np.mean([decode_bytes([int(n) + s + 1 for n in lens], n_ret, n_str, d, 2, n_sink, window)
                  for s in range(steps)])
    resident = sum((c.k.numel() + c.v.numel()) for c in (full, ring) if c is not None) * 2
    del full, ring, out, qs, kvs
    return {"steps": steps, "ms_per_step": round(ms, 4), "tokens_per_s": round(B / (ms * 1e-3), 1),
            "kv_gb_per_step": round(by / 1e9, 4), "kv_gbps": round(by / (ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(by / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "allocated_kv_gb": round(resident / 1e9, 4)}


def classify_leg(args, torch, synth):
    """Offline head classification of a whole Qwen2.5-7B-shaped model (28
    layers, 28 query / 4 KV heads, d_head 128, d_model 3584, bf16 weights):
    Gram matrices, Cholesky, spectra, effective ranks and labels on the GPU."""
    from paper_2608_06849_amd import aoh_classify, aoh_classify_workspace_bytes, aoh_retrieval_group_count
    name = "qwen25_classify"
    c = synth.CONFIGS[name]
    L, hq, hkv, d, dm = c["layers"], c["hq"], c["hkv"], c["d"], c["d_model"]
    t0 = time.time()
    wq = torch.empty((L, hq * d, dm), dtype=torch.bfloat16, device="cuda")
    wk = torch.empty((L, hkv * d, dm), dtype=torch.bfloat16, device="cuda")
    for l in range(L):
        a, b = synth.projection_weights(name, l)
        wq[l].copy_(torch.from_numpy(a).to(torch.bfloat16))
        wk[l].copy_(torch.from_numpy(b).to(torch.bfloat16))
    k = aoh_retrieval_group_count(hkv, c["sparsity"])
    hr = torch.empty((L, hq), dtype=torch.float64, device="cuda")
    gsc = torch.empty((L, hkv), dtype=torch.float64, device="cuda")
    lab = torch.empty((L, hkv), dtype=torch.uint8, device="cuda")
    ws = torch.empty(aoh_classify_workspace_bytes(L, hq, hkv, d), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    log(f"classifier weights ready in {time.time() - t0:.1f}s")
    for _ in range(2):
        aoh_classify(wq, wk, d, k, hr, gsc, lab, workspace=ws)
    n = max(3, args.steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(n):
        aoh_classify(wq, wk, d, k, hr, gsc, lab, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n
    wbytes = (wq.numel() + wk.numel()) * 2
    log(f"classify {L} layers: {ms:.3f} ms ({wbytes / (ms * 1e-3) / 1e12:.2f} TB/s of weights)")
    return {
        "workload": f"Qwen2.5-7B-shaped projections: {L} layers x ({hq} q + {hkv} KV heads), d_head {d}, "
                    f"d_model {dm}, bf16; {k} of {hkv} groups retrieval per layer",
        "ms": round(ms, 4),
        "heads_per_s": round(L * hq / (ms * 1e-3)),
        "weight_bytes": wbytes,
        "weight_tb_per_s": round(wbytes / (ms * 1e-3) / 1e12, 3),
        "streaming_groups": int(lab.sum().item()),
    }


def cpu_baseline(q, k, v, mask, n_sink, window, T, D, gs, target_s=15.0):
    """The oracle (float64 numpy, untuned) on a bounded sample of the same
    workload: a set of query rows (mask boundaries plus seeded random rows)
    for all 28 heads of the 32K prefill.  Reported in the metric's unit."""
    import threadpoolctl

    from oracle import accounting as C
    from oracle import attention as OA

    cores = len(os.sched_getaffinity(0))
    limiter = threadpoolctl.threadpool_limits(limits=cores)
    qh = q.float().cpu().numpy().astype(np.float64)
    kh = k.float().cpu().numpy().astype(np.float64)
    vh = v.float().cpu().numpy().astype(np.float64)
    boundary = [0, n_sink - 1, n_sink, window - 1, window, n_sink + window, T - 1]
    rng = np.random.default_rng(12345)
    n_rows = 16
    while True:
        rows = np.unique(np.concatenate([boundary, rng.integers(0, T, n_rows)])).astype(np.int64)
        t0 = time.perf_counter()
        OA.prefill(qh, kh, vh, mask, n_sink, window, rows=rows)
        dt = time.perf_counter() - t0
        if dt >= target_s * 2 / 3 or n_rows >= 8192:
            break
        n_rows = int(n_rows * max(2.0, target_s / max(dt, 1e-3)))
    limiter.restore_original_limits()
    flops = 0
    for g, st in enumerate(mask):
        per_row = sum(C.visible_pairs_row(int(i), bool(st), n_sink, window) for i in rows)
        flops += 4 * D * gs * per_row
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "seconds": round(dt, 2),
            "sample": f"{len(rows)} query rows (mask boundaries + seeded random) x {q.shape[2]} heads of the "
                      f"{T}-token prefill, float64 numpy, BLAS threads limited to the {cores} cores this "
                      "process may run on"}


if __name__ == "__main__":
    main()
