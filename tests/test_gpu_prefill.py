"""Prefill parity on the GPU: libaoh (through the C interface) against the
float64 oracle, on seeded inputs, at sizes that span several tiles and a
ragged tail, plus exact special cases."""
import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2608_06849_amd import aoh_prefill, aoh_prefill_chunked
from tests.helpers import assert_parity, bits, f64, to_dtype

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _inputs(B, T, Hq, Hkv, D, dtype, seed, k_scale=1.0):
    q = to_dtype(synth.gaussian((B, T, Hq, D), seed, "q"), dtype).to(DEV)
    k = to_dtype(synth.gaussian((B, T, Hkv, D), seed, "k", scale=k_scale), dtype).to(DEV)
    v = to_dtype(synth.gaussian((B, T, Hkv, D), seed, "v"), dtype).to(DEV)
    return q, k, v


def test_tiny_fp32_workload():
    # batch 1, 4 query heads over 2 KV heads, d 64, fp32, 256 tokens; KV head 1
    # streaming with 4 sink tokens and a 32-token window
    cfg = synth.CONFIGS["tiny"]
    q, k, v = _inputs(1, 256, 4, 2, 64, torch.float32, cfg["seed"])
    mask = cfg["streaming"]
    out = aoh_prefill(q, k, v, mask, cfg["n_sink"], cfg["window"])
    torch.cuda.synchronize()
    want = OA.prefill(f64(q), f64(k), f64(v), mask, cfg["n_sink"], cfg["window"])
    assert_parity(out, want, torch.float32, "tiny fp32 prefill")


CASES = [
    # B, T, Hq, Hkv, D, mask, n_sink, window
    (2, 300, 8, 2, 128, [1, 0], 4, 100),      # ragged tail, GQA 4
    (1, 513, 14, 2, 128, [0, 1], 64, 128),    # GQA 7 (Qwen-like), tile-skipping band
    (1, 700, 4, 4, 64, [1, 0, 1, 1], 0, 1),   # d 64, window of one token, no sink
    (1, 1, 4, 2, 128, [1, 0], 4, 32),         # single token
    (3, 129, 8, 8, 128, [1] * 8, 130, 5),     # sink covers the sequence -> dense
    (1, 1000, 4, 2, 128, [1, 1], 70, 200),    # sink spans two tiles, band far away
    (1, 640, 2, 1, 64, [1], 0, 64),           # window exactly one tile
    (1, 257, 4, 1, 128, [0], 4, 32),          # all retrieval
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("B,T,Hq,Hkv,D,mask,n_sink,window", CASES)
def test_prefill_matches_oracle(B, T, Hq, Hkv, D, mask, n_sink, window, dtype):
    q, k, v = _inputs(B, T, Hq, Hkv, D, dtype, seed=T * 7 + Hq)
    out = aoh_prefill(q, k, v, mask, n_sink, window)
    torch.cuda.synchronize()
    want = OA.prefill(f64(q), f64(k), f64(v), mask, n_sink, window)
    assert_parity(out, want, dtype, f"prefill {B,T,Hq,Hkv,D,mask,n_sink,window}")


def test_prefill_fp32_output_and_strided_inputs():
    # q, k, v as column slices of one fused [B, T, Hq + 2 Hkv, D] buffer
    B, T, Hq, Hkv, D = 2, 333, 8, 2, 128
    qkv = to_dtype(synth.gaussian((B, T, Hq + 2 * Hkv, D), 5, "qkv"), torch.bfloat16).to(DEV)
    q, k, v = qkv[:, :, :Hq], qkv[:, :, Hq:Hq + Hkv], qkv[:, :, Hq + Hkv:]
    assert not q.is_contiguous()
    out = torch.empty((B, T, Hq, D), dtype=torch.float32, device=DEV)
    aoh_prefill(q, k, v, [0, 1], 16, 64, out=out)
    torch.cuda.synchronize()
    want = OA.prefill(f64(q), f64(k), f64(v), [0, 1], 16, 64)
    mx, _ = assert_parity(out, want, torch.bfloat16, "strided prefill, fp32 out")
    assert mx < 5e-3  # no bf16 rounding of the output


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_window_one_returns_own_value_exactly(dtype):
    B, T, Hq, Hkv, D = 1, 300, 4, 2, 128
    q, k, v = _inputs(B, T, Hq, Hkv, D, dtype, seed=11)
    out = aoh_prefill(q, k, v, [1, 1], 0, 1)
    torch.cuda.synchronize()
    for h in range(Hq):
        got, want = out[:, :, h], v[:, :, h // 2]
        if not np.array_equal(bits(got), bits(want)):
            d = np.abs(f64(got) - f64(want))
            bad = np.argwhere(d > 0)
            raise AssertionError(f"head {h}: {len(bad)} elements differ, max {d.max():.3e}, first {bad[:5].tolist()}")


def test_zero_keys_average_visible_values():
    # K = 0: every visible key has weight exactly 1/count; V[j] = j mod 64 is
    # exact in bf16, so with an fp32 output the only error is fp32 summation
    B, T, Hq, Hkv, D = 1, 1000, 4, 2, 128
    q = to_dtype(synth.gaussian((B, T, Hq, D), 3, "q"), torch.bfloat16).to(DEV)
    k = torch.zeros((B, T, Hkv, D), dtype=torch.bfloat16, device=DEV)
    vv = np.broadcast_to((np.arange(T) % 64).astype(np.float32)[None, :, None, None], (B, T, Hkv, D))
    v = to_dtype(vv, torch.bfloat16).to(DEV)
    out = torch.empty((B, T, Hq, D), dtype=torch.float32, device=DEV)
    for n_sink, window in [(4, 32), (0, 100), (70, 64), (3, 1)]:
        aoh_prefill(q, k, v, [0, 1], n_sink, window, out=out)
        torch.cuda.synchronize()
        want = OA.prefill(f64(q), f64(k), f64(v), [0, 1], n_sink, window)
        err = np.abs(f64(out) - want).max()
        assert err < 1e-4, (n_sink, window, err)


@pytest.mark.parametrize("T,n_sink,window", [(2048, 4, 600), (1500, 64, 1000), (777, 0, 300)])
def test_score_spikes_far_from_the_diagonal(T, n_sink, window):
    # Every query shares a direction u; a few keys far before the diagonal
    # (and the first sink key) carry a large multiple of u, so their scores
    # sit ~40 log2 units above the rest.  The running max a query block has
    # when it reaches them (from its diagonal tiles) is far too low: the
    # kernel must raise it and rescale what it has accumulated.  Retrieval
    # and streaming heads, d_head 128, bf16 (Sec. 5 attention, oracle in fp64).
    B, Hq, Hkv, D = 1, 4, 2, 128
    rng_q = synth.gaussian((B, T, Hq, D), 31, "spike-q")
    rng_k = synth.gaussian((B, T, Hkv, D), 31, "spike-k", scale=0.5)
    rng_v = synth.gaussian((B, T, Hkv, D), 31, "spike-v")
    u = np.zeros(D, dtype=np.float32)
    u[::2] = 1.0 / np.sqrt(D / 2)
    qn = rng_q + 10.0 * u
    kn = rng_k.copy()
    for p_ in (0, 5, 300, T // 2, T - 700):
        if 0 <= p_ < T:
            kn[:, p_] += 31.0 * u
    q = to_dtype(qn, torch.bfloat16).to(DEV)
    k = to_dtype(kn, torch.bfloat16).to(DEV)
    v = to_dtype(rng_v, torch.bfloat16).to(DEV)
    mask = [0, 1]
    out = aoh_prefill(q, k, v, mask, n_sink, window, out=torch.empty((B, T, Hq, D), dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
    want = OA.prefill(f64(q), f64(k), f64(v), mask, n_sink, window)
    assert_parity(out, want, torch.bfloat16, f"score spikes T={T}")


def test_deterministic():
    q, k, v = _inputs(1, 777, 8, 2, 128, torch.bfloat16, seed=9)
    a = aoh_prefill(q, k, v, [0, 1], 4, 50)
    b = aoh_prefill(q, k, v, [0, 1], 4, 50)
    torch.cuda.synchronize()
    assert np.array_equal(bits(a), bits(b))


CHUNK_CASES = [
    # B, T, Hq, Hkv, D, mask, n_sink, window, chunk
    (1, 700, 8, 2, 128, [1, 0], 4, 100, 1),       # one-token chunks
    (2, 300, 8, 2, 128, [0, 1], 4, 32, 7),        # chunk not a divisor of any tile size
    (1, 1000, 14, 2, 128, [1, 1], 64, 128, 64),   # chunk = a quarter of a query block
    (1, 1300, 4, 4, 64, [1, 0, 1, 1], 0, 50, 100),
    (1, 2500, 4, 1, 128, [1], 16, 256, 1024),     # chunk spans four query blocks
    (1, 513, 4, 2, 128, [1, 0], 8, 64, 600),      # one chunk covers the prompt -> dense
    (1, 1, 4, 2, 128, [1, 0], 4, 32, 16),         # single token
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("B,T,Hq,Hkv,D,mask,n_sink,window,chunk", CHUNK_CASES)
def test_chunked_prefill_matches_oracle(B, T, Hq, Hkv, D, mask, n_sink, window, chunk, dtype):
    q, k, v = _inputs(B, T, Hq, Hkv, D, dtype, seed=T * 5 + chunk)
    out = aoh_prefill_chunked(q, k, v, mask, n_sink, window, chunk)
    torch.cuda.synchronize()
    want = OA.prefill(f64(q), f64(k), f64(v), mask, n_sink, window, chunk=chunk)
    assert_parity(out, want, dtype, f"chunked prefill {B,T,Hq,Hkv,D,mask,n_sink,window,chunk}")


def test_chunk_one_equals_band_one_wider():
    # with one-token chunks a query sees the window tokens before it plus itself
    q, k, v = _inputs(1, 900, 8, 2, 128, torch.bfloat16, seed=21)
    a = aoh_prefill_chunked(q, k, v, [1, 0], 4, 63, 1)
    b = aoh_prefill(q, k, v, [1, 0], 4, 64)
    torch.cuda.synchronize()
    assert np.array_equal(bits(a), bits(b))


def test_chunk_at_least_prompt_is_full_causal():
    q, k, v = _inputs(1, 600, 4, 2, 128, torch.bfloat16, seed=22)
    a = aoh_prefill_chunked(q, k, v, [1, 1], 4, 32, 600)
    b = aoh_prefill(q, k, v, [0, 0], 4, 32)
    torch.cuda.synchronize()
    assert np.array_equal(bits(a), bits(b))


@pytest.mark.parametrize("B,T,Hq,Hkv,mask", [
    (1, 513, 14, 2, [0, 1]),          # 21 retrieval items: the streaming items start after 3 idle pads
    (2, 700, 8, 4, [1, 0, 0, 1]),
    (1, 2000, 28, 4, [0, 1, 0, 1]),   # Qwen-shaped heads
])
def test_one_launch_equals_per_type_launches(B, T, Hq, Hkv, mask):
    # A layer with both head types runs its prefill as one launch (retrieval
    # items, then streaming items).  Each head's output must be bit-identical
    # to a call holding only the heads of its type (Sec. 5 attention per head).
    D, gs, n_sink, window = 128, Hq // Hkv, 4, 100
    q, k, v = _inputs(B, T, Hq, Hkv, D, torch.bfloat16, seed=T + Hq)
    out = aoh_prefill(q, k, v, mask, n_sink, window)
    for typ in (0, 1):
        qi = torch.tensor([h for h in range(Hq) if mask[h // gs] == typ], device=DEV)
        ki = torch.tensor([g for g in range(Hkv) if mask[g] == typ], device=DEV)
        one = aoh_prefill(q.index_select(2, qi).contiguous(), k.index_select(2, ki).contiguous(),
                          v.index_select(2, ki).contiguous(), [typ] * len(ki), n_sink, window)
        torch.cuda.synchronize()
        assert np.array_equal(bits(one), bits(out.index_select(2, qi))), f"head type {typ}"


def test_one_launch_queue_slots_across_calls_streams_and_graph_replays():
    # The one-launch form hands its streaming items out through work-queue
    # counters in one of 64 slots per launch, cleared by the launch's last
    # workgroup.  Every later launch must see its slot cleared: more calls
    # than slots on one stream, calls overlapping on two streams, and replays
    # of a captured call all give the output of a first call, bit for bit.
    B, T, Hq, Hkv, D, mask, n_sink, window = 1, 2000, 28, 4, 128, [0, 1, 0, 1], 64, 256
    q, k, v = _inputs(B, T, Hq, Hkv, D, torch.bfloat16, seed=77)
    ref = bits(aoh_prefill(q, k, v, mask, n_sink, window))
    out = torch.empty_like(q)
    for i in range(70):
        aoh_prefill(q, k, v, mask, n_sink, window, out=out)
        torch.cuda.synchronize()
        assert np.array_equal(bits(out), ref), f"call {i} on one stream"
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = [torch.empty_like(q) for _ in range(2)]
    torch.cuda.synchronize()
    for i in range(8):
        for st, o in zip((s1, s2), outs):
            with torch.cuda.stream(st):
                aoh_prefill(q, k, v, mask, n_sink, window, out=o)
    torch.cuda.synchronize()
    for j, o in enumerate(outs):
        assert np.array_equal(bits(o), ref), f"stream {j}"
    g_out = torch.empty_like(q)
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        aoh_prefill(q, k, v, mask, n_sink, window, out=g_out)  # warm-up outside the graph
        with torch.cuda.graph(g, stream=cap):
            aoh_prefill(q, k, v, mask, n_sink, window, out=g_out)
    torch.cuda.synchronize()
    for r in range(5):
        g_out.zero_()
        aoh_prefill(q, k, v, mask, n_sink, window, out=out)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(g_out), ref), f"graph replay {r}"
        assert np.array_equal(bits(out), ref), f"eager call after replay {r}"


@pytest.mark.parametrize("T,n_sink,window,step", [(1500, 4, 600, 20.0), (1100, 64, 300, 3.0), (700, 0, 1000, 40.0)])
def test_rising_scores_raise_the_max_every_tile(T, n_sink, window, step):
    # Scores that grow along the sequence: key p carries (p / 64) * step
    # along the queries' shared direction u, so every 64-key tile a query
    # block reaches lifts the row max by about step * 10 * log2(e) / sqrt(D)
    # (log2 units): with step 20 or 40 each tile exceeds any trailing reference
    # max by far and must be rescaled; with step 3 the growth stays below the
    # acceptance bound for several tiles.  Retrieval and streaming heads,
    # d_head 128, bf16 against the fp64 oracle (Sec. 5 attention).
    B, Hq, Hkv, D = 1, 4, 2, 128
    rng_q = synth.gaussian((B, T, Hq, D), 37, "rise-q")
    rng_k = synth.gaussian((B, T, Hkv, D), 37, "rise-k", scale=0.5)
    rng_v = synth.gaussian((B, T, Hkv, D), 37, "rise-v")
    u = np.zeros(D, dtype=np.float32)
    u[1::2] = 1.0 / np.sqrt(D / 2)
    qn = rng_q + 10.0 * u
    kn = rng_k + (np.arange(T, dtype=np.float32) / 64.0 * step)[None, :, None, None] * u
    q = to_dtype(qn, torch.bfloat16).to(DEV)
    k = to_dtype(kn, torch.bfloat16).to(DEV)
    v = to_dtype(rng_v, torch.bfloat16).to(DEV)
    mask = [1, 0]
    out = aoh_prefill(q, k, v, mask, n_sink, window, out=torch.empty((B, T, Hq, D), dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
    want = OA.prefill(f64(q), f64(k), f64(v), mask, n_sink, window)
    assert_parity(out, want, torch.bfloat16, f"rising scores T={T} step={step}")
