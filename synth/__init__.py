"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke run.

This module only draws random numbers and lays them out; it holds none of the
attention arithmetic.  Every draw comes from numpy's counter-based Philox
generator keyed by (seed, purpose, index...), so a tensor can be regenerated
piecewise and identically on any host.

The workloads stand in for the paper's long-context runs (LongBench, passkey,
and the latency tables) whose data and model weights are not used here: the
shapes follow the models the paper evaluates (Qwen2.5-7B: 28 query heads, 4 KV
heads, d_head 128; a Llama-3.1-8B-like shape: 32 query heads, 8 KV heads,
d_head 128), values are N(0, 1) (optionally scaled), and "needles" are planted
keys that a retrieval head can find far from the query.
"""
import hashlib

import numpy as np

_PURPOSES = {}


def _purpose_id(name):
    if name not in _PURPOSES:
        _PURPOSES[name] = int.from_bytes(hashlib.sha256(name.encode()).digest()[:4], "little")
    return _PURPOSES[name]


def rng(seed, purpose, *index):
    """Philox generator for (seed, purpose, index...)."""
    key = [int(seed) & 0xFFFFFFFF, _purpose_id(purpose)] + [int(i) & 0xFFFFFFFF for i in index]
    while len(key) < 4:
        key.append(0)
    if len(key) > 4:
        h = hashlib.sha256(np.asarray(key, dtype=np.uint64).tobytes()).digest()
        key = list(np.frombuffer(h[:16], dtype=np.uint32))
    k = np.asarray(key[:4], dtype=np.uint32).view(np.uint64)
    return np.random.Generator(np.random.Philox(key=k))


def gaussian(shape, seed, purpose, *index, scale=1.0, dtype=np.float32):
    """N(0, scale^2) samples, float32."""
    x = rng(seed, purpose, *index).standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x.astype(dtype, copy=False)


def choose_streaming(n_kv_heads, n_streaming, seed, purpose="streaming", *index):
    """0/1 mask of length n_kv_heads with n_streaming ones, seeded choice."""
    sel = rng(seed, purpose, *index).choice(n_kv_heads, size=n_streaming, replace=False)
    m = np.zeros(n_kv_heads, dtype=np.uint8)
    m[sel] = 1
    return m


def n_streaming_for(n_kv_heads, sparsity_pct):
    """Streaming KV heads for a target sparsity: G - ceil((1 - s) G), in exact
    integer arithmetic on a percentage."""
    retrieval = -(-(100 - sparsity_pct) * n_kv_heads // 100)
    return n_kv_heads - retrieval


def page_permutation(n_pages, seed, purpose="pages"):
    """A seeded shuffle of physical page ids (so logical order != physical)."""
    return rng(seed, purpose).permutation(n_pages).astype(np.int32)


def lengths_uniform(n, lo, hi, seed, purpose="lengths"):
    """n integer lengths drawn uniformly from [lo, hi]."""
    return rng(seed, purpose).integers(lo, hi + 1, size=n).astype(np.int64)


def plant_needles(k, lens, n_needles, n_sink, window_max, seed, scale=4.0, seq_ids=None):
    """Overwrite n_needles rows per (sequence, KV head) of k [B, L, Hkv, D]
    in place with scale * |k_row| * u, u a seeded unit direction, at positions
    drawn from [n_sink, len - window_max) so the needles are outside every
    streaming head's window and only retrieval heads can see them.
    Returns the positions [B, Hkv, n_needles]."""
    b_n, _, hkv, d = k.shape
    seq_ids = list(range(b_n)) if seq_ids is None else list(seq_ids)
    pos = np.zeros((b_n, hkv, n_needles), dtype=np.int64)
    for b in range(b_n):
        hi = int(lens[b]) - window_max
        if hi <= n_sink:
            continue
        for g in range(hkv):
            r = rng(seed, "needle", seq_ids[b], g)
            u = r.standard_normal(d).astype(np.float64)
            u /= np.linalg.norm(u)
            p = np.sort(r.choice(np.arange(n_sink, hi), size=n_needles, replace=False))
            pos[b, g] = p
            for q in p:
                nrm = float(np.linalg.norm(k[b, q, g].astype(np.float64)))
                k[b, q, g] = (scale * nrm * u).astype(k.dtype)
    return pos


# Workloads.  Sizes follow the models the paper evaluates; see the module doc.
CONFIGS = {
    "tiny": dict(batch=1, hq=4, hkv=2, d=64, dtype="f32", seq=256, streaming=[0, 1],
                 n_sink=4, window=32, decode_steps=16, seed=0),
    "qwen25_prefill_32k": dict(batch=1, hq=28, hkv=4, d=128, dtype="bf16", seq=32768,
                               streaming=[0, 1, 0, 1], n_sink=64, window=1024, k_scale=0.5, seed=1),
    "llama_decode_b8_128k": dict(batch=8, hq=32, hkv=8, d=128, dtype="bf16", context=131072,
                                 n_streaming=4, n_sink=64, window=1024, page=16, steps=64, seed=2),
    "qwen25_stack_256k": dict(layers=28, batch=1, hq=28, hkv=4, d=128, dtype="bf16", seq=262144,
                              n_streaming=2, n_sink=64, window=2048, decode_steps=128, seed=3),
    "varlen_sweep": dict(n_seq=16, len_lo=4096, len_hi=65536, hq=32, hkv=8, d=128, dtype="bf16",
                         sparsity_pct=[25, 50, 75], windows=[512, 4096], n_sink=64, needles=8,
                         decode_steps=32, seed=4),
    # Projection weights for the head classifier (bf16, PyTorch Linear layout).
    "classify_tiny": dict(layers=2, hq=4, hkv=2, d=64, d_model=256, sparsity=0.5, seed=5),
    "qwen25_classify": dict(layers=28, hq=28, hkv=4, d=128, d_model=3584, sparsity=0.5, seed=6),
    "llama31_classify": dict(layers=32, hq=32, hkv=8, d=128, d_model=4096, sparsity=0.5, seed=7),
}


def gaussian_blocks(shape, seed, purpose, block_dims, scale=1.0, workers=None):
    """N(0, scale^2) float32 array whose sub-arrays over the leading
    `block_dims` indices are drawn independently, key (seed, purpose, *index),
    in a thread pool.  The result depends only on the keys, not on the pool."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    from itertools import product

    out = np.empty(shape, dtype=np.float32)
    lead = shape[:block_dims]
    tail = shape[block_dims:]
    idx = list(product(*[range(n) for n in lead]))
    if workers is None:
        workers = min(16, len(os.sched_getaffinity(0)))

    def fill(i):
        out[i] = gaussian(tail, seed, purpose, *i, scale=scale)

    with ThreadPoolExecutor(max(1, workers)) as ex:
        list(ex.map(fill, idx))
    return out


def gaussian_bthd(B, T, H, D, seed, purpose, scale=1.0):
    """N(0, scale^2) float32 [B, T, H, D] (contiguous), drawn as independent
    [T, D] blocks per (batch, head) keyed (seed, purpose, b, h)."""
    x = gaussian_blocks((B, H, T, D), seed, purpose, 2, scale=scale)
    return np.ascontiguousarray(x.transpose(0, 2, 1, 3))


def qwen_prefill_inputs():
    """Q, K, V (float32, [1, T, H, D]) of the Qwen2.5-7B-shaped 32K prefill
    workload and its head labels / mask sizes."""
    c = CONFIGS["qwen25_prefill_32k"]
    T, hq, hkv, d, seed = c["seq"], c["hq"], c["hkv"], c["d"], c["seed"]
    q = gaussian_bthd(1, T, hq, d, seed, "q")
    k = gaussian_bthd(1, T, hkv, d, seed, "k", scale=c["k_scale"])
    v = gaussian_bthd(1, T, hkv, d, seed, "v")
    return dict(q=q, k=k, v=v, mask=list(c["streaming"]), n_sink=c["n_sink"], window=c["window"])


def llama_decode_inputs(steps=None):
    """The batch-8 x 131072-token decode workload (Llama-3-8B-shaped heads):
    context K/V as [B, Hkv, L, D] float32 blocks (view them as [B, L, Hkv, D]),
    the streaming labels, the page permutation, and the per-step queries and
    new K/V."""
    c = CONFIGS["llama_decode_b8_128k"]
    B, hq, hkv, d, L0, seed = c["batch"], c["hq"], c["hkv"], c["d"], c["context"], c["seed"]
    steps = c["steps"] if steps is None else steps
    mask = choose_streaming(hkv, c["n_streaming"], seed).tolist()
    max_pages = (L0 + steps + 15) // 16
    return dict(
        k_ctx=gaussian_blocks((B, hkv, L0, d), seed, "kctx", 2),
        v_ctx=gaussian_blocks((B, hkv, L0, d), seed, "vctx", 2),
        mask=mask, n_sink=c["n_sink"], window=c["window"], max_pages=max_pages,
        pages=page_permutation(B * max_pages, seed).reshape(B, max_pages),
        q_steps=gaussian((steps, B, hq, d), seed, "qsteps"),
        kv_steps=gaussian((steps, 2, B, 1, hkv, d), seed, "kvsteps"),
    )


def stack_layer_inputs(layer):
    """Q, K, V (float32, [1, T, H, D]) and head labels of one layer of the
    28-layer Qwen2.5-7B-shaped 262144-token stack; every layer is regenerated
    from (seed, layer)."""
    c = CONFIGS["qwen25_stack_256k"]
    T, hq, hkv, d, seed = c["seq"], c["hq"], c["hkv"], c["d"], c["seed"]
    return dict(
        q=gaussian_bthd(1, T, hq, d, seed * 1000 + layer, "q"),
        k=gaussian_bthd(1, T, hkv, d, seed * 1000 + layer, "k"),
        v=gaussian_bthd(1, T, hkv, d, seed * 1000 + layer, "v"),
        mask=choose_streaming(hkv, c["n_streaming"], seed, "streaming", layer).tolist(),
    )


def stack_decode_inputs(layer, steps):
    """Per-step query and new K/V of one stack layer: q [steps, 1, Hq, D],
    kv [steps, 2, 1, 1, Hkv, D]."""
    c = CONFIGS["qwen25_stack_256k"]
    seed = c["seed"] * 1000 + layer
    return (gaussian((steps, 1, c["hq"], c["d"]), seed, "qdec"),
            gaussian((steps, 2, 1, 1, c["hkv"], c["d"]), seed, "kvdec"))


def sweep_sequence(b, length):
    """Q, K, V (float32 [1, len, H, D]) of sequence b of the variable-length
    sweep, with 8 needles planted in K (outside every window of the sweep)."""
    c = CONFIGS["varlen_sweep"]
    hq, hkv, d, seed = c["hq"], c["hkv"], c["d"], c["seed"]
    q = gaussian_bthd(1, length, hq, d, seed * 1000 + b, "q")
    k = gaussian_bthd(1, length, hkv, d, seed * 1000 + b, "k")
    v = gaussian_bthd(1, length, hkv, d, seed * 1000 + b, "v")
    needles = plant_needles(k, [length], c["needles"], c["n_sink"], max(c["windows"]), seed, seq_ids=[b])
    return dict(q=q, k=k, v=v, needles=needles[0])


def projection_weights(name, layer):
    """W_Q [hq * d, d_model] and W_K [hkv * d, d_model] (float32) of one layer
    of a classifier workload.  Every head's d x d_model slice is a Gaussian
    matrix / sqrt(d_model) whose row r is scaled by (r + 1) ** -alpha, with
    alpha ~ U[0.05, 1.2] drawn per (layer, head), so the heads' spectra range
    from nearly flat to steeply decaying.  Keys (seed, "wq"/"wk", layer, head)."""
    c = CONFIGS[name]
    d, dm = c["d"], c["d_model"]
    out = []
    for kind, n in (("wq", c["hq"]), ("wk", c["hkv"])):
        w = gaussian_blocks((n, d, dm), c["seed"] * 1000 + layer, kind, 1, scale=dm ** -0.5)
        alpha = rng(c["seed"], kind + "-alpha", layer).uniform(0.05, 1.2, n)
        w *= (np.arange(1, d + 1)[None, :, None] ** -alpha[:, None, None]).astype(np.float32)
        out.append(w.reshape(n * d, dm))
    return out[0], out[1]
