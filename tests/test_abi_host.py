"""Host-side checks of the C interface: the library loads, exports every symbol
the header declares, and rejects invalid arguments before launching anything.
No GPU is needed: every call here fails validation, which runs on the host."""
import ctypes
import os
import re

import pytest

from paper_2608_06849_amd import aoh as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # 16-byte aligned stand-in for a device pointer; never dereferenced


def _declared():
    src = open(os.path.join(ROOT, "include", "aoh.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(aoh_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert set(names) == set(A.EXPORTS)
    L = A.lib()
    for n in names:
        assert getattr(L, n) is not None


def test_version():
    assert A.aoh_version() == 100


def _t(shape, dtype=A.AOH_BF16, data=FAKE, stride=None):
    d = A.AohTensor()
    d.data = data
    d.dtype = dtype
    d.ndim = len(shape)
    if stride is None:
        stride, acc = [], 1
        for s in reversed(shape):
            stride.insert(0, acc)
            acc *= s
    for i, (s, st) in enumerate(zip(shape, stride)):
        d.shape[i] = s
        d.stride[i] = st
    return d


def _prefill(q, k, v, out, mask=b"\x00\x01", n_sink=4, window=32):
    buf = ctypes.create_string_buffer(mask, len(mask))
    st = A.lib().aoh_prefill(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v),
                             ctypes.cast(buf, ctypes.c_void_p), n_sink, window, ctypes.byref(out), None)
    return st, A.aoh_last_error()


def _good():
    return _t((1, 256, 4, 64)), _t((1, 256, 2, 64)), _t((1, 256, 2, 64)), _t((1, 256, 4, 64))


@pytest.mark.parametrize("case,status,msg", [
    ("null_q_data", A.AOH_ERR_INVALID_ARG, "null data"),
    ("bad_rank", A.AOH_ERR_INVALID_ARG, "dimensions"),
    ("bad_dtype", A.AOH_ERR_UNSUPPORTED, "dtype"),
    ("d96", A.AOH_ERR_UNSUPPORTED, "supported: 64, 128"),
    ("gqa", A.AOH_ERR_UNSUPPORTED, "multiple"),
    ("window0", A.AOH_ERR_INVALID_ARG, "window"),
    ("sink_neg", A.AOH_ERR_INVALID_ARG, "n_sink"),
    ("mask2", A.AOH_ERR_INVALID_ARG, "not 0/1"),
    ("misaligned", A.AOH_ERR_INVALID_ARG, "aligned"),
    ("noncontig", A.AOH_ERR_INVALID_ARG, "contiguous"),
    ("out_shape", A.AOH_ERR_INVALID_ARG, "shape of q"),
    ("kv_mismatch", A.AOH_ERR_INVALID_ARG, "k/v"),
    ("mixed_dtype", A.AOH_ERR_UNSUPPORTED, "dtype"),
])
def test_prefill_validation(case, status, msg):
    q, k, v, out = _good()
    kw = {}
    if case == "null_q_data":
        q.data = None
    elif case == "bad_rank":
        q.ndim = 3
    elif case == "bad_dtype":
        q.dtype = 7
    elif case == "d96":
        q, k, v, out = _t((1, 8, 4, 96)), _t((1, 8, 2, 96)), _t((1, 8, 2, 96)), _t((1, 8, 4, 96))
    elif case == "gqa":
        q, out = _t((1, 256, 3, 64)), _t((1, 256, 3, 64))
    elif case == "window0":
        kw["window"] = 0
    elif case == "sink_neg":
        kw["n_sink"] = -1
    elif case == "mask2":
        kw["mask"] = b"\x00\x02"
    elif case == "misaligned":
        q.data = FAKE + 2
    elif case == "noncontig":
        q = _t((1, 256, 4, 64), stride=(256 * 4 * 128, 4 * 128, 128, 2))
    elif case == "out_shape":
        out = _t((1, 256, 2, 64))
    elif case == "kv_mismatch":
        k = _t((1, 128, 2, 64))
    elif case == "mixed_dtype":
        k = _t((1, 256, 2, 64), dtype=A.AOH_F32)
    st, err = _prefill(q, k, v, out, **kw)
    assert st == status, err
    assert msg in err


@pytest.mark.parametrize("chunk,status,msg", [
    (0, A.AOH_ERR_INVALID_ARG, "chunk"),
    (-3, A.AOH_ERR_INVALID_ARG, "chunk"),
    (64, A.AOH_ERR_INVALID_ARG, "window"),   # chunk valid, window 0 still rejected
])
def test_prefill_chunked_validation(chunk, status, msg):
    q, k, v, out = _good()
    buf = ctypes.create_string_buffer(b"\x00\x01", 2)
    st = A.lib().aoh_prefill_chunked(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v),
                                     ctypes.cast(buf, ctypes.c_void_p), 4, 0 if chunk == 64 else 32, chunk,
                                     ctypes.byref(out), None)
    err = A.aoh_last_error()
    assert st == status, err
    assert msg in err


def test_decode_workspace_size_and_checks():
    L = A.lib()
    n = A.aoh_decode_workspace_bytes(8, 32, 128, 8196, 1088)
    assert n > 0 and n % 4 == 0
    # grows with batch and heads, zero on invalid input
    assert A.aoh_decode_workspace_bytes(8, 32, 128, 8196, 1088) >= A.aoh_decode_workspace_bytes(4, 32, 128, 8196, 1088)
    assert A.aoh_decode_workspace_bytes(0, 32, 128, 16, 64) == 0
    assert A.aoh_decode_workspace_bytes(1, 32, 96, 16, 64) == 0
    # a decode call with a too-small workspace fails before launching
    q, out = _t((2, 8, 128)), _t((2, 8, 128))
    full = A.AohPagedCache(k=FAKE, v=FAKE, block_table=FAKE, num_pages=8, max_pages_per_seq=4, n_heads=1, n_seqs=2)
    ring = A.AohRingCache(k=FAKE, v=FAKE, n_heads=1, capacity=4 + 32, batch=2)
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    need = A.aoh_decode_workspace_bytes(2, 8, 128, 4, 36)
    st = L.aoh_decode(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring), ctypes.cast(mask, ctypes.c_void_p),
                      ctypes.c_void_p(FAKE), 4, 32, ctypes.byref(out), ctypes.c_void_p(FAKE), need - 4, None)
    assert st == A.AOH_ERR_WORKSPACE, A.aoh_last_error()
    # ring capacity must equal n_sink + window
    st = L.aoh_decode(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring), ctypes.cast(mask, ctypes.c_void_p),
                      ctypes.c_void_p(FAKE), 4, 33, ctypes.byref(out), ctypes.c_void_p(FAKE), need, None)
    assert st == A.AOH_ERR_INVALID_ARG and "capacity" in A.aoh_last_error()
    # head counts of the caches must match the labels
    full.n_heads = 2
    st = L.aoh_decode(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring), ctypes.cast(mask, ctypes.c_void_p),
                      ctypes.c_void_p(FAKE), 4, 32, ctypes.byref(out), ctypes.c_void_p(FAKE), need, None)
    assert st != A.AOH_OK
    # group size above 16 is not supported by the bf16 decode kernel
    q2, out2 = _t((2, 34, 128)), _t((2, 34, 128))
    full.n_heads = 1
    st = L.aoh_decode(ctypes.byref(q2), ctypes.byref(full), ctypes.byref(ring), ctypes.cast(mask, ctypes.c_void_p),
                      ctypes.c_void_p(FAKE), 4, 32, ctypes.byref(out2), ctypes.c_void_p(FAKE), 1 << 30, None)
    assert st == A.AOH_ERR_UNSUPPORTED and "16" in A.aoh_last_error()


def test_decode_step_validation():
    # the fused step validates its new-token tensors on top of the decode checks
    L = A.lib()
    q, out = _t((2, 8, 128)), _t((2, 8, 128))
    full = A.AohPagedCache(k=FAKE, v=FAKE, block_table=FAKE, num_pages=8, max_pages_per_seq=4, n_heads=1, n_seqs=2)
    ring = A.AohRingCache(k=FAKE, v=FAKE, n_heads=1, capacity=4 + 32, batch=2)
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    need = A.aoh_decode_workspace_bytes(2, 8, 128, 4, 36)

    def step(kn, vn, ws=need):
        st = L.aoh_decode_step(ctypes.byref(q), ctypes.byref(kn) if kn is not None else None,
                               ctypes.byref(vn) if vn is not None else None, ctypes.byref(full), ctypes.byref(ring),
                               ctypes.cast(mask, ctypes.c_void_p), ctypes.c_void_p(FAKE), 4, 32, ctypes.byref(out),
                               ctypes.c_void_p(FAKE), ws, None)
        return st, A.aoh_last_error()

    good = _t((2, 2, 128))
    st, err = step(None, good)
    assert st == A.AOH_ERR_INVALID_ARG and "k_new" in err
    st, err = step(good, None)
    assert st == A.AOH_ERR_INVALID_ARG and "v_new" in err
    st, err = step(_t((2, 1, 2, 128)), _t((2, 1, 2, 128)))        # [B, 1, Hkv, D]: one dimension too many
    assert st == A.AOH_ERR_INVALID_ARG and "dimensions" in err
    st, err = step(_t((2, 3, 128)), _t((2, 3, 128)))              # Hkv 3, the caches hold 2 KV heads
    assert st == A.AOH_ERR_INVALID_ARG and "k_new / v_new" in err
    st, err = step(_t((2, 2, 128), A.AOH_F32), _t((2, 2, 128), A.AOH_F32))  # dtype of q required
    assert st == A.AOH_ERR_UNSUPPORTED and "k_new" in err
    st, err = step(good, _t((2, 2, 128), stride=[256, 128, 2]))   # last dimension not contiguous
    assert st == A.AOH_ERR_INVALID_ARG and "contiguous" in err
    st, err = step(good, good, need - 4)                          # workspace as for aoh_decode
    assert st == A.AOH_ERR_WORKSPACE, err


def test_append_validation():
    L = A.lib()
    k, v = _t((2, 5, 2, 128)), _t((2, 5, 2, 128))
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    ring = A.AohRingCache(k=FAKE, v=FAKE, n_heads=1, capacity=36, batch=2)
    # retrieval head present but no paged cache
    st = L.aoh_kv_append(ctypes.byref(k), ctypes.byref(v), ctypes.cast(mask, ctypes.c_void_p),
                         ctypes.c_void_p(FAKE), None, ctypes.byref(ring), 4, 32, None)
    assert st == A.AOH_ERR_INVALID_ARG and "kv_full" in A.aoh_last_error()
    # null start positions
    full = A.AohPagedCache(k=FAKE, v=FAKE, block_table=FAKE, num_pages=8, max_pages_per_seq=4, n_heads=1, n_seqs=2)
    st = L.aoh_kv_append(ctypes.byref(k), ctypes.byref(v), ctypes.cast(mask, ctypes.c_void_p),
                         None, ctypes.byref(full), ctypes.byref(ring), 4, 32, None)
    assert st == A.AOH_ERR_INVALID_ARG and "start_pos" in A.aoh_last_error()


def _classify(wq, wk, d_head=64, k=1, ws=FAKE, ws_bytes=1 << 40, outs=(FAKE, FAKE, FAKE)):
    st = A.lib().aoh_classify(ctypes.byref(wq), ctypes.byref(wk), d_head, k,
                              *[ctypes.c_void_p(o) for o in outs], ctypes.c_void_p(ws), ws_bytes, None)
    return st, A.aoh_last_error()


@pytest.mark.parametrize("case,status,msg", [
    ("f32", A.AOH_ERR_UNSUPPORTED, "dtype"),
    ("d96", A.AOH_ERR_UNSUPPORTED, "d_head"),
    ("rows", A.AOH_ERR_INVALID_ARG, "multiple of d_head"),
    ("gqa", A.AOH_ERR_UNSUPPORTED, "multiple"),
    ("dmodel", A.AOH_ERR_UNSUPPORTED, "multiple of 64"),
    ("layers", A.AOH_ERR_INVALID_ARG, "same layers"),
    ("k_big", A.AOH_ERR_INVALID_ARG, "n_retrieval"),
    ("k_neg", A.AOH_ERR_INVALID_ARG, "n_retrieval"),
    ("no_ws", A.AOH_ERR_WORKSPACE, "null"),
    ("small_ws", A.AOH_ERR_WORKSPACE, "needed"),
    ("null_out", A.AOH_ERR_INVALID_ARG, "null output"),
])
def test_classify_validation(case, status, msg):
    wq, wk = _t((2, 4 * 64, 256)), _t((2, 2 * 64, 256))
    kw = {}
    if case == "f32":
        wq = _t((2, 4 * 64, 256), dtype=A.AOH_F32)
    elif case == "d96":
        kw["d_head"] = 96
    elif case == "rows":
        wq = _t((2, 4 * 64 + 8, 256))
    elif case == "gqa":
        wq = _t((2, 3 * 64, 256))
    elif case == "dmodel":
        wq, wk = _t((2, 4 * 64, 200)), _t((2, 2 * 64, 200))
    elif case == "layers":
        wk = _t((3, 2 * 64, 256))
    elif case == "k_big":
        kw["k"] = 3
    elif case == "k_neg":
        kw["k"] = -1
    elif case == "no_ws":
        kw["ws"] = 0
    elif case == "small_ws":
        kw["ws_bytes"] = A.aoh_classify_workspace_bytes(2, 4, 2, 64) - 1
    elif case == "null_out":
        kw["outs"] = (FAKE, 0, FAKE)
    st, err = _classify(wq, wk, **kw)
    assert st == status, err
    assert msg in err


def test_classify_workspace_and_group_count():
    assert A.aoh_classify_workspace_bytes(28, 28, 4, 128) == 28 * 32 * 128 * 128 * 4 + 28 * 4 * 128 * 128 * 8
    assert A.aoh_classify_workspace_bytes(1, 4, 2, 96) == 0
    from oracle import accounting as ACC
    for g in (1, 2, 4, 8, 10, 28, 64):
        for s in (0.0, 0.1, 0.25, 0.3, 0.5, 0.7, 0.75, 0.9, 1.0):
            assert A.aoh_retrieval_group_count(g, s) == ACC.n_retrieval_groups(g, s), (g, s)
    assert A.lib().aoh_retrieval_group_count(4, 1.5) == -1


def test_prefill_append_validation():
    q, k, v, out = _good()
    buf = ctypes.create_string_buffer(b"\x00\x01", 2)
    fn = A.lib().aoh_prefill_append
    st = fn(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v), ctypes.cast(buf, ctypes.c_void_p), 4, 32, -1,
            None, None, ctypes.byref(out), None)
    assert st == A.AOH_ERR_INVALID_ARG and "chunk" in A.aoh_last_error()
    st = fn(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v), ctypes.cast(buf, ctypes.c_void_p), 4, 32, 0,
            None, None, ctypes.byref(out), None)
    assert st == A.AOH_ERR_INVALID_ARG and "kv_full is null" in A.aoh_last_error()
    full = A.AohPagedCache(FAKE, FAKE, FAKE, 10, 20, 1, 1)
    st = fn(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v), ctypes.cast(buf, ctypes.c_void_p), 4, 32, 0,
            ctypes.byref(full), None, ctypes.byref(out), None)
    assert st == A.AOH_ERR_INVALID_ARG and "kv_ring is null" in A.aoh_last_error()
    ring = A.AohRingCache(FAKE, FAKE, 1, 35, 1)
    st = fn(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v), ctypes.cast(buf, ctypes.c_void_p), 4, 32, 0,
            ctypes.byref(full), ctypes.byref(ring), ctypes.byref(out), None)
    assert st == A.AOH_ERR_INVALID_ARG and "capacity" in A.aoh_last_error()


# Checks that depend on the whole request run before the first launch: with
# fake device pointers and no GPU, a launch would return AOH_ERR_HIP, so a
# validation status here also shows that nothing was enqueued.

def test_cache_batch_must_cover_the_call():
    L = A.lib()
    q, out = _t((3, 8, 128)), _t((3, 8, 128))
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    need = A.aoh_decode_workspace_bytes(3, 8, 128, 4, 36)

    def dec(full, ring):
        st = L.aoh_decode(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring), ctypes.cast(mask, ctypes.c_void_p),
                          ctypes.c_void_p(FAKE), 4, 32, ctypes.byref(out), ctypes.c_void_p(FAKE), need, None)
        return st, A.aoh_last_error()

    full = A.AohPagedCache(k=FAKE, v=FAKE, block_table=FAKE, num_pages=8, max_pages_per_seq=4, n_heads=1, n_seqs=2)
    ring = A.AohRingCache(k=FAKE, v=FAKE, n_heads=1, capacity=36, batch=3)
    st, err = dec(full, ring)
    assert st == A.AOH_ERR_INVALID_ARG and "n_seqs" in err
    full.n_seqs = 3
    ring.batch = 2
    st, err = dec(full, ring)
    assert st == A.AOH_ERR_INVALID_ARG and "kv_ring.batch" in err
    # the same rule for an append of 3 sequences
    k, v = _t((3, 5, 2, 128)), _t((3, 5, 2, 128))
    st = L.aoh_kv_append(ctypes.byref(k), ctypes.byref(v), ctypes.cast(mask, ctypes.c_void_p),
                         ctypes.c_void_p(FAKE), ctypes.byref(full), ctypes.byref(ring), 4, 32, None)
    assert st == A.AOH_ERR_INVALID_ARG and "kv_ring.batch" in A.aoh_last_error()
    # and for a prefill that fills the caches
    q4, k4, v4, o4 = _t((3, 64, 4, 128)), _t((3, 64, 2, 128)), _t((3, 64, 2, 128)), _t((3, 64, 4, 128))
    st = L.aoh_prefill_append(ctypes.byref(q4), ctypes.byref(k4), ctypes.byref(v4), ctypes.cast(mask, ctypes.c_void_p),
                              4, 32, 0, ctypes.byref(full), ctypes.byref(ring), ctypes.byref(o4), None)
    assert st == A.AOH_ERR_INVALID_ARG and "kv_ring.batch" in A.aoh_last_error()


def test_packed_fp32_append_rejected_before_launch():
    q, k, v, out = _t((300, 4, 64), A.AOH_F32), _t((300, 2, 64), A.AOH_F32), _t((300, 2, 64), A.AOH_F32), \
        _t((300, 4, 64), A.AOH_F32)
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    full = A.AohPagedCache(FAKE, FAKE, FAKE, 64, 20, 1, 2)
    ring = A.AohRingCache(FAKE, FAKE, 1, 36, 2)
    st = A.lib().aoh_prefill_varlen(ctypes.byref(q), ctypes.byref(k), ctypes.byref(v), ctypes.c_void_p(FAKE), 2, 200,
                                    ctypes.cast(mask, ctypes.c_void_p), 4, 32, 0, ctypes.byref(full),
                                    ctypes.byref(ring), ctypes.byref(out), None)
    assert st == A.AOH_ERR_UNSUPPORTED and "needs bf16" in A.aoh_last_error()


def test_anchor_large_batch_rejected_before_launch():
    B = 65536
    q, out = _t((B, 8, 128)), _t((B, 8, 128))
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    full = A.AohPagedCache(FAKE, FAKE, FAKE, 8, 4, 1, B)
    ring = A.AohRingCache(FAKE, FAKE, 1, 36, B)
    st = A.lib().aoh_decode_anchor(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring),
                                   ctypes.cast(mask, ctypes.c_void_p), ctypes.c_void_p(FAKE), 4, 32, 16,
                                   ctypes.c_void_p(FAKE), ctypes.byref(out), ctypes.c_void_p(FAKE), 1 << 62, None)
    assert st == A.AOH_ERR_UNSUPPORTED and "batch" in A.aoh_last_error()


def test_noalloc_step_rejects_a_workspace_beyond_the_static_area():
    # batch 8192 x 16 query heads of width 128: the split partials need more
    # than the 64 MiB static area (checked before any GPU call)
    B, Hq = 8192, 16
    q, out, kn, vn = _t((B, Hq, 128)), _t((B, Hq, 128)), _t((B, 2, 128)), _t((B, 2, 128))
    full = A.AohPagedCache(FAKE, FAKE, FAKE, 1 << 20, 1 << 14, 1, B)
    ring = A.AohRingCache(FAKE, FAKE, 1, 36, B)
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    assert A.aoh_decode_workspace_bytes(B, Hq, 128, 1 << 14, 36) > 64 << 20
    st = A.lib().aoh_decode_step_noalloc(ctypes.byref(q), ctypes.byref(kn), ctypes.byref(vn), ctypes.byref(full),
                                         ctypes.byref(ring), ctypes.cast(mask, ctypes.c_void_p), ctypes.c_void_p(FAKE),
                                         4, 32, ctypes.byref(out), None)
    assert st == A.AOH_ERR_UNSUPPORTED and "static scratch" in A.aoh_last_error()


def test_token_major_v_pages_only_for_append_and_reuse():
    # a cache with token-major V pages is rejected, before any launch, by the
    # calls that read or write dimension-major pages; an invalid flag is an
    # argument error everywhere
    L = A.lib()
    q, out = _t((2, 8, 128)), _t((2, 8, 128))
    mask = ctypes.create_string_buffer(b"\x00\x01", 2)
    full = A.AohPagedCache(k=FAKE, v=FAKE, block_table=FAKE, num_pages=8, max_pages_per_seq=4, n_heads=1, n_seqs=2,
                           v_token_major=1)
    ring = A.AohRingCache(k=FAKE, v=FAKE, n_heads=1, capacity=36, batch=2)
    need = A.aoh_decode_workspace_bytes(2, 8, 128, 4, 36)
    m = ctypes.cast(mask, ctypes.c_void_p)
    st = L.aoh_decode(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring), m, ctypes.c_void_p(FAKE), 4, 32,
                      ctypes.byref(out), ctypes.c_void_p(FAKE), need, None)
    assert st == A.AOH_ERR_UNSUPPORTED and "aoh_decode needs dimension-major" in A.aoh_last_error()
    kn = _t((2, 2, 128))
    st = L.aoh_decode_step(ctypes.byref(q), ctypes.byref(kn), ctypes.byref(kn), ctypes.byref(full),
                           ctypes.byref(ring), m, ctypes.c_void_p(FAKE), 4, 32, ctypes.byref(out),
                           ctypes.c_void_p(FAKE), need, None)
    assert st == A.AOH_ERR_UNSUPPORTED and "aoh_decode_step" in A.aoh_last_error()
    st = L.aoh_decode_anchor(ctypes.byref(q), ctypes.byref(full), ctypes.byref(ring), m, ctypes.c_void_p(FAKE), 4,
                             32, 16, ctypes.c_void_p(FAKE), ctypes.byref(out), ctypes.c_void_p(FAKE), 1 << 40, None)
    assert st == A.AOH_ERR_UNSUPPORTED and "aoh_decode_anchor" in A.aoh_last_error()
    q4, k4, v4, o4 = _t((2, 64, 4, 128)), _t((2, 64, 2, 128)), _t((2, 64, 2, 128)), _t((2, 64, 4, 128))
    st = L.aoh_prefill_append(ctypes.byref(q4), ctypes.byref(k4), ctypes.byref(v4), m, 4, 32, 0, ctypes.byref(full),
                              ctypes.byref(ring), ctypes.byref(o4), None)
    assert st == A.AOH_ERR_UNSUPPORTED and "prefill" in A.aoh_last_error()
    full.v_token_major = 2
    k5, v5 = _t((2, 5, 2, 128)), _t((2, 5, 2, 128))
    st = L.aoh_kv_append(ctypes.byref(k5), ctypes.byref(v5), m, ctypes.c_void_p(FAKE), ctypes.byref(full),
                         ctypes.byref(ring), 4, 32, None)
    assert st == A.AOH_ERR_INVALID_ARG and "v_token_major" in A.aoh_last_error()
