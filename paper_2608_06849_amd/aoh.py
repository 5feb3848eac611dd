"""Thin ctypes binding of libaoh (include/aoh.h).

Every function here only marshals arguments: torch tensors become aoh_tensor
descriptors (pointer, dtype, shape, strides) and the call goes to the C entry
point of the same name, on the current HIP stream.  All arithmetic runs in the
library's HIP kernels.  If libaoh.so is missing or cannot be loaded, every call
raises: there is no fallback path.

Cache helpers allocate the two cache layouts with torch (the library itself
never allocates device memory).
"""
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libaoh.so")

AOH_OK, AOH_ERR_INVALID_ARG, AOH_ERR_UNSUPPORTED, AOH_ERR_HIP, AOH_ERR_WORKSPACE = range(5)
AOH_BF16, AOH_F32 = 0, 1
PAGE_TOKENS = 16

_DTYPES = {torch.bfloat16: AOH_BF16, torch.float32: AOH_F32}


class AohError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"aoh status {status}: {message}")
        self.status = status


class AohTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 4), ("stride", ctypes.c_int64 * 4)]


class AohPagedCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("block_table", ctypes.c_void_p),
                ("num_pages", ctypes.c_int64), ("max_pages_per_seq", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_seqs", ctypes.c_int32), ("v_token_major", ctypes.c_int32)]


class AohRingCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("n_heads", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("batch", ctypes.c_int32)]


_lib = None

EXPORTS = ("aoh_prefill", "aoh_prefill_chunked", "aoh_prefill_append", "aoh_prefill_varlen", "aoh_kv_append", "aoh_decode_workspace_bytes", "aoh_decode", "aoh_decode_step",
           "aoh_decode_step_noalloc",
           "aoh_classify_workspace_bytes", "aoh_classify", "aoh_retrieval_group_count",
           "aoh_head_mapping_workspace_bytes", "aoh_head_mapping", "aoh_decode_anchor_workspace_bytes",
           "aoh_decode_anchor", "aoh_decode_reuse_workspace_bytes", "aoh_decode_reuse",
           "aoh_last_error", "aoh_version")


def lib():
    """Load libaoh.so once; raise if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_06849_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.aoh_prefill.argtypes = [P(AohTensor), P(AohTensor), P(AohTensor), ctypes.c_void_p,
                                  ctypes.c_int32, ctypes.c_int32, P(AohTensor), ctypes.c_void_p]
        L.aoh_prefill.restype = ctypes.c_int
        L.aoh_prefill_chunked.argtypes = [P(AohTensor), P(AohTensor), P(AohTensor), ctypes.c_void_p,
                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P(AohTensor),
                                          ctypes.c_void_p]
        L.aoh_prefill_chunked.restype = ctypes.c_int
        L.aoh_prefill_append.argtypes = [P(AohTensor), P(AohTensor), P(AohTensor), ctypes.c_void_p,
                                         ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P(AohPagedCache),
                                         P(AohRingCache), P(AohTensor), ctypes.c_void_p]
        L.aoh_prefill_append.restype = ctypes.c_int
        L.aoh_prefill_varlen.argtypes = [P(AohTensor), P(AohTensor), P(AohTensor), ctypes.c_void_p, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, P(AohPagedCache), P(AohRingCache), P(AohTensor),
                                         ctypes.c_void_p]
        L.aoh_prefill_varlen.restype = ctypes.c_int
        L.aoh_kv_append.argtypes = [P(AohTensor), P(AohTensor), ctypes.c_void_p, ctypes.c_void_p,
                                    P(AohPagedCache), P(AohRingCache), ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_void_p]
        L.aoh_kv_append.restype = ctypes.c_int
        L.aoh_decode_workspace_bytes.argtypes = [ctypes.c_int32] * 5
        L.aoh_decode_workspace_bytes.restype = ctypes.c_size_t
        L.aoh_decode.argtypes = [P(AohTensor), P(AohPagedCache), P(AohRingCache), ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, P(AohTensor),
                                 ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.aoh_decode.restype = ctypes.c_int
        L.aoh_decode_step.argtypes = [P(AohTensor), P(AohTensor), P(AohTensor), P(AohPagedCache), P(AohRingCache),
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                      P(AohTensor), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.aoh_decode_step.restype = ctypes.c_int
        L.aoh_decode_step_noalloc.argtypes = [P(AohTensor), P(AohTensor), P(AohTensor), P(AohPagedCache),
                                              P(AohRingCache), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                              ctypes.c_int32, P(AohTensor), ctypes.c_void_p]
        L.aoh_decode_step_noalloc.restype = ctypes.c_int
        L.aoh_classify_workspace_bytes.argtypes = [ctypes.c_int32] * 4
        L.aoh_classify_workspace_bytes.restype = ctypes.c_size_t
        L.aoh_classify.argtypes = [P(AohTensor), P(AohTensor), ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_size_t, ctypes.c_void_p]
        L.aoh_classify.restype = ctypes.c_int
        L.aoh_retrieval_group_count.argtypes = [ctypes.c_int32, ctypes.c_double]
        L.aoh_retrieval_group_count.restype = ctypes.c_int32
        L.aoh_head_mapping_workspace_bytes.argtypes = [ctypes.c_int32] * 3
        L.aoh_head_mapping_workspace_bytes.restype = ctypes.c_size_t
        L.aoh_head_mapping.argtypes = [P(AohTensor)] * 4 + [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                            ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.aoh_head_mapping.restype = ctypes.c_int
        L.aoh_decode_anchor_workspace_bytes.argtypes = [ctypes.c_int32] * 5
        L.aoh_decode_anchor_workspace_bytes.restype = ctypes.c_size_t
        L.aoh_decode_anchor.argtypes = [P(AohTensor), P(AohPagedCache), P(AohRingCache), ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, P(AohTensor), ctypes.c_void_p, ctypes.c_size_t,
                                        ctypes.c_void_p]
        L.aoh_decode_anchor.restype = ctypes.c_int
        L.aoh_decode_reuse_workspace_bytes.argtypes = [ctypes.c_int32] * 5
        L.aoh_decode_reuse_workspace_bytes.restype = ctypes.c_size_t
        L.aoh_decode_reuse.argtypes = [P(AohTensor), P(AohPagedCache), P(AohRingCache), ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, P(AohTensor),
                                       ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.aoh_decode_reuse.restype = ctypes.c_int
        L.aoh_last_error.argtypes = []
        L.aoh_last_error.restype = ctypes.c_char_p
        L.aoh_version.argtypes = []
        L.aoh_version.restype = ctypes.c_int32
        _lib = L
    return _lib


def _check(status):
    if status != AOH_OK:
        raise AohError(status, lib().aoh_last_error().decode())


def tensor_desc(t):
    """aoh_tensor descriptor of a torch tensor (no copy)."""
    if t.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {t.dtype}")
    if t.dim() > 4:
        raise ValueError("at most 4 dimensions")
    d = AohTensor()
    d.data = t.data_ptr()
    d.dtype = _DTYPES[t.dtype]
    d.ndim = t.dim()
    for i in range(t.dim()):
        d.shape[i] = t.shape[i]
        d.stride[i] = t.stride(i)
    return d


class _Mask:
    """Host byte array of head labels, kept alive for the duration of a call."""

    def __init__(self, head_is_streaming):
        m = bytes(int(x) for x in head_is_streaming)
        self.buf = ctypes.create_string_buffer(m, max(len(m), 1))

    @property
    def ptr(self):
        return ctypes.cast(self.buf, ctypes.c_void_p)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


# ----------------------------------------------------------------------------- caches

class PagedCache:
    """Retrieval-head cache: 16-token pages, K token-major and V dimension-major
    inside a page (or token-major with v_token_major, for reuse layers), and a
    per-sequence block table (device int32)."""

    def __init__(self, k, v, block_table, v_token_major=False):
        self.k, self.v, self.block_table = k, v, block_table
        self.v_token_major = bool(v_token_major)

    @classmethod
    def allocate(cls, num_pages, n_heads, d, dtype, block_table, device="cuda", v_token_major=False):
        k = torch.empty((num_pages, n_heads, PAGE_TOKENS, d), dtype=dtype, device=device)
        vshape = (num_pages, n_heads, PAGE_TOKENS, d) if v_token_major else (num_pages, n_heads, d, PAGE_TOKENS)
        v = torch.empty(vshape, dtype=dtype, device=device)
        return cls(k, v, block_table.to(device=device, dtype=torch.int32).contiguous(), v_token_major)

    def rows(self, b0, b1):
        """The same pages with block-table rows b0 .. b1-1 (sequences b0 .. b1-1)."""
        return PagedCache(self.k, self.v, self.block_table[b0:b1], self.v_token_major)

    def desc(self):
        c = AohPagedCache()
        c.k, c.v = self.k.data_ptr(), self.v.data_ptr()
        c.block_table = self.block_table.data_ptr()
        c.num_pages = self.k.shape[0]
        c.max_pages_per_seq = self.block_table.shape[1]
        c.n_heads = self.k.shape[1]
        c.n_seqs = self.block_table.shape[0]
        c.v_token_major = int(self.v_token_major)
        return c


class RingCache:
    """Streaming-head cache: n_sink + window slots per (sequence, head), padded
    to whole 16-slot blocks; K token-major and V dimension-major per block."""

    def __init__(self, k, v, capacity):
        self.k, self.v, self.capacity = k, v, capacity

    @classmethod
    def allocate(cls, batch, n_heads, n_sink, window, d, dtype, device="cuda"):
        cap = n_sink + window
        nblk = (cap + PAGE_TOKENS - 1) // PAGE_TOKENS
        k = torch.empty((batch, n_heads, nblk, PAGE_TOKENS, d), dtype=dtype, device=device)
        v = torch.empty((batch, n_heads, nblk, d, PAGE_TOKENS), dtype=dtype, device=device)
        return cls(k, v, cap)

    def desc(self):
        c = AohRingCache()
        c.k, c.v = self.k.data_ptr(), self.v.data_ptr()
        c.n_heads = self.k.shape[1]
        c.capacity = self.capacity
        c.batch = self.k.shape[0]
        return c


# ----------------------------------------------------------------------------- entry points

def aoh_prefill(q, k, v, head_is_streaming, n_sink, window, out=None, stream=None):
    """out[B,T,Hq,D] = head-mixed causal attention (see aoh.h)."""
    if out is None:
        out = torch.empty_like(q)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    m = _Mask(head_is_streaming)
    _check(lib().aoh_prefill(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), m.ptr,
                             n_sink, window, ctypes.byref(od), _stream(stream)))
    return out


def aoh_prefill_chunked(q, k, v, head_is_streaming, n_sink, window, chunk, out=None, stream=None):
    """Prefill with chunk eviction of `chunk` tokens for streaming heads (see aoh.h)."""
    if out is None:
        out = torch.empty_like(q)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    m = _Mask(head_is_streaming)
    _check(lib().aoh_prefill_chunked(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), m.ptr,
                                     n_sink, window, chunk, ctypes.byref(od), _stream(stream)))
    return out


def aoh_prefill_append(q, k, v, head_is_streaming, n_sink, window, kv_full, kv_ring, chunk=0, out=None,
                       stream=None):
    """Prefill of a new prompt that also writes its K/V into the caches (see aoh.h)."""
    if out is None:
        out = torch.empty_like(q)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    m = _Mask(head_is_streaming)
    _check(lib().aoh_prefill_append(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), m.ptr, n_sink, window,
                                    chunk, ctypes.byref(fd) if fd else None, ctypes.byref(rd) if rd else None,
                                    ctypes.byref(od), _stream(stream)))
    return out


def aoh_prefill_varlen(q, k, v, cu_seqlens, max_seqlen, head_is_streaming, n_sink, window, chunk=0, kv_full=None,
                       kv_ring=None, out=None, stream=None):
    """Packed variable-length prefill: q [total, Hq, D], k/v [total, Hkv, D], cu_seqlens device int32 [B + 1]."""
    if out is None:
        out = torch.empty_like(q)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    m = _Mask(head_is_streaming)
    _check(lib().aoh_prefill_varlen(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), _ptr(cu_seqlens),
                                    cu_seqlens.numel() - 1, max_seqlen, m.ptr, n_sink, window, chunk,
                                    ctypes.byref(fd) if fd else None, ctypes.byref(rd) if rd else None,
                                    ctypes.byref(od), _stream(stream)))
    return out


def aoh_kv_append(k_new, v_new, head_is_streaming, start_pos, kv_full, kv_ring, n_sink, window,
                  stream=None):
    """Append k_new/v_new [B,n_new,Hkv,D] at positions start_pos[b] + t."""
    kd, vd = tensor_desc(k_new), tensor_desc(v_new)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    m = _Mask(head_is_streaming)
    _check(lib().aoh_kv_append(ctypes.byref(kd), ctypes.byref(vd), m.ptr,
                               _ptr(start_pos), ctypes.byref(fd) if fd else None,
                               ctypes.byref(rd) if rd else None, n_sink, window, _stream(stream)))


def aoh_decode_workspace_bytes(batch, n_q_heads, d_head, max_pages_per_seq, ring_capacity):
    return int(lib().aoh_decode_workspace_bytes(batch, n_q_heads, d_head, max_pages_per_seq,
                                                ring_capacity))


def aoh_decode(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out=None,
               workspace=None, stream=None):
    """One decode step: out[B,Hq,D] for queries at positions lens[b]-1."""
    if out is None:
        out = torch.empty_like(q)
    qd, od = tensor_desc(q), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) \
        if workspace is not None else (0, 0)
    m = _Mask(head_is_streaming)
    _check(lib().aoh_decode(ctypes.byref(qd), ctypes.byref(fd) if fd else None,
                            ctypes.byref(rd) if rd else None, m.ptr,
                            _ptr(lens), n_sink, window, ctypes.byref(od), ctypes.c_void_p(ws_ptr),
                            ws_bytes, _stream(stream)))
    return out


def aoh_decode_step(q, k_new, v_new, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out=None,
                    workspace=None, stream=None):
    """Append the token at position lens[b]-1 (k_new, v_new [B,Hkv,D]) and decode
    with it in one call: the same result and caches as aoh_kv_append + aoh_decode."""
    if out is None:
        out = torch.empty_like(q)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k_new), tensor_desc(v_new), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) \
        if workspace is not None else (0, 0)
    m = _Mask(head_is_streaming)
    _check(lib().aoh_decode_step(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd),
                                 ctypes.byref(fd) if fd else None, ctypes.byref(rd) if rd else None, m.ptr,
                                 _ptr(lens), n_sink, window, ctypes.byref(od), ctypes.c_void_p(ws_ptr),
                                 ws_bytes, _stream(stream)))
    return out


def aoh_decode_step_noalloc(q, k_new, v_new, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out=None,
                            stream=None):
    """aoh_decode_step without a workspace: the library's static scratch area
    holds the split partials (calls on one GPU must not overlap)."""
    if out is None:
        out = torch.empty_like(q)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k_new), tensor_desc(v_new), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    m = _Mask(head_is_streaming)
    _check(lib().aoh_decode_step_noalloc(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd),
                                         ctypes.byref(fd) if fd else None, ctypes.byref(rd) if rd else None, m.ptr,
                                         _ptr(lens), n_sink, window, ctypes.byref(od), _stream(stream)))
    return out


def aoh_classify_workspace_bytes(n_layers, n_q_heads, n_kv_heads, d_head):
    return int(lib().aoh_classify_workspace_bytes(n_layers, n_q_heads, n_kv_heads, d_head))


def aoh_retrieval_group_count(n_kv_heads, sparsity):
    """Retrieval groups per layer for a target sparsity s (the library's ceil((1 - s) G))."""
    k = int(lib().aoh_retrieval_group_count(n_kv_heads, float(sparsity)))
    if k < 0:
        raise AohError(AOH_ERR_INVALID_ARG, aoh_last_error())
    return k


def aoh_classify(w_q, w_k, d_head, n_retrieval, head_rank=None, group_score=None, head_is_streaming=None,
                 workspace=None, stream=None):
    """Head classification of every layer: w_q [L, Hq*d_head, d_model], w_k
    [L, Hkv*d_head, d_model] (bf16, device).  Returns (head_rank [L, Hq] f64,
    group_score [L, Hkv] f64, head_is_streaming [L, Hkv] u8), device tensors."""
    L, hq, hkv = w_q.shape[0], w_q.shape[1] // d_head, w_k.shape[1] // d_head
    dev = w_q.device
    if head_rank is None:
        head_rank = torch.empty((L, hq), dtype=torch.float64, device=dev)
    if group_score is None:
        group_score = torch.empty((L, hkv), dtype=torch.float64, device=dev)
    if head_is_streaming is None:
        head_is_streaming = torch.empty((L, hkv), dtype=torch.uint8, device=dev)
    if workspace is None:
        n = aoh_classify_workspace_bytes(L, hq, hkv, d_head)
        workspace = torch.empty(max(n, 16), dtype=torch.uint8, device=dev)
    qd, kd = tensor_desc(w_q), tensor_desc(w_k)
    _check(lib().aoh_classify(ctypes.byref(qd), ctypes.byref(kd), d_head, n_retrieval, _ptr(head_rank),
                              _ptr(group_score), _ptr(head_is_streaming), _ptr(workspace),
                              workspace.numel() * workspace.element_size(), _stream(stream)))
    return head_rank, group_score, head_is_streaming


def _ws(workspace, n_bytes, device):
    if workspace is None:
        workspace = torch.empty(max(n_bytes, 16), dtype=torch.uint8, device=device)
    return workspace, workspace.numel() * workspace.element_size()


def aoh_head_mapping_workspace_bytes(n_q_heads, n_kv_heads, d_head):
    return int(lib().aoh_head_mapping_workspace_bytes(n_q_heads, n_kv_heads, d_head))


def aoh_head_mapping(w_q_anchor, w_k_anchor, w_q_reuse, w_k_reuse, d_head, anchor_is_streaming,
                     reuse_is_streaming, workspace=None, stream=None):
    """Cross-layer head/group similarity and the group mapping (see aoh.h).
    Returns device tensors (head_sim [Hq, Hq] f64, group_sim [Hkv, Hkv] f64, mapping [Hkv] i32)."""
    hq, hkv = w_q_anchor.shape[0] // d_head, w_k_anchor.shape[0] // d_head
    dev = w_q_anchor.device
    head_sim = torch.empty((hq, hq), dtype=torch.float64, device=dev)
    group_sim = torch.empty((hkv, hkv), dtype=torch.float64, device=dev)
    mapping = torch.empty(hkv, dtype=torch.int32, device=dev)
    workspace, wsb = _ws(workspace, aoh_head_mapping_workspace_bytes(hq, hkv, d_head), dev)
    ds = [tensor_desc(t) for t in (w_q_anchor, w_k_anchor, w_q_reuse, w_k_reuse)]
    ma, mr = _Mask(anchor_is_streaming), _Mask(reuse_is_streaming)
    _check(lib().aoh_head_mapping(*[ctypes.byref(d) for d in ds], d_head, ma.ptr, mr.ptr, _ptr(head_sim),
                                  _ptr(group_sim), _ptr(mapping), _ptr(workspace), wsb, _stream(stream)))
    return head_sim, group_sim, mapping


def aoh_decode_anchor_workspace_bytes(batch, n_q_heads, d_head, max_pages_per_seq, ring_capacity):
    return int(lib().aoh_decode_anchor_workspace_bytes(batch, n_q_heads, d_head, max_pages_per_seq, ring_capacity))


def aoh_decode_anchor(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, top_k, indices=None, out=None,
                      workspace=None, stream=None):
    """Anchor-layer decode step; returns (out, indices [B, n_retrieval_groups, top_k] int32)."""
    if out is None:
        out = torch.empty_like(q)
    n_ret = sum(1 for x in head_is_streaming if not x)
    if indices is None:
        indices = torch.empty((q.shape[0], max(n_ret, 1), top_k), dtype=torch.int32, device=q.device)
    max_pages = kv_full.block_table.shape[1] if kv_full is not None else 1
    cap = kv_ring.capacity if kv_ring is not None else n_sink + window
    workspace, wsb = _ws(workspace, aoh_decode_anchor_workspace_bytes(q.shape[0], q.shape[1], q.shape[2], max_pages,
                                                                      cap), q.device)
    qd, od = tensor_desc(q), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    m = _Mask(head_is_streaming)
    _check(lib().aoh_decode_anchor(ctypes.byref(qd), ctypes.byref(fd) if fd else None,
                                   ctypes.byref(rd) if rd else None, m.ptr, _ptr(lens), n_sink, window, top_k,
                                   _ptr(indices), ctypes.byref(od), _ptr(workspace), wsb, _stream(stream)))
    return out, indices


def aoh_decode_reuse_workspace_bytes(batch, n_q_heads, d_head, top_k, ring_capacity):
    return int(lib().aoh_decode_reuse_workspace_bytes(batch, n_q_heads, d_head, top_k, ring_capacity))


def aoh_decode_reuse(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, indices, mapping, out=None,
                     workspace=None, stream=None):
    """Reuse-layer decode step with borrowed positions indices [B, n_lists, top_k] (device int32) and
    mapping (host sequence of Hkv list rows)."""
    if out is None:
        out = torch.empty_like(q)
    n_lists, top_k = indices.shape[1], indices.shape[2]
    cap = kv_ring.capacity if kv_ring is not None else n_sink + window
    workspace, wsb = _ws(workspace, aoh_decode_reuse_workspace_bytes(q.shape[0], q.shape[1], q.shape[2], top_k, cap),
                         q.device)
    mp = (ctypes.c_int32 * len(mapping))(*[int(x) for x in mapping])
    qd, od = tensor_desc(q), tensor_desc(out)
    fd = kv_full.desc() if kv_full is not None else None
    rd = kv_ring.desc() if kv_ring is not None else None
    m = _Mask(head_is_streaming)
    _check(lib().aoh_decode_reuse(ctypes.byref(qd), ctypes.byref(fd) if fd else None,
                                  ctypes.byref(rd) if rd else None, m.ptr, _ptr(lens), n_sink, window, _ptr(indices),
                                  n_lists, top_k, ctypes.cast(mp, ctypes.c_void_p), ctypes.byref(od), _ptr(workspace),
                                  wsb, _stream(stream)))
    return out


def aoh_last_error():
    return lib().aoh_last_error().decode()


def aoh_version():
    return int(lib().aoh_version())
