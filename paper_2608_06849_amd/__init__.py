"""Autonomy-of-Heads head-mixed attention for MI355X (gfx950).

The compute lives in libaoh.so (HIP kernels behind the C interface of
include/aoh.h); ``aoh`` is its ctypes binding.
"""
from .aoh import (AohError, PagedCache, RingCache, aoh_classify, aoh_classify_workspace_bytes,  # noqa: F401
                  aoh_decode, aoh_decode_step, aoh_decode_step_noalloc, aoh_decode_anchor, aoh_decode_anchor_workspace_bytes, aoh_decode_reuse,
                  aoh_decode_reuse_workspace_bytes, aoh_decode_workspace_bytes, aoh_head_mapping,
                  aoh_head_mapping_workspace_bytes, aoh_kv_append, aoh_last_error, aoh_prefill,
                  aoh_prefill_append, aoh_prefill_chunked, aoh_prefill_varlen, aoh_retrieval_group_count, aoh_version, lib)
