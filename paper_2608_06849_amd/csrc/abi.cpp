// Host side of libaoh: argument validation, the head-scheduling pass and the
// launch plan for every entry point of aoh.h.
//
// Head-scheduling pass.  The paper reorders the Q/K/V projection weights
// offline so that retrieval and streaming heads form contiguous slices and no
// gather is needed (Sec. 5 "Reordering"; Appendix "GQA Extension", weight
// reordering at KV-group and query-head granularity).  Here the caller's head
// order is kept: the pass splits the KV heads by label into two lists that
// travel by value in the kernel arguments, and each kernel maps its work item
// to (KV head, query head) through its list.  Outputs land in the caller's
// head order, so the concatenation of Eq. 8 needs no copy.  Each head type
// gets its own launch, sized for its own work: causal query blocks of the
// retrieval launch are issued longest first; the decode cache is cut into
// splits so each launch has enough independent waves to fill the GPU.
#include <cstdarg>
#include <cstdio>
#include <atomic>
#include <cstring>
#include <algorithm>
#include <cmath>

#include "aoh.h"
#include "aoh_internal.h"

using namespace aoh;

namespace {

thread_local char g_err[512] = "";

aoh_status fail(aoh_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

aoh_status ok() {
  g_err[0] = '\0';
  return AOH_OK;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Compute units of the current device, queried once per device (256 on an
// MI355X, also the answer when the query fails).
int compute_units() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cached[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  cached[dev].store(n, std::memory_order_relaxed);
  return n;
}

int elt_size(int dtype) { return dtype == AOH_BF16 ? 2 : 4; }

// Checks a tensor descriptor: rank, dtype, positive sizes, unit last stride,
// positive strides, alignment of the base pointer and strides for 16-byte
// vector access.
aoh_status check_tensor(const aoh_tensor* t, const char* name, int ndim, int dtype_a, int dtype_b) {
  if (!t) return fail(AOH_ERR_INVALID_ARG, "%s: null descriptor", name);
  if (!t->data) return fail(AOH_ERR_INVALID_ARG, "%s: null data pointer", name);
  if (t->ndim != ndim) return fail(AOH_ERR_INVALID_ARG, "%s: expected %d dimensions, got %d", name, ndim, t->ndim);
  if (t->dtype != dtype_a && t->dtype != dtype_b)
    return fail(AOH_ERR_UNSUPPORTED, "%s: unsupported dtype %d", name, t->dtype);
  for (int i = 0; i < ndim; ++i) {
    if (t->shape[i] < 1) return fail(AOH_ERR_INVALID_ARG, "%s: dimension %d has size %lld", name, i, (long long)t->shape[i]);
    if (t->stride[i] < 1) return fail(AOH_ERR_INVALID_ARG, "%s: stride %d must be positive", name, i);
  }
  if (t->stride[ndim - 1] != 1) return fail(AOH_ERR_INVALID_ARG, "%s: last dimension must be contiguous", name);
  const int64_t vec = 16 / elt_size(t->dtype);
  if (reinterpret_cast<uintptr_t>(t->data) % 16)
    return fail(AOH_ERR_INVALID_ARG, "%s: data pointer must be 16-byte aligned", name);
  for (int i = 0; i < ndim - 1; ++i)
    if (t->stride[i] % vec)
      return fail(AOH_ERR_INVALID_ARG, "%s: stride %d must be a multiple of %lld elements", name, i, (long long)vec);
  return AOH_OK;
}

// Head-scheduling pass: KV-head lists by label (ascending id) and each KV
// head's rank inside its cache.
struct HeadSchedule {
  int n_ret = 0, n_str = 0;
  uint8_t ret[kMaxKvHeads];
  uint8_t str[kMaxKvHeads];
  uint8_t rank[kMaxKvHeads];
  uint64_t streaming_mask = 0;
};

aoh_status schedule_heads(const uint8_t* head_is_streaming, int hkv, HeadSchedule* hs) {
  if (!head_is_streaming) return fail(AOH_ERR_INVALID_ARG, "head_is_streaming: null pointer");
  if (hkv < 1 || hkv > kMaxKvHeads) return fail(AOH_ERR_UNSUPPORTED, "Hkv=%d outside [1, %d]", hkv, kMaxKvHeads);
  for (int g = 0; g < hkv; ++g) {
    const uint8_t s = head_is_streaming[g];
    if (s > 1) return fail(AOH_ERR_INVALID_ARG, "head_is_streaming[%d]=%d is not 0/1", g, (int)s);
    if (s) {
      hs->rank[g] = (uint8_t)hs->n_str;
      hs->str[hs->n_str++] = (uint8_t)g;
      hs->streaming_mask |= (1ull << g);
    } else {
      hs->rank[g] = (uint8_t)hs->n_ret;
      hs->ret[hs->n_ret++] = (uint8_t)g;
    }
  }
  return AOH_OK;
}

aoh_status check_mask_params(int n_sink, int window) {
  if (n_sink < 0) return fail(AOH_ERR_INVALID_ARG, "n_sink=%d must be >= 0", n_sink);
  if (window < 1) return fail(AOH_ERR_INVALID_ARG, "window=%d must be >= 1", window);
  if ((int64_t)n_sink + window > (1ll << 30)) return fail(AOH_ERR_UNSUPPORTED, "n_sink + window too large");
  return AOH_OK;
}

// Decode split plan from the cache capacity.  A paged split is
// split_blocks_full 16-token blocks (even, so a wave always reads whole
// 32-token chunks).  The split count per (sequence, KV head) aims at
// ~kDecodeTargetWaves paged waves over the whole launch (enough loads in
// flight to stream HBM), never above kMaxSplits; the ring is cut the same way
// (its wave count below).  n_ret (retrieval KV heads) may be unknown
// (workspace sizing): then the plan for n_ret = 0, n_str = 1 is used,
// which has the most splits of either type (its paged items are cut as for
// one KV head, its ring as the whole step) and so bounds every real plan.
struct SplitPlan {
  int split_blocks_full, n_splits_full;
  int split_blocks_ring, n_splits_ring;
  int ring_blocks;
  int max_splits;
};

SplitPlan plan_splits(int batch, int max_pages, int ring_cap, int n_ret, int n_str) {
  SplitPlan p;
  const int64_t per_head = std::max<int64_t>(1, (int64_t)kDecodeTargetWaves / ((int64_t)batch * std::max(n_ret, 1)));
  const int target_full = (int)std::min<int64_t>(per_head, kMaxSplits);
  int sb = (int)std::max<int64_t>(2, ceil_div(max_pages, target_full));
  sb += sb & 1;
  p.split_blocks_full = sb;
  p.n_splits_full = (int)ceil_div(max_pages, sb);
  p.ring_blocks = (int)ceil_div(std::max(ring_cap, 1), kPageTokens);
  // Ring waves: at least kDecodeTargetWaves / 8, more when the rings hold a
  // larger share of the step's blocks at full length (up to kRingTargetWaves
  // for rings alone), so a ring wave does not outlast the paged ones.
  const int64_t ring_work = (int64_t)std::max(n_str, 1) * p.ring_blocks;
  const int64_t paged_work = (int64_t)n_ret * max_pages;
  const int64_t ring_target = std::max<int64_t>(kDecodeTargetWaves / 8,
                                                kRingTargetWaves * ring_work / (ring_work + paged_work));
  const int64_t per_head_ring = std::max<int64_t>(1, ring_target / ((int64_t)batch * std::max(n_str, 1)));
  const int target_ring = (int)std::min<int64_t>(per_head_ring, kMaxSplits);
  int sbr = (int)std::max<int64_t>(2, ceil_div(p.ring_blocks, target_ring));
  sbr += sbr & 1;
  p.split_blocks_ring = sbr;
  p.n_splits_ring = (int)ceil_div(p.ring_blocks, sbr);
  p.max_splits = std::max(p.n_splits_full, p.n_splits_ring);  // <= kMaxSplits by construction
  return p;
}

// Split partials: fixed splits hold [B][Hq][max_splits] partials; the
// work-space pass (batches up to kWsMaxBatch) at most kWsMaxWgs + B x Hkv
// slots of gs heads, bounded by (kWsMaxWgs + B) x Hq, and two int32 per item
// (B x Hkv <= B x Hq) after them.
size_t workspace_bytes(int batch, int hq, int d, const SplitPlan& p) {
  const size_t fixed = (size_t)batch * hq * p.max_splits * (d + 2) * sizeof(float);
  if (batch > kWsMaxBatch) return fixed;
  const size_t ws = (size_t)(kWsMaxWgs + batch) * hq * (d + 2) * sizeof(float) + (size_t)batch * hq * 2 * sizeof(int32_t);
  return std::max(fixed, ws);
}

}  // namespace

extern "C" {

int32_t aoh_version(void) { return 100; }

const char* aoh_last_error(void) { return g_err; }

static aoh_status check_paged(const aoh_paged_cache* c, int n_ret, int64_t B);
static aoh_status check_v_dim_major(const aoh_paged_cache* c, int n_ret, const char* call);
static aoh_status check_ring(const aoh_ring_cache* c, int n_str, int n_sink, int window, int64_t B);

// Prefill; with append set, also writes the prompt's K/V (positions 0..T-1 of
// every sequence) into kv_full / kv_ring.
constexpr int64_t kSeqMajorMaxBatch = 64;

// Varlen (packed) form of a prefill call: cu_seqlens != nullptr.
struct Varlen {
  const int32_t* cu_seqlens = nullptr;  // DEVICE [batch + 1]
  int32_t batch = 0, max_seqlen = 0;
};

static aoh_status prefill_impl(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                               const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                               int32_t chunk, bool append, const aoh_paged_cache* kv_full,
                               const aoh_ring_cache* kv_ring, aoh_tensor* out, void* stream,
                               const Varlen& vl = Varlen()) {
  aoh_status st;
  const bool packed = vl.cu_seqlens != nullptr;
  const int nd = packed ? 3 : 4;  // packed tensors are [total][H][D]
  if ((st = check_tensor(q, "q", nd, AOH_BF16, AOH_F32))) return st;
  const int dt = q->dtype;
  if ((st = check_tensor(k, "k", nd, dt, dt))) return st;
  if ((st = check_tensor(v, "v", nd, dt, dt))) return st;
  if ((st = check_tensor(out, "out", nd, dt, AOH_F32))) return st;
  // as [B][T][H][D]; packed: B = batch, T = max_seqlen, rows = total tokens
  const int64_t n_rows = packed ? q->shape[0] : q->shape[1];
  const int64_t B = packed ? vl.batch : q->shape[0], T = packed ? vl.max_seqlen : q->shape[1];
  const int64_t Hq = q->shape[nd - 2], D = q->shape[nd - 1];
  const int64_t Hkv = k->shape[nd - 2];
  if (packed) {
    if (B < 1) return fail(AOH_ERR_INVALID_ARG, "batch=%lld must be >= 1", (long long)B);
    if (T < 1) return fail(AOH_ERR_INVALID_ARG, "max_seqlen=%lld must be >= 1", (long long)T);
    if (n_rows > (1ll << 31) - 1) return fail(AOH_ERR_UNSUPPORTED, "too many packed tokens");
    for (const aoh_tensor* t : {k, v})
      if (t->shape[0] != n_rows || t->shape[1] != Hkv || t->shape[2] != D)
        return fail(AOH_ERR_INVALID_ARG, "k/v must be [total=%lld, Hkv, D=%lld] with equal shapes",
                    (long long)n_rows, (long long)D);
    if (out->shape[0] != n_rows || out->shape[1] != Hq || out->shape[2] != D)
      return fail(AOH_ERR_INVALID_ARG, "out must have the shape of q");
  } else {
    for (const aoh_tensor* t : {k, v})
      if (t->shape[0] != B || t->shape[1] != T || t->shape[2] != Hkv || t->shape[3] != D)
        return fail(AOH_ERR_INVALID_ARG, "k/v must be [B=%lld, T=%lld, Hkv, D=%lld] with equal shapes",
                    (long long)B, (long long)T, (long long)D);
    if (out->shape[0] != B || out->shape[1] != T || out->shape[2] != Hq || out->shape[3] != D)
      return fail(AOH_ERR_INVALID_ARG, "out must have the shape of q");
  }
  if (D != 64 && D != 128) return fail(AOH_ERR_UNSUPPORTED, "D=%lld; supported: 64, 128", (long long)D);
  if (Hq % Hkv) return fail(AOH_ERR_UNSUPPORTED, "Hq=%lld is not a multiple of Hkv=%lld", (long long)Hq, (long long)Hkv);
  if (T > (1ll << 30)) return fail(AOH_ERR_UNSUPPORTED, "T=%lld too large", (long long)T);
  if ((st = check_mask_params(n_sink, window))) return st;
  HeadSchedule hs;
  if ((st = schedule_heads(head_is_streaming, (int)Hkv, &hs))) return st;
  const int gs = (int)(Hq / Hkv);
  const int rows = dt == AOH_BF16 ? kPrefillRows : kPrefillRowsF32;
  const int64_t n_qblocks = ceil_div(T, rows);
  if (n_qblocks * Hq * B >= (1ll << 31)) return fail(AOH_ERR_UNSUPPORTED, "grid too large");
  if (append) {
    if ((st = check_paged(kv_full, hs.n_ret, B))) return st;
    if ((st = check_v_dim_major(kv_full, hs.n_ret, "a prefill that fills the caches"))) return st;
    if ((st = check_ring(kv_ring, hs.n_str, n_sink, window, B))) return st;
    if (B > 65535) return fail(AOH_ERR_UNSUPPORTED, "batch too large");
    // fp32 prompts are appended by a separate launch, which has no packed form
    if (packed && dt != AOH_BF16) return fail(AOH_ERR_UNSUPPORTED, "packed prefill with cache append needs bf16");
  }

  PrefillArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q->data; a.k = k->data; a.v = v->data; a.out = out->data;
  if (packed) {
    a.q_st = q->stride[0]; a.q_sh = q->stride[1];
    a.k_st = k->stride[0]; a.k_sh = k->stride[1];
    a.v_st = v->stride[0]; a.v_sh = v->stride[1];
    a.o_st = out->stride[0]; a.o_sh = out->stride[1];
    a.cu_seqlens = vl.cu_seqlens;
    a.total = (int)n_rows;
    // sequence-major order for the bf16 kernel when the per-workgroup walk
    // over the sequences stays short
    a.seq_major = (dt == AOH_BF16 && B <= kSeqMajorMaxBatch) ? 1 : 0;
  } else {
    a.q_sb = q->stride[0]; a.q_st = q->stride[1]; a.q_sh = q->stride[2];
    a.k_sb = k->stride[0]; a.k_st = k->stride[1]; a.k_sh = k->stride[2];
    a.v_sb = v->stride[0]; a.v_st = v->stride[1]; a.v_sh = v->stride[2];
    a.o_sb = out->stride[0]; a.o_st = out->stride[1]; a.o_sh = out->stride[2];
  }
  a.B = (int)B; a.T = (int)T; a.gs = gs;
  a.n_sink = n_sink; a.window = window; a.chunk = chunk;
  a.n_qblocks = (int)n_qblocks;
  a.scale = (float)(1.0 / std::sqrt((double)D));
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  const int out_f32 = out->dtype == AOH_F32 && dt == AOH_BF16;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // The bf16 kernel writes the caches itself; the fp32 path appends after.
  const bool fused = append && dt == AOH_BF16;
  // Per-type arguments: the retrieval heads (and the paged cache), the
  // streaming heads (and the ring).
  PrefillArgs ar = a, as = a;
  if (hs.n_ret) {
    ar.n_kv = hs.n_ret;
    std::memcpy(ar.kv_heads, hs.ret, hs.n_ret);
    if (fused) {
      ar.append = 1;
      ar.ck = kv_full->k; ar.cv = kv_full->v; ar.block_table = kv_full->block_table;
      ar.max_pages = kv_full->max_pages_per_seq; ar.num_pages = (int)kv_full->num_pages;
      ar.n_cache = hs.n_ret; ar.ring_blocks = 0;
    }
  }
  if (hs.n_str) {
    as.n_kv = hs.n_str;
    std::memcpy(as.kv_heads, hs.str, hs.n_str);
    if (fused) {
      as.append = 1;
      as.ck = kv_ring->k; as.cv = kv_ring->v; as.block_table = nullptr;
      as.max_pages = 0; as.num_pages = 0;
      as.n_cache = hs.n_str; as.ring_blocks = (int)ceil_div(kv_ring->capacity, kPageTokens);
    }
  }
  if (hs.n_ret && hs.n_str && prefill_mixed_preferred(ar, dt, (int)D)) {
    // One launch, retrieval items first: their causal work dominates
    // (O(T^2) vs O(T(n_sink+window))); the streaming items fill the tail.
    hipError_t e = launch_prefill_mixed(ar, as, out_f32, s);
    if (e != hipSuccess) return fail(AOH_ERR_HIP, "prefill launch: %s", hipGetErrorString(e));
  } else {
    if (hs.n_ret) {
      hipError_t e = launch_prefill(ar, dt, out_f32, (int)D, false, s);
      if (e != hipSuccess) return fail(AOH_ERR_HIP, "prefill retrieval launch: %s", hipGetErrorString(e));
    }
    if (hs.n_str) {
      hipError_t e = launch_prefill(as, dt, out_f32, (int)D, true, s);
      if (e != hipSuccess) return fail(AOH_ERR_HIP, "prefill streaming launch: %s", hipGetErrorString(e));
    }
  }
  if (append && !fused) {
    AppendArgs ap;
    std::memset(&ap, 0, sizeof(ap));
    ap.k_new = k->data; ap.v_new = v->data;
    ap.k_sb = k->stride[0]; ap.k_st = k->stride[1]; ap.k_sh = k->stride[2];
    ap.v_sb = v->stride[0]; ap.v_st = v->stride[1]; ap.v_sh = v->stride[2];
    ap.start_pos = nullptr;  // the prompt starts at position 0
    ap.B = (int)B; ap.n_new = (int)T; ap.Hkv = (int)Hkv;
    if (hs.n_ret) {
      ap.pk = kv_full->k; ap.pv = kv_full->v; ap.block_table = kv_full->block_table;
      ap.max_pages = kv_full->max_pages_per_seq; ap.num_pages = (int)kv_full->num_pages; ap.n_ret = hs.n_ret;
    }
    if (hs.n_str) {
      ap.rk = kv_ring->k; ap.rv = kv_ring->v; ap.n_str = hs.n_str;
      ap.ring_blocks = (int)ceil_div(kv_ring->capacity, kPageTokens);
    }
    ap.n_sink = n_sink; ap.window = window;
    ap.n_chunks = (int)ceil_div(T, kPageTokens);
    ap.streaming_mask = hs.streaming_mask;
    std::memcpy(ap.rank, hs.rank, sizeof(ap.rank));
    hipError_t e = launch_append(ap, dt, (int)D, s);
    if (e != hipSuccess) return fail(AOH_ERR_HIP, "append launch: %s", hipGetErrorString(e));
  }
  return ok();
}

aoh_status aoh_prefill(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                       const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                       aoh_tensor* out, void* stream) {
  return prefill_impl(q, k, v, head_is_streaming, n_sink, window, 0, false, nullptr, nullptr, out, stream);
}

aoh_status aoh_prefill_chunked(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                               const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                               int32_t chunk, aoh_tensor* out, void* stream) {
  if (chunk < 1) return fail(AOH_ERR_INVALID_ARG, "chunk=%d must be >= 1", chunk);
  return prefill_impl(q, k, v, head_is_streaming, n_sink, window, chunk, false, nullptr, nullptr, out, stream);
}

aoh_status aoh_prefill_varlen(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                              const int32_t* cu_seqlens, int32_t batch, int32_t max_seqlen,
                              const uint8_t* head_is_streaming, int32_t n_sink, int32_t window, int32_t chunk,
                              const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring, aoh_tensor* out,
                              void* stream) {
  if (chunk < 0) return fail(AOH_ERR_INVALID_ARG, "chunk=%d must be >= 0", chunk);
  if (!cu_seqlens) return fail(AOH_ERR_INVALID_ARG, "cu_seqlens: null pointer");
  Varlen vl;
  vl.cu_seqlens = cu_seqlens; vl.batch = batch; vl.max_seqlen = max_seqlen;
  const bool append = kv_full != nullptr || kv_ring != nullptr;
  return prefill_impl(q, k, v, head_is_streaming, n_sink, window, chunk, append, kv_full, kv_ring, out, stream, vl);
}

aoh_status aoh_prefill_append(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                              const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                              int32_t chunk, const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                              aoh_tensor* out, void* stream) {
  if (chunk < 0) return fail(AOH_ERR_INVALID_ARG, "chunk=%d must be >= 0", chunk);
  return prefill_impl(q, k, v, head_is_streaming, n_sink, window, chunk, true, kv_full, kv_ring, out, stream);
}

static aoh_status check_paged(const aoh_paged_cache* c, int n_ret, int64_t B) {
  if (!n_ret) return AOH_OK;
  if (!c) return fail(AOH_ERR_INVALID_ARG, "kv_full is null but %d retrieval heads exist", n_ret);
  if (!c->k || !c->v || !c->block_table) return fail(AOH_ERR_INVALID_ARG, "kv_full: null pointer");
  if (c->n_heads != n_ret)
    return fail(AOH_ERR_INVALID_ARG, "kv_full.n_heads=%d but the mask has %d retrieval heads", c->n_heads, n_ret);
  if (c->num_pages < 1 || c->max_pages_per_seq < 1) return fail(AOH_ERR_INVALID_ARG, "kv_full: empty cache");
  if (c->num_pages > (1ll << 31) - 1) return fail(AOH_ERR_UNSUPPORTED, "kv_full: too many pages");
  if ((int64_t)c->max_pages_per_seq * kPageTokens > (1ll << 30)) return fail(AOH_ERR_UNSUPPORTED, "kv_full: too many pages per sequence");
  if (c->n_seqs < B)
    return fail(AOH_ERR_INVALID_ARG, "kv_full.n_seqs=%d: the block table has fewer rows than the %lld sequences",
                c->n_seqs, (long long)B);
  if (reinterpret_cast<uintptr_t>(c->k) % 16 || reinterpret_cast<uintptr_t>(c->v) % 16)
    return fail(AOH_ERR_INVALID_ARG, "kv_full: cache pointers must be 16-byte aligned");
  if (c->v_token_major != 0 && c->v_token_major != 1)
    return fail(AOH_ERR_INVALID_ARG, "kv_full.v_token_major=%d; must be 0 or 1", c->v_token_major);
  return AOH_OK;
}

// Token-major V pages are written by aoh_kv_append and read by the reuse layer
// only; the other readers and writers take dimension-major pages.
static aoh_status check_v_dim_major(const aoh_paged_cache* c, int n_ret, const char* call) {
  if (n_ret && c->v_token_major)
    return fail(AOH_ERR_UNSUPPORTED, "%s needs dimension-major V pages (kv_full.v_token_major=0); "
                "token-major pages are for aoh_kv_append and aoh_decode_reuse", call);
  return AOH_OK;
}

static aoh_status check_ring(const aoh_ring_cache* c, int n_str, int n_sink, int window, int64_t B) {
  if (!n_str) return AOH_OK;
  if (!c) return fail(AOH_ERR_INVALID_ARG, "kv_ring is null but %d streaming heads exist", n_str);
  if (!c->k || !c->v) return fail(AOH_ERR_INVALID_ARG, "kv_ring: null pointer");
  if (c->n_heads != n_str)
    return fail(AOH_ERR_INVALID_ARG, "kv_ring.n_heads=%d but the mask has %d streaming heads", c->n_heads, n_str);
  if (c->capacity != n_sink + window)
    return fail(AOH_ERR_INVALID_ARG, "kv_ring.capacity=%d must equal n_sink + window = %d", c->capacity, n_sink + window);
  if (c->batch < B)
    return fail(AOH_ERR_INVALID_ARG, "kv_ring.batch=%d: the ring holds fewer than the %lld sequences", c->batch,
                (long long)B);
  if (reinterpret_cast<uintptr_t>(c->k) % 16 || reinterpret_cast<uintptr_t>(c->v) % 16)
    return fail(AOH_ERR_INVALID_ARG, "kv_ring: cache pointers must be 16-byte aligned");
  return AOH_OK;
}

aoh_status aoh_kv_append(const aoh_tensor* k_new, const aoh_tensor* v_new,
                         const uint8_t* head_is_streaming, const int32_t* start_pos,
                         const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                         int32_t n_sink, int32_t window, void* stream) {
  aoh_status st;
  if ((st = check_tensor(k_new, "k_new", 4, AOH_BF16, AOH_F32))) return st;
  const int dt = k_new->dtype;
  if ((st = check_tensor(v_new, "v_new", 4, dt, dt))) return st;
  for (int i = 0; i < 4; ++i)
    if (v_new->shape[i] != k_new->shape[i]) return fail(AOH_ERR_INVALID_ARG, "k_new and v_new shapes differ");
  const int64_t B = k_new->shape[0], n_new = k_new->shape[1], Hkv = k_new->shape[2], D = k_new->shape[3];
  if (D != 64 && D != 128) return fail(AOH_ERR_UNSUPPORTED, "D=%lld; supported: 64, 128", (long long)D);
  if (n_new > (1ll << 30)) return fail(AOH_ERR_UNSUPPORTED, "n_new too large");
  if (B > 65535) return fail(AOH_ERR_UNSUPPORTED, "batch too large");
  if (!start_pos) return fail(AOH_ERR_INVALID_ARG, "start_pos: null pointer");
  if ((st = check_mask_params(n_sink, window))) return st;
  HeadSchedule hs;
  if ((st = schedule_heads(head_is_streaming, (int)Hkv, &hs))) return st;
  if ((st = check_paged(kv_full, hs.n_ret, B))) return st;
  if ((st = check_ring(kv_ring, hs.n_str, n_sink, window, B))) return st;

  AppendArgs a;
  std::memset(&a, 0, sizeof(a));
  a.k_new = k_new->data; a.v_new = v_new->data;
  a.k_sb = k_new->stride[0]; a.k_st = k_new->stride[1]; a.k_sh = k_new->stride[2];
  a.v_sb = v_new->stride[0]; a.v_st = v_new->stride[1]; a.v_sh = v_new->stride[2];
  a.start_pos = start_pos;
  a.B = (int)B; a.n_new = (int)n_new; a.Hkv = (int)Hkv;
  if (hs.n_ret) {
    a.pk = kv_full->k; a.pv = kv_full->v; a.block_table = kv_full->block_table;
    a.max_pages = kv_full->max_pages_per_seq; a.num_pages = (int)kv_full->num_pages; a.n_ret = hs.n_ret;
    a.v_token_major = kv_full->v_token_major;
  }
  if (hs.n_str) {
    a.rk = kv_ring->k; a.rv = kv_ring->v; a.n_str = hs.n_str;
    a.ring_blocks = (int)ceil_div(kv_ring->capacity, kPageTokens);
  }
  a.n_sink = n_sink; a.window = window;
  a.n_chunks = (int)ceil_div(n_new, kPageTokens) + 1;
  a.streaming_mask = hs.streaming_mask;
  std::memcpy(a.rank, hs.rank, sizeof(a.rank));
  hipError_t e = launch_append(a, dt, (int)D, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(AOH_ERR_HIP, "append launch: %s", hipGetErrorString(e));
  return ok();
}

size_t aoh_decode_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t d_head,
                                  int32_t max_pages_per_seq, int32_t ring_capacity) {
  if (batch < 1 || n_q_heads < 1 || (d_head != 64 && d_head != 128) || max_pages_per_seq < 1 ||
      ring_capacity < 0)
    return 0;
  return workspace_bytes(batch, n_q_heads, d_head, plan_splits(batch, max_pages_per_seq, ring_capacity, 0, 1));
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Anchor extras: score codes [B][Hq][16 * max_pages] (16-bit) and their
// references [B][Hq][max_pages], final (m, l) [B][Hq][2], and the top-k keys
// and partial histograms per (sequence, KV head) list (sized with Hq lists per
// sequence, a bound on the retrieval KV heads).
static size_t anchor_codes_bytes(int64_t B, int64_t Hq, int64_t max_pages) {
  return align256((size_t)(B * Hq * max_pages * kPageTokens) * sizeof(uint16_t));
}
static size_t anchor_refs_bytes(int64_t B, int64_t Hq, int64_t max_pages) {
  return align256((size_t)(B * Hq * max_pages) * sizeof(float));
}
static size_t anchor_keys_bytes(int64_t B, int64_t Hq, int64_t max_pages) {
  return align256((size_t)(B * Hq * max_pages * kPageTokens) * sizeof(uint32_t));
}
static size_t anchor_ml_bytes(int64_t B, int64_t Hq) { return align256((size_t)(B * Hq * 2) * sizeof(float)); }
static size_t anchor_part_bytes(int64_t B, int64_t Hq) {
  return align256((size_t)(B * Hq * kTopkPasses * kTopkParts * 2048) * sizeof(uint32_t));
}
// dummy targets of the score stores: 64 x 8 codes, then 64 references
static constexpr size_t kCodeDummyBytes = 64 * 8 * sizeof(uint16_t);
static constexpr size_t kScoreDummyBytes = kCodeDummyBytes + 64 * sizeof(float);
static size_t anchor_extra(int64_t B, int64_t Hq, int64_t max_pages) {
  return anchor_codes_bytes(B, Hq, max_pages) + anchor_refs_bytes(B, Hq, max_pages) +
         anchor_keys_bytes(B, Hq, max_pages) + anchor_ml_bytes(B, Hq) + anchor_part_bytes(B, Hq) +
         kScoreDummyBytes;
}

// H2Share roles of a decode call (Sec. "AoH-Guided Sparse Attention"): plain,
// anchor layer (also selects top-k positions), reuse layer (retrieval heads
// attend to borrowed positions).
enum DecodeMode { kPlain = 0, kAnchor = 1, kReuse = 2 };

struct DecodeExtra {
  int mode = kPlain;
  int32_t top_k = 0;          // anchor: positions to select; reuse: entries per list
  int32_t* sel_out = nullptr; // anchor output [B][n_ret][top_k]
  const int32_t* sel_in = nullptr;  // reuse input [B][n_lists][top_k]
  int32_t n_lists = 0;
  const int32_t* mapping = nullptr;  // reuse: HOST [Hkv], list rank per retrieval group
  const aoh_tensor* k_new = nullptr;  // fused step: token at lens - 1, [B][Hkv][D]
  const aoh_tensor* v_new = nullptr;
  size_t* need_only = nullptr;  // validate only: store the workspace bytes needed, launch nothing
};

static aoh_status decode_impl(const aoh_tensor* q, const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                              const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                              int32_t window, aoh_tensor* out, void* workspace, size_t workspace_bytes_given,
                              void* stream, const DecodeExtra& x) {
  aoh_status st;
  if ((st = check_tensor(q, "q", 3, AOH_BF16, AOH_F32))) return st;
  const int dt = q->dtype;
  if ((st = check_tensor(out, "out", 3, dt, AOH_F32))) return st;
  const int64_t B = q->shape[0], Hq = q->shape[1], D = q->shape[2];
  if (out->shape[0] != B || out->shape[1] != Hq || out->shape[2] != D)
    return fail(AOH_ERR_INVALID_ARG, "out must have the shape of q");
  if (D != 64 && D != 128) return fail(AOH_ERR_UNSUPPORTED, "D=%lld; supported: 64, 128", (long long)D);
  if (!lens) return fail(AOH_ERR_INVALID_ARG, "lens: null pointer");
  if ((st = check_mask_params(n_sink, window))) return st;
  // The label array has one entry per KV head; its length is Hkv.  The
  // caches tell how many heads of each type exist, so Hkv = n_ret + n_str.
  const int n_ret_c = kv_full ? kv_full->n_heads : 0;
  const int n_str_c = kv_ring ? kv_ring->n_heads : 0;
  const int64_t Hkv = (int64_t)n_ret_c + n_str_c;
  if (Hkv < 1) return fail(AOH_ERR_INVALID_ARG, "no cache given");
  if (Hq % Hkv) return fail(AOH_ERR_UNSUPPORTED, "Hq=%lld is not a multiple of Hkv=%lld", (long long)Hq, (long long)Hkv);
  HeadSchedule hs;
  if ((st = schedule_heads(head_is_streaming, (int)Hkv, &hs))) return st;
  if ((st = check_paged(kv_full, hs.n_ret, B))) return st;
  if (x.mode != kReuse) {
    const char* call = x.k_new ? "aoh_decode_step" : x.mode == kAnchor ? "aoh_decode_anchor" : "aoh_decode";
    if ((st = check_v_dim_major(kv_full, hs.n_ret, call))) return st;
  }
  if ((st = check_ring(kv_ring, hs.n_str, n_sink, window, B))) return st;
  const int gs = (int)(Hq / Hkv);
  if (dt == AOH_BF16 && gs > 16) return fail(AOH_ERR_UNSUPPORTED, "Hq/Hkv=%d > 16", gs);
  const bool step = x.k_new != nullptr;
  if (step) {
    if ((st = check_tensor(x.k_new, "k_new", 3, dt, dt))) return st;
    if ((st = check_tensor(x.v_new, "v_new", 3, dt, dt))) return st;
    for (const aoh_tensor* t : {x.k_new, x.v_new})
      if (t->shape[0] != B || t->shape[1] != Hkv || t->shape[2] != D)
        return fail(AOH_ERR_INVALID_ARG, "k_new / v_new must be [B=%lld][Hkv=%lld][D=%lld]", (long long)B,
                    (long long)Hkv, (long long)D);
  }
  if (x.mode != kPlain) {
    if (dt != AOH_BF16) return fail(AOH_ERR_UNSUPPORTED, "anchor/reuse decode needs bf16");
    if (x.top_k < 1 || x.top_k > (1 << 30)) return fail(AOH_ERR_INVALID_ARG, "top_k=%d must be >= 1", x.top_k);
  }
  if (x.mode == kAnchor && hs.n_ret && !x.sel_out) return fail(AOH_ERR_INVALID_ARG, "indices: null pointer");
  // the append of an fp32 step and the top-k launch put the batch in grid.z
  if ((x.mode == kAnchor || (step && dt == AOH_F32)) && B > 65535)
    return fail(AOH_ERR_UNSUPPORTED, "batch too large");
  uint8_t sel_rank[kMaxKvHeads] = {0};
  if (x.mode == kReuse && hs.n_ret) {
    if (!x.sel_in) return fail(AOH_ERR_INVALID_ARG, "indices: null pointer");
    if (!x.mapping) return fail(AOH_ERR_INVALID_ARG, "mapping: null pointer");
    if (x.n_lists < 1 || x.n_lists > kMaxKvHeads) return fail(AOH_ERR_INVALID_ARG, "n_lists=%d outside [1, 64]", x.n_lists);
    for (int j = 0; j < hs.n_ret; ++j) {
      const int32_t r = x.mapping[hs.ret[j]];
      if (r < 0 || r >= x.n_lists)
        return fail(AOH_ERR_INVALID_ARG, "mapping[%d]=%d: a retrieval group needs a list in [0, %d)", hs.ret[j], r,
                    x.n_lists);
      sel_rank[j] = (uint8_t)r;
    }
  }
  const int max_pages = hs.n_ret ? kv_full->max_pages_per_seq : 1;
  const int ring_cap = n_sink + window;
  // Reuse: the paged items run over the borrowed list, cut like a cache of
  // ceil(top_k / 16) blocks.
  const int plan_pages = x.mode == kReuse ? (int)ceil_div(x.top_k, kPageTokens) : max_pages;
  const SplitPlan sp = plan_splits((int)B, plan_pages, ring_cap, hs.n_ret, hs.n_str);
  // The workspace is sized for the n_ret = 0, n_str = 1 plan, which bounds this one.
  const SplitPlan sp_bound = plan_splits((int)B, plan_pages, ring_cap, 0, 1);

  DecodeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q->data; a.q_sb = q->stride[0]; a.q_sh = q->stride[1];
  a.lens = lens;
  a.B = (int)B; a.Hq = (int)Hq; a.gs = gs;
  a.ring_cap = ring_cap;
  a.scale = (float)(1.0 / std::sqrt((double)D));
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)D));
  if (hs.n_ret) {
    CacheView& c = a.full;
    c.k = kv_full->k; c.v = kv_full->v; c.block_table = kv_full->block_table;
    c.max_pages = kv_full->max_pages_per_seq; c.num_pages = (int)kv_full->num_pages;
    c.v_token_major = kv_full->v_token_major;
    c.n_kv = hs.n_ret;
    c.split_blocks = sp.split_blocks_full; c.n_splits = sp.n_splits_full;
    c.n_groups = (int)ceil_div(sp.n_splits_full, kSplitWaves);
    c.n_items = (int)(B * hs.n_ret * c.n_groups);
    std::memcpy(c.kv_heads, hs.ret, hs.n_ret);
  }
  if (hs.n_str) {
    CacheView& c = a.ring;
    c.k = kv_ring->k; c.v = kv_ring->v;
    c.ring_blocks = sp.ring_blocks;
    c.n_kv = hs.n_str;
    c.split_blocks = sp.split_blocks_ring; c.n_splits = sp.n_splits_ring;
    c.n_groups = (int)ceil_div(sp.n_splits_ring, kSplitWaves);
    c.n_items = (int)(B * hs.n_str * c.n_groups);
    std::memcpy(c.kv_heads, hs.str, hs.n_str);
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((int64_t)a.full.n_items + a.ring.n_items >= (1ll << 31)) return fail(AOH_ERR_UNSUPPORTED, "grid too large");
  // Workspace: split partials (bf16 only; fp32 decodes directly).
  const size_t base_need = dt == AOH_F32 ? 0 : workspace_bytes((int)B, (int)Hq, (int)D, sp_bound);
  const size_t need = x.mode == kAnchor ? align256(base_need) + anchor_extra(B, Hq, max_pages) : base_need;
  if (x.need_only) {
    *x.need_only = need;
    return ok();
  }
  if (dt == AOH_BF16) {
    if (!workspace) return fail(AOH_ERR_WORKSPACE, "workspace is null; %zu bytes needed", need);
    if (workspace_bytes_given < need)
      return fail(AOH_ERR_WORKSPACE, "workspace has %zu bytes; %zu needed", workspace_bytes_given, need);
    if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(AOH_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  }

  if (step) {
    a.k_new = x.k_new->data; a.v_new = x.v_new->data;
    a.kn_sb = x.k_new->stride[0]; a.kn_sh = x.k_new->stride[1];
    a.vn_sb = x.v_new->stride[0]; a.vn_sh = x.v_new->stride[1];
    a.n_sink = n_sink; a.window = window;
  }
  if (step && dt == AOH_F32) {
    // fp32 step: a separate append at position lens - 1 before the decode.
    AppendArgs ap;
    std::memset(&ap, 0, sizeof(ap));
    ap.k_new = x.k_new->data; ap.v_new = x.v_new->data;
    ap.k_sb = x.k_new->stride[0]; ap.k_st = 0; ap.k_sh = x.k_new->stride[1];
    ap.v_sb = x.v_new->stride[0]; ap.v_st = 0; ap.v_sh = x.v_new->stride[1];
    ap.start_pos = lens; ap.start_bias = -1;
    ap.B = (int)B; ap.n_new = 1; ap.Hkv = (int)Hkv;
    if (hs.n_ret) {
      ap.pk = kv_full->k; ap.pv = kv_full->v; ap.block_table = kv_full->block_table;
      ap.max_pages = kv_full->max_pages_per_seq; ap.num_pages = (int)kv_full->num_pages; ap.n_ret = hs.n_ret;
    }
    if (hs.n_str) {
      ap.rk = kv_ring->k; ap.rv = kv_ring->v; ap.n_str = hs.n_str;
      ap.ring_blocks = (int)ceil_div(kv_ring->capacity, kPageTokens);
    }
    ap.n_sink = n_sink; ap.window = window;
    ap.n_chunks = 2;
    ap.streaming_mask = hs.streaming_mask;
    std::memcpy(ap.rank, hs.rank, sizeof(ap.rank));
    hipError_t e = launch_append(ap, dt, (int)D, s);
    if (e != hipSuccess) return fail(AOH_ERR_HIP, "append launch: %s", hipGetErrorString(e));
  }

  if (dt == AOH_F32) {
    // fp32: direct per-head kernel, no workspace.
    hipError_t e = launch_decode_f32(a, (int)D, out->data, out->stride[0], out->stride[1], s);
    if (e != hipSuccess) return fail(AOH_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
    return ok();
  }

  // Plain, anchor and fused steps of up to kWsMaxBatch sequences split the
  // step's work space on the device (two workgroups per CU), which follows any
  // mix of lengths and of cache types; larger batches and the reuse layer take
  // fixed splits from the cache capacity.
  const int64_t ws_blocks = std::max<int64_t>(max_pages, sp.ring_blocks);
  if (x.mode != kReuse && B <= kWsMaxBatch && B * Hkv * ws_blocks < (1ll << 30))
    a.ws_cu = std::min(compute_units(), kWsMaxWgs / 2);
  float* part_acc = reinterpret_cast<float*>(workspace);
  const size_t acc_floats = a.ws_cu ? (size_t)(2 * a.ws_cu + B * Hkv) * gs * D
                                    : (size_t)B * Hq * sp_bound.max_splits * D;
  float* part_ml = part_acc + acc_floats;
  a.part_acc = part_acc; a.part_ml = part_ml; a.max_splits = sp_bound.max_splits;
  if (a.ws_cu) a.ws_items = reinterpret_cast<int32_t*>(part_ml + acc_floats / D * 2);
  uint16_t* codes = nullptr;
  float* refs = nullptr;
  uint32_t* keys = nullptr;
  float* ml = nullptr;
  uint32_t* part = nullptr;
  if (x.mode == kAnchor) {
    char* w = reinterpret_cast<char*>(workspace) + align256(base_need);
    codes = reinterpret_cast<uint16_t*>(w);
    w += anchor_codes_bytes(B, Hq, max_pages);
    refs = reinterpret_cast<float*>(w);
    w += anchor_refs_bytes(B, Hq, max_pages);
    keys = reinterpret_cast<uint32_t*>(w);
    w += anchor_keys_bytes(B, Hq, max_pages);
    ml = reinterpret_cast<float*>(w);
    w += anchor_ml_bytes(B, Hq);
    part = reinterpret_cast<uint32_t*>(w);
    w += anchor_part_bytes(B, Hq);
    a.code_dummy = reinterpret_cast<uint16_t*>(w);
    a.ref_dummy = reinterpret_cast<float*>(w + kCodeDummyBytes);
    a.score_codes = codes;
    a.score_refs = refs;
    a.score_len = max_pages * kPageTokens;
  }
  if (x.mode == kReuse) {
    a.sel = x.sel_in; a.n_sel = x.top_k; a.n_lists = x.n_lists;
    std::memcpy(a.sel_rank, sel_rank, sizeof(sel_rank));
  }
  {
    hipError_t e = launch_decode_split(a, (int)D, step ? 3 : x.mode, s);
    if (e != hipSuccess) return fail(AOH_ERR_HIP, "decode split launch: %s", hipGetErrorString(e));
  }
  MergeArgs m;
  std::memset(&m, 0, sizeof(m));
  m.part_acc = part_acc; m.part_ml = part_ml; m.lens = lens;
  m.out = out->data; m.o_sb = out->stride[0]; m.o_sh = out->stride[1];
  m.B = (int)B; m.Hq = (int)Hq; m.gs = gs; m.max_splits = sp_bound.max_splits;
  // One partial per split workgroup (kSplitWaves consecutive splits).
  m.n_splits_full = a.full.n_groups;
  m.n_splits_ring = a.ring.n_groups;
  // reuse: a retrieval head's "length" is its number of borrowed entries
  m.max_len = x.mode == kReuse ? x.top_k : max_pages * kPageTokens;
  m.ring_cap = ring_cap;
  m.ws_cu = a.ws_cu; m.ws_n_ret = hs.n_ret; m.ws_n_str = hs.n_str; m.ws_items = a.ws_items;
  m.streaming_mask = hs.streaming_mask;
  m.ml_out = ml;
  const int out_f32 = out->dtype == AOH_F32;
  hipError_t e = launch_decode_merge(m, dt, out_f32, (int)D, s);
  if (e != hipSuccess) return fail(AOH_ERR_HIP, "decode merge launch: %s", hipGetErrorString(e));
  if (x.mode == kAnchor && hs.n_ret) {
    TopkArgs t;
    std::memset(&t, 0, sizeof(t));
    t.score_codes = codes; t.score_refs = refs; t.keys = keys; t.ml = ml; t.lens = lens; t.sel = x.sel_out;
    t.B = (int)B; t.Hq = (int)Hq; t.gs = gs; t.n_kv = hs.n_ret;
    t.score_len = max_pages * kPageTokens;
    t.n_sel = x.top_k;
    t.part = part;
    std::memcpy(t.kv_heads, hs.ret, hs.n_ret);
    e = launch_topk(t, s);
    if (e != hipSuccess) return fail(AOH_ERR_HIP, "top-k launch: %s", hipGetErrorString(e));
  }
  return ok();
}

aoh_status aoh_decode(const aoh_tensor* q, const aoh_paged_cache* kv_full,
                      const aoh_ring_cache* kv_ring, const uint8_t* head_is_streaming,
                      const int32_t* lens, int32_t n_sink, int32_t window, aoh_tensor* out,
                      void* workspace, size_t workspace_bytes_given, void* stream) {
  return decode_impl(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out, workspace,
                     workspace_bytes_given, stream, DecodeExtra());
}

aoh_status aoh_decode_step(const aoh_tensor* q, const aoh_tensor* k_new, const aoh_tensor* v_new,
                           const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                           const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                           int32_t window, aoh_tensor* out, void* workspace, size_t workspace_bytes_given,
                           void* stream) {
  if (!k_new) return fail(AOH_ERR_INVALID_ARG, "k_new: null descriptor");
  if (!v_new) return fail(AOH_ERR_INVALID_ARG, "v_new: null descriptor");
  DecodeExtra x;
  x.k_new = k_new; x.v_new = v_new;
  return decode_impl(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out, workspace,
                     workspace_bytes_given, stream, x);
}

}  // extern "C"

// Validation of a fused decode step without launching: on AOH_OK, *need is
// the workspace aoh_decode_step needs for these arguments.
aoh_status aoh::decode_step_workspace_need(const aoh_tensor* q, const aoh_tensor* k_new, const aoh_tensor* v_new,
                                           const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                                           const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                                           int32_t window, aoh_tensor* out, size_t* need) {
  if (!k_new) return fail(AOH_ERR_INVALID_ARG, "k_new: null descriptor");
  if (!v_new) return fail(AOH_ERR_INVALID_ARG, "v_new: null descriptor");
  DecodeExtra x;
  x.k_new = k_new; x.v_new = v_new; x.need_only = need;
  return decode_impl(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out, nullptr, 0, nullptr, x);
}

aoh_status aoh::report(aoh_status st, const char* msg) { return st == AOH_OK ? ok() : fail(st, "%s", msg); }

extern "C" {

size_t aoh_decode_anchor_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t d_head,
                                         int32_t max_pages_per_seq, int32_t ring_capacity) {
  const size_t base = aoh_decode_workspace_bytes(batch, n_q_heads, d_head, max_pages_per_seq, ring_capacity);
  if (!base) return 0;
  return align256(base) + anchor_extra(batch, n_q_heads, max_pages_per_seq);
}

aoh_status aoh_decode_anchor(const aoh_tensor* q, const aoh_paged_cache* kv_full,
                             const aoh_ring_cache* kv_ring, const uint8_t* head_is_streaming,
                             const int32_t* lens, int32_t n_sink, int32_t window, int32_t top_k,
                             int32_t* indices, aoh_tensor* out, void* workspace, size_t workspace_bytes_given,
                             void* stream) {
  DecodeExtra x;
  x.mode = kAnchor; x.top_k = top_k; x.sel_out = indices;
  return decode_impl(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out, workspace,
                     workspace_bytes_given, stream, x);
}

size_t aoh_decode_reuse_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t d_head, int32_t top_k,
                                        int32_t ring_capacity) {
  if (top_k < 1) return 0;
  return aoh_decode_workspace_bytes(batch, n_q_heads, d_head, (int32_t)ceil_div(top_k, kPageTokens), ring_capacity);
}

aoh_status aoh_decode_reuse(const aoh_tensor* q, const aoh_paged_cache* kv_full,
                            const aoh_ring_cache* kv_ring, const uint8_t* head_is_streaming,
                            const int32_t* lens, int32_t n_sink, int32_t window, const int32_t* indices,
                            int32_t n_lists, int32_t top_k, const int32_t* mapping, aoh_tensor* out,
                            void* workspace, size_t workspace_bytes_given, void* stream) {
  DecodeExtra x;
  x.mode = kReuse; x.top_k = top_k; x.sel_in = indices; x.n_lists = n_lists; x.mapping = mapping;
  return decode_impl(q, kv_full, kv_ring, head_is_streaming, lens, n_sink, window, out, workspace,
                     workspace_bytes_given, stream, x);
}

static size_t mapping_ws(int64_t hq, int64_t hkv, int64_t d) {
  return align256((size_t)(2 * (hq + hkv) * d * d) * sizeof(float)) +
         align256((size_t)(hkv * hkv * d * d) * sizeof(float)) + align256((size_t)(hq * hq) * sizeof(double)) +
         align256((size_t)(2 * hq) * sizeof(double));
}

size_t aoh_head_mapping_workspace_bytes(int32_t n_q_heads, int32_t n_kv_heads, int32_t d_head) {
  if (n_q_heads < 1 || n_kv_heads < 1 || (d_head != 64 && d_head != 128)) return 0;
  return mapping_ws(n_q_heads, n_kv_heads, d_head);
}

aoh_status aoh_head_mapping(const aoh_tensor* w_q_anchor, const aoh_tensor* w_k_anchor,
                            const aoh_tensor* w_q_reuse, const aoh_tensor* w_k_reuse, int32_t d_head,
                            const uint8_t* anchor_is_streaming, const uint8_t* reuse_is_streaming,
                            double* head_sim, double* group_sim, int32_t* mapping, void* workspace,
                            size_t workspace_bytes_given, void* stream) {
  aoh_status st;
  const aoh_tensor* ws4[4] = {w_q_anchor, w_k_anchor, w_q_reuse, w_k_reuse};
  const char* names[4] = {"w_q_anchor", "w_k_anchor", "w_q_reuse", "w_k_reuse"};
  for (int i = 0; i < 4; ++i)
    if ((st = check_tensor(ws4[i], names[i], 2, AOH_BF16, AOH_BF16))) return st;
  if (d_head != 64 && d_head != 128) return fail(AOH_ERR_UNSUPPORTED, "d_head=%d; supported: 64, 128", d_head);
  const int64_t dm = w_q_anchor->shape[1];
  for (int i = 1; i < 4; ++i)
    if (ws4[i]->shape[1] != dm) return fail(AOH_ERR_INVALID_ARG, "all weights need the same d_model");
  if (w_q_reuse->shape[0] != w_q_anchor->shape[0] || w_k_reuse->shape[0] != w_k_anchor->shape[0])
    return fail(AOH_ERR_INVALID_ARG, "anchor and reuse layers need the same head counts");
  if (w_q_anchor->shape[0] % d_head || w_k_anchor->shape[0] % d_head)
    return fail(AOH_ERR_INVALID_ARG, "rows of w_q / w_k must be a multiple of d_head");
  const int64_t Hq = w_q_anchor->shape[0] / d_head, Hkv = w_k_anchor->shape[0] / d_head;
  if (Hq % Hkv) return fail(AOH_ERR_UNSUPPORTED, "Hq=%lld is not a multiple of Hkv=%lld", (long long)Hq, (long long)Hkv);
  if (Hkv > kMaxKvHeads) return fail(AOH_ERR_UNSUPPORTED, "Hkv=%lld > %d", (long long)Hkv, kMaxKvHeads);
  if (Hq * Hq >= (1ll << 31)) return fail(AOH_ERR_UNSUPPORTED, "too many heads");
  if (dm % 64) return fail(AOH_ERR_UNSUPPORTED, "d_model=%lld must be a multiple of 64", (long long)dm);
  if (!head_sim || !group_sim || !mapping) return fail(AOH_ERR_INVALID_ARG, "null output pointer");
  if (reinterpret_cast<uintptr_t>(head_sim) % 8 || reinterpret_cast<uintptr_t>(group_sim) % 8)
    return fail(AOH_ERR_INVALID_ARG, "head_sim / group_sim must be 8-byte aligned");
  HeadSchedule ha, hr;
  if ((st = schedule_heads(anchor_is_streaming, (int)Hkv, &ha))) return st;
  if ((st = schedule_heads(reuse_is_streaming, (int)Hkv, &hr))) return st;
  if (ha.n_ret == 0) return fail(AOH_ERR_INVALID_ARG, "the anchor layer has no retrieval group");
  const size_t need = mapping_ws(Hq, Hkv, d_head);
  if (!workspace) return fail(AOH_ERR_WORKSPACE, "workspace is null; %zu bytes needed", need);
  if (workspace_bytes_given < need)
    return fail(AOH_ERR_WORKSPACE, "workspace has %zu bytes; %zu needed", workspace_bytes_given, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(AOH_ERR_INVALID_ARG, "workspace must be 16-byte aligned");

  SimilarityArgs a;
  std::memset(&a, 0, sizeof(a));
  a.wq_a = w_q_anchor->data; a.wk_a = w_k_anchor->data; a.wq_r = w_q_reuse->data; a.wk_r = w_k_reuse->data;
  a.wq_a_sr = w_q_anchor->stride[0]; a.wk_a_sr = w_k_anchor->stride[0];
  a.wq_r_sr = w_q_reuse->stride[0]; a.wk_r_sr = w_k_reuse->stride[0];
  a.Hq = (int)Hq; a.Hkv = (int)Hkv; a.gs = (int)(Hq / Hkv); a.d_model = (int)dm;
  char* w = reinterpret_cast<char*>(workspace);
  a.gram = reinterpret_cast<float*>(w);
  w += align256((size_t)(2 * (Hq + Hkv) * d_head * d_head) * sizeof(float));
  a.kx = reinterpret_cast<float*>(w);
  w += align256((size_t)(Hkv * Hkv * d_head * d_head) * sizeof(float));
  a.num = reinterpret_cast<double*>(w);
  w += align256((size_t)(Hq * Hq) * sizeof(double));
  a.n2 = reinterpret_cast<double*>(w);
  a.head_sim = head_sim; a.group_sim = group_sim; a.mapping = mapping;
  a.anchor_streaming = ha.streaming_mask; a.reuse_streaming = hr.streaming_mask;
  hipError_t e = launch_similarity(a, d_head, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(AOH_ERR_HIP, "head mapping launch: %s", hipGetErrorString(e));
  return ok();
}

static size_t classify_ws(int64_t L, int64_t hq, int64_t hkv, int64_t d) {
  const size_t gram = (size_t)(L * (hq + hkv) * d * d) * sizeof(float);
  return gram + (size_t)(L * hkv * d * d) * sizeof(double);
}

int32_t aoh_retrieval_group_count(int32_t n_kv_heads, double sparsity) {
  if (n_kv_heads < 1 || !(sparsity >= 0.0 && sparsity <= 1.0)) {
    fail(AOH_ERR_INVALID_ARG, "need n_kv_heads >= 1 and 0 <= sparsity <= 1");
    return -1;
  }
  // k = ceil((1 - s) G); the small offset keeps e.g. (1 - 0.7) * 10 = 3.0000000000000004 at 3
  const double x = (1.0 - sparsity) * n_kv_heads;
  return (int32_t)std::ceil(x - 1e-9 * n_kv_heads);
}

size_t aoh_classify_workspace_bytes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads, int32_t d_head) {
  if (n_layers < 1 || n_q_heads < 1 || n_kv_heads < 1 || (d_head != 64 && d_head != 128)) return 0;
  return classify_ws(n_layers, n_q_heads, n_kv_heads, d_head);
}

aoh_status aoh_classify(const aoh_tensor* w_q, const aoh_tensor* w_k, int32_t d_head, int32_t n_retrieval,
                        double* head_rank, double* group_score, uint8_t* head_is_streaming,
                        void* workspace, size_t workspace_bytes_given, void* stream) {
  aoh_status st;
  if ((st = check_tensor(w_q, "w_q", 3, AOH_BF16, AOH_BF16))) return st;
  if ((st = check_tensor(w_k, "w_k", 3, AOH_BF16, AOH_BF16))) return st;
  if (d_head != 64 && d_head != 128) return fail(AOH_ERR_UNSUPPORTED, "d_head=%d; supported: 64, 128", d_head);
  const int64_t L = w_q->shape[0], dm = w_q->shape[2];
  if (w_k->shape[0] != L || w_k->shape[2] != dm)
    return fail(AOH_ERR_INVALID_ARG, "w_q and w_k must have the same layers and d_model");
  if (w_q->shape[1] % d_head || w_k->shape[1] % d_head)
    return fail(AOH_ERR_INVALID_ARG, "rows of w_q / w_k must be a multiple of d_head");
  const int64_t Hq = w_q->shape[1] / d_head, Hkv = w_k->shape[1] / d_head;
  if (Hq % Hkv) return fail(AOH_ERR_UNSUPPORTED, "Hq=%lld is not a multiple of Hkv=%lld", (long long)Hq, (long long)Hkv);
  if (Hkv > kMaxKvHeads) return fail(AOH_ERR_UNSUPPORTED, "Hkv=%lld > %d", (long long)Hkv, kMaxKvHeads);
  if (dm % 64) return fail(AOH_ERR_UNSUPPORTED, "d_model=%lld must be a multiple of 64", (long long)dm);
  if (n_retrieval < 0 || n_retrieval > Hkv)
    return fail(AOH_ERR_INVALID_ARG, "n_retrieval=%d outside [0, %lld]", n_retrieval, (long long)Hkv);
  if (!head_rank || !group_score || !head_is_streaming)
    return fail(AOH_ERR_INVALID_ARG, "null output pointer");
  if (reinterpret_cast<uintptr_t>(head_rank) % 8 || reinterpret_cast<uintptr_t>(group_score) % 8)
    return fail(AOH_ERR_INVALID_ARG, "head_rank / group_score must be 8-byte aligned");
  if (L * (Hq + Hkv) >= (1ll << 31)) return fail(AOH_ERR_UNSUPPORTED, "too many layers");
  const size_t need = classify_ws(L, Hq, Hkv, d_head);
  if (!workspace) return fail(AOH_ERR_WORKSPACE, "workspace is null; %zu bytes needed", need);
  if (workspace_bytes_given < need)
    return fail(AOH_ERR_WORKSPACE, "workspace has %zu bytes; %zu needed", workspace_bytes_given, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 16) return fail(AOH_ERR_INVALID_ARG, "workspace must be 16-byte aligned");

  ClassifyArgs a;
  std::memset(&a, 0, sizeof(a));
  a.wq = w_q->data; a.wq_sl = w_q->stride[0]; a.wq_sr = w_q->stride[1];
  a.wk = w_k->data; a.wk_sl = w_k->stride[0]; a.wk_sr = w_k->stride[1];
  a.L = (int)L; a.Hq = (int)Hq; a.Hkv = (int)Hkv; a.gs = (int)(Hq / Hkv);
  a.d_model = (int)dm; a.n_retrieval = n_retrieval;
  a.gram = reinterpret_cast<float*>(workspace);
  a.chol = reinterpret_cast<double*>(reinterpret_cast<char*>(workspace) +
                                     (size_t)(L * (Hq + Hkv) * d_head * d_head) * sizeof(float));
  a.head_rank = head_rank; a.group_score = group_score; a.head_is_streaming = head_is_streaming;
  hipError_t e = launch_classify(a, d_head, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(AOH_ERR_HIP, "classify launch: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
