/*
 * aoh.h -- C interface of libaoh: head-mixed attention for Autonomy-of-Heads
 * (AoH) on AMD Instinct MI355X (gfx950).
 *
 * The method (paper: "Autonomy-of-Heads: Data-Free Sparse Attention from Frozen
 * Query-Key Geometry") labels every KV group of a layer as a retrieval group or
 * a streaming group (Sec. 4, group-level classification; Appendix "GQA
 * Extension").  At inference, retrieval heads attend to the whole causal
 * prefix and keep an O(T) KV cache; streaming heads keep only s_sink sink
 * tokens and s_recent recent tokens (Sec. 5, decode stage and chunked-prefill
 * stage).  The two outputs are concatenated along the head axis in the
 * original head order (Sec. 5, Eq. 8).  This library computes that attention
 * -- the softmax(Q K^T / sqrt(d)) V of each head under its mask -- for a batch
 * of prefills and for single-token decode steps, and maintains the two caches.
 *
 * Conventions common to every call
 *   - Q, K and V arrive after any positional encoding; no scale other than
 *     1/sqrt(D) is applied.
 *   - GQA: query head h reads KV head g = h / (Hq / Hkv) (contiguous groups).
 *   - head_is_streaming is a HOST array of Hkv bytes (0 = retrieval,
 *     1 = streaming); the label is per KV group and every query head of the
 *     group inherits it.
 *   - Streaming mask: key j is visible to the query at position i when
 *     j <= i and (j < n_sink or i - j < window).  The window includes the
 *     current token, so a streaming query sees at most n_sink + window keys.
 *     aoh_prefill applies this per-token sink + band mask to every row (the
 *     chunk-size-independent form of the paper's chunked eviction, and what
 *     decode sees); aoh_prefill_chunked applies the chunk-eviction form with a
 *     given chunk size.  Retrieval mask: j <= i.
 *   - Supported: dtype bf16 (fp32 accumulation and softmax) or fp32
 *     (fp32 throughout); D in {64, 128}; Hq a multiple of Hkv with
 *     Hq / Hkv <= 16; Hkv <= 64.  n_sink >= 0, window >= 1.
 *   - Every device pointer is owned by the caller.  The library allocates no
 *     device memory, performs no host<->device copy and no synchronisation in
 *     these calls, and keeps no pointer after returning.  All work is enqueued
 *     on `stream` (a hipStream_t; NULL = the default stream), in order.
 *   - Errors: arguments are validated before anything is enqueued; on any
 *     non-OK status nothing was launched and aoh_last_error() returns a
 *     message (thread-local, valid until the next call on the same thread).
 *     A failed launch returns AOH_ERR_HIP.  Faults inside a kernel surface at
 *     the caller's next synchronisation.  No C++ exception crosses this
 *     interface.
 *   - Calls are thread-safe; calls that write the same cache or workspace
 *     concurrently race, as any two kernels writing one buffer would.
 *   - The prefill calls (aoh_prefill, aoh_prefill_chunked, aoh_prefill_append,
 *     aoh_prefill_varlen) hand the streaming items of their one-launch form
 *     (both head types in one kernel, at d_head 128) out through work-queue
 *     counters in the library's own device memory (a static array per GPU,
 *     not an allocation): each such launch takes the next of 64 counter slots
 *     and leaves it cleared when it ends.  Prefill launches may run at the
 *     same time on different streams unless 64 others were enqueued between
 *     them; a prefill launch captured in a HIP graph must not run at the same
 *     time as another replay of that graph.
 */
#ifndef AOH_H_
#define AOH_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AOH_OK = 0,
  AOH_ERR_INVALID_ARG = 1, /* null pointer, inconsistent shapes, bad strides */
  AOH_ERR_UNSUPPORTED = 2, /* valid request outside the supported set above */
  AOH_ERR_HIP = 3,         /* a HIP runtime call or kernel launch failed */
  AOH_ERR_WORKSPACE = 4    /* decode workspace missing or too small */
} aoh_status;

typedef enum { AOH_BF16 = 0, AOH_F32 = 1 } aoh_dtype;

/* Tokens per page of the paged cache and per block of the ring cache. */
#define AOH_PAGE_TOKENS 16

/*
 * A strided dense tensor in device memory.  Strides are in elements; the last
 * dimension must have stride 1.  Unused trailing shape/stride entries are
 * ignored.
 */
typedef struct {
  void* data;
  int32_t dtype; /* aoh_dtype */
  int32_t ndim;
  int64_t shape[4];
  int64_t stride[4];
} aoh_tensor;

/*
 * Paged cache of the retrieval KV heads (the paper's O(T) cache, Sec. 5).
 * Only retrieval KV heads are stored, indexed by rank r = position of the head
 * among the retrieval KV heads in ascending KV-head id, so resident KV shrinks
 * with the streaming fraction.  Token p of sequence b lives in physical page
 * block_table[b * max_pages_per_seq + p / 16], row p % 16.  Layouts
 * (contiguous, dtype = the call's dtype):
 *   k: [num_pages][n_heads][16][D]   token-major inside a page
 *   v: [num_pages][n_heads][D][16]   dimension-major inside a page, or, with
 *      v_token_major = 1, [num_pages][n_heads][16][D] like k
 * block_table is a DEVICE int32 array [n_seqs][max_pages_per_seq]; the caller
 * allocates pages and fills it for every page a call touches.  A call with B
 * sequences requires n_seqs >= B (AOH_ERR_INVALID_ARG otherwise), so no row
 * outside the table is ever read.
 * Token-major V pages are for the caches of H2Share reuse layers, which are
 * only read at scattered borrowed positions: aoh_kv_append writes them and
 * aoh_decode_reuse reads them (a borrowed token's V is then one contiguous
 * row instead of a column spread over its page); aoh_decode, aoh_decode_step,
 * aoh_decode_anchor and the prefill calls that fill caches return
 * AOH_ERR_UNSUPPORTED for them.
 */
typedef struct {
  void* k;
  void* v;
  const int32_t* block_table;
  int64_t num_pages;
  int32_t max_pages_per_seq;
  int32_t n_heads;
  int32_t n_seqs;        /* rows of block_table */
  int32_t v_token_major; /* 0: dimension-major V pages; 1: token-major */
} aoh_paged_cache;

/*
 * Ring cache of the streaming KV heads: the paper's fixed sink + recent cache
 * (Sec. 5; 128 + 256 tokens in its experiments).  capacity must equal
 * n_sink + window; storage is padded to Cpad = capacity rounded up to a
 * multiple of 16 slots.  Token p goes to slot p if p < n_sink, else to
 * n_sink + (p - n_sink) % window; slot c lives in block c / 16, row c % 16.
 * Layouts (contiguous, rank s among the streaming KV heads):
 *   k: [B][n_heads][Cpad/16][16][D]
 *   v: [B][n_heads][Cpad/16][D][16]
 * After any sequence of appends each slot holds the token of greatest
 * position that maps to it.  A call with B sequences requires batch >= B
 * (AOH_ERR_INVALID_ARG otherwise), so no write leaves the ring.
 */
typedef struct {
  void* k;
  void* v;
  int32_t n_heads;
  int32_t capacity;
  int32_t batch; /* sequences the ring holds (its first dimension) */
} aoh_ring_cache;

/*
 * Head-mixed causal prefill (Sec. 5 chunked-prefill stage; Appendix H2Share
 * "Inference Phase", prefill).  For every batch b, query head h and position i
 * of the prompt:
 *   out[b,i,h,:] = sum_{j visible} softmax_j(q[b,i,h,:] . k[b,j,g,:] / sqrt(D)) v[b,j,g,:]
 * with g = h / (Hq/Hkv) and the mask of g's type.
 *   q:   [B][T][Hq][D]   k, v: [B][T][Hkv][D]   out: [B][T][Hq][D]
 * q, k, v share one dtype; out has the same dtype, or fp32 for bf16 inputs.
 * T may be any value >= 1 (a ragged last tile is handled); B >= 1.
 * Streaming heads only visit the sink tiles and the diagonal band of tiles;
 * tiles outside the mask are never loaded.
 */
aoh_status aoh_prefill(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                       const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                       aoh_tensor* out, void* stream);

/*
 * Prefill with the paper's chunk eviction for streaming heads (Sec. 5,
 * chunked-prefill stage): the prompt is processed in chunks of `chunk` tokens
 * and after each chunk a streaming head keeps only its n_sink sink tokens and
 * its `window` most recent tokens.  A query at position i, in the chunk that
 * starts at c = (i / chunk) * chunk, therefore sees the keys j <= i with
 * j < n_sink or j >= c - window.  Retrieval heads are unaffected.  Arguments,
 * layouts and errors as aoh_prefill; chunk >= 1 (chunk = 1 equals the per-token
 * band of aoh_prefill with window + 1).
 */
aoh_status aoh_prefill_chunked(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                               const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                               int32_t chunk, aoh_tensor* out, void* stream);

/*
 * Prefill of a new prompt that also fills the caches (Sec. 5: the prefill stage
 * leaves retrieval heads with their O(T) K/V states and streaming heads with
 * their sink + recent cache).  Output as aoh_prefill (chunk = 0) or
 * aoh_prefill_chunked (chunk >= 1); in addition the prompt's K/V occupy
 * positions 0..T-1 of every sequence b, written exactly as
 * aoh_kv_append(k, v, head_is_streaming, start_pos = 0, kv_full, kv_ring, ...)
 * would write them (bit-exact; the paged cache needs pages mapped for
 * positions 0..T-1).  For bf16 the prefill kernels write the caches from the
 * K/V tiles they already stage, so the prompt's K/V are read once; fp32 runs
 * the append as a separate launch.  Errors as aoh_prefill and aoh_kv_append.
 */
aoh_status aoh_prefill_append(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                              const uint8_t* head_is_streaming, int32_t n_sink, int32_t window,
                              int32_t chunk, const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                              aoh_tensor* out, void* stream);

/*
 * Prefill of a batch of prompts of different lengths packed along the token
 * axis (no padding): sequence b is rows cu_seqlens[b] .. cu_seqlens[b+1]-1 of
 *   q: [total][Hq][D]   k, v: [total][Hkv][D]   out: [total][Hq][D]
 * and attends only within itself (positions restart at 0).  Each sequence's
 * rows are computed exactly as by aoh_prefill (chunk = 0) or
 * aoh_prefill_chunked (chunk >= 1) on that sequence alone.
 *   cu_seqlens: DEVICE int32 [batch + 1], non-decreasing, cu_seqlens[0] = 0,
 *     cu_seqlens[batch] <= total (entries are clamped into [0, total]).
 *   max_seqlen: HOST bound on every sequence length; it sizes the grid (rows
 *     past it are not computed), so the call reads nothing back from the device.
 * With kv_full or kv_ring given, the prompts' K/V are also written to the
 * caches as aoh_prefill_append does (sequence b into block-table row b / ring
 * row b, positions 0..len_b-1; bf16 only).  Errors as aoh_prefill.
 */
aoh_status aoh_prefill_varlen(const aoh_tensor* q, const aoh_tensor* k, const aoh_tensor* v,
                              const int32_t* cu_seqlens, int32_t batch, int32_t max_seqlen,
                              const uint8_t* head_is_streaming, int32_t n_sink, int32_t window, int32_t chunk,
                              const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring, aoh_tensor* out,
                              void* stream);

/*
 * Append n_new tokens per sequence to the caches (Sec. 5: retrieval heads
 * retain every token; streaming heads evict all but the sink and recent
 * tokens).  Token t of k_new/v_new has position start_pos[b] + t.
 *   k_new, v_new: [B][n_new][Hkv][D]; start_pos: DEVICE int32 [B] (the
 *   sequence length before the append).
 * Retrieval KV heads are written to kv_full, streaming KV heads to kv_ring;
 * either cache may be NULL when no head of its type exists.  Copies are
 * bit-exact.  The paged cache must have pages mapped for every position
 * written.  Only the last window tokens of a bulk append (and any sink
 * positions) are written to the ring, so the result does not depend on
 * write order.
 */
aoh_status aoh_kv_append(const aoh_tensor* k_new, const aoh_tensor* v_new,
                         const uint8_t* head_is_streaming, const int32_t* start_pos,
                         const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                         int32_t n_sink, int32_t window, void* stream);

/*
 * Device workspace (bytes) that aoh_decode needs for its split-K partial
 * results, for a batch of `batch` sequences, Hq query heads of width d_head,
 * a paged cache of max_pages_per_seq pages per sequence and a ring of
 * ring_capacity slots.  Returns 0 for invalid arguments.
 */
size_t aoh_decode_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t d_head,
                                  int32_t max_pages_per_seq, int32_t ring_capacity);

/*
 * One single-token decode step (Sec. 5 decode stage, Eq. 8): for each
 * sequence b and query head h, with the query at position lens[b] - 1,
 *   out[b,h,:] = Attn(q[b,h,:], cache of KV group g)
 * where a retrieval group's cache holds tokens 0..lens[b]-1 and a streaming
 * group's ring holds its sink and recent tokens.  The step's own K/V must have
 * been appended already (lens counts it).
 *   q: [B][Hq][D]; out: [B][Hq][D] (dtype of q, or fp32 for bf16 q);
 *   lens: DEVICE int32 [B], 1 <= lens[b] <= 16 * max_pages_per_seq.
 * The grid is sized from the cache capacity, never from lens, so the host
 * reads nothing back and the call can be captured in a HIP graph.
 * workspace: DEVICE buffer of at least aoh_decode_workspace_bytes(...) bytes,
 * owned by the caller; its contents are scratch.
 */
aoh_status aoh_decode(const aoh_tensor* q, const aoh_paged_cache* kv_full,
                      const aoh_ring_cache* kv_ring, const uint8_t* head_is_streaming,
                      const int32_t* lens, int32_t n_sink, int32_t window, aoh_tensor* out,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Fused decode step (Sec. 5 decode stage, Eq. 8, with the cache policy of the
 * same section): the result and the final caches equal those of
 * aoh_kv_append of the step's token at start_pos = lens[b] - 1 followed by
 * aoh_decode with the same lens, bit for bit.
 *   k_new, v_new: [B][Hkv][D], dtype of q, the key / value of the token at
 *   position lens[b] - 1; the other arguments as for aoh_decode (lens counts
 *   the new token; the workspace is sized by aoh_decode_workspace_bytes).
 * bf16: one launch fewer than the two calls; the decode wave that reads the
 * token's page (ring block) writes the token there first.  This needs the
 * page of position lens[b] - 1 to be referenced by no other block-table entry
 * read in the call (pages are not shared across sequences at the write
 * position), which paged serving guarantees by copy-on-write.  fp32: the two
 * operations run as separate launches.
 * Errors: as aoh_decode, plus AOH_ERR_INVALID_ARG for a null or misshapen
 * k_new / v_new.
 */
aoh_status aoh_decode_step(const aoh_tensor* q, const aoh_tensor* k_new, const aoh_tensor* v_new,
                           const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                           const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                           int32_t window, aoh_tensor* out, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * aoh_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same call without a workspace argument.  The split-K partials go to a
 * static 64 MiB device array of the library (one per GPU, held until the
 * process ends); this call allocates nothing and calls no allocating routine.
 * Results and caches are bit-identical to aoh_decode_step.
 * Errors: as aoh_decode_step; AOH_ERR_UNSUPPORTED when the step would need
 * more than 64 MiB of workspace (aoh_decode_workspace_bytes > 64 MiB, e.g. a
 * batch far above 8 x 131072 tokens at 32 query heads of width 128);
 * AOH_ERR_HIP when the array's device address cannot be obtained.  All calls
 * on one GPU share its array, which keeps the last call's contents: calls
 * that overlap on one GPU (other streams, other threads) race and must be
 * serialised by the caller.
 */
aoh_status aoh_decode_step_noalloc(const aoh_tensor* q, const aoh_tensor* k_new, const aoh_tensor* v_new,
                                   const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                                   const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                                   int32_t window, aoh_tensor* out, void* stream);

/*
 * ---------------------------------------------------------------- H2Share
 * AoH-guided cross-layer sparse attention (paper section "AoH-Guided Sparse
 * Attention: H2Share" and its Inference Phase; GQA appendix, group-level head
 * mapping).  Layers are grouped into blocks; the first layer of a block (the
 * anchor) runs full attention for its retrieval heads and selects, per
 * retrieval KV group, the top_k token positions of highest attention; the
 * other layers of the block (reuse layers) let each retrieval group attend
 * only to its OWN K/V at the positions selected by its mapped anchor group.
 * Only integer positions cross layers.  Streaming groups use sink + window in
 * every layer.  Readings taken where the paper is open: a group's selection
 * score is the mean over its query heads of the attention probabilities of
 * the step; ties go to the lower position; selection happens on every step.
 */

/*
 * Offline head mapping between an anchor layer and a reuse layer (Eq. sim,
 * evaluated in d_head space by the trace identities of the trace-reduction
 * appendix):
 *   head_sim[h][h'] = <M_h, M_h'>_F / (|M_h|_F |M_h'|_F),  M_h = W_K^g^T W_Q^h,
 *   group_sim[g][g'] = mean of head_sim over the query heads of g and g',
 *   mapping[g'] = rank (among the anchor's retrieval groups, ascending id) of
 *                 the anchor retrieval group g maximising group_sim[g][g']
 *                 (lower g on ties); -1 for streaming reuse groups.
 *   w_q_*: [Hq * d_head][d_model] bf16, w_k_*: [Hkv * d_head][d_model] bf16,
 *   DEVICE, one layer each (PyTorch Linear layout), same shapes in both layers;
 *   d_head in {64, 128}; d_model a multiple of 64; Hkv <= 64.
 *   anchor_is_streaming, reuse_is_streaming: HOST, Hkv bytes; the anchor needs
 *   at least one retrieval group.
 *   head_sim: DEVICE double [Hq][Hq]; group_sim: DEVICE double [Hkv][Hkv];
 *   mapping: DEVICE int32 [Hkv] (all written).
 *   workspace: DEVICE, aoh_head_mapping_workspace_bytes(Hq, Hkv, d_head) bytes.
 */
size_t aoh_head_mapping_workspace_bytes(int32_t n_q_heads, int32_t n_kv_heads, int32_t d_head);
aoh_status aoh_head_mapping(const aoh_tensor* w_q_anchor, const aoh_tensor* w_k_anchor,
                            const aoh_tensor* w_q_reuse, const aoh_tensor* w_k_reuse, int32_t d_head,
                            const uint8_t* anchor_is_streaming, const uint8_t* reuse_is_streaming,
                            double* head_sim, double* group_sim, int32_t* mapping, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Anchor-layer decode step: exactly aoh_decode (same arguments, same out),
 * and in addition, for every sequence b and the r-th retrieval KV group g
 * (ascending id), indices[b][r][0..top_k) = the top_k positions p < lens[b]
 * of highest score sum_{h in g} P_h(p) / (Hq/Hkv), P_h the attention
 * probabilities of query head h in this step, in ascending order; when
 * lens[b] <= top_k every position, then -1.  The ranking uses each score as
 * the decode pass keeps it: rounded to 2^-11 log2 units (each P_h within
 * 1.7e-4 of its relative value; equal scores stay equal) and stored as a
 * 16-bit distance below the rounded maximum of its 32-token chunk, which
 * saturates just under 32 units, so probabilities below ~2^-32 of their
 * chunk's maximum rank as that bound (at most 2.3e-10 of the head's
 * probability mass: only such positions can trade places).  The group's
 * score is ranked with 13 mantissa bits (within 1.2e-4 of its value); equal
 * ranked scores go to the lower position.
 *   indices: DEVICE int32 [B][n_retrieval_groups][top_k]; top_k >= 1; bf16 only.
 *   workspace: aoh_decode_anchor_workspace_bytes(B, Hq, D, max_pages, ring_capacity).
 */
size_t aoh_decode_anchor_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t d_head,
                                         int32_t max_pages_per_seq, int32_t ring_capacity);
aoh_status aoh_decode_anchor(const aoh_tensor* q, const aoh_paged_cache* kv_full,
                             const aoh_ring_cache* kv_ring, const uint8_t* head_is_streaming,
                             const int32_t* lens, int32_t n_sink, int32_t window, int32_t top_k,
                             int32_t* indices, aoh_tensor* out, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * Reuse-layer decode step: streaming groups as aoh_decode; retrieval group g
 * (query heads of g) attends to this layer's own cache at the positions
 * indices[b][mapping[g]][0..top_k) (entries < 0 or >= lens[b] are skipped):
 *   out[b,h,:] = sum_{p in list} softmax_p(q[b,h] . k[b,p,g] / sqrt(D)) v[b,p,g].
 *   indices: DEVICE int32 [B][n_lists][top_k] (an anchor step's output);
 *   mapping: HOST int32 [Hkv], list row for each retrieval group (as written
 *   by aoh_head_mapping), ignored for streaming groups.
 *   Lists are expected in the anchor's form: valid entries first (the first
 *   min(lens[b], top_k)).  bf16 only.
 *   workspace: aoh_decode_reuse_workspace_bytes(B, Hq, D, top_k, ring_capacity).
 */
size_t aoh_decode_reuse_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t d_head, int32_t top_k,
                                        int32_t ring_capacity);
aoh_status aoh_decode_reuse(const aoh_tensor* q, const aoh_paged_cache* kv_full,
                            const aoh_ring_cache* kv_ring, const uint8_t* head_is_streaming,
                            const int32_t* lens, int32_t n_sink, int32_t window, const int32_t* indices,
                            int32_t n_lists, int32_t top_k, const int32_t* mapping, aoh_tensor* out,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * The AoH head classifier (Sec. 4, Eqs. 2-7 and Algorithm 1; group-level
 * classification in the "GQA Extension" appendix).  It is offline work: it
 * produces the head_is_streaming arrays that the calls above take.
 *
 * For query head h of layer l, with KV group g = h / (Hq/Hkv), the score is
 * the effective rank of the kernel attention matrix M_h = W_K^g^T W_Q^h:
 *   sigma_k = sqrt(max(lambda_k((W_Q W_Q^T)(W_K W_K^T)), 0)),
 *   p_k = sigma_k / sum_j sigma_j,  eff_rank = exp(-sum_{p_k > 0} p_k log p_k).
 * A group's score is the mean of its query heads' scores; in every layer the
 * n_retrieval groups with the lowest scores are retrieval groups (0), the rest
 * streaming (1).  On equal scores the lower group index is taken first, so
 * exactly n_retrieval groups are retrieval (the paper's k = ceil((1 - s) G)
 * for a target sparsity s is the caller's choice of n_retrieval).
 *
 *   w_q: [L][Hq * d_head][d_model] bf16, DEVICE; query head h owns rows
 *        h*d_head .. h*d_head + d_head - 1 of each layer (PyTorch Linear
 *        weight layout: output features x input features).
 *   w_k: [L][Hkv * d_head][d_model] bf16, DEVICE; group g owns rows likewise.
 *   d_head in {64, 128}; d_model a multiple of 64; Hq a multiple of Hkv;
 *   Hkv <= 64; 0 <= n_retrieval <= Hkv.
 *   head_rank:         DEVICE double [L][Hq]   (written)
 *   group_score:       DEVICE double [L][Hkv]  (written)
 *   head_is_streaming: DEVICE uint8  [L][Hkv]  (written, 0/1)
 *   workspace: DEVICE, at least aoh_classify_workspace_bytes(L, Hq, Hkv,
 *   d_head) bytes, 16-byte aligned, caller-owned scratch.
 * The Gram matrices W W^T are formed from the bf16 weights with fp32
 * accumulation; everything after them is fp64.  Errors as for the calls above.
 */
size_t aoh_classify_workspace_bytes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads, int32_t d_head);

/*
 * Retrieval groups per layer for a target sparsity s in [0, 1]:
 * k = ceil((1 - s) G) (Sec. 4, group-level classification), with products
 * that land within 1e-9 G above an integer rounded down to it.  Returns -1 for
 * invalid arguments (message in aoh_last_error).
 */
int32_t aoh_retrieval_group_count(int32_t n_kv_heads, double sparsity);

aoh_status aoh_classify(const aoh_tensor* w_q, const aoh_tensor* w_k, int32_t d_head, int32_t n_retrieval,
                        double* head_rank, double* group_score, uint8_t* head_is_streaming,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* aoh_last_error(void);

/* Interface version: 100 * major + minor. */
int32_t aoh_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AOH_H_ */
