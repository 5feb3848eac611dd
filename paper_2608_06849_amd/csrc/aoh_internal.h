// Kernel argument blocks and launchers shared by the host layer (abi.cpp) and
// the kernel translation units.  Arguments travel by value in kernargs: the
// head lists produced by the scheduling pass are small fixed arrays, so no
// device memory is needed to describe a launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aoh {

constexpr int kMaxKvHeads = 64;
constexpr int kPageTokens = 16;  // tokens per cache page / ring block

// One prefill launch covers every query head of the KV heads in kv_heads[]
// (all of one type).  Work item = (batch, query head, 128-row query block).
struct PrefillArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  int64_t q_sb, q_st, q_sh;
  int64_t k_sb, k_st, k_sh;
  int64_t v_sb, v_st, v_sh;
  int64_t o_sb, o_st, o_sh;
  int32_t B, T, gs;      // gs = query heads per KV head; T = the longest sequence (varlen)
  // Packed variable-length batch: sequence b is rows cu_seqlens[b] ..
  // cu_seqlens[b+1] - 1 of the tensors (token stride *_st; *_sb unused);
  // nullptr for the dense [B][T] layout.  total = rows of the tensors.
  const int32_t* cu_seqlens;
  int32_t total;
  int32_t seq_major;     // varlen: visit sequences in order (heaviest block first in each)
  int32_t n_kv;          // KV heads in this launch
  int32_t n_sink, window;
  int32_t chunk;         // streaming mask: 0 = per-token band, K >= 1 = chunk eviction
  int32_t n_qblocks;     // ceil(T / rows per block)
  float scale_log2;      // log2(e) / sqrt(D)
  float scale;           // 1 / sqrt(D)
  // Fused append of the prompt (positions 0..T-1) into this launch's cache:
  // the paged cache for the retrieval launch, the ring for the streaming one.
  // The cache rank of kv_heads[j] is j.
  int32_t append;
  void* ck;
  void* cv;
  const int32_t* block_table;   // paged cache only
  int32_t max_pages, num_pages; // paged cache only
  int32_t n_cache;              // KV heads stored in the cache
  int32_t ring_blocks;          // ring only: Cpad / 16
  uint8_t kv_heads[kMaxKvHeads];
};

// One cache type as seen by the decode split pass.  Work item = (batch, KV
// head of the list, split of split_blocks 16-token blocks).
struct CacheView {
  const void* k;
  const void* v;
  const int32_t* block_table;   // paged cache only (nullptr for the ring)
  int32_t max_pages;            // paged: pages per sequence row of block_table
  int32_t num_pages;            // paged: physical pages (entries outside are never read)
  int32_t ring_blocks;          // ring: Cpad / 16
  int32_t n_kv;                 // KV heads of this type (= heads stored in the cache)
  int32_t split_blocks;         // 16-token blocks per split
  int32_t n_splits;             // splits per (batch, KV head)
  int32_t n_groups;             // workgroups per (batch, KV head): ceil(n_splits / kSplitWaves)
  int32_t n_items;              // workgroups of the launch: B * n_kv * n_groups
  int32_t v_token_major;        // paged: V pages [16][D] (read by the reuse layer only)
  uint8_t kv_heads[kMaxKvHeads];  // KV head ids; rank in the cache = index here
};

// Anchor score codes: scores rounded to 2^-11 log2 units (a probability moves
// by at most 2^(2^-12) - 1 < 1.7e-4 of itself); the 16-bit code saturates just
// under 32 log2 units below the reference, so probabilities below ~2^-32 of
// their chunk's maximum all read as that bound.
constexpr float kScoreCodeScale = 2048.f;

// The decode split launch: paged-cache work items first (long), ring work items
// after them (short, they fill the tail of the launch).
struct DecodeArgs {
  const void* q;
  int64_t q_sb, q_sh;
  const int32_t* lens;
  float* part_acc;              // [B][Hq][max_splits][D]
  float* part_ml;               // [B][Hq][max_splits][2]  (m in log2 units, l)
  int32_t B, Hq, gs;
  int32_t ring_cap;             // n_sink + window
  int32_t max_splits;
  // > 0: the work-space split pass (decode_ws_kernel) with 2 * ws_cu
  // workgroups; part_acc / part_ml then hold [slot][gs][D] / [slot][gs][2],
  // and ws_items [B * Hkv][2] each item's first partial slot and count.
  int32_t ws_cu;
  int32_t* ws_items;
  float scale_log2;
  float scale;
  CacheView full;
  CacheView ring;
  // Anchor layer (H2Share): the scaled scores (log2 units) of the paged-cache
  // heads for positions < lens, rounded to multiples of 1 / kScoreCodeScale,
  // each as a 16-bit distance below a reference: score = ref - code /
  // kScoreCodeScale, with codes [B][Hq][score_len] and one reference per
  // 16-token block, refs [B][Hq][score_len / 16] (the rounded maximum of the
  // 32-token chunk the block was scored in).  Distances of 65535 steps and
  // more saturate at 65535.
  uint16_t* score_codes;
  float* score_refs;
  uint16_t* code_dummy;         // 64 x 8 codes written by lanes without a query head
  float* ref_dummy;             // 64 references written by those lanes
  int32_t score_len;
  // Reuse layer (H2Share): paged-cache items attend to borrowed positions
  // sel[b][sel_rank[j]][0..n_sel) (ascending, -1 = none) of KV head j of the
  // list, in chunks of split_blocks * 16 list entries per split.
  const int32_t* sel;
  int32_t n_sel, n_lists;
  uint8_t sel_rank[kMaxKvHeads];
  // Fused decode step: the key / value of the token at position lens - 1,
  // [B][Hkv][D], written into its cache slot by the one wave that reads it.
  const void* k_new;
  const void* v_new;
  int64_t kn_sb, kn_sh, vn_sb, vn_sh;
  int32_t n_sink, window;
};

struct MergeArgs {
  const float* part_acc;
  const float* part_ml;
  const int32_t* lens;
  void* out;
  int64_t o_sb, o_sh;
  int32_t B, Hq, gs;
  int32_t max_splits;
  int32_t n_splits_full;        // partials written per (b, head), paged cache
  int32_t n_splits_ring;        // partials written per (b, head), ring
  int32_t max_len;              // 16 * pages per sequence: lens are clamped to it
  int32_t ring_cap;
  // > 0: partials of the work-space split pass (DecodeArgs::ws_cu) over
  // ws_n_ret paged KV heads and ws_n_str rings, located through ws_items.
  int32_t ws_cu, ws_n_ret, ws_n_str;
  const int32_t* ws_items;
  uint64_t streaming_mask;      // bit g set = KV head g streaming
  float* ml_out;                // anchor layer: final (m, l) of each paged-cache head, [B][Hq][2]
};

struct AppendArgs {
  const void* k_new;
  const void* v_new;
  int64_t k_sb, k_st, k_sh;
  int64_t v_sb, v_st, v_sh;
  const int32_t* start_pos;     // device [B]; nullptr: every sequence starts at 0
  int32_t start_bias;           // added to start_pos[b] (-n_new: start_pos holds the end)
  int32_t B, n_new, Hkv;
  // paged cache
  void* pk;
  void* pv;
  const int32_t* block_table;
  int32_t max_pages;
  int32_t num_pages;
  int32_t n_ret;
  int32_t v_token_major;        // V pages [16][D] instead of [D][16]
  // ring cache
  void* rk;
  void* rv;
  int32_t n_str;
  int32_t ring_blocks;
  int32_t n_sink, window;
  int32_t n_chunks;             // 16-position chunks launched per (b, head)
  uint64_t streaming_mask;
  uint8_t rank[kMaxKvHeads];    // rank of each KV head inside its cache
};

// The head classifier over L layers.  Weights are bf16 [L][H * D][d_model]
// slices (layer stride *_sl, row stride *_sr, unit column stride).
struct ClassifyArgs {
  const void* wq;
  const void* wk;
  int64_t wq_sl, wq_sr;
  int64_t wk_sl, wk_sr;
  int32_t L, Hq, Hkv, gs;
  int32_t d_model;             // multiple of 64
  int32_t n_retrieval;         // retrieval groups per layer
  float* gram;                 // workspace [L][Hq + Hkv][D][D]
  double* chol;                // workspace [L][Hkv][D][D]
  double* head_rank;           // [L][Hq]
  double* group_score;         // [L][Hkv]
  uint8_t* head_is_streaming;  // [L][Hkv]
};

// Launchers (return the launch status; no synchronisation).
hipError_t launch_prefill(const PrefillArgs& a, int dtype, int out_f32, int d, bool streaming,
                          hipStream_t s);
// One launch for a layer with both head types (bf16, d_head 128, short
// retrieval launches; see prefill.hip).
bool prefill_mixed_preferred(const PrefillArgs& ar, int dtype, int d);
hipError_t launch_prefill_mixed(const PrefillArgs& ar, const PrefillArgs& as, int out_f32, hipStream_t s);
// mode: 0 plain, 1 anchor (also writes scores), 2 reuse (sparse paged items)
hipError_t launch_decode_split(const DecodeArgs& a, int d, int mode, hipStream_t s);
hipError_t launch_decode_merge(const MergeArgs& a, int dtype, int out_f32, int d, hipStream_t s);
hipError_t launch_decode_f32(const DecodeArgs& a, int d, void* out, int64_t o_sb, int64_t o_sh, hipStream_t s);
hipError_t launch_append(const AppendArgs& a, int dtype, int d, hipStream_t s);
hipError_t launch_classify(const ClassifyArgs& a, int d, hipStream_t s);

// Top-k selection of an anchor decode step (H2Share): per (sequence, paged
// KV head j of the list), the n_sel positions of highest group-mean attention
// probability, ascending, padded with -1.
struct TopkArgs {
  const uint16_t* score_codes;  // [B][Hq][score_len] (DecodeArgs::score_codes)
  const float* score_refs;      // [B][Hq][score_len / 16]
  uint32_t* keys;               // [B][n_kv][score_len] ranking keys of the lists
  const float* ml;              // [B][Hq][2] final (m, l)
  const int32_t* lens;
  int32_t* sel;                 // [B][n_kv][n_sel]
  int32_t B, Hq, gs, n_kv;
  int32_t score_len;            // positions per row (16 * pages per sequence)
  int32_t n_sel;
  uint32_t* part;               // [B][n_kv][kTopkPasses][kTopkParts][2048] partial histograms
  uint8_t kv_heads[kMaxKvHeads];
};
constexpr int kTopkParts = 8;   // workgroups per (sequence, KV head) list
constexpr int kTopkPasses = 2;  // 11-bit digits of the 22-bit ranking keys
hipError_t launch_topk(const TopkArgs& a, hipStream_t s);

// Cross-layer head similarity (H2Share): grams of both layers are in gram
// ([2][Hq + Hkv][D][D]: anchor, reuse), KX[g][g'] = W_K^g W_K'^g'^T in kx,
// num[h][h'] = <W_Q^h W_Q'^h'^T, KX[g(h)][g(h')]>_F.
struct SimilarityArgs {
  const void* wq_a; const void* wk_a; const void* wq_r; const void* wk_r;
  int64_t wq_a_sr, wk_a_sr, wq_r_sr, wk_r_sr;   // row strides
  int32_t Hq, Hkv, gs, d_model;
  float* gram;
  float* kx;                    // [Hkv][Hkv][D][D]
  double* num;                  // [Hq][Hq]
  double* n2;                   // [2][Hq] squared Frobenius norms (anchor, reuse)
  double* head_sim;             // [Hq][Hq] out
  double* group_sim;            // [Hkv][Hkv] out
  int32_t* mapping;             // [Hkv] out: anchor retrieval rank, -1 for streaming reuse groups
  uint64_t anchor_streaming, reuse_streaming;
};
hipError_t launch_similarity(const SimilarityArgs& a, int d, hipStream_t s);

// Largest number of splits per (sequence, head) the merge pass accepts.
constexpr int kMaxSplits = 1024;
// Decode split pass: waves per workgroup, one split each; the workgroup merges
// its waves' partial results in LDS and writes one partial per group.
constexpr int kSplitWaves = 4;
// Fixed decode splits: ~kDecodeTargetWaves paged waves (8 per CU), and ring
// waves up to kRingTargetWaves by the rings' share of the work.
constexpr int kDecodeTargetWaves = 2048;
constexpr int kRingTargetWaves = 4096;
// Work-space decode split pass: batches of up to kWsMaxBatch sequences (one
// lane per sequence), at most kWsMaxWgs workgroups (two per CU), so at most
// that many partials per item for the merge pass.
constexpr int kWsMaxBatch = 64;
constexpr int kWsMaxWgs = 512;

// Query rows per bf16 prefill workgroup, and 32-row MFMA blocks per wave
// (the workgroup has kPrefillRows / (32 * kPrefillRB) waves).
constexpr int kPrefillRB = 1;
constexpr int kPrefillRows = 256;
constexpr int kPrefillRowsF32 = 64;

// Host layer (abi.cpp) services for entry points defined in other units.
// The aoh_* types come from aoh.h, which the including unit includes first.
#ifdef AOH_H_
aoh_status decode_step_workspace_need(const aoh_tensor* q, const aoh_tensor* k_new, const aoh_tensor* v_new,
                                      const aoh_paged_cache* kv_full, const aoh_ring_cache* kv_ring,
                                      const uint8_t* head_is_streaming, const int32_t* lens, int32_t n_sink,
                                      int32_t window, aoh_tensor* out, size_t* need);
// Sets the thread's last-error text for a status (clears it for AOH_OK) and returns the status.
aoh_status report(aoh_status st, const char* msg);
#endif

}  // namespace aoh
