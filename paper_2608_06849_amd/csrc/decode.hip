// Single-token decode over the two caches (paper Sec. 5, decode stage, Eq. 8).
//
// Split-K ("flash-decoding") structure:
//   pass 1 (decode_split): one wave per (sequence, KV head, split of the
//     cache).  The wave reads the split's K/V once for the whole GQA group and
//     keeps fp32 partial results (running max m, sum l, unnormalised acc[D])
//     for every query head of the group.  Four consecutive splits share a
//     workgroup, which merges their partials in LDS and writes one.
//   pass 2 (decode_merge): per (sequence, query head), log-sum-exp merge of
//     the partials of the splits that hold tokens, normalise, store in the
//     caller's head order.
//
// bf16 pass 1 works on chunks of 32 tokens = two 16-token cache blocks with
// v_mfma_f32_16x16x32_bf16:
//   S^T[16 tokens x 16 heads] = K[16 x 32 dims] . Q^T  (x2 token blocks, D/32 k-steps)
//   O^T[16 dims x 16 heads]  += V^T[16 dims x 32 tokens] . P^T   (D/16 dim blocks)
// Query heads of the group sit in the 16 MFMA columns (group size <= 16), so
// softmax statistics are per lane column.  Lane group G = lane / 16 holds,
// for both token blocks, chunk tokens 8G..8G+7, which makes the P^T operand
// lane-local and lets the V^T operand be one 16-byte load from the
// dimension-major V page ([D][16] per page).  K rows are read with 16-byte
// loads covering 64 contiguous bytes per token row per instruction.
#include "aoh_device.h"
#include "aoh_internal.h"

namespace aoh {

// Folds one 32-token chunk (token blocks c and c + 1 of the cache row; tokens
// at or past tok_end masked, none of them at or past blk_end * 16 kept as a
// score) into a wave's running softmax state: K rows in kcur, the V^T operand
// in vcur (zeroed where masked), Q^T in qreg.
template <int D, bool SCORES>
__device__ __forceinline__ void fold_chunk(const DecodeArgs& a, const u32x4 (&kcur)[2][D / 32],
                                           u32x4 (&vcur)[D / 16], const bf16x8 (&qreg)[D / 32], int c, int tok_end,
                                           int blk_end, bool head_ok, uint16_t* code_row, float* ref_row,
                                           f32x4 (&acc)[D / 16], float& m_run, float& l_run) {
  constexpr int kKSteps = D / 32;
  constexpr int kDimBlocks = D / 16;
  const int lane = threadIdx.x & (kWave - 1);
  const int G = lane >> 4;
  // S^T for the two 16-token blocks.
  f32x4 sc[2];
#pragma unroll
  for (int X = 0; X < 2; ++X) {
    sc[X] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kKSteps; ++s) sc[X] = mfma16(__builtin_bit_cast(bf16x8, kcur[X][s]), qreg[s], sc[X]);
  }
  // This lane's 8 scores: chunk tokens 8G + j, j = 4X + i.
  const int tok0 = c * kPage + 8 * G;
  const bool partial = (c * kPage + 2 * kPage) > tok_end;
  float x[8];
  float mx = -INFINITY;
#pragma unroll
  for (int X = 0; X < 2; ++X)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = sc[X][i] * a.scale_log2;
      if (partial && tok0 + 4 * X + i >= tok_end) v = -INFINITY;
      x[4 * X + i] = v;
      mx = fmaxf(mx, v);
    }
  mx = wave_xor_max(mx, 16);
  mx = wave_xor_max(mx, 32);
  if (SCORES) {
    // Anchor layer: keep the scaled scores for the top-k selection.  Each
    // score is rounded to the code grid (kScoreCodeScale steps per log2 unit)
    // and kept as its 16-bit distance below the grid point of the chunk's
    // maximum for this head, which is the reference of each of the chunk's two
    // blocks; a kept score therefore reads back as its own grid point
    // whatever chunk it was scored in (equal scores stay equal), unless its
    // distance saturates.  Masked positions (beyond the valid length, never
    // read by the selection) saturate.  Every lane issues the same stores in
    // every chunk (a fixed count, so the compiler's wait for the prefetched
    // chunk stays exact): lanes without a query head, and lanes whose tokens
    // lie past the range's last block (the missing second block of a range
    // with an odd block count, which at the end of a full row would be the
    // next row's first positions), write to a dummy area.
    const bool keep = head_ok && tok0 < blk_end * kPage;
    // grid points are integer-valued floats; mx is one of the scores, so
    // every distance is >= 0; -inf scores give +inf, clamped before the
    // conversion
    const float top = rintf(mx * kScoreCodeScale);
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo = (uint32_t)fminf(top - rintf(x[2 * j] * kScoreCodeScale), 65535.f);
      const uint32_t hi = (uint32_t)fminf(top - rintf(x[2 * j + 1] * kScoreCodeScale), 65535.f);
      w[j] = lo | (hi << 16);
    }
    uint16_t* cp = keep ? code_row + tok0 : a.code_dummy + 8 * lane;
    *reinterpret_cast<u32x4*>(cp) = u32x4{w[0], w[1], w[2], w[3]};
    // lane groups 0 and 2 start the chunk's two blocks
    if ((G & 1) == 0) *(keep ? ref_row + tok0 / kPage : a.ref_dummy + lane) = top * (1.f / kScoreCodeScale);
  }
  const float m_new = fmaxf(m_run, mx);  // finite: every chunk holds a valid token
  const float alpha = fast_exp2(m_run - m_new);
  m_run = m_new;
  bf16x8 pop;
  float psum = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float p = fast_exp2(x[j] - m_new);
    psum += p;
    pop[j] = f32_to_bf16(p);
  }
  l_run = l_run * alpha + psum;
  if (partial) {
    // Slots past the valid range may hold stale or uninitialised data: zero
    // their V so 0 * garbage cannot poison the product.
#pragma unroll
    for (int nb = 0; nb < kDimBlocks; ++nb) {
      bf16x8 vv = __builtin_bit_cast(bf16x8, vcur[nb]);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (tok0 + j >= tok_end) vv[j] = (bf16)0.f;
      vcur[nb] = __builtin_bit_cast(u32x4, vv);
    }
  }
#pragma unroll
  for (int nb = 0; nb < kDimBlocks; ++nb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[nb][i] *= alpha;
    acc[nb] = mfma16(__builtin_bit_cast(bf16x8, vcur[nb]), pop, acc[nb]);
  }
}

// Blocks [blk0, blk_lim) of the cache row of (sequence b, KV head kvl) for
// one wave (blk0 even in the row or at the start of a workgroup's share); its
// partial results (unnormalised acc, running max m in log2 units, sum l) are
// left in acc / m_out / l_out (unchanged when the split holds no token).
template <int D, bool RING, bool SCORES = false, bool APPEND = false>
__device__ __forceinline__ void decode_split_body(const DecodeArgs& a, const CacheView& cv, int b, int kvl,
                                                  int len, int blk0, int blk_lim, f32x4 (&acc)[D / 16],
                                                  float& m_out, float& l_out) {
  constexpr int kKSteps = D / 32;   // 32-dim k-steps for Q K^T
  constexpr int kDimBlocks = D / 16;
  const int g = cv.kv_heads[kvl];
  const int rank = kvl;
  const int lane = threadIdx.x & (kWave - 1);
  const int col = lane & 15;   // query head within the group (MFMA column)
  const int G = lane >> 4;     // lane group

  // Lengths beyond the cache capacity are clamped so no read leaves the cache.
  const int n_valid = RING ? min(len, a.ring_cap) : min(len, cv.max_pages * kPage);
  const int n_blocks_valid = (n_valid + kPage - 1) / kPage;
  const int blk_end = min(blk_lim, n_blocks_valid);
  if (blk0 >= blk_end) return;
  const int tok_end = min(n_valid, blk_end * kPage);

  // Q^T operand: column = query head g*gs + col (zero beyond the group).
  const bool head_ok = col < a.gs;
  const int hq = g * a.gs + col;
  bf16x8 qreg[kKSteps];
  {
    const uint16_t* qp = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)b * a.q_sb + (int64_t)hq * a.q_sh;
#pragma unroll
    for (int s = 0; s < kKSteps; ++s) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (head_ok) x = ld16(qp + 32 * s + 8 * G);
      qreg[s] = __builtin_bit_cast(bf16x8, x);
    }
  }

  const uint16_t* kc = reinterpret_cast<const uint16_t*>(cv.k);
  const uint16_t* vc = reinterpret_cast<const uint16_t*>(cv.v);
  // Cache unit of a block: ring block, or the page of the block table (an
  // invalid entry reads page 0, never outside the cache).
  auto unit_of = [&](int entry) -> int64_t {
    if (RING) return ((int64_t)b * cv.n_kv + rank) * cv.ring_blocks + entry;
    const int page = (entry < 0 || entry >= cv.num_pages) ? 0 : entry;
    return (int64_t)page * cv.n_kv + rank;
  };
  // Block-table entries of the two blocks of chunk c (block ids for the ring);
  // they are fetched one chunk ahead of their use, so waiting for them never
  // waits for anything issued later (the score stores of the anchor layer).
  auto fetch_entries = [&](int c, int (&e)[2]) {
    const int c1 = min(c + 1, blk_end - 1);  // a chunk's second block may not exist
    if (RING) {
      e[0] = c;
      e[1] = c1;
    } else {
      const int32_t* bt = cv.block_table + (int64_t)b * cv.max_pages;
      e[0] = bt[c];
      e[1] = bt[c1];  // two independent loads: nothing waits for the first
    }
  };

  // K row of MFMA row m = lane & 15 for token block X: chunk token
  // 8*(m/4) + 4X + (m%4), i.e. page (m/4)/2, row 8*((m/4)%2) + 4X + (m%4).
  const int m = lane & 15;
  const int k_half = (m >> 2) >> 1;           // 0: first page of the chunk, 1: second
  const int k_row0 = 8 * ((m >> 2) & 1) + (m & 3);
  // V^T operand: dim = 16*nb + (lane & 15), tokens 8G..8G+7 of the chunk.
  const int v_half = G >> 1;
  const int v_off = 8 * (G & 1);

  u32x4 kreg[2][kKSteps];
  u32x4 vreg[kDimBlocks];
  auto load_chunk = [&](const int (&e)[2]) {
    const int64_t kb = unit_of(e[k_half]) * (kPage * D);
    const int64_t vb = unit_of(e[v_half]) * (kPage * D);
#pragma unroll
    for (int X = 0; X < 2; ++X)
#pragma unroll
      for (int s = 0; s < kKSteps; ++s)
        kreg[X][s] = ld16_stream(kc + kb + (int64_t)(k_row0 + 4 * X) * D + 32 * s + 8 * G);
#pragma unroll
    for (int nb = 0; nb < kDimBlocks; ++nb)
      vreg[nb] = ld16_stream(vc + vb + (int64_t)(16 * nb + (lane & 15)) * kPage + v_off);
  };

  float m_run = -INFINITY;
  float l_run = 0.f;

  if (APPEND) {
    // Fused step: position lens - 1 receives the new key / value (ring: its
    // slot, sink positions kept, others modulo the window).  Its block lies in
    // exactly one split, and only the wave of that split reads the unit (page
    // or ring block) of this (sequence, KV head), so that wave stores the
    // token, waits for the stores, then streams its range as usual.  A block
    // beyond the table or an invalid page entry gets no write, as in a
    // separate append.
    const int p = len - 1;
    if (p >= 0) {
      const int slot = RING ? (p < a.n_sink ? p : a.n_sink + (p - a.n_sink) % a.window) : p;
      const int blk = slot / kPage, row = slot % kPage;
      if (blk >= blk0 && blk < blk_end) {
        int64_t unit = -1;
        if (RING) {
          unit = ((int64_t)b * cv.n_kv + rank) * cv.ring_blocks + blk;
        } else {
          const int page = cv.block_table[(int64_t)b * cv.max_pages + blk];
          if (page >= 0 && page < cv.num_pages) unit = (int64_t)page * cv.n_kv + rank;
        }
        if (unit >= 0) {
          const uint16_t* kn = reinterpret_cast<const uint16_t*>(a.k_new) + (int64_t)b * a.kn_sb + (int64_t)g * a.kn_sh;
          const uint16_t* vn = reinterpret_cast<const uint16_t*>(a.v_new) + (int64_t)b * a.vn_sb + (int64_t)g * a.vn_sh;
          uint16_t* kdst = const_cast<uint16_t*>(kc) + unit * (kPage * D) + (int64_t)row * D;
          uint16_t* vdst = const_cast<uint16_t*>(vc) + unit * (kPage * D) + row;
          if (lane < D / 8) st16(kdst + 8 * lane, ld16(kn + 8 * lane));
#pragma unroll
          for (int i = 0; i < D / kWave; ++i) vdst[(int64_t)(lane + kWave * i) * kPage] = vn[lane + kWave * i];
          // The stores must reach the cache before this wave's loads of it.
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
      }
    }
  }

  int ent[2];
  fetch_entries(blk0, ent);
  load_chunk(ent);
  if (blk0 + 2 < blk_end) fetch_entries(blk0 + 2, ent);
  for (int c = blk0; c < blk_end; c += 2) {
    u32x4 kcur[2][kKSteps];
    u32x4 vcur[kDimBlocks];
#pragma unroll
    for (int X = 0; X < 2; ++X)
#pragma unroll
      for (int s = 0; s < kKSteps; ++s) kcur[X][s] = kreg[X][s];
#pragma unroll
    for (int nb = 0; nb < kDimBlocks; ++nb) vcur[nb] = vreg[nb];
    if (c + 2 < blk_end) {
      load_chunk(ent);                                // chunk c + 2
      if (c + 4 < blk_end) fetch_entries(c + 4, ent);  // entries of chunk c + 4
    }

    fold_chunk<D, SCORES>(a, kcur, vcur, qreg, c, tok_end, blk_end, head_ok,
                          SCORES ? a.score_codes + ((int64_t)b * a.Hq + hq) * a.score_len : nullptr,
                          SCORES ? a.score_refs + ((int64_t)b * a.Hq + hq) * (a.score_len / kPage) : nullptr, acc,
                          m_run, l_run);
  }

  // Partial results of this split: m (log2 units), l, acc[D] for each head.
  float l_tot = wave_xor_sum(l_run, 16);
  l_tot = wave_xor_sum(l_tot, 32);
  m_out = m_run;
  l_out = l_tot;
}


// Reuse layer of H2Share: one wave per (sequence, paged KV head, split of its
// borrowed position list).  The same 16x16x32 MFMA structure as the dense
// body, on gathered tokens: each lane loads the K rows of its two MFMA rows
// from their own pages (16-byte loads), and the V^T operand element by
// element (the 8 tokens of a lane group are in general on 8 different pages).
// With dimension-major V pages every element sits in its own 32-byte sector;
// with token-major ones the 16 lanes of a group read 32 contiguous bytes of
// one token's row per load.  List entries < 0 or beyond the sequence are
// masked out.
template <int D>
__device__ __forceinline__ void decode_sparse_body(const DecodeArgs& a, const CacheView& cv, int b, int kvl,
                                                   int split, f32x4 (&acc)[D / 16], float& m_out, float& l_out) {
  constexpr int kKSteps = D / 32;
  constexpr int kDimBlocks = D / 16;
  const int g = cv.kv_heads[kvl];
  const int lane = threadIdx.x & (kWave - 1);
  const int col = lane & 15;
  const int G = lane >> 4;
  const int len = a.lens[b];
  const int n_valid = min(len, cv.max_pages * kPage);
  const int split_len = cv.split_blocks * kPage;
  const int e0 = split * split_len;
  const int e_end = min(e0 + split_len, a.n_sel);
  if (e0 >= e_end) return;
  const int32_t* list = a.sel + ((int64_t)b * a.n_lists + a.sel_rank[kvl]) * a.n_sel;

  const bool head_ok = col < a.gs;
  const int hq = g * a.gs + col;
  bf16x8 qreg[kKSteps];
  {
    const uint16_t* qp = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)b * a.q_sb + (int64_t)hq * a.q_sh;
#pragma unroll
    for (int s = 0; s < kKSteps; ++s) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (head_ok) x = ld16(qp + 32 * s + 8 * G);
      qreg[s] = __builtin_bit_cast(bf16x8, x);
    }
  }
  const uint16_t* kc = reinterpret_cast<const uint16_t*>(cv.k);
  const uint16_t* vc = reinterpret_cast<const uint16_t*>(cv.v);
  // cache unit of a position (page of the block table); invalid -> unit 0
  auto unit_of = [&](int pos) -> int64_t {
    if (pos < 0 || pos >= n_valid) return 0;
    int page = cv.block_table[(int64_t)b * cv.max_pages + pos / kPage];
    page = (page < 0 || page >= cv.num_pages) ? 0 : page;
    return (int64_t)page * cv.n_kv + kvl;
  };
  const int m = lane & 15;
  const int slot_k0 = 8 * (m >> 2) + (m & 3);  // chunk slot of MFMA row m, token block 0 (+4 for block 1)

  float m_run = -INFINITY;
  float l_run = 0.f;

  for (int c0 = e0; c0 < e_end; c0 += 32) {
    // the chunk's 32 list entries, one per lane of the low half
    const int my_e = c0 + (lane & 31);
    const int my_pos = my_e < e_end ? list[my_e] : -1;
    u32x4 kcur[2][kKSteps];
#pragma unroll
    for (int X = 0; X < 2; ++X) {
      const int pos = __shfl(my_pos, slot_k0 + 4 * X, kWave);
      const int64_t kb = unit_of(pos) * (kPage * D) + (int64_t)((pos < 0 ? 0 : pos) % kPage) * D;
#pragma unroll
      for (int s = 0; s < kKSteps; ++s) kcur[X][s] = ld16(kc + kb + 32 * s + 8 * G);
    }
    int vpos[8];
    bool vok[8];
    int64_t vb[8];
    // element (token row r, dimension d) of a V page: r + 16 d (dimension-major)
    // or D r + d (token-major)
    const int v_row = cv.v_token_major ? D : 1;
    const int v_dim = cv.v_token_major ? 1 : kPage;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      vpos[j] = __shfl(my_pos, 8 * G + j, kWave);
      vok[j] = vpos[j] >= 0 && vpos[j] < n_valid;
      vb[j] = unit_of(vpos[j]) * (kPage * D) + (vok[j] ? vpos[j] % kPage : 0) * v_row;
    }
    bf16x8 vcur[kDimBlocks];
#pragma unroll
    for (int nb = 0; nb < kDimBlocks; ++nb)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint16_t raw = vc[vb[j] + (int64_t)(16 * nb + (lane & 15)) * v_dim];
        vcur[nb][j] = vok[j] ? __builtin_bit_cast(bf16, raw) : (bf16)0.f;
      }

    f32x4 sc[2];
#pragma unroll
    for (int X = 0; X < 2; ++X) {
      sc[X] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < kKSteps; ++s) sc[X] = mfma16(__builtin_bit_cast(bf16x8, kcur[X][s]), qreg[s], sc[X]);
    }
    float x[8];
    float mx = -INFINITY;
#pragma unroll
    for (int X = 0; X < 2; ++X)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 4 * X + i;  // chunk slot 8G + j
        float v = sc[X][i] * a.scale_log2;
        if (!vok[j]) v = -INFINITY;
        x[j] = v;
        mx = fmaxf(mx, v);
      }
    mx = wave_xor_max(mx, 16);
    mx = wave_xor_max(mx, 32);
    const float m_new = fmaxf(m_run, mx);
    if (m_new == -INFINITY) continue;  // no valid entry in this chunk (wave-uniform)
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    bf16x8 pop;
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = fast_exp2(x[j] - m_new);
      psum += p;
      pop[j] = f32_to_bf16(p);
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int nb = 0; nb < kDimBlocks; ++nb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[nb][i] *= alpha;
      acc[nb] = mfma16(vcur[nb], pop, acc[nb]);
    }
  }

  float l_tot = wave_xor_sum(l_run, 16);
  l_tot = wave_xor_sum(l_tot, 32);
  m_out = m_run;
  l_out = l_tot;
}

// One launch for both cache types: paged-cache items first, ring items last.
// MODE 0: plain decode; 1: anchor layer (paged items also keep their scores);
// 2: reuse layer (paged items attend to borrowed positions only); 3: plain
// decode that first stores the new token at position lens - 1 (fused step).
// A workgroup holds kSplitWaves consecutive splits of one (sequence, KV
// head), one per wave; the waves' partials are merged in LDS (log-sum-exp
// weights, as in the merge pass) and the group writes one partial, so the
// merge pass reads kSplitWaves times fewer.  Each wave then combines a share
// of the dimension blocks.
// The kSplitWaves waves' partial states (acc, m in log2 units, l) merged in
// LDS with log-sum-exp weights; lane (col, G) holds query head col of the
// group, and each wave writes a share of the dimension blocks of the merged
// partial to row `row` of part_acc / part_ml (lanes with lane_ok).  A wave
// without tokens has m = -inf and weight 0; if no wave has tokens the row gets
// m = -inf (the merge pass never reads such a row).  Starts with a barrier so
// a workgroup can call it once per segment.
template <int D>
__device__ __forceinline__ void merge_waves_store(const DecodeArgs& a, f32x4 (&acc)[D / 16], float m, float l,
                                                  f32x4 (*s_acc)[D / 16][kWave], float (*s_m)[kWave],
                                                  float (*s_l)[kWave], bool lane_ok, int64_t row) {
  constexpr int kDimBlocks = D / 16;
  static_assert(kDimBlocks % kSplitWaves == 0, "dimension blocks split evenly over the waves");
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  __syncthreads();
#pragma unroll
  for (int nb = 0; nb < kDimBlocks; ++nb) s_acc[wave][nb][lane] = acc[nb];
  s_m[wave][lane] = m;
  s_l[wave][lane] = l;
  __syncthreads();
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kSplitWaves; ++w) M = fmaxf(M, s_m[w][lane]);
  float wt[kSplitWaves];
  float L = 0.f;
#pragma unroll
  for (int w = 0; w < kSplitWaves; ++w) {
    const float mw = s_m[w][lane];
    wt[w] = (mw == -INFINITY) ? 0.f : fast_exp2(mw - M);
    L += wt[w] * s_l[w][lane];
  }
  if (lane_ok) {
    const int G = lane >> 4;
    float* pa = a.part_acc + row * D;
#pragma unroll
    for (int k = 0; k < kDimBlocks / kSplitWaves; ++k) {
      const int nb = wave * (kDimBlocks / kSplitWaves) + k;
      f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < kSplitWaves; ++w) {
        const f32x4 x = s_acc[w][nb][lane];
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] += wt[w] * x[i];
      }
      *reinterpret_cast<f32x4*>(pa + 16 * nb + 4 * G) = o;
    }
    if (wave == 0 && G == 0) {
      a.part_ml[row * 2 + 0] = M;
      a.part_ml[row * 2 + 1] = L;
    }
  }
}

// Fixed splits from the cache capacity (batches over kWsMaxBatch sequences,
// and the reuse layer).  One launch for both cache types: paged-cache items
// first, ring items last.  MODE 0: plain decode; 1: anchor layer (paged items
// also keep their scores); 2: reuse layer (paged items attend to borrowed
// positions only); 3: plain decode that first stores the new token at
// position lens - 1 (fused step).  A workgroup holds kSplitWaves consecutive
// splits of one (sequence, KV head), one per wave, and writes one merged
// partial, so the merge pass reads kSplitWaves times fewer.
template <int D, int MODE>
__global__ __launch_bounds__(kSplitWaves * kWave, 2) void decode_split_bf16_kernel(DecodeArgs a) {
  constexpr int kDimBlocks = D / 16;
  __shared__ f32x4 s_acc[kSplitWaves][kDimBlocks][kWave];
  __shared__ float s_m[kSplitWaves][kWave];
  __shared__ float s_l[kSplitWaves][kWave];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  int wg = blockIdx.x;
  const bool ring = wg >= a.full.n_items;
  if (ring) wg -= a.full.n_items;
  const CacheView& cv = ring ? a.ring : a.full;
  const int sg = wg % cv.n_groups;
  const int rest = wg / cv.n_groups;
  const int kvl = rest % cv.n_kv;
  const int b = rest / cv.n_kv;
  const int split = sg * kSplitWaves + wave;
  const int blk0 = split * cv.split_blocks;

  f32x4 acc[kDimBlocks];
#pragma unroll
  for (int nb = 0; nb < kDimBlocks; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  if (split < cv.n_splits) {
    const int len = a.lens[b];
    if (ring)
      decode_split_body<D, true, false, MODE == 3>(a, a.ring, b, kvl, len, blk0, blk0 + cv.split_blocks, acc, m, l);
    else if (MODE == 2)
      decode_sparse_body<D>(a, a.full, b, kvl, split, acc, m, l);
    else
      decode_split_body<D, false, MODE == 1, MODE == 3>(a, a.full, b, kvl, len, blk0, blk0 + cv.split_blocks, acc,
                                                        m, l);
  }
  const int col = lane & 15;
  const int hq = cv.kv_heads[kvl] * a.gs + col;
  merge_waves_store<D>(a, acc, m, l, s_acc, s_m, s_l, col < a.gs,
                       ((int64_t)b * a.Hq + hq) * a.max_splits + sg);
}

// ---------------------------------------------------------------------------
// Split pass over the step's work space (bf16 plain, anchor and fused-step
// decode of up to kWsMaxBatch sequences).
//
// Work space: the valid 16-token blocks of every item (cache type, sequence,
// KV head) laid end to end, paged items first, each type in (sequence, KV
// head) order, so one plan covers any mix of lengths and of the two cache
// types.  Each workgroup takes one contiguous range of it and each of its
// waves a consecutive quarter of every item segment in that range; the waves'
// states are merged in LDS and the workgroup writes one partial per segment.
// The launch has two workgroups per CU: the first n_cu are placed one per CU,
// and a CU's second workgroup runs about a third slower (its waves lose issue
// arbitration on every SIMD to the older ones), so first-round ranges hold 4
// shares and second-round ranges 3, and both rounds end together.  Item i,
// covered by workgroups first_i..last_i, has its partials in slots
// first_i + i .. last_i + i (items are contiguous, so no two items share a
// slot): at most workgroups + items slots of gs heads each.
constexpr int kWsMinBlocks = 16;  // smallest range a workgroup takes

struct WsPlan {
  int nb_tot, nbr_tot;  // paged / ring blocks summed over the sequences
  int total;            // blocks of all items
  int n_old, n_young;   // workgroups of the first and second round
  int r_old, r_young;   // blocks per range of each round
  int g_young;          // first block of the second round's ranges
};

// The plan from the sequence lengths.  Every lane of a wave calls it; lane b
// gets sequence b's length, its valid block counts in the paged cache (nb)
// and the ring (nbr), and their exclusive prefix sums over the sequences
// (P, Q); lanes >= B get zeros.
__device__ __forceinline__ WsPlan ws_plan(const int32_t* lens, int B, int max_pages, int n_ret, int ring_cap,
                                          int n_str, int n_cu, int& len, int& nb, int& nbr, int& P, int& Q) {
  const int lane = threadIdx.x & (kWave - 1);
  len = 0;
  nb = 0;
  nbr = 0;
  if (lane < B) {
    len = lens[lane];
    const int l = max(len, 0);
    if (n_ret) nb = (min(l, max_pages * kPage) + kPage - 1) / kPage;
    if (n_str) nbr = (min(l, ring_cap) + kPage - 1) / kPage;
  }
  int ip = nb, iq = nbr;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int tp = __shfl_up(ip, o, kWave), tq = __shfl_up(iq, o, kWave);
    if (lane >= o) {
      ip += tp;
      iq += tq;
    }
  }
  P = ip - nb;
  Q = iq - nbr;
  WsPlan p;
  p.nb_tot = __builtin_amdgcn_readlane(ip, kWave - 1);
  p.nbr_tot = __builtin_amdgcn_readlane(iq, kWave - 1);
  p.total = n_ret * p.nb_tot + n_str * p.nbr_tot;
  const int n_wg = min(2 * n_cu, max(1, (p.total + kWsMinBlocks - 1) / kWsMinBlocks));
  p.n_old = min(n_wg, n_cu);
  p.n_young = n_wg - p.n_old;
  const int64_t weight = 4 * (int64_t)p.n_old + 3 * (int64_t)p.n_young;
  p.r_old = (int)((4 * (int64_t)p.total + weight - 1) / weight);
  p.g_young = min(p.total, p.n_old * p.r_old);
  p.r_young = p.n_young ? (p.total - p.g_young + p.n_young - 1) / p.n_young : 0;
  return p;
}

// Workgroup whose range holds block g (g < total).
__device__ __forceinline__ int ws_wg_of(int g, const WsPlan& p) {
  return g < p.g_young ? g / p.r_old : p.n_old + (g - p.g_young) / p.r_young;
}

// The item holding block g of the work space (g < total): its type, sequence,
// KV head rank, first block in the work space, valid blocks and item index.
struct WsItem {
  bool ring;
  int b, kvl, off, len, idx;
};

__device__ __forceinline__ WsItem ws_item(int g, const WsPlan& p, int B, int n_ret, int n_str, int nb, int nbr, int P,
                                          int Q) {
  const int lane = threadIdx.x & (kWave - 1);
  WsItem it;
  const int paged_end = n_ret * p.nb_tot;
  it.ring = g >= paged_end;
  const int heads = it.ring ? n_str : n_ret;
  const int blocks = it.ring ? nbr : nb;
  const int start = (it.ring ? paged_end : 0) + heads * (it.ring ? Q : P);
  const uint64_t hit = __ballot(lane < B && g >= start && g < start + heads * blocks);
  if (hit == 0) {  // not reached for g < total
    it.b = it.kvl = it.off = it.idx = it.len = 0;
    return it;
  }
  it.b = __builtin_amdgcn_readfirstlane((int)__builtin_ctzll(hit));
  const int first = __builtin_amdgcn_readlane(start, it.b);
  it.len = __builtin_amdgcn_readlane(blocks, it.b);
  it.kvl = (g - first) / it.len;
  it.off = first + it.kvl * it.len;
  it.idx = it.ring ? B * n_ret + it.b * n_str + it.kvl : it.b * n_ret + it.kvl;
  return it;
}

template <int D, int MODE>
__global__ __launch_bounds__(kSplitWaves * kWave, 2) void decode_ws_kernel(DecodeArgs a) {
  constexpr int kDimBlocks = D / 16;
  __shared__ f32x4 s_acc[kSplitWaves][kDimBlocks][kWave];
  __shared__ float s_m[kSplitWaves][kWave];
  __shared__ float s_l[kSplitWaves][kWave];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  int len_l, nb_l, nbr_l, P_l, Q_l;
  const WsPlan p = ws_plan(a.lens, a.B, a.full.max_pages, a.full.n_kv, a.ring_cap, a.ring.n_kv, a.ws_cu, len_l, nb_l,
                           nbr_l, P_l, Q_l);
  const int w = blockIdx.x;
  int g0, g1;
  if (w < p.n_old) {
    g0 = w * p.r_old;
    g1 = min(g0 + p.r_old, p.g_young);
  } else {
    g0 = p.g_young + (w - p.n_old) * p.r_young;
    g1 = w < p.n_old + p.n_young ? min(g0 + p.r_young, p.total) : g0;
  }
  for (int g = g0; g < g1;) {  // uniform: every wave walks the same segments
    const WsItem it = ws_item(g, p, a.B, a.full.n_kv, a.ring.n_kv, nb_l, nbr_l, P_l, Q_l);
    if (it.len == 0) break;
    const int s0 = g - it.off, s1 = min(g1 - it.off, it.len);
    const int len = __builtin_amdgcn_readlane(len_l, it.b);
    // This wave's consecutive quarter of the segment's 32-token chunks.
    const int per = ((s1 - s0 + 1) / 2 + kSplitWaves - 1) / kSplitWaves;
    const int c0 = min(s1, s0 + 2 * per * wave), c1 = min(s1, c0 + 2 * per);
    f32x4 acc[kDimBlocks];
#pragma unroll
    for (int nb = 0; nb < kDimBlocks; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m = -INFINITY, l = 0.f;
    if (c0 < c1) {
      if (it.ring) decode_split_body<D, true, false, MODE == 3>(a, a.ring, it.b, it.kvl, len, c0, c1, acc, m, l);
      else decode_split_body<D, false, MODE == 1, MODE == 3>(a, a.full, it.b, it.kvl, len, c0, c1, acc, m, l);
    }
    const int col = lane & 15;
    merge_waves_store<D>(a, acc, m, l, s_acc, s_m, s_l, col < a.gs, (int64_t)(w + it.idx) * a.gs + col);
    if (s0 == 0 && threadIdx.x == 0) {
      // The workgroup holding the item's first block records where the item's
      // partials are for the merge pass: first slot and count.
      a.ws_items[2 * it.idx + 0] = w + it.idx;
      a.ws_items[2 * it.idx + 1] = ws_wg_of(it.off + it.len - 1, p) - w + 1;
    }
    g = it.off + s1;
  }
}

// fp32 decode: one workgroup of 64 threads per (sequence, query head) of the
// listed KV heads; threads stride over the valid tokens, then combine through
// LDS.  Writes the final output directly (no split partials).
template <int D, bool RING>
__device__ __forceinline__ void decode_f32_body(const DecodeArgs& a, const CacheView& cv, int item, void* out,
                                                int64_t o_sb, int64_t o_sh) {
#pragma clang fp contract(off)
  __shared__ float sh_acc[kWave][D + 1];
  __shared__ float sh_m[kWave], sh_l[kWave];
  const int n_qh = cv.n_kv * a.gs;
  const int qhl = item % n_qh;
  const int b = item / n_qh;
  const int kvl = qhl / a.gs;
  const int g = cv.kv_heads[kvl];
  const int hq = g * a.gs + qhl % a.gs;
  const int t = threadIdx.x;
  const int len = a.lens[b];
  const int n_valid = RING ? min(len, a.ring_cap) : min(len, cv.max_pages * kPage);
  const float* qp = reinterpret_cast<const float*>(a.q) + (int64_t)b * a.q_sb + (int64_t)hq * a.q_sh;
  const float* kc = reinterpret_cast<const float*>(cv.k);
  const float* vc = reinterpret_cast<const float*>(cv.v);
  float q[D], o[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = qp[d];
    o[d] = 0.f;
  }
  float mrun = -INFINITY, lrun = 0.f;
  for (int tok = t; tok < n_valid; tok += kWave) {
    const int blk = tok / kPage, row = tok % kPage;
    int64_t unit;
    if (RING) {
      unit = ((int64_t)b * cv.n_kv + kvl) * cv.ring_blocks + blk;
    } else {
      int page = cv.block_table[(int64_t)b * cv.max_pages + blk];
      page = (page < 0 || page >= cv.num_pages) ? 0 : page;
      unit = (int64_t)page * cv.n_kv + kvl;
    }
    const float* kr = kc + unit * (kPage * D) + (int64_t)row * D;
    const float* vr = vc + unit * (kPage * D) + row;
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) s = fmaf(q[d], kr[d], s);
    s *= a.scale;
    const float mn = fmaxf(mrun, s);
    const float al = expf(mrun - mn);
    const float p = expf(s - mn);
    lrun = lrun * al + p;
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] = o[d] * al + p * vr[(int64_t)d * kPage];
    mrun = mn;
  }
  sh_m[t] = mrun;
  sh_l[t] = lrun;
#pragma unroll
  for (int d = 0; d < D; ++d) sh_acc[t][d] = o[d];
  __syncthreads();
  float mx = -INFINITY;
  for (int i = 0; i < kWave; ++i) mx = fmaxf(mx, sh_m[i]);
  float L = 0.f;
  for (int i = 0; i < kWave; ++i)
    if (sh_m[i] != -INFINITY) L += expf(sh_m[i] - mx) * sh_l[i];
  float* op = reinterpret_cast<float*>(out) + (int64_t)b * o_sb + (int64_t)hq * o_sh;
  for (int d = t; d < D; d += kWave) {
    float acc = 0.f;
    for (int i = 0; i < kWave; ++i)
      if (sh_m[i] != -INFINITY) acc += expf(sh_m[i] - mx) * sh_acc[i][d];
    op[d] = acc / L;
  }
}

// fp32 decode: one workgroup of 64 threads per (sequence, query head); threads
// stride over the valid tokens, then combine through LDS.  Writes the final
// output directly (no split partials).  Paged items first, ring items after.
template <int D>
__global__ __launch_bounds__(kWave) void decode_f32_kernel(DecodeArgs a, void* out, int64_t o_sb, int64_t o_sh) {
  const int wg = blockIdx.x;
  const int n_full = a.B * a.full.n_kv * a.gs;
  if (wg < n_full) decode_f32_body<D, false>(a, a.full, wg, out, o_sb, o_sh);
  else decode_f32_body<D, true>(a, a.ring, wg - n_full, out, o_sb, o_sh);
}

constexpr int kMergeDims = 32;      // output dimensions per merge workgroup
constexpr int kMergeThreads = 512;  // kMergeDims x 16 split groups
constexpr int kMergeGroups = kMergeThreads / kMergeDims;

// Log-sum-exp merge of the split partials of one (sequence, query head), for
// one slice of kMergeDims output dimensions.  Every load the workgroup needs
// (each partial's (m, l), and acc[d] of this slice for all partials, spread
// over 16 groups of 32 threads reading coalesced 128-byte rows) is issued up
// front, so the pass costs one round trip to memory; the statistics are then
// reduced in LDS and the weighted sums combined.
// Loads and log-sum-exp merge of ns partials (rows base + s * stride, at most
// kMergeGroups * PER_GROUP of them) for slice `slice` of (sequence b, query
// head hq), and the output store.
template <int D, bool OUT_F32, int PER_GROUP>
__device__ __forceinline__ void merge_partials(const MergeArgs& a, int b, int hq, int slice, bool streaming, int ns,
                                               int64_t base, int64_t stride, float* s_w, float* s_red,
                                               float (*s_acc)[kMergeDims]) {
  constexpr int kWaves = kMergeThreads / kWave;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int dd = tid % kMergeDims, grp = tid / kMergeDims;
  const int d = slice * kMergeDims + dd;

  // All loads first.
  float m = -INFINITY, l = 0.f;
  if (tid < ns) {
    m = a.part_ml[(base + tid * stride) * 2];
    l = a.part_ml[(base + tid * stride) * 2 + 1];
  }
  float av[PER_GROUP];
#pragma unroll
  for (int k = 0; k < PER_GROUP; ++k) {
    const int s = grp + kMergeGroups * k;
    av[k] = s < ns ? a.part_acc[(base + s * stride) * D + d] : 0.f;
  }

  float mloc = m;
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, o, kWave));
  if (lane == 0) s_red[wave] = mloc;
  __syncthreads();
  float mx = s_red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) mx = fmaxf(mx, s_red[i]);
  __syncthreads();
  const float w = tid < ns ? fast_exp2(m - mx) : 0.f;
  if (tid < ns) s_w[tid] = w;
  float lloc = w * l;
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) lloc += __shfl_xor(lloc, o, kWave);
  if (lane == 0) s_red[wave] = lloc;
  __syncthreads();
  float L = 0.f;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) L += s_red[i];

  float acc = 0.f;
#pragma unroll
  for (int k = 0; k < PER_GROUP; ++k) {
    const int s = grp + kMergeGroups * k;
    if (s < ns) acc += s_w[s] * av[k];
  }
  s_acc[grp][dd] = acc;
  __syncthreads();
  if (a.ml_out && !streaming && slice == 0 && tid == 0) {
    a.ml_out[((int64_t)b * a.Hq + hq) * 2 + 0] = mx;
    a.ml_out[((int64_t)b * a.Hq + hq) * 2 + 1] = L;
  }
  if (grp == 0) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kMergeGroups; ++i) tot += s_acc[i][dd];
    const float o = tot / L;
    if (OUT_F32) {
      reinterpret_cast<float*>(a.out)[(int64_t)b * a.o_sb + (int64_t)hq * a.o_sh + d] = o;
    } else {
      reinterpret_cast<uint16_t*>(a.out)[(int64_t)b * a.o_sb + (int64_t)hq * a.o_sh + d] = f32_to_bf16_bits(o);
    }
  }
}

template <int D, bool OUT_F32, bool WS>
__global__ __launch_bounds__(kMergeThreads) void decode_merge_kernel(MergeArgs a) {
  constexpr int kSlices = D / kMergeDims;
  // Partials per (sequence, head): fixed splits write up to kMaxSplits /
  // kSplitWaves, the work-space pass up to kWsMaxWgs (in practice no more than
  // that first bound unless an item spans most of the launch).
  constexpr int kFewPartials = kMaxSplits / kSplitWaves;
  constexpr int kMaxPartials = WS ? kWsMaxWgs : kFewPartials;
  static_assert(kFewPartials % kMergeGroups == 0 && kMaxPartials % kMergeGroups == 0, "merge covers every partial");
  static_assert(kMergeThreads >= kMaxPartials, "one (m, l) pair per thread");
  __shared__ float s_w[kMaxPartials];
  __shared__ float s_red[kMergeThreads / kWave];
  __shared__ float s_acc[kMergeGroups][kMergeDims];
  const int wg = blockIdx.x;
  const int slice = wg % kSlices;
  const int hq = (wg / kSlices) % a.Hq;
  const int b = wg / (kSlices * a.Hq);
  const int g = hq / a.gs;
  const bool streaming = (a.streaming_mask >> g) & 1ull;
  if constexpr (WS) {
    // Partials of the work-space split pass: the item's slots, as recorded by
    // the workgroup that held its first block (an item without valid blocks
    // has none and records nothing).
    const int len = a.lens[b];
    const int n_valid = streaming ? min(len, a.ring_cap) : min(len, a.max_len);
    const uint64_t below = (1ull << g) - 1;
    const int rank = __builtin_popcountll((streaming ? a.streaming_mask : ~a.streaming_mask) & below);
    const int idx = streaming ? a.B * a.ws_n_ret + b * a.ws_n_str + rank : b * a.ws_n_ret + rank;
    const int slot0 = a.ws_items[2 * idx + 0];
    const int ns = n_valid > 0 ? a.ws_items[2 * idx + 1] : 0;
    const int64_t base = (int64_t)slot0 * a.gs + (hq - g * a.gs);
    if (ns <= kFewPartials)
      merge_partials<D, OUT_F32, kFewPartials / kMergeGroups>(a, b, hq, slice, streaming, ns, base, a.gs, s_w, s_red,
                                                              s_acc);
    else
      merge_partials<D, OUT_F32, kMaxPartials / kMergeGroups>(a, b, hq, slice, streaming, ns, base, a.gs, s_w, s_red,
                                                              s_acc);
  } else {
    // Every split workgroup writes its partial, one without tokens m = -inf
    // (weight 0), so all of them are merged and the length is not needed.
    const int ns = streaming ? a.n_splits_ring : a.n_splits_full;
    merge_partials<D, OUT_F32, kFewPartials / kMergeGroups>(a, b, hq, slice, streaming, ns,
                                                            ((int64_t)b * a.Hq + hq) * a.max_splits, 1, s_w, s_red,
                                                            s_acc);
  }
}

template <int D>
static void launch_split_d(const DecodeArgs& a, int mode, int grid, hipStream_t s) {
  const dim3 blk(kSplitWaves * kWave);
  if (mode == 1) hipLaunchKernelGGL((decode_split_bf16_kernel<D, 1>), dim3(grid), blk, 0, s, a);
  else if (mode == 2) hipLaunchKernelGGL((decode_split_bf16_kernel<D, 2>), dim3(grid), blk, 0, s, a);
  else if (mode == 3) hipLaunchKernelGGL((decode_split_bf16_kernel<D, 3>), dim3(grid), blk, 0, s, a);
  else hipLaunchKernelGGL((decode_split_bf16_kernel<D, 0>), dim3(grid), blk, 0, s, a);
}

template <int D>
void launch_ws_d(const DecodeArgs& a, int mode, hipStream_t s) {
  const dim3 grid(2 * a.ws_cu), blk(kSplitWaves * kWave);
  if (mode == 1) hipLaunchKernelGGL((decode_ws_kernel<D, 1>), grid, blk, 0, s, a);
  else if (mode == 3) hipLaunchKernelGGL((decode_ws_kernel<D, 3>), grid, blk, 0, s, a);
  else hipLaunchKernelGGL((decode_ws_kernel<D, 0>), grid, blk, 0, s, a);
}

hipError_t launch_decode_split(const DecodeArgs& a, int d, int mode, hipStream_t s) {
  if (a.ws_cu) {
    if (d == 64) launch_ws_d<64>(a, mode, s);
    else launch_ws_d<128>(a, mode, s);
    return hipGetLastError();
  }
  const int grid = a.full.n_items + a.ring.n_items;
  if (d == 64) launch_split_d<64>(a, mode, grid, s);
  else launch_split_d<128>(a, mode, grid, s);
  return hipGetLastError();
}

hipError_t launch_decode_f32(const DecodeArgs& a, int d, void* out, int64_t o_sb, int64_t o_sh, hipStream_t s) {
  const int grid = a.B * (a.full.n_kv + a.ring.n_kv) * a.gs;
  if (d == 64) hipLaunchKernelGGL((decode_f32_kernel<64>), dim3(grid), dim3(kWave), 0, s, a, out, o_sb, o_sh);
  else hipLaunchKernelGGL((decode_f32_kernel<128>), dim3(grid), dim3(kWave), 0, s, a, out, o_sb, o_sh);
  return hipGetLastError();
}

template <int D, bool WS>
void launch_merge_d(const MergeArgs& a, int out_f32, int grid, hipStream_t s) {
  if (out_f32) hipLaunchKernelGGL((decode_merge_kernel<D, true, WS>), dim3(grid), dim3(kMergeThreads), 0, s, a);
  else hipLaunchKernelGGL((decode_merge_kernel<D, false, WS>), dim3(grid), dim3(kMergeThreads), 0, s, a);
}

hipError_t launch_decode_merge(const MergeArgs& a, int dtype, int out_f32, int d, hipStream_t s) {
  (void)dtype;
  const int grid = a.B * a.Hq * (d / kMergeDims);
  if (d == 64) {
    if (a.ws_cu) launch_merge_d<64, true>(a, out_f32, grid, s);
    else launch_merge_d<64, false>(a, out_f32, grid, s);
  } else {
    if (a.ws_cu) launch_merge_d<128, true>(a, out_f32, grid, s);
    else launch_merge_d<128, false>(a, out_f32, grid, s);
  }
  return hipGetLastError();
}

}  // namespace aoh
