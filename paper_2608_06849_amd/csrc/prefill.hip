// Head-mixed causal prefill on gfx950.
//
// Computes, per (batch, query head, query row i), the attention of the paper's
// Sec. 5 (chunked-prefill stage): softmax over the visible keys of
// q_i . k_j / sqrt(D), times V.  Retrieval heads see j <= i; streaming heads
// see j <= i with j < n_sink or j >= lo(i), where lo(i) = i - window + 1 for
// the per-token band and lo(i) = floor(i / K) K - window for chunk eviction
// with chunks of K tokens (the cache before a chunk keeps the sink and the
// window most recent tokens; the chunk sees those and itself).
//
// bf16 kernel (the hot one).  One workgroup = 4 waves = 128 query rows of one
// query head; each wave owns 32 rows.  Key/value tiles of 64 keys are staged
// in LDS and shared by the 4 waves.  Per tile and wave:
//   S^T[64 keys x 32 rows] = K_tile . Q^T        (v_mfma_f32_32x32x16_bf16)
//   online softmax in fp32, one query row per lane column, so the row max is a
//   lane-local reduction plus one exchange with the partner lane (lane ^ 32)
//   O^T[D x 32 rows] += V_tile^T . P^T           (same MFMA)
// P never leaves registers: the S^T accumulator layout is already the B
// operand layout of the P^T product.  V^T operands come straight out of the
// row-major V tile through the gfx950 LDS transpose read (ds_read_b64_tr_b16).
// Streaming heads iterate only over the sink tiles and the diagonal band of
// tiles; other tiles are never loaded.  Tiles that are fully visible skip the
// per-element mask.
//
// fp32 kernel: a plain per-row kernel (one thread per query row) kept exact
// for fp32 inputs; it has no performance role.
#include <type_traits>

#include "aoh_device.h"
#include "aoh_internal.h"

namespace aoh {

constexpr int kBN = 64;          // keys per tile
constexpr int kRB = kPrefillRB;                 // 32-row MFMA blocks per wave
constexpr int kRowsPerWave = 32 * kRB;
constexpr int kWaves = kPrefillRows / kRowsPerWave;  // waves per workgroup

#ifndef AOH_PREFILL_V_PAD
#define AOH_PREFILL_V_PAD 32
#endif
#ifndef AOH_PREFILL_STAGE_TILES
#define AOH_PREFILL_STAGE_TILES 1
#endif
// 64-key tiles per LDS stage (one barrier per stage).
constexpr int kStageTiles = AOH_PREFILL_STAGE_TILES;

template <int D>
struct PrefillLds {
  // Row paddings (bf16 elements): K rows are read 16 bytes per lane down 32
  // rows; V rows are read by the transpose read as 4 rows x 32 bytes per
  // 16 lanes.  Each padding spreads its access pattern over distinct banks.
  static constexpr int kStrideK = D + 8;
  static constexpr int kStrideV = D + AOH_PREFILL_V_PAD;
  uint16_t k[kBN * kStageTiles][kStrideK];
  uint16_t v[kBN * kStageTiles][kStrideV];
};

// Lazy rescaling threshold (log2 units): the running max used for the
// exponentials is only raised when a row's true max exceeds it by more than
// this, so P stays below 2^8 and the O rescale is skipped on most tiles.
constexpr float kRescaleThreshold = 8.0f;

// First non-sink key visible to row i of a streaming head (may be negative).
__device__ __forceinline__ int lo_of(int i, int chunk, int window) {
  return chunk ? (i / chunk) * chunk - window : i - window + 1;
}

// Tile visit plan of one query block [i0, i0 + kPrefillRows).
struct TilePlan {
  int n_sink_tiles;  // leading sink tiles visited before the band
  int band_first;    // first band tile
  int n_visit;       // total tiles
  __device__ __forceinline__ int tile(int it) const {
    return it < n_sink_tiles ? it : band_first + (it - n_sink_tiles);
  }
};

template <bool STREAM>
__device__ __forceinline__ TilePlan make_plan(int i0, int rows, int T, int n_sink, int window, int chunk) {
  const int last_row = min(i0 + rows - 1, T - 1);
  const int last_tile = last_row / kBN;
  TilePlan p;
  if (!STREAM) {
    p.n_sink_tiles = 0;
    p.band_first = 0;
    p.n_visit = last_tile + 1;
  } else {
    const int band_lo = max(0, lo_of(i0, chunk, window));  // lo is non-decreasing in i
    p.band_first = band_lo / kBN;
    const int sink_tiles = (n_sink + kBN - 1) / kBN;
    p.n_sink_tiles = min(sink_tiles, p.band_first);
    p.n_visit = p.n_sink_tiles + (last_tile - p.band_first + 1);
  }
  return p;
}

template <int D, bool STREAM, bool OUT_F32, bool APPEND>
__global__ __launch_bounds__(kWaves * kWave, kRB == 1 ? 2 : 1) void prefill_bf16_kernel(PrefillArgs a) {
  __shared__ __align__(16) PrefillLds<D> lds[2];
  constexpr int kChunksPerRow = D / 8;                     // 16-byte chunks per key row
  constexpr int kChunksPerThread = kBN * kChunksPerRow / (kWaves * kWave);
  constexpr int kKSteps = D / 16;                          // MFMA k-steps over D
  constexpr int kMBlocks = D / 32;                         // 32-dim blocks of O^T

  const int n_qh = a.n_kv * a.gs;
  const int per_block = n_qh * a.B;
  const int wg = blockIdx.x;
  // Heaviest query blocks first (longest-processing-time order) for causal work.
  int qb = a.n_qblocks - 1 - wg / per_block;
  const int rem = wg % per_block;
  int qh_local = rem % n_qh;
  int b = rem / n_qh;
  if (a.seq_major) {
    // Packed batch, sequence-major: the workgroups in flight share one or two
    // sequences' K/V (cache reuse); heaviest block first within a sequence.
    int unit = wg / n_qh;
    qh_local = wg % n_qh;
    b = -1;
    for (int s2 = 0; s2 < a.B; ++s2) {
      const int s0 = min(max(a.cu_seqlens[s2], 0), a.total);
      const int s1 = min(max(a.cu_seqlens[s2 + 1], s0), a.total);
      const int nb = (min(s1 - s0, a.T) + kPrefillRows - 1) / kPrefillRows;
      if (unit < nb) {
        b = s2;
        qb = nb - 1 - unit;
        break;
      }
      unit -= nb;
    }
    if (b < 0) return;  // past the last sequence's blocks
  }
  const int g = a.kv_heads[qh_local / a.gs];
  const int h = g * a.gs + (qh_local % a.gs);

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int h2 = lane >> 5;
  int T = a.T;
  int64_t tok0 = 0;  // varlen: first row of this sequence in the packed tensors
  if (a.cu_seqlens) {
    const int s0 = min(max(a.cu_seqlens[b], 0), a.total);
    const int s1 = min(max(a.cu_seqlens[b + 1], s0), a.total);
    T = min(s1 - s0, a.T);
    tok0 = s0;
  }
  const int i0 = qb * kPrefillRows;
  if (i0 >= T) return;  // query block past this sequence's end (whole workgroup)
  const int r0 = i0 + wave * kRowsPerWave;      // first row of this wave
  int my_row[kRB];                              // row of this lane in each 32-row block
  int my_lo[kRB];                               // its first visible non-sink key (streaming)
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    my_row[rb] = r0 + 32 * rb + l32;
    my_lo[rb] = lo_of(my_row[rb], a.chunk, a.window);
  }

  const int64_t qoff = a.cu_seqlens ? tok0 * a.q_st : (int64_t)b * a.q_sb;
  const int64_t koff = a.cu_seqlens ? tok0 * a.k_st : (int64_t)b * a.k_sb;
  const int64_t voff = a.cu_seqlens ? tok0 * a.v_st : (int64_t)b * a.v_sb;
  const int64_t ooff = a.cu_seqlens ? tok0 * a.o_st : (int64_t)b * a.o_sb;
  const uint16_t* qp = reinterpret_cast<const uint16_t*>(a.q) + qoff + (int64_t)h * a.q_sh;
  const uint16_t* kp = reinterpret_cast<const uint16_t*>(a.k) + koff + (int64_t)g * a.k_sh;
  const uint16_t* vp = reinterpret_cast<const uint16_t*>(a.v) + voff + (int64_t)g * a.v_sh;

  // Q^T operands: lane holds row my_row[rb], dims 8*h2 + 16*s .. +8.
  bf16x8 qreg[kRB][kKSteps];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
    for (int s = 0; s < kKSteps; ++s) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (my_row[rb] < T) x = ld16(qp + (int64_t)my_row[rb] * a.q_st + 8 * h2 + 16 * s);
      qreg[rb][s] = __builtin_bit_cast(bf16x8, x);
    }

  f32x16 acc_o[kRB][kMBlocks];
  float m_run[kRB];  // reference max (log2 units) of this lane's row
  float l_run[kRB];  // this lane's partial row sum (partner lane has the rest)
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
#pragma unroll
    for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc_o[rb][mb][i] = 0.f;
  }

  const TilePlan plan = make_plan<STREAM>(i0, kPrefillRows, T, a.n_sink, a.window, a.chunk);

  // Cooperative staging of one stage (kStageTiles tiles of 64 keys): global ->
  // registers -> LDS (double buffered).  Per-thread row/column are fixed, so
  // the global address of a tile is one scalar offset away.
  u32x4 kst[kStageTiles][kChunksPerThread], vst[kStageTiles][kChunksPerThread];
  int st_row[kChunksPerThread], st_col[kChunksPerThread];
#pragma unroll
  for (int r = 0; r < kChunksPerThread; ++r) {
    const int cidx = tid + r * kWaves * kWave;
    st_row[r] = cidx / kChunksPerRow;
    st_col[r] = (cidx % kChunksPerRow) * 8;
  }
  auto load_tile = [&](int u, int kb) {
    if (kb + kBN <= T) {
#pragma unroll
      for (int r = 0; r < kChunksPerThread; ++r) {
        kst[u][r] = ld16(kp + (int64_t)(kb + st_row[r]) * a.k_st + st_col[r]);
        vst[u][r] = ld16(vp + (int64_t)(kb + st_row[r]) * a.v_st + st_col[r]);
      }
    } else {
      // Ragged last tile: rows past T read row T-1 and are zeroed.
#pragma unroll
      for (int r = 0; r < kChunksPerThread; ++r) {
        const int key = kb + st_row[r];
        const int key_c = min(key, T - 1);
        const u32x4 kx = ld16(kp + (int64_t)key_c * a.k_st + st_col[r]);
        const u32x4 vx = ld16(vp + (int64_t)key_c * a.v_st + st_col[r]);
        const bool in = key < T;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kst[u][r][e] = in ? kx[e] : 0u;
          vst[u][r][e] = in ? vx[e] : 0u;
        }
      }
    }
  };
  auto load_stage = [&](int stage) {
#pragma unroll
    for (int u = 0; u < kStageTiles; ++u) {
      const int it = stage * kStageTiles + u;
      if (it < plan.n_visit) load_tile(u, plan.tile(it) * kBN);
    }
  };
  auto store_stage = [&](PrefillLds<D>& buf) {
#pragma unroll
    for (int u = 0; u < kStageTiles; ++u)
#pragma unroll
      for (int r = 0; r < kChunksPerThread; ++r) {
        *reinterpret_cast<u32x4*>(&buf.k[kBN * u + st_row[r]][st_col[r]]) = kst[u][r];
        *reinterpret_cast<u32x4*>(&buf.v[kBN * u + st_row[r]][st_col[r]]) = vst[u][r];
      }
  };

  // Fused append: the first query head of each group writes the K/V tiles of
  // its block's own rows [i0, i0 + rows) into the cache, from the LDS stage
  // that already holds them, so every position is written exactly once.
  // Retrieval: paged cache (K token-major, V dimension-major per page; pages
  // outside the block table are skipped).  Streaming: the ring keeps a
  // position only if no later prompt position maps to its slot.
  const bool writer = APPEND && (qh_local % a.gs) == 0;
  const int crank = qh_local / a.gs;
  auto write_tile = [&](const PrefillLds<D>& buf, int u, int kb) {
    constexpr int kCh = D / 8;
    uint16_t* ck = static_cast<uint16_t*>(a.ck);
    uint16_t* cv = static_cast<uint16_t*>(a.cv);
    if (!STREAM) {
      for (int e = tid; e < kBN * kCh; e += kWaves * kWave) {
        const int row = e / kCh, col = (e % kCh) * 8;
        const int p = kb + row;
        const int lp = p / kPageTokens;
        if (p >= T || lp >= a.max_pages) continue;
        const int page = a.block_table[(int64_t)b * a.max_pages + lp];
        if (page < 0 || page >= a.num_pages) continue;
        uint16_t* dst = ck + (((int64_t)page * a.n_cache + crank) * kPageTokens + p % kPageTokens) * D + col;
        st16(dst, *reinterpret_cast<const u32x4*>(&buf.k[kBN * u + row][col]));
      }
      for (int e = tid; e < (kBN / kPageTokens) * D * 2; e += kWaves * kWave) {
        const int pg = e / (2 * D), d = (e / 2) % D, hf = e % 2;
        const int p0 = kb + kPageTokens * pg + 8 * hf;
        const int lp = p0 / kPageTokens;
        if (p0 >= T || lp >= a.max_pages) continue;
        const int page = a.block_table[(int64_t)b * a.max_pages + lp];
        if (page < 0 || page >= a.num_pages) continue;
        uint16_t* dst = cv + (((int64_t)page * a.n_cache + crank) * D + d) * kPageTokens + 8 * hf;
        const int row0 = kBN * u + kPageTokens * pg + 8 * hf;
        if (p0 + 8 <= T) {
          u32x4 w;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            w[j] = (uint32_t)buf.v[row0 + 2 * j][d] | ((uint32_t)buf.v[row0 + 2 * j + 1][d] << 16);
          st16(dst, w);
        } else {
          for (int j = 0; p0 + j < T; ++j) dst[j] = buf.v[row0 + j][d];
        }
      }
    } else {
      for (int e = tid; e < kBN * kCh; e += kWaves * kWave) {
        const int row = e / kCh, col = (e % kCh) * 8;
        const int p = kb + row;
        if (p >= T || !(p < a.n_sink || p >= T - a.window)) continue;
        const int slot = p < a.n_sink ? p : a.n_sink + (p - a.n_sink) % a.window;
        const int64_t unit = ((int64_t)b * a.n_cache + crank) * a.ring_blocks + slot / kPageTokens;
        const int r = slot % kPageTokens;
        st16(ck + unit * (kPageTokens * D) + r * D + col, *reinterpret_cast<const u32x4*>(&buf.k[kBN * u + row][col]));
        uint16_t* rv = cv + unit * (kPageTokens * D);
#pragma unroll
        for (int j = 0; j < 8; ++j) rv[(col + j) * kPageTokens + r] = buf.v[kBN * u + row][col + j];
      }
    }
  };

  const float c = a.scale_log2;
  // Softmax of one 32-key block of S^T for row block rb, in two halves so the
  // caller can put independent MFMAs between them:
  //   block_max:  mask, row max, lazy rescale decision (a wave-uniform branch)
  //   block_exp:  exponentials into the two P^T operands of the block's key steps
  auto block_max = [&](int rb, f32x16& sb, int key0, auto masked) {
    constexpr bool MASKED = decltype(masked)::value;
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float x = sb[i];
      if (MASKED) {
        const int key = key0 + 8 * (i >> 2) + 4 * h2 + (i & 3);
        bool vis = key <= my_row[rb];
        if (STREAM) vis = vis && (key < a.n_sink || key >= my_lo[rb]);
        x = vis ? x : -INFINITY;
        sb[i] = x;
      }
      mx = fmaxf(mx, x);
    }
    mx = wave_xor_max(mx, 32) * c;  // log2 units (c > 0 keeps the order)
    // Raise the reference max only when some row needs it (wave-uniform).
    if (__any(mx > m_run[rb] + kRescaleThreshold)) {
      const float m_new = fmaxf(m_run[rb], mx);
      // 0 when only m_run is -inf; 1 when the row has seen no visible key yet.
      const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_run[rb] - m_new);
      m_run[rb] = m_new;
      l_run[rb] *= alpha;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc_o[rb][mb][i] *= alpha;
    }
  };
#ifndef AOH_PREFILL_DOT2_SUM
#define AOH_PREFILL_DOT2_SUM 1
#endif
  auto block_exp = [&](int rb, const f32x16& sb, bf16x8& p_lo, bf16x8& p_hi) {
    const float m_use = (m_run[rb] == -INFINITY) ? 0.f : m_run[rb];
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float p = fast_exp2(fmaf(sb[i], c, -m_use));
#if !AOH_PREFILL_DOT2_SUM
      psum += p;
#endif
      if (i < 8) p_lo[i] = f32_to_bf16(p);
      else p_hi[i - 8] = f32_to_bf16(p);
    }
#if AOH_PREFILL_DOT2_SUM
    // Row sum of the bf16 P actually fed to P.V: one dot2 with (1, 1) per pair.
    const bf16x2 ones = {(bf16)1.f, (bf16)1.f};
#define AOH_DOT2_PAIR(v, j) \
  psum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(v, v, j, j + 1), ones, psum, false)
    AOH_DOT2_PAIR(p_lo, 0);
    AOH_DOT2_PAIR(p_lo, 2);
    AOH_DOT2_PAIR(p_lo, 4);
    AOH_DOT2_PAIR(p_lo, 6);
    AOH_DOT2_PAIR(p_hi, 0);
    AOH_DOT2_PAIR(p_hi, 2);
    AOH_DOT2_PAIR(p_hi, 4);
    AOH_DOT2_PAIR(p_hi, 6);
#undef AOH_DOT2_PAIR
#endif
    l_run[rb] += psum;
  };

  // S^T of one 32-key block for every row block: each K operand read from LDS
  // feeds kRB MFMAs.
  auto qk_block = [&](const PrefillLds<D>& buf, int u, int blk, f32x16 (&sb)[kRB]) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sb[rb][i] = 0.f;
#pragma unroll
    for (int s = 0; s < kKSteps; ++s) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(&buf.k[kBN * u + 32 * blk + l32][8 * h2 + 16 * s]);
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) sb[rb] = mfma32(kop, qreg[rb][s], sb[rb]);
    }
  };
  // O^T += V^T . P^T for key step t (keys 16t..16t+15 of the tile): the k
  // index 8*h2 + j maps to key 16t + 4*h2 + j (j < 4) or 16t + 8 + 4*h2 + (j-4).
  // Each V^T operand (two transpose reads) feeds kRB MFMAs.
  const int q16 = lane >> 4;        // 16-lane block
  const int i16 = lane & 15;
  auto pv_step = [&](const PrefillLds<D>& buf, int u, int t, const bf16x8 (&pop)[kRB]) {
    const int vrow = kBN * u + 16 * t + 4 * h2 + (i16 >> 2);
#pragma unroll
    for (int mb = 0; mb < kMBlocks; ++mb) {
      const int vcol = 32 * mb + 16 * (q16 & 1) + 4 * (i16 & 3);
      const i16x4 lo = lds_read_tr16(&buf.v[vrow][vcol]);
      const i16x4 hi = lds_read_tr16(&buf.v[vrow + 8][vcol]);
      // Whole-vector concatenation: per-element bf16 insertion of the
      // transposed halves is avoided on purpose (it was lowered to a
      // broadcast of the first element by this toolchain).
      const i16x8 cat = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      const bf16x8 vop = __builtin_bit_cast(bf16x8, cat);
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) acc_o[rb][mb] = mfma32(vop, pop[rb], acc_o[rb][mb]);
    }
  };

  // One 64-key tile for this wave.  MASKED selects the per-element mask; full
  // tiles carry no mask code.  Order: S^T of block 0, its max; then the S^T
  // MFMAs of block 1 next to the exponentials of block 0 and the P.V MFMAs of
  // block 0 next to the max of block 1 (same scheduling region, independent
  // work for the matrix core and the vector ALU); then block 1.
#ifndef AOH_PREFILL_SETPRIO
#define AOH_PREFILL_SETPRIO 1
#endif
  // Wave issue priority (s_setprio, inside this wave only): raised while a wave
  // issues its MFMA clusters so the matrix core is fed first and the other
  // wave's vector work fills the gaps.
  auto prio = [&](int p) {
#if AOH_PREFILL_SETPRIO
    if (p) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
#else
    (void)p;
#endif
  };
  auto tile_step = [&](const PrefillLds<D>& buf, int u, int kb, auto masked) {
    f32x16 s0[kRB], s1[kRB];
    bf16x8 p0[kRB], p1[kRB], p2[kRB], p3[kRB];  // P^T operands of the 4 key steps
    prio(1);
    qk_block(buf, u, 0, s0);
    prio(0);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) block_max(rb, s0[rb], kb, masked);
    prio(1);
    qk_block(buf, u, 1, s1);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) block_exp(rb, s0[rb], p0[rb], p1[rb]);
    pv_step(buf, u, 0, p0);
    pv_step(buf, u, 1, p1);
    prio(0);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) block_max(rb, s1[rb], kb + 32, masked);
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) block_exp(rb, s1[rb], p2[rb], p3[rb]);
    prio(1);
    pv_step(buf, u, 2, p2);
    pv_step(buf, u, 3, p3);
    prio(0);
  };

  // Double-buffered main loop: one barrier per stage of kStageTiles tiles.
  // While stage `st` is computed from lds[st & 1], stage st+1 waits in
  // registers and is written to the other buffer afterwards; stage st+2 is
  // fetched from global memory.
  const int n_stage = (plan.n_visit + kStageTiles - 1) / kStageTiles;
  if (n_stage > 0) {
    load_stage(0);
    store_stage(lds[0]);
    if (n_stage > 1) load_stage(1);
  }
  __syncthreads();
  for (int st = 0; st < n_stage; ++st) {
    const PrefillLds<D>& buf = lds[st & 1];
    if (APPEND && writer)
      for (int u = 0; u < kStageTiles; ++u) {
        const int it = st * kStageTiles + u;
        if (it < plan.n_visit) {
          const int kb = plan.tile(it) * kBN;
          if (kb >= i0 && kb < i0 + kPrefillRows) write_tile(buf, u, kb);
        }
      }
#pragma unroll
    for (int u = 0; u < kStageTiles; ++u) {
      const int it = st * kStageTiles + u;
      if (it < plan.n_visit) {
        const int kb = plan.tile(it) * kBN;
        // Is any element of this wave's rows x 64 keys visible?  Is every element?
        const bool wave_dead = (kb > r0 + kRowsPerWave - 1) ||
                               (STREAM && kb >= a.n_sink && kb + kBN - 1 < lo_of(r0, a.chunk, a.window));
        if (!wave_dead) {
          const bool need_mask =
              (kb + kBN - 1 > r0) ||
              (STREAM && !(kb + kBN - 1 < a.n_sink || kb >= lo_of(r0 + kRowsPerWave - 1, a.chunk, a.window)));
          if (need_mask) tile_step(buf, u, kb, std::true_type{});
          else tile_step(buf, u, kb, std::false_type{});
        }
      }
    }
    if (st + 1 < n_stage) {
      store_stage(lds[(st + 1) & 1]);
      if (st + 2 < n_stage) load_stage(st + 2);
    }
    __syncthreads();
  }

  // Epilogue: normalise by the row sum, store.
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    const float l_tot = wave_xor_sum(l_run[rb], 32);
    const float inv = 1.f / l_tot;
    if (my_row[rb] >= T) continue;
    if (OUT_F32) {
      float* op = reinterpret_cast<float*>(a.out) + ooff + (int64_t)my_row[rb] * a.o_st +
                  (int64_t)h * a.o_sh;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          f32x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = acc_o[rb][mb][4 * q4 + e] * inv;
          *reinterpret_cast<f32x4*>(op + 32 * mb + 8 * q4 + 4 * h2) = w;
        }
    } else {
      uint16_t* op = reinterpret_cast<uint16_t*>(a.out) + ooff + (int64_t)my_row[rb] * a.o_st +
                     (int64_t)h * a.o_sh;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          u32x2 w;
          w[0] = (uint32_t)f32_to_bf16_bits(acc_o[rb][mb][4 * q4 + 0] * inv) |
                 ((uint32_t)f32_to_bf16_bits(acc_o[rb][mb][4 * q4 + 1] * inv) << 16);
          w[1] = (uint32_t)f32_to_bf16_bits(acc_o[rb][mb][4 * q4 + 2] * inv) |
                 ((uint32_t)f32_to_bf16_bits(acc_o[rb][mb][4 * q4 + 3] * inv) << 16);
          *reinterpret_cast<u32x2*>(op + 32 * mb + 8 * q4 + 4 * h2) = w;
        }
    }
  }
}

// fp32 reference-grade kernel: one thread per query row, keys visited in
// order (sink part, then the recent band), exact expf.
template <int D, bool STREAM>
__global__ __launch_bounds__(kPrefillRowsF32) void prefill_f32_kernel(PrefillArgs a) {
  // No implicit FMA contraction: a lone visible key must get weight exactly 1.
#pragma clang fp contract(off)
  const int n_qh = a.n_kv * a.gs;
  const int per_block = n_qh * a.B;
  const int wg = blockIdx.x;
  const int qb = a.n_qblocks - 1 - wg / per_block;
  const int rem = wg % per_block;
  const int qh_local = rem % n_qh;
  const int b = rem / n_qh;
  const int g = a.kv_heads[qh_local / a.gs];
  const int h = g * a.gs + (qh_local % a.gs);
  const int i = qb * kPrefillRowsF32 + threadIdx.x;
  int T = a.T;
  int64_t tok0 = 0;
  if (a.cu_seqlens) {
    const int s0 = min(max(a.cu_seqlens[b], 0), a.total);
    const int s1 = min(max(a.cu_seqlens[b + 1], s0), a.total);
    T = min(s1 - s0, a.T);
    tok0 = s0;
  }
  if (i >= T) return;
  const int64_t qoff = a.cu_seqlens ? tok0 * a.q_st : (int64_t)b * a.q_sb;
  const int64_t koff = a.cu_seqlens ? tok0 * a.k_st : (int64_t)b * a.k_sb;
  const int64_t voff = a.cu_seqlens ? tok0 * a.v_st : (int64_t)b * a.v_sb;
  const int64_t ooff = a.cu_seqlens ? tok0 * a.o_st : (int64_t)b * a.o_sb;
  const float* qp = reinterpret_cast<const float*>(a.q) + qoff + (int64_t)i * a.q_st +
                    (int64_t)h * a.q_sh;
  const float* kp = reinterpret_cast<const float*>(a.k) + koff + (int64_t)g * a.k_sh;
  const float* vp = reinterpret_cast<const float*>(a.v) + voff + (int64_t)g * a.v_sh;
  float q[D], o[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = qp[d];
    o[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  int lo = 0, sink_end = 0;
  if (STREAM) {
    lo = max(0, lo_of(i, a.chunk, a.window));
    sink_end = min(a.n_sink, lo);
  }
  auto visit = [&](int j) {
    float s = 0.f;
    const float* kr = kp + (int64_t)j * a.k_st;
#pragma unroll
    for (int d = 0; d < D; ++d) s = fmaf(q[d], kr[d], s);
    s *= a.scale;
    const float m_new = fmaxf(m, s);
    const float alpha = expf(m - m_new);
    const float p = expf(s - m_new);
    l = l * alpha + p;
    const float* vr = vp + (int64_t)j * a.v_st;
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] = o[d] * alpha + p * vr[d];
    m = m_new;
  };
  for (int j = 0; j < sink_end; ++j) visit(j);
  for (int j = lo; j <= i; ++j) visit(j);
  float* op = reinterpret_cast<float*>(a.out) + ooff + (int64_t)i * a.o_st + (int64_t)h * a.o_sh;
  const float inv = 1.f / l;
#pragma unroll
  for (int d = 0; d < D; ++d) op[d] = o[d] * inv;
}

template <int D, bool STREAM, bool OUT_F32>
static hipError_t launch_bf16(const PrefillArgs& a, hipStream_t s) {
  const int grid = a.n_qblocks * a.n_kv * a.gs * a.B;
  if (a.append)
    hipLaunchKernelGGL((prefill_bf16_kernel<D, STREAM, OUT_F32, true>), dim3(grid), dim3(kWaves * kWave), 0, s, a);
  else
    hipLaunchKernelGGL((prefill_bf16_kernel<D, STREAM, OUT_F32, false>), dim3(grid), dim3(kWaves * kWave), 0, s, a);
  return hipGetLastError();
}

template <int D, bool STREAM>
static hipError_t launch_f32(const PrefillArgs& a, hipStream_t s) {
  const int grid = a.n_qblocks * a.n_kv * a.gs * a.B;
  hipLaunchKernelGGL((prefill_f32_kernel<D, STREAM>), dim3(grid), dim3(kPrefillRowsF32), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int out_f32, int d, bool streaming,
                          hipStream_t s) {
  if (dtype == 1) {  // fp32
    if (d == 64) return streaming ? launch_f32<64, true>(a, s) : launch_f32<64, false>(a, s);
    return streaming ? launch_f32<128, true>(a, s) : launch_f32<128, false>(a, s);
  }
  if (d == 64) {
    if (out_f32) return streaming ? launch_bf16<64, true, true>(a, s) : launch_bf16<64, false, true>(a, s);
    return streaming ? launch_bf16<64, true, false>(a, s) : launch_bf16<64, false, false>(a, s);
  }
  if (out_f32) return streaming ? launch_bf16<128, true, true>(a, s) : launch_bf16<128, false, true>(a, s);
  return streaming ? launch_bf16<128, true, false>(a, s) : launch_bf16<128, false, false>(a, s);
}

}  // namespace aoh
