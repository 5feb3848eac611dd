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
// bf16 kernels.  One workgroup = 8 waves = 256 query rows of one query head;
// each wave owns 32 rows.  Key/value tiles of 64 keys are staged in LDS and
// shared by the 8 waves.  Per tile and wave:
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
//   prefill_pp_kernel (d_head 128): direct global->LDS tile loads into a
//     4-stage ring, swizzled LDS rows, two phase-shifted wave groups,
//     XCD-aware workgroup order (see its own comment).  A layer with both
//     head types runs as one launch (prefill_pp_mixed_kernel): retrieval
//     items first, streaming items after them.
//   prefill_bf16_kernel (d_head 64): register-staged, double-buffered, padded
//     LDS tiles.
//
// fp32 kernel: a plain per-row kernel (one thread per query row) kept exact
// for fp32 inputs; it has no performance role.
#include <atomic>
#include <type_traits>

#include "aoh_device.h"
#include "aoh_internal.h"

namespace aoh {

constexpr int kBN = 64;          // keys per tile
constexpr int kRB = kPrefillRB;                 // 32-row MFMA blocks per wave
constexpr int kRowsPerWave = 32 * kRB;
constexpr int kWaves = kPrefillRows / kRowsPerWave;  // waves per workgroup

// 64-key tiles per LDS stage (one barrier per stage).
constexpr int kStageTiles = 1;

template <int D>
struct PrefillLds {
  // Row paddings (bf16 elements): K rows are read 16 bytes per lane down 32
  // rows; V rows are read by the transpose read as 4 rows x 32 bytes per
  // 16 lanes.  Each padding spreads its access pattern over distinct banks.
  static constexpr int kStrideK = D + 8;
  static constexpr int kStrideV = D + 32;
  uint16_t k[kBN * kStageTiles][kStrideK];
  uint16_t v[kBN * kStageTiles][kStrideV];
};

// Lazy rescaling threshold (log2 units): the running max used for the
// exponentials is only raised when a row's true max exceeds it by more than
// this, so P stays below 2^8 and the O rescale is skipped on most tiles.
constexpr float kRescaleThreshold = 8.0f;

// d_head-128 kernel: largest sum of a lane's 32 exponentials of one tile,
// taken against the trailing reference max, that is accepted as it is.
constexpr float kSumHi = 65536.f;

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
  auto block_exp = [&](int rb, const f32x16& sb, bf16x8& p_lo, bf16x8& p_hi) {
    const float m_use = (m_run[rb] == -INFINITY) ? 0.f : m_run[rb];
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float p = fast_exp2(fmaf(sb[i], c, -m_use));
      if (i < 8) p_lo[i] = f32_to_bf16(p);
      else p_hi[i - 8] = f32_to_bf16(p);
    }
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
  // Wave issue priority (s_setprio, inside this wave only): raised while a wave
  // issues its MFMA clusters so the matrix core is fed first and the other
  // wave's vector work fills the gaps.
  auto prio = [&](int p) {
    if (p) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
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

// ---------------------------------------------------------------------------
// D = 128 bf16 kernel, phase-shifted wave groups.
//
// Same work item and products as prefill_bf16_kernel (256 query rows of one
// query head, 32 rows per wave, S^T = K.Q^T and O^T += V^T.P^T on the 32x32x16
// bf16 MFMA, online softmax in fp32); differences:
//  * K/V tiles move global -> LDS with direct loads (global_load_lds_dwordx4),
//    no register staging, into a K ring and a V ring of four 16 KB tiles
//    each, issued two tiles ahead of their first use.
//  * Rows hold 16 chunks of 16 bytes with no padding; chunk c of row r sits
//    at c ^ (r & 15) for K and c ^ 4 (r & 3) for V, which keeps the K row
//    reads and the V transpose reads free of bank conflicts.  Every operand
//    address is one of 12 per-lane base registers plus a constant, and the
//    tile loop runs four tiles per pass so that each ring slot is a
//    compile-time constant too: the operand reads take it as an immediate
//    offset, with no address arithmetic per tile.
//  * Per tile t a wave runs an MFMA phase (P(t-1).V(t-1) then K(t).Q^T, at
//    raised wave priority) and a vector phase (mask, exponentials of S(t)
//    against a trailing reference max, no max pass unless the tile's
//    exponentials grow too large); waves 0-3 and waves 4-7 (one of each per
//    SIMD) run one phase apart, with one workgroup barrier per tile (after
//    the vector phase for waves 0-3, after the MFMA phase for waves 4-7).
//    The loop has a single path (a tile with no visible key for a wave
//    yields P = 0), so the accumulators never move between registers.
//  * The fused cache append writes the block's own (diagonal) tiles after
//    the loop, from the ring, which still holds them.
//  * Workgroups are ordered so that the query heads of one KV group and query
//    block run on the same XCD (one L2); the light items at the end of a
//    launch are taken from per-XCD work queues, so that faster XCDs take over
//    part of the slower ones' share.
constexpr int kPPStages = 4;  // slots of the K and V rings
constexpr int kPPD = 128;
constexpr int kPPRows = kPrefillRows;     // query rows per workgroup (8 waves x 32)
static_assert(kPPRows == 256 && kPrefillRB == 1, "phase-shifted kernel: 8 waves x 32 rows");

// The LDS rings of the d_head-128 kernel: the K tiles of the kPPStages slots,
// then their V tiles (a slot's offset within a ring fits the 16-bit immediate
// offset of an LDS read).
struct PPRing {
  uint16_t k[kPPStages][kBN * kPPD];
  uint16_t v[kPPStages][kBN * kPPD];
};
constexpr uint32_t kPPTileBytes = kBN * kPPD * 2;  // one K or V tile
// Element offset of 16-byte chunk c of row r in a stage's K / V tile.
__device__ __forceinline__ int pp_koff(int r, int c) { return r * kPPD + 8 * (c ^ (r & 15)); }
__device__ __forceinline__ int pp_voff(int r, int c) { return r * kPPD + 8 * (c ^ (4 * (r & 3))); }

// Direct global -> LDS load of 16 bytes per lane: lane L's bytes land at
// lds_row + 16 L (one contiguous 1 KB block per wave).  Issued as inline
// assembly so that the compiler does not treat every later LDS read as
// possibly depending on it (it would wait for all outstanding loads before
// each one); the kernel orders these loads itself with s_waitcnt and barriers.
__device__ __forceinline__ void lds_dma16(const void* gptr, const void* lds_row) {
  const uint32_t m0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds_row));
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(gptr), "{m0}"(m0) : "memory");
}

// s_waitcnt immediates (gfx9 encoding: vmcnt [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]); a field at its maximum does not wait.
constexpr int kWaitVm0 = 0x0 | (0x7 << 4) | (0xF << 8);
constexpr int kWaitVm4 = 0x4 | (0x7 << 4) | (0xF << 8);
constexpr int kWaitLgkm0 = 0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14);


// Work item of a workgroup of the d_head-128 kernels: query block qb (rows
// qb * rows ..), local query head qh_local of the launch's KV-head list and
// sequence b.  Dense batches use the XCD-aware order below; packed batches
// with sequence-major order walk cu_seqlens.  Returns false when the
// workgroup has no work (past the last sequence's blocks).
__device__ __forceinline__ bool pp_work_item(const PrefillArgs& a, int rows, int wg, int& qb, int& qh_local,
                                             int& b) {
  const int n_qh = a.n_kv * a.gs;
  const int per_block = n_qh * a.B;
  qb = a.n_qblocks - 1 - wg / per_block;
  const int rem = wg % per_block;
  qh_local = rem % n_qh;
  b = rem / n_qh;
  if (!a.seq_major) {
    // XCD-aware order.  Workgroups go to the 8 XCDs (each with its own L2)
    // in turn; work item group j = (query block, sequence, KV head), heaviest
    // block first, holds the gs query heads that read the same K/V tiles.
    // Round m of 8 groups runs as gs consecutive workgroups on each XCD, so a
    // group's tiles are fetched into one L2 once.  Groups get lighter along
    // the order, so odd rounds deal them in reverse, which keeps each XCD's
    // total work level (dealt one way, XCD 0 would take the heaviest group of
    // every round).  When a round holds whole query blocks (the per-block
    // group count divides 8) only the blocks' order is reversed: each XCD
    // keeps serving one (sequence, KV head), whose causal prefix stays in its
    // L2.  The trailing groups that do not fill a round of 8 are dealt in
    // plain order.
    const int n_groups = a.n_qblocks * a.n_kv * a.B;
    const int full = 8 * a.gs * (n_groups / 8);
    const int pq = a.n_kv * a.B;
    int j, hl;
    if (wg < full) {
      const int slot = wg >> 3;
      const int m = slot / a.gs;
      int x = wg & 7;
      if (m & 1) x = (8 % pq == 0) ? (8 - pq) - (x - x % pq) + x % pq : 7 - x;
      j = 8 * m + x;
      hl = slot % a.gs;
    } else {
      j = (full / a.gs) + (wg - full) / a.gs;
      hl = (wg - full) % a.gs;
    }
    const int per_qb = a.n_kv * a.B;
    qb = a.n_qblocks - 1 - j / per_qb;
    const int r2 = j % per_qb;
    b = r2 / a.n_kv;
    qh_local = (r2 % a.n_kv) * a.gs + hl;
  }
  if (a.seq_major) {
    int unit = wg / n_qh;
    qh_local = wg % n_qh;
    b = -1;
    for (int s2 = 0; s2 < a.B; ++s2) {
      const int s0 = min(max(a.cu_seqlens[s2], 0), a.total);
      const int s1 = min(max(a.cu_seqlens[s2 + 1], s0), a.total);
      const int nb = (min(s1 - s0, a.T) + rows - 1) / rows;
      if (unit < nb) {
        b = s2;
        qb = nb - 1 - unit;
        break;
      }
      unit -= nb;
    }
    if (b < 0) return false;
  }
  return true;
}

// Fused append of one resident tile (keys kb .. kb+63) into the cache of the
// launch: the paged cache (K token-major, V dimension-major per page; pages
// outside the block table are skipped) or the ring (a position is kept only
// if no later prompt position maps to its slot).  Threads tid, tid + nthr, ..
// take the 16-byte chunks of the tile; crank = the KV head's rank in the cache.
template <bool STREAM>
__device__ __forceinline__ void pp_write_tile(const PrefillArgs& a, const uint16_t* tk, const uint16_t* tv, int kb,
                                              int b, int crank, int T, int tid, int nthr) {
  constexpr int D = kPPD;
  constexpr int kCh = D / 8;
  uint16_t* ck = static_cast<uint16_t*>(a.ck);
  uint16_t* cv = static_cast<uint16_t*>(a.cv);
  if (!STREAM) {
    for (int e = tid; e < kBN * kCh; e += nthr) {
      const int row = e / kCh, ch = e % kCh;
      const int p = kb + row;
      const int lp = p / kPageTokens;
      if (p >= T || lp >= a.max_pages) continue;
      const int page = a.block_table[(int64_t)b * a.max_pages + lp];
      if (page < 0 || page >= a.num_pages) continue;
      uint16_t* dst = ck + (((int64_t)page * a.n_cache + crank) * kPageTokens + p % kPageTokens) * D + 8 * ch;
      st16(dst, *reinterpret_cast<const u32x4*>(&tk[pp_koff(row, ch)]));
    }
    for (int e = tid; e < (kBN / kPageTokens) * D * 2; e += nthr) {
      const int pg = e / (2 * D), d = (e / 2) % D, hf = e % 2;
      const int p0 = kb + kPageTokens * pg + 8 * hf;
      const int lp = p0 / kPageTokens;
      if (p0 >= T || lp >= a.max_pages) continue;
      const int page = a.block_table[(int64_t)b * a.max_pages + lp];
      if (page < 0 || page >= a.num_pages) continue;
      uint16_t* dst = cv + (((int64_t)page * a.n_cache + crank) * D + d) * kPageTokens + 8 * hf;
      const int row0 = kPageTokens * pg + 8 * hf;
      const int dc = d >> 3, de = d & 7;
      if (p0 + 8 <= T) {
        u32x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          w[j] = (uint32_t)tv[pp_voff(row0 + 2 * j, dc) + de] |
                 ((uint32_t)tv[pp_voff(row0 + 2 * j + 1, dc) + de] << 16);
        st16(dst, w);
      } else {
        for (int j = 0; p0 + j < T; ++j) dst[j] = tv[pp_voff(row0 + j, dc) + de];
      }
    }
  } else {
    for (int e = tid; e < kBN * kCh; e += nthr) {
      const int row = e / kCh, ch = e % kCh;
      const int p = kb + row;
      if (p >= T || !(p < a.n_sink || p >= T - a.window)) continue;
      const int slot = p < a.n_sink ? p : a.n_sink + (p - a.n_sink) % a.window;
      const int64_t unit = ((int64_t)b * a.n_cache + crank) * a.ring_blocks + slot / kPageTokens;
      const int r = slot % kPageTokens;
      st16(ck + unit * (kPageTokens * D) + r * D + 8 * ch, *reinterpret_cast<const u32x4*>(&tk[pp_koff(row, ch)]));
      uint16_t* rv = cv + unit * (kPageTokens * D);
      const int vo = pp_voff(row, ch);
#pragma unroll
      for (int j = 0; j < 8; ++j) rv[(8 * ch + j) * kPageTokens + r] = tv[vo + j];
    }
  }
}

// One work item (workgroup index wg of its launch's item space) of the
// d_head-128 kernel; ring = the workgroup's LDS rings.
template <bool STREAM, bool OUT_F32, bool APPEND>
__device__ __forceinline__ void prefill_pp_body(const PrefillArgs& a, int wg, PPRing& ring) {
  constexpr int D = kPPD;
  constexpr int kKSteps = D / 16;
  constexpr int kMBlocks = D / 32;

  int qb, qh_local, b;
  if (!pp_work_item(a, kPPRows, wg, qb, qh_local, b)) return;
  const int g = a.kv_heads[qh_local / a.gs];
  const int h = g * a.gs + (qh_local % a.gs);

  const int tid = threadIdx.x;
  // Wave index as a scalar: every branch that decides a barrier is uniform.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int h2 = lane >> 5;
  int T = a.T;
  int64_t tok0 = 0;
  if (a.cu_seqlens) {
    const int s0 = min(max(a.cu_seqlens[b], 0), a.total);
    const int s1 = min(max(a.cu_seqlens[b + 1], s0), a.total);
    T = min(s1 - s0, a.T);
    tok0 = s0;
  }
  T = __builtin_amdgcn_readfirstlane(T);
  const int i0 = qb * kPPRows;
  if (i0 >= T) return;
  const int r0 = i0 + wave * 32;
  const int my_row = r0 + l32;
  const int my_lo = lo_of(my_row, a.chunk, a.window);

  const int64_t qoff = a.cu_seqlens ? tok0 * a.q_st : (int64_t)b * a.q_sb;
  const int64_t koff = a.cu_seqlens ? tok0 * a.k_st : (int64_t)b * a.k_sb;
  const int64_t voff = a.cu_seqlens ? tok0 * a.v_st : (int64_t)b * a.v_sb;
  const int64_t ooff = a.cu_seqlens ? tok0 * a.o_st : (int64_t)b * a.o_sb;
  const uint16_t* qp = reinterpret_cast<const uint16_t*>(a.q) + qoff + (int64_t)h * a.q_sh;
  const uint16_t* kp = reinterpret_cast<const uint16_t*>(a.k) + koff + (int64_t)g * a.k_sh;
  const uint16_t* vp = reinterpret_cast<const uint16_t*>(a.v) + voff + (int64_t)g * a.v_sh;

  const TilePlan plan = make_plan<STREAM>(i0, kPPRows, T, a.n_sink, a.window, a.chunk);
  const int n = __builtin_amdgcn_readfirstlane(plan.n_visit);
  if (n < 1) return;  // a block with rows below T always has its diagonal tile

  // Direct loads of tile `it` into stage it % 4: wave w fills rows 8w .. 8w+7
  // of K and of V, one 4-row (1 KB) instruction at a time; lane L writes
  // physical chunk L % 16 of row 4j + L / 16 and therefore fetches the
  // logical chunk that the swizzle puts there.  Rows past the sequence end
  // repeat its last row (those keys are masked for every query row).
  // Per-lane element offsets of the two 4-row blocks this wave loads, relative
  // to the tile's first key (full tiles), and the rows themselves (the ragged
  // last tile clamps them).
  int64_t dma_k[2], dma_v[2];
  int dma_r[2];
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    const int j = 2 * wave + jj;
    const int r = 4 * j + (lane >> 4);
    const int pc = lane & 15;
    dma_r[jj] = r;
    dma_k[jj] = (int64_t)r * a.k_st + 8 * (pc ^ (r & 15));
    dma_v[jj] = (int64_t)r * a.v_st + 8 * (pc ^ (4 * (r & 3)));
  }
  auto issue_tile = [&](int it) {
    const int kb = plan.tile(it) * kBN;
    uint16_t* sk = ring.k[it % kPPStages];
    uint16_t* sv = ring.v[it % kPPStages];
    if (kb + kBN <= T) {
      const uint16_t* kt = kp + (int64_t)kb * a.k_st;
      const uint16_t* vt = vp + (int64_t)kb * a.v_st;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * wave + jj;
        lds_dma16(kt + dma_k[jj], &sk[4 * j * kPPD]);
        lds_dma16(vt + dma_v[jj], &sv[4 * j * kPPD]);
      }
    } else {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * wave + jj;
        const int r = dma_r[jj];
        const int pc = lane & 15;
        const int64_t row = min(kb + r, T - 1);
        lds_dma16(kp + row * a.k_st + 8 * (pc ^ (r & 15)), &sk[4 * j * kPPD]);
        lds_dma16(vp + row * a.v_st + 8 * (pc ^ (4 * (r & 3))), &sv[4 * j * kPPD]);
      }
    }
  };

  bf16x8 qreg[kKSteps];  // Q^T operands: lane holds row my_row, dims 8*h2 + 16*s .. +8
  f32x16 acc_o[kMBlocks];
#pragma unroll
  for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc_o[mb][i] = 0.f;
  float m_run = -INFINITY;  // reference max (log2 units) of this lane's row
  float m_use = 0.f;        // m_run, or 0 while the row has seen no visible key
  float l_run = 0.f;        // this lane's partial row sum (partner lane has the rest)
  f32x16 sacc[2];           // S^T of the current tile, two 32-key blocks
  bf16x8 pop[4];            // P^T operands of the previous tile's 4 key steps

  const float c = a.scale_log2;

  // Per-lane LDS byte addresses.  K operand of step s, block blk: row
  // 32 blk + l32, logical chunk 2 s + h2; with the swizzle that is
  // kaddr0 ^ 32 s (+ 8 KB per block).  V^T operand of key step ks, 32-dim
  // block mb (transpose reads): row 16 ks + 4 h2 + i16 / 4 (+ 8 rows for the
  // second half), logical chunk 4 mb + 2 (q16 & 1) + (i16 & 3) / 2, 4 more
  // elements for odd i16; that is vaddr0 ^ 64 mb (+ 4 KB per key step).
  const int q16 = lane >> 4;
  const int i16 = lane & 15;
  const uint32_t kring0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&ring.k[0][0]));
  const uint32_t vring0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&ring.v[0][0]));
  const uint32_t kaddr0 = 2u * (uint32_t)pp_koff(l32, h2);
  const int vrow0 = 4 * h2 + (i16 >> 2);
  const uint32_t vaddr0 = 2u * (uint32_t)(pp_voff(vrow0, 2 * (q16 & 1) + ((i16 & 3) >> 1)) + 4 * (i16 & 1));
  // The swizzle XORs touch bits below 256 and the rings are 1 KB aligned, so
  // a slot offset adds after them: operand addresses are these per-lane bases
  // plus constants (immediate offsets once the slot is known at compile time).
  uint32_t kx[kKSteps], vx[kMBlocks];
#pragma unroll
  for (int s = 0; s < kKSteps; ++s) kx[s] = (kring0 + kaddr0) ^ (32u * s);
#pragma unroll
  for (int mb = 0; mb < kMBlocks; ++mb) vx[mb] = (vring0 + vaddr0) ^ (64u * mb);
  auto k_operand = [&](int st, int s, int blk) {
    typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;
    return *reinterpret_cast<lds_bf16x8*>(kx[s] + (uint32_t)st * kPPTileBytes + 8192u * blk);
  };
  auto v_operand = [&](int st, int ks, int mb) {
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const uint32_t a = vx[mb] + (uint32_t)st * kPPTileBytes + 4096u * ks;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_i16x4*>(a));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_i16x4*>(a + 2048u));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  auto wave_dead = [&](int kb) {
    return (kb > r0 + 31) || (STREAM && kb >= a.n_sink && kb + kBN - 1 < lo_of(r0, a.chunk, a.window));
  };
  auto need_mask = [&](int kb) {
    return (kb + kBN - 1 > r0) ||
           (STREAM && !(kb + kBN - 1 < a.n_sink || kb >= lo_of(r0 + 31, a.chunk, a.window)));
  };

  // Fused append: the first query head of each group copies its block's own
  // K/V rows from LDS into the cache.  They are the block's diagonal tiles,
  // the last (up to four) tiles of the loop, which the ring still holds when
  // the loop ends; the workgroup writes them then.
  const bool writer = APPEND && (qh_local % a.gs) == 0;
  const int crank = qh_local / a.gs;
  auto write_tile = [&](int st, int kb) {
    pp_write_tile<STREAM>(a, ring.k[st], ring.v[st], kb, b, crank, T, tid, 512);
  };

  // MFMA phase of tile t (stage st = t % kPPStages): O^T += V(t-1)^T
  // P(t-1)^T (stage vst), then S^T(t) = K(t) Q^T.
  auto pv_part = [&](int vst) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb) acc_o[mb] = mfma32(v_operand(vst, ks, mb), pop[ks], acc_o[mb]);
  };
  auto qk_part = [&](int st) {
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[blk][i] = 0.f;
#pragma unroll
    for (int s = 0; s < kKSteps; ++s)
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) sacc[blk] = mfma32(k_operand(st, s, blk), qreg[s], sacc[blk]);
  };
  auto append_tile = [&](int t, int st) {
    if (APPEND && writer) {
      const int kb = plan.tile(t) * kBN;
      if (kb >= i0 && kb < i0 + kPPRows) write_tile(st, kb);
    }
  };
  // Steady-state MFMA phase.  Both products run unconditionally (a wave with
  // no visible key in a tile gets P = 0 from its vector phase), so the loop
  // has one path and the O accumulators stay in place.
  // The MFMA phase runs at raised wave priority (s_setprio, this wave only):
  // its SIMD also holds a wave of the other group in its vector phase, and
  // the matrix core is kept fed first (2-3% faster than equal priority).
  auto mfma_phase = [&](int t, int st) {
    __builtin_amdgcn_s_setprio(1);
    pv_part((st + kPPStages - 1) % kPPStages);
    qk_part(st);
    // Operands are read four MFMAs ahead of their products, the first K
    // operands while the last P.V products run.
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
  };

  // Vector phase of tile t: mask, exponentials into the P^T operands, row
  // sums (and, rarely, a new reference max with the rescale).
  auto apply_mask = [&](int kb) {
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kb + 32 * blk + 8 * (i >> 2) + 4 * h2 + (i & 3);
        bool vis = key <= my_row;
        if (STREAM) vis = vis && (key < a.n_sink || key >= my_lo);
        sacc[blk][i] = vis ? sacc[blk][i] : -INFINITY;
      }
  };
  // Softmax of a tile without a max pass: the exponentials are taken against
  // the reference max m_use as it stands (it trails the true row max) and the
  // tile is accepted when each lane's 32 exponentials sum to at most kSumHi,
  // which bounds every P by it (P, l and O stay far from fp32 overflow and P
  // keeps bf16's relative precision).  A lane whose row has seen no visible
  // key yet, or whose sum is larger or NaN, sends the wave through the exact
  // step: the true row max of the tile becomes the reference, O and l are
  // rescaled and the exponentials are taken again.  Row sums of the fp32
  // exponentials are added as balanced trees: the phase ends on its longest
  // dependency chain, and a running accumulator, a chain of bf16 dot products
  // or a max pass ahead of the exponentials lengthens it.
  auto softmax_tile = [&]() {
    auto exps = [&]() {
      float psum[4];
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          bf16x8 pv;
          float pf[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            pf[i] = fast_exp2(fmaf(sacc[blk][8 * hf + i], c, -m_use));
            pv[i] = f32_to_bf16(pf[i]);
          }
          psum[2 * blk + hf] = ((pf[0] + pf[1]) + (pf[2] + pf[3])) + ((pf[4] + pf[5]) + (pf[6] + pf[7]));
          pop[2 * blk + hf] = pv;
        }
      return (psum[0] + psum[1]) + (psum[2] + psum[3]);
    };
    float tsum = exps();
    if (__any(!(tsum <= kSumHi) || m_run == -INFINITY)) {
      float mx = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[blk][i]);
      const float m_new = fmaxf(m_run, xor32_max(mx) * c);
      const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc_o[mb][i] *= alpha;
      m_use = (m_run == -INFINITY) ? 0.f : m_run;
      tsum = exps();
    }
    l_run += tsum;
  };
  auto valu_phase = [&](int t) {
    const int kb = plan.tile(t) * kBN;
    if (wave_dead(kb)) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) pop[ks][i] = (bf16)0.f;
      return;
    }
    if (need_mask(kb)) apply_mask(kb);
    softmax_tile();
  };

  // One workgroup barrier per tile.  Every wave runs MFMA(0) V(0) MFMA(1)
  // V(1) ..; waves 0-3 take the barrier of tile t after V(t), waves 4-7 after
  // MFMA(t), so a SIMD's two waves alternate without a barrier between their
  // phases.  The barrier of tile t follows each wave's wait for its loads of
  // tile t+1 (those of tile t+2 may stay in flight); after it, tile t+3 goes
  // into the stage of tile t-1, whose last reads (P.V of tile t-1, in MFMA(t))
  // every wave has completed by then.
  auto barrier = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  auto sync_tile = [&](int t) {
    if (t + 2 < n) __builtin_amdgcn_s_waitcnt(kWaitVm4);
    else __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    barrier();
    if (t + kPPStages - 1 < n) issue_tile(t + kPPStages - 1);
  };

  // Prologue: tiles 0 .. kPPStages-2 and this wave's Q rows in flight, then
  // everything complete (the explicit full wait also tells the compiler that
  // the Q registers are ready, so it adds no wait of its own inside the loop).
  for (int u = 0; u < kPPStages - 1 && u < n; ++u) issue_tile(u);
#pragma unroll
  for (int s = 0; s < kKSteps; ++s) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (my_row < T) x = ld16(qp + (int64_t)my_row * a.q_st + 8 * h2 + 16 * s);
    qreg[s] = __builtin_bit_cast(bf16x8, x);
  }
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  barrier();

  qk_part(0);
  if (grp == 1) sync_tile(0);
  valu_phase(0);
  if (grp == 0) sync_tile(0);
  // Tiles 1, 2, 3, 4, 5, .. use stages 1, 2, 3, 0, 1, ..: the loop runs four
  // tiles per pass with each stage a compile-time constant (its operand
  // addresses are then immediate offsets), the last n - 1 mod 4 tiles with
  // the stage computed.
  auto tile_step = [&](int t, int st) {
    mfma_phase(t, st);
    if (grp == 1) sync_tile(t);
    valu_phase(t);
    if (grp == 0) sync_tile(t);
  };
  int t = 1;
  for (; t + 3 < n; t += 4) {
    tile_step(t, 1);
    tile_step(t + 1, 2);
    tile_step(t + 2, 3);
    tile_step(t + 3, 0);
  }
  for (; t < n; ++t) tile_step(t, t % kPPStages);
  pv_part((n - 1) % kPPStages);
  // every wave passed the barrier of tile n-1 after its loads of the last
  // tiles completed, so the ring holds them
  if (APPEND && writer)
    for (int u = max(n - kPPStages, 0); u < n; ++u) append_tile(u, u % kPPStages);

  // Epilogue: normalise by the row sum, store.
  const float l_tot = xor32_sum(l_run);
  const float inv = 1.f / l_tot;
  if (my_row < T) {
    if (OUT_F32) {
      float* op = reinterpret_cast<float*>(a.out) + ooff + (int64_t)my_row * a.o_st + (int64_t)h * a.o_sh;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          f32x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = acc_o[mb][4 * q4 + e] * inv;
          *reinterpret_cast<f32x4*>(op + 32 * mb + 8 * q4 + 4 * h2) = w;
        }
    } else {
      uint16_t* op = reinterpret_cast<uint16_t*>(a.out) + ooff + (int64_t)my_row * a.o_st + (int64_t)h * a.o_sh;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          u32x2 w;
          w[0] = (uint32_t)f32_to_bf16_bits(acc_o[mb][4 * q4 + 0] * inv) |
                 ((uint32_t)f32_to_bf16_bits(acc_o[mb][4 * q4 + 1] * inv) << 16);
          w[1] = (uint32_t)f32_to_bf16_bits(acc_o[mb][4 * q4 + 2] * inv) |
                 ((uint32_t)f32_to_bf16_bits(acc_o[mb][4 * q4 + 3] * inv) << 16);
          *reinterpret_cast<u32x2*>(op + 32 * mb + 8 * q4 + 4 * h2) = w;
        }
    }
  }
}

// Dynamic tail of the d_head-128 launches.  The XCDs run at different speeds
// under this load (several percent apart), and the slowest sets the end of a
// launch whose items are dealt to them in equal shares.  The first items keep
// their static XCD-aware order; the light items at the end (the streaming
// items of the one-launch form, the second half of the items of a one-type
// launch) are taken dynamically: queue x holds the items the XCD-aware order
// puts on XCD x (index w with w % 8 == x), a workgroup takes the next item of
// the queue of the XCD it runs on (read from the XCC_ID register) or, once
// that is empty, of another queue, and the launch has kStreamSlack more
// workgroups than tail items so that a fast XCD can take over a slow one's
// share.  Workgroups that find every queue empty exit.
// The queue counters live in one of kSchedSlots slots of a device array,
// chosen per launch by the host; the last workgroup to take (or fail to take)
// an item clears the slot.  Launches that run at the same time therefore
// need different slots: consecutive launches take consecutive slots.
constexpr int kSchedSlots = 64;
constexpr float kStreamSlack = 0.25f;
__device__ uint32_t g_pp_sched[kSchedSlots][16];  // [0, 8): queue heads; [8]: workgroups served

// XCD (0..7) the calling wave runs on: bits 3:0 of hardware register XCC_ID.
__device__ __forceinline__ int pp_xcc() { return __builtin_amdgcn_s_getreg((3 << 11) | 20) & 7; }

// Next item for a workgroup on XCD x, or -1 when every queue is empty.
// Queue y holds ceil((n - y) / 8) items.
__device__ __forceinline__ int pp_grab(uint32_t* q, int n, int x) {
  {
    const int n_x = (n - x + 7) >> 3;
    if (n_x > 0) {
      const uint32_t k = atomicAdd(&q[x], 1u);
      if (k < (uint32_t)n_x) return 8 * (int)k + x;
    }
  }
  for (;;) {
    uint32_t head[8];
#pragma unroll
    for (int y = 0; y < 8; ++y) head[y] = __hip_atomic_load(&q[y], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int pick = -1;
    for (int d = 1; d < 8 && pick < 0; ++d) {
      const int y = (x + d) & 7;
      if (head[y] < (uint32_t)((n - y + 7) >> 3)) pick = y;
    }
    if (pick < 0) return -1;
    const uint32_t k = atomicAdd(&q[pick], 1u);
    if (k < (uint32_t)((n - pick + 7) >> 3)) return 8 * (int)k + pick;
  }
}

// Both head types of a layer in one launch: workgroups [0, n_ret) take the
// retrieval items, [ret_pad, ret_pad + n_dyn) the n_str streaming ones
// through the queues above (ret_pad = n_ret rounded up to the 8 XCDs, so both
// item spaces keep their XCD-aware order).  The light streaming items are
// dispatched last and fill the CUs that the causal retrieval items leave
// idle at the end.
// One tail item for this workgroup (every thread gets it), or -1: n tail
// items, n_dyn workgroups of the launch take part.  The last of them to take
// (or fail to take) an item clears the slot.
__device__ __forceinline__ int pp_take(int slot, int n, int n_dyn) {
  __shared__ int s_item;
  uint32_t* q = g_pp_sched[slot];
  if (threadIdx.x == 0) {
    s_item = pp_grab(q, n, pp_xcc());
    if (atomicAdd(&q[8], 1u) == (uint32_t)n_dyn - 1) {
#pragma unroll
      for (int y = 0; y < 9; ++y) atomicExch(&q[y], 0u);
    }
  }
  __syncthreads();
  return __builtin_amdgcn_readfirstlane(s_item);
}

// One head type: workgroups [0, n_static) take items [0, n_static) in the
// XCD-aware order, the n_dyn others the tail items [n_static, n_static + n_tail).
template <bool STREAM, bool OUT_F32, bool APPEND>
__global__ __launch_bounds__(512, 1) void prefill_pp_kernel(PrefillArgs a, int n_static, int n_tail, int n_dyn,
                                                            int slot) {
  __shared__ __align__(1024) PPRing ring;
  int w = blockIdx.x;
  if (w >= n_static) {
    w = pp_take(slot, n_tail, n_dyn);
    if (w < 0) return;
    w += n_static;
  }
  prefill_pp_body<STREAM, OUT_F32, APPEND>(a, w, ring);
}

// Both head types of a layer in one launch: workgroups [0, n_ret) take the
// retrieval items, [ret_pad, ret_pad + n_dyn) the n_str streaming ones
// through the queues (ret_pad = n_ret rounded up to the 8 XCDs, so both item
// spaces keep their XCD-aware order).  The light streaming items are
// dispatched last and fill the CUs that the causal retrieval items leave
// idle at the end.
template <bool OUT_F32, bool APPEND>
__global__ __launch_bounds__(512, 1) void prefill_pp_mixed_kernel(PrefillArgs ar, PrefillArgs as, int n_ret,
                                                                  int ret_pad, int n_str, int n_dyn, int slot) {
  __shared__ __align__(1024) PPRing ring;
  const int wg = blockIdx.x;
  if (wg < n_ret) {
    prefill_pp_body<false, OUT_F32, APPEND>(ar, wg, ring);
    return;
  }
  if (wg < ret_pad) return;
  const int w = pp_take(slot, n_str, n_dyn);
  if (w >= 0) prefill_pp_body<true, OUT_F32, APPEND>(as, w, ring);
}

static std::atomic<uint32_t> g_sched_next{0};
static int pp_slot() { return (int)(g_sched_next.fetch_add(1, std::memory_order_relaxed) % kSchedSlots); }
// Workgroups that take part in a dynamic tail of n items.
static int pp_n_dyn(int n) { return (int)((1.f + kStreamSlack) * n / 8 + 1) * 8; }

template <int D, bool STREAM, bool OUT_F32>
static hipError_t launch_bf16(const PrefillArgs& a, hipStream_t s) {
  const int grid = a.n_qblocks * a.n_kv * a.gs * a.B;
  if constexpr (D == kPPD) {
    // the first half of the items (a multiple of 8) static, the rest dynamic
    const int n_static = grid / 16 * 8, n_tail = grid - n_static, n_dyn = pp_n_dyn(n_tail);
    const int slot = pp_slot();
    if (a.append)
      hipLaunchKernelGGL((prefill_pp_kernel<STREAM, OUT_F32, true>), dim3(n_static + n_dyn), dim3(512), 0, s, a,
                         n_static, n_tail, n_dyn, slot);
    else
      hipLaunchKernelGGL((prefill_pp_kernel<STREAM, OUT_F32, false>), dim3(n_static + n_dyn), dim3(512), 0, s, a,
                         n_static, n_tail, n_dyn, slot);
  } else {
    if (a.append)
      hipLaunchKernelGGL((prefill_bf16_kernel<D, STREAM, OUT_F32, true>), dim3(grid), dim3(kWaves * kWave), 0, s, a);
    else
      hipLaunchKernelGGL((prefill_bf16_kernel<D, STREAM, OUT_F32, false>), dim3(grid), dim3(kWaves * kWave), 0, s, a);
  }
  return hipGetLastError();
}

template <int D, bool STREAM>
static hipError_t launch_f32(const PrefillArgs& a, hipStream_t s) {
  const int grid = a.n_qblocks * a.n_kv * a.gs * a.B;
  hipLaunchKernelGGL((prefill_f32_kernel<D, STREAM>), dim3(grid), dim3(kPrefillRowsF32), 0, s, a);
  return hipGetLastError();
}

// The mixed launch pays where the retrieval items fill only a few rounds of
// the 256 CUs (one 512-thread workgroup per CU): their causal tail is then a
// sizeable part of the launch.  Its retrieval path is compiled together with
// the streaming one and runs ~1-2% slower per tile, so long launches keep two
// kernels: measured on the 28/4-head d_head-128 layer, 1.6% faster at 32768
// tokens (7 rounds), even at 65536, 0.5-1.7% slower from 131072 on.
constexpr int kMixedMaxRetItems = 8 * 256;

bool prefill_mixed_preferred(const PrefillArgs& ar, int dtype, int d) {
  const int64_t n_ret = (int64_t)ar.n_qblocks * ar.n_kv * ar.gs * ar.B;
  return dtype == 0 && d == kPPD && n_ret <= kMixedMaxRetItems;
}

hipError_t launch_prefill_mixed(const PrefillArgs& ar, const PrefillArgs& as, int out_f32, hipStream_t s) {
  const int n_ret = ar.n_qblocks * ar.n_kv * ar.gs * ar.B;
  const int n_str = as.n_qblocks * as.n_kv * as.gs * as.B;
  const int ret_pad = (n_ret + 7) / 8 * 8;
  const int n_dyn = pp_n_dyn(n_str);
  const int slot = pp_slot();
  const dim3 grid(ret_pad + n_dyn), blk(512);
  const bool app = ar.append;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, blk, 0, s, ar, as, n_ret, ret_pad, n_str, n_dyn, slot);
  };
  if (out_f32) {
    if (app) go(prefill_pp_mixed_kernel<true, true>);
    else go(prefill_pp_mixed_kernel<true, false>);
  } else {
    if (app) go(prefill_pp_mixed_kernel<false, true>);
    else go(prefill_pp_mixed_kernel<false, false>);
  }
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
