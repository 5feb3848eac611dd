// Head-mixed causal prefill on gfx950.
//
// Computes, per (batch, query head, query row i), the attention of the paper's
// Sec. 5 (chunked-prefill stage): softmax over the visible keys of
// q_i . k_j / sqrt(D), times V.  Retrieval heads see j <= i; streaming heads
// see j <= i with j < n_sink or i - j < window.
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
constexpr int kWaves = kPrefillWaves;  // waves per workgroup
constexpr int kRowsPerWave = 32;

#ifndef AOH_PREFILL_V_PAD
#define AOH_PREFILL_V_PAD 32
#endif
template <int D>
struct PrefillLds {
  // Row paddings (bf16 elements): K rows are read 16 bytes per lane down 32
  // rows; V rows are read by the transpose read as 4 rows x 32 bytes per
  // 16 lanes.  Each padding spreads its access pattern over distinct banks.
  static constexpr int kStrideK = D + 8;
  static constexpr int kStrideV = D + AOH_PREFILL_V_PAD;
  uint16_t k[kBN][kStrideK];
  uint16_t v[kBN][kStrideV];
};

// Lazy rescaling threshold (log2 units): the running max used for the
// exponentials is only raised when a row's true max exceeds it by more than
// this, so P stays below 2^8 and the O rescale is skipped on most tiles.
constexpr float kRescaleThreshold = 8.0f;

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
__device__ __forceinline__ TilePlan make_plan(int i0, int rows, int T, int n_sink, int window) {
  const int last_row = min(i0 + rows - 1, T - 1);
  const int last_tile = last_row / kBN;
  TilePlan p;
  if (!STREAM) {
    p.n_sink_tiles = 0;
    p.band_first = 0;
    p.n_visit = last_tile + 1;
  } else {
    const int band_lo = max(0, i0 - window + 1);
    p.band_first = band_lo / kBN;
    const int sink_tiles = (n_sink + kBN - 1) / kBN;
    p.n_sink_tiles = min(sink_tiles, p.band_first);
    p.n_visit = p.n_sink_tiles + (last_tile - p.band_first + 1);
  }
  return p;
}

template <int D, bool STREAM, bool OUT_F32>
__global__ __launch_bounds__(kWaves * kWave, 2) void prefill_bf16_kernel(PrefillArgs a) {
  __shared__ __align__(16) PrefillLds<D> lds;
  constexpr int kChunksPerRow = D / 8;                     // 16-byte chunks per key row
  constexpr int kChunksPerThread = kBN * kChunksPerRow / (kWaves * kWave);
  constexpr int kKSteps = D / 16;                          // MFMA k-steps over D
  constexpr int kMBlocks = D / 32;                         // 32-dim blocks of O^T

  const int n_qh = a.n_kv * a.gs;
  const int per_block = n_qh * a.B;
  const int wg = blockIdx.x;
  // Heaviest query blocks first (longest-processing-time order) for causal work.
  const int qb = a.n_qblocks - 1 - wg / per_block;
  const int rem = wg % per_block;
  const int qh_local = rem % n_qh;
  const int b = rem / n_qh;
  const int g = a.kv_heads[qh_local / a.gs];
  const int h = g * a.gs + (qh_local % a.gs);

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int h2 = lane >> 5;
  const int T = a.T;
  const int i0 = qb * kPrefillRows;
  const int r0 = i0 + wave * kRowsPerWave;
  const int my_row = r0 + l32;

  const uint16_t* qp = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh;
  const uint16_t* kp = reinterpret_cast<const uint16_t*>(a.k) + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh;
  const uint16_t* vp = reinterpret_cast<const uint16_t*>(a.v) + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh;

  // Q^T operand: lane holds row my_row, dims 8*h2 + 16*s .. +8.
  bf16x8 qreg[kKSteps];
#pragma unroll
  for (int s = 0; s < kKSteps; ++s) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (my_row < T) x = ld16(qp + (int64_t)my_row * a.q_st + 8 * h2 + 16 * s);
    qreg[s] = __builtin_bit_cast(bf16x8, x);
  }

  f32x16 acc_o[kMBlocks];
#pragma unroll
  for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc_o[mb][i] = 0.f;
  float m_run = -INFINITY;  // reference max (log2 units) of this lane's row
  float l_run = 0.f;        // this lane's partial row sum (partner lane has the rest)

  const TilePlan plan = make_plan<STREAM>(i0, kPrefillRows, T, a.n_sink, a.window);

  // Cooperative tile staging: registers -> LDS.
  u32x4 kst[kChunksPerThread], vst[kChunksPerThread];
  auto load_tile = [&](int kb) {
#pragma unroll
    for (int r = 0; r < kChunksPerThread; ++r) {
      const int c = tid + r * kWaves * kWave;
      const int row = c / kChunksPerRow;
      const int col = (c % kChunksPerRow) * 8;
      const int key = kb + row;
      if (key < T) {
        kst[r] = ld16(kp + (int64_t)key * a.k_st + col);
        vst[r] = ld16(vp + (int64_t)key * a.v_st + col);
      } else {
        kst[r] = u32x4{0u, 0u, 0u, 0u};
        vst[r] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int r = 0; r < kChunksPerThread; ++r) {
      const int c = tid + r * kWaves * kWave;
      const int row = c / kChunksPerRow;
      const int col = (c % kChunksPerRow) * 8;
      *reinterpret_cast<u32x4*>(&lds.k[row][col]) = kst[r];
      *reinterpret_cast<u32x4*>(&lds.v[row][col]) = vst[r];
    }
  };

  const float c = a.scale_log2;
  // One 64-key tile for this wave: S^T, online softmax, O^T += V^T P^T.
  // MASKED selects the per-element mask; full tiles carry no mask code.
  auto tile_step = [&](int kb, auto masked) {
    constexpr bool MASKED = decltype(masked)::value;
    f32x16 s_acc[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int i = 0; i < 16; ++i) s_acc[blk][i] = 0.f;
#pragma unroll
      for (int s = 0; s < kKSteps; ++s) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8*>(&lds.k[32 * blk + l32][8 * h2 + 16 * s]);
        s_acc[blk] = mfma32(kop, qreg[s], s_acc[blk]);
      }
    }
    // Mask (raw scores), row max of the raw scores.
    float mx = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float x = s_acc[blk][i];
        if (MASKED) {
          const int key = kb + 32 * blk + 8 * (i >> 2) + 4 * h2 + (i & 3);
          bool vis = key <= my_row;
          if (STREAM) vis = vis && (key < a.n_sink || my_row - key < a.window);
          x = vis ? x : -INFINITY;
          s_acc[blk][i] = x;
        }
        mx = fmaxf(mx, x);
      }
    mx = wave_xor_max(mx, 32) * c;  // log2 units (c > 0 keeps the order)
    // Raise the reference max only when some row needs it (wave-uniform).
    if (__any(mx > m_run + kRescaleThreshold)) {
      const float m_new = fmaxf(m_run, mx);
      // 0 when only m_run is -inf; 1 when the row has seen no visible key yet.
      const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc_o[mb][i] *= alpha;
    }
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    float psum = 0.f;
    bf16x8 pop[4];  // P^T operands for the 4 key steps of 16 keys
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = fast_exp2(fmaf(s_acc[blk][i], c, -m_use));
        psum += p;
        pop[blk * 2 + (i >> 3)][i & 7] = f32_to_bf16(p);
      }
    l_run += psum;

    // O^T += V^T . P^T.  Key step t covers keys 16t..16t+15; the k index
    // 8*h2 + j maps to key 16t + 4*h2 + j (j < 4) or 16t + 8 + 4*h2 + (j-4).
    const int q16 = lane >> 4;        // 16-lane block
    const int i16 = lane & 15;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int vrow = 16 * t + 4 * h2 + (i16 >> 2);
#pragma unroll
      for (int mb = 0; mb < kMBlocks; ++mb) {
        const int vcol = 32 * mb + 16 * (q16 & 1) + 4 * (i16 & 3);
        const i16x4 lo = lds_read_tr16(&lds.v[vrow][vcol]);
        const i16x4 hi = lds_read_tr16(&lds.v[vrow + 8][vcol]);
        // Whole-vector concatenation: per-element bf16 insertion of the
        // transposed halves is avoided on purpose (it was lowered to a
        // broadcast of the first element by this toolchain).
        const i16x8 cat = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        acc_o[mb] = mfma32(__builtin_bit_cast(bf16x8, cat), pop[t], acc_o[mb]);
      }
    }
  };

  if (plan.n_visit > 0) load_tile(plan.tile(0) * kBN);

  for (int it = 0; it < plan.n_visit; ++it) {
    const int kb = plan.tile(it) * kBN;
    store_tile();
    __syncthreads();
    if (it + 1 < plan.n_visit) load_tile(plan.tile(it + 1) * kBN);

    // Is any element of this wave's 32 x 64 block visible?  Is every element?
    const bool wave_dead = (kb > r0 + kRowsPerWave - 1) ||
                           (STREAM && kb >= a.n_sink && (r0 - (kb + kBN - 1)) >= a.window);
    if (!wave_dead) {
      const bool need_mask = (kb + kBN - 1 > r0) ||
                             (STREAM && !(kb + kBN - 1 < a.n_sink ||
                                          (r0 + kRowsPerWave - 1) - kb < a.window));
      if (need_mask) tile_step(kb, std::true_type{});
      else tile_step(kb, std::false_type{});
    }
    __syncthreads();
  }

  // Epilogue: combine the two half-row sums, normalise, store.
  const float l_tot = wave_xor_sum(l_run, 32);
  const float inv = 1.f / l_tot;
  if (my_row < T) {
    if (OUT_F32) {
      float* op = reinterpret_cast<float*>(a.out) + (int64_t)b * a.o_sb + (int64_t)my_row * a.o_st +
                  (int64_t)h * a.o_sh;
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
      uint16_t* op = reinterpret_cast<uint16_t*>(a.out) + (int64_t)b * a.o_sb + (int64_t)my_row * a.o_st +
                     (int64_t)h * a.o_sh;
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
  if (i >= a.T) return;
  const float* qp = reinterpret_cast<const float*>(a.q) + (int64_t)b * a.q_sb + (int64_t)i * a.q_st +
                    (int64_t)h * a.q_sh;
  const float* kp = reinterpret_cast<const float*>(a.k) + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh;
  const float* vp = reinterpret_cast<const float*>(a.v) + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh;
  float q[D], o[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = qp[d];
    o[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  int lo = 0, sink_end = 0;
  if (STREAM) {
    lo = max(0, i - a.window + 1);
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
  float* op = reinterpret_cast<float*>(a.out) + (int64_t)b * a.o_sb + (int64_t)i * a.o_st + (int64_t)h * a.o_sh;
  const float inv = 1.f / l;
#pragma unroll
  for (int d = 0; d < D; ++d) op[d] = o[d] * inv;
}

template <int D, bool STREAM, bool OUT_F32>
static hipError_t launch_bf16(const PrefillArgs& a, hipStream_t s) {
  const int grid = a.n_qblocks * a.n_kv * a.gs * a.B;
  hipLaunchKernelGGL((prefill_bf16_kernel<D, STREAM, OUT_F32>), dim3(grid), dim3(kWaves * kWave), 0, s, a);
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
