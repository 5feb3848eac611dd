// Top-k positions of an H2Share anchor decode step (paper Sec. "AoH-Guided
// Sparse Attention: H2Share": anchor retrieval heads select the important
// token indices from their attention scores; GQA appendix: a group's query
// heads share one index set).
//
// One workgroup of 1024 threads per (sequence, retrieval KV head).  The score
// of position j is the sum over the group's query heads of their attention
// probability exp2(s_hj - m_h) / l_h (the mean up to the constant 1/gs, so the
// same ranking), from the scaled scores the split pass kept and the final
// (m, l) of the merge.  Probabilities are non-negative, so their fp32 bit
// patterns order like the values; the k-th largest bit pattern is found by a
// three-digit (11 + 11 + 10 bits) radix select over histograms in LDS, and the
// positions are then compacted in ascending order: every key above the
// threshold, and as many keys equal to it as still needed, lowest positions
// first.  Sequences with at most k positions select all of them; unused
// entries are -1.
#include "aoh_device.h"
#include "aoh_internal.h"

namespace aoh {
namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / kWave;

// Exclusive prefix sum over the workgroup (thread order) of one value per
// thread; also returns the total.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* wsum, uint32_t& total) {
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  __syncthreads();  // wsum may still be read by a previous scan
  if (lane == kWave - 1) wsum[wave] = x;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) {
    const uint32_t s = wsum[w];
    if (w < wave) before += s;
    tot += s;
  }
  total = tot;
  return before + x - v;
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(TopkArgs a) {
  __shared__ uint32_t hist[2048];
  __shared__ uint32_t wsum[kTopkWaves];
  __shared__ uint32_t s_bin, s_above;
  __shared__ float s_m[kMaxKvHeads], s_il[kMaxKvHeads];
  const int kvl = blockIdx.x, b = blockIdx.y;
  const int g = a.kv_heads[kvl];
  const int t = threadIdx.x;
  const int n = max(0, min(a.lens[b], a.score_len));
  const int k = a.n_sel;
  int32_t* out = a.sel + ((int64_t)b * a.n_kv + kvl) * k;
  if (n <= k) {
    for (int j = t; j < k; j += kTopkThreads) out[j] = j < n ? j : -1;
    return;
  }
  const int64_t row_stride = a.score_len;
  float* row0 = a.scores + ((int64_t)b * a.Hq + (int64_t)g * a.gs) * row_stride;
  uint32_t* keys = reinterpret_cast<uint32_t*>(row0);  // written over the first head's row
  if (t < a.gs) {
    const float* ml = a.ml + ((int64_t)b * a.Hq + g * a.gs + t) * 2;
    s_m[t] = ml[0];
    s_il[t] = 1.f / ml[1];
  }
  __syncthreads();
  for (int j = t; j < n; j += kTopkThreads) {
    float p = 0.f;
    for (int h = 0; h < a.gs; ++h) p += fast_exp2(row0[h * row_stride + j] - s_m[h]) * s_il[h];
    keys[j] = __builtin_bit_cast(uint32_t, p);
  }
  __syncthreads();

  // radix select of the k-th largest key
  uint32_t prefix = 0, pmask = 0;
  uint32_t kk = (uint32_t)k;  // rank (from the top, 1-based) still to find among keys matching prefix
#pragma unroll 1
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const int nb = pass == 2 ? 1024 : 2048;
    for (int i = t; i < 2048; i += kTopkThreads) hist[i] = 0;
    __syncthreads();
    for (int j = t; j < n; j += kTopkThreads) {
      const uint32_t key = keys[j];
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & (nb - 1)], 1u);
    }
    __syncthreads();
    // thread t owns the bins of descending rank 2t, 2t+1
    const int b_hi = nb - 1 - 2 * t, b_lo = nb - 2 - 2 * t;
    const uint32_t h_hi = b_hi >= 0 ? hist[b_hi] : 0u;
    const uint32_t h_lo = b_lo >= 0 ? hist[b_lo] : 0u;
    uint32_t total;
    const uint32_t above = block_excl_scan(h_hi + h_lo, wsum, total);
    if (above < kk && kk <= above + h_hi) {
      s_bin = (uint32_t)b_hi;
      s_above = above;
    } else if (above + h_hi < kk && kk <= above + h_hi + h_lo) {
      s_bin = (uint32_t)b_lo;
      s_above = above + h_hi;
    }
    __syncthreads();
    prefix |= s_bin << shift;
    pmask |= (uint32_t)(nb - 1) << shift;
    kk -= s_above;
    __syncthreads();  // s_bin / s_above are rewritten by the next pass
  }
  const uint32_t thr = prefix;
  const uint32_t need_eq = kk;  // keys equal to thr still to take

  // ascending compaction: each thread owns a contiguous segment of positions
  const int seg = (n + kTopkThreads - 1) / kTopkThreads;
  const int j0 = min(n, t * seg), j1 = min(n, j0 + seg);
  uint32_t gt = 0, eq = 0;
  for (int j = j0; j < j1; ++j) {
    const uint32_t key = keys[j];
    gt += key > thr;
    eq += key == thr;
  }
  uint32_t tot_gt, tot_eq;
  const uint32_t gt_before = block_excl_scan(gt, wsum, tot_gt);
  const uint32_t eq_before = block_excl_scan(eq, wsum, tot_eq);
  uint32_t pos = gt_before + min(eq_before, need_eq);
  uint32_t eq_seen = eq_before;
  for (int j = j0; j < j1; ++j) {
    const uint32_t key = keys[j];
    if (key > thr) {
      out[pos++] = j;
    } else if (key == thr) {
      if (eq_seen < need_eq) out[pos++] = j;
      ++eq_seen;
    }
  }
}

}  // namespace

hipError_t launch_topk(const TopkArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(topk_kernel, dim3(a.n_kv, a.B), dim3(kTopkThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace aoh
