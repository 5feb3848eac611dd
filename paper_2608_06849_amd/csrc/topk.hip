// Top-k positions of an H2Share anchor decode step (paper Sec. "AoH-Guided
// Sparse Attention: H2Share": anchor retrieval heads select the important
// token indices from their attention scores; GQA appendix: a group's query
// heads share one index set).
//
// Each (sequence, retrieval KV head) list is cut into kTopkParts segments, one
// workgroup of 1024 threads each, over three launches that exchange partial
// histograms through the workspace (no atomics in memory).  The score
// of position j is the sum over the group's query heads of their attention
// probability exp2(s_hj - m_h) / l_h (the mean up to the constant 1/gs, so the
// same ranking), from the scaled scores the split pass kept (16-bit offsets
// below a per-block reference) and the final (m, l) of the merge.  Probabilities are non-negative, so their fp32 bit
// patterns order like the values.  Keys keep the top 22 bits of the pattern
// (8 exponent and 13 mantissa bits: 1.2e-4 relative), so the k-th largest key
// is found by a two-digit (11 + 11 bits) radix select over per-segment
// histograms, and the
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

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

constexpr int kHistCopies = 4;  // lanes spread their increments over 4 copies (hot bins)
constexpr int kTile = 4 * kTopkThreads;  // positions per compaction tile

struct ListView {
  int n;                 // positions of the list (lens clamped to the score row)
  int seg0, seg1;        // this workgroup's segment [seg0, seg1)
  uint32_t* keys;        // key row of the list
  const uint32_t* part;  // partial histograms of the list [kTopkPasses][kTopkParts][2048]
  uint32_t* my_part;     // this workgroup's [kTopkPasses][...] slot base
  int32_t* out;
};

__device__ __forceinline__ ListView list_view(const TopkArgs& a) {
  ListView v;
  const int p = blockIdx.x, kvl = blockIdx.y, b = blockIdx.z;
  v.n = max(0, min(a.lens[b], a.score_len));
  // segments are whole compaction tiles
  const int per = (v.n + kTopkParts - 1) / kTopkParts;
  const int seg = ((per + kTile - 1) / kTile) * kTile;
  v.seg0 = min(v.n, p * seg);
  v.seg1 = min(v.n, v.seg0 + seg);
  const int64_t list = (int64_t)b * a.n_kv + kvl;
  v.keys = a.keys + list * a.score_len;
  v.part = a.part + list * kTopkPasses * kTopkParts * 2048;
  v.my_part = a.part + list * kTopkPasses * kTopkParts * 2048 + (int64_t)p * 2048;
  v.out = a.sel + list * a.n_sel;
  return v;
}

// The digit of the k-th largest key among those matching the earlier digits:
// sum the partial histograms of `pass` over the parts, then scan from the top.
__device__ __forceinline__ void find_digit(const uint32_t* part, int pass, int nb, uint32_t& kk, uint32_t& bin,
                                           uint32_t* wsum, uint32_t* s_bin) {
  const int t = threadIdx.x;
  const int b_hi = nb - 1 - 2 * t, b_lo = nb - 2 - 2 * t;
  uint32_t h_hi = 0, h_lo = 0;
  for (int q = 0; q < kTopkParts; ++q) {
    const uint32_t* h = part + ((int64_t)pass * kTopkParts + q) * 2048;
    if (b_hi >= 0) h_hi += h[b_hi];
    if (b_lo >= 0) h_lo += h[b_lo];
  }
  uint32_t total;
  const uint32_t above = block_excl_scan(h_hi + h_lo, wsum, total);
  if (above < kk && kk <= above + h_hi) {
    s_bin[0] = (uint32_t)b_hi;
    s_bin[1] = above;
  } else if (above + h_hi < kk && kk <= above + h_hi + h_lo) {
    s_bin[0] = (uint32_t)b_lo;
    s_bin[1] = above + h_hi;
  }
  __syncthreads();
  bin = s_bin[0];
  kk -= s_bin[1];
  __syncthreads();
}

constexpr int kShift[kTopkPasses] = {21, 10};
constexpr int kBins[kTopkPasses] = {2048, 2048};
constexpr uint32_t kKeyMask = 0xFFFFFC00u;  // the key bits the two digits cover

// Threshold key (the k-th largest) and the number of keys equal to it to take,
// from the histograms of both digits.
__device__ __forceinline__ void threshold(const ListView& v, int k, uint32_t& thr, uint32_t& need_eq,
                                          uint32_t* wsum, uint32_t* s_bin) {
  uint32_t kk = (uint32_t)k, prefix = 0, bin;
#pragma unroll
  for (int pass = 0; pass < kTopkPasses; ++pass) {
    find_digit(v.part, pass, kBins[pass], kk, bin, wsum, s_bin);
    prefix |= bin << kShift[pass];
  }
  thr = prefix;
  need_eq = kk;
}

// Pass PASS: keys (PASS 0 only) and the histogram of digit PASS of this
// workgroup's segment, among keys matching the digits already found.
template <int PASS>
__global__ __launch_bounds__(kTopkThreads) void topk_hist_kernel(TopkArgs a) {
  __shared__ uint32_t hist[kHistCopies][2048];
  __shared__ uint32_t wsum[kTopkWaves];
  __shared__ uint32_t s_bin[2];
  __shared__ float s_m[16], s_il[16];
  const ListView v = list_view(a);
  if (v.n <= a.n_sel) return;  // everything is selected: nothing to rank
  const int t = threadIdx.x;
  const int b = blockIdx.z, g = a.kv_heads[blockIdx.y];
  uint32_t prefix = 0, pmask = 0;
  if (PASS > 0) {
    uint32_t kk = (uint32_t)a.n_sel, bin;
#pragma unroll
    for (int q = 0; q < PASS; ++q) {
      find_digit(v.part, q, kBins[q], kk, bin, wsum, s_bin);
      prefix |= bin << kShift[q];
      pmask |= (uint32_t)(kBins[q] - 1) << kShift[q];
    }
  }
  for (int i = t; i < kHistCopies * 2048; i += kTopkThreads) (&hist[0][0])[i] = 0;
  if (PASS == 0 && t < a.gs) {
    const float* ml = a.ml + ((int64_t)b * a.Hq + g * a.gs + t) * 2;
    s_m[t] = ml[0];
    s_il[t] = 1.f / ml[1];
  }
  __syncthreads();
  uint32_t* my_hist = hist[t & (kHistCopies - 1)];
  const int64_t row = a.score_len;
  const int64_t head0 = (int64_t)b * a.Hq + (int64_t)g * a.gs;
  const uint16_t* c0 = a.score_codes + head0 * row;
  const float* r0 = a.score_refs + head0 * (row / 16);
  for (int j = v.seg0 + t; j < v.seg1; j += kTopkThreads) {
    uint32_t key;
    if (PASS == 0) {
      // score = ref - code / kScoreCodeScale (log2 units): a grid point,
      // computed exactly, so equal kept scores give equal keys
      float p = 0.f;
      for (int h = 0; h < a.gs; ++h) {
        const float xq = r0[h * (row / 16) + j / 16] - (float)c0[h * row + j] * (1.f / kScoreCodeScale);
        p += fast_exp2(xq - s_m[h]) * s_il[h];
      }
      key = __builtin_bit_cast(uint32_t, p) & kKeyMask;
      v.keys[j] = key;
    } else {
      key = v.keys[j];
    }
    if ((key & pmask) == prefix) atomicAdd(&my_hist[(key >> kShift[PASS]) & (kBins[PASS] - 1)], 1u);
  }
  __syncthreads();
  uint32_t* dst = v.my_part + (int64_t)PASS * kTopkParts * 2048;
  for (int i = t; i < 2048; i += kTopkThreads) {
    uint32_t c = 0;
#pragma unroll
    for (int q = 0; q < kHistCopies; ++q) c += hist[q][i];
    dst[i] = c;
  }
}

// Keys above and equal to the threshold in the segments before this
// workgroup's, from their partial histograms: keys carry exactly the two
// digits, so a key above the threshold has a larger first digit, or the same
// first digit and a larger second one, and a key equal to it has both digits.
__device__ __forceinline__ void counts_before(const ListView& v, uint32_t thr, uint32_t& gt, uint32_t& eq,
                                              uint32_t* wsum) {
  const int t = threadIdx.x;
  const uint32_t d0 = thr >> kShift[0], d1 = (thr >> kShift[1]) & (kBins[1] - 1);
  uint32_t my_gt = 0, my_eq = 0;
  for (int q = 0; q < (int)blockIdx.x; ++q) {
    const uint32_t* h0 = v.part + (int64_t)q * 2048;
    const uint32_t* h1 = v.part + ((int64_t)kTopkParts + q) * 2048;
    for (int b = t; b < 2048; b += kTopkThreads) {
      if ((uint32_t)b > d0) my_gt += h0[b];
      if ((uint32_t)b > d1) my_gt += h1[b];
    }
    if (t == 0) my_eq += h1[d1];
  }
  block_excl_scan(my_gt, wsum, gt);
  block_excl_scan(my_eq, wsum, eq);
}

// Ascending compaction of this workgroup's segment into the list: tiles of
// 4 x 1024 consecutive positions (4 per thread, coalesced); tied keys are
// ranked from the counts of the earlier segments and wave scans.
__global__ __launch_bounds__(kTopkThreads) void topk_compact_kernel(TopkArgs a) {
  __shared__ uint32_t wsum[kTopkWaves];
  __shared__ uint32_t s_bin[2];
  __shared__ uint32_t s_weq[kTopkWaves], s_wsel[kTopkWaves];
  const ListView v = list_view(a);
  const int t = threadIdx.x;
  const int k = a.n_sel;
  if (v.n <= k) {
    if (blockIdx.x == 0)
      for (int j = t; j < k; j += kTopkThreads) v.out[j] = j < v.n ? j : -1;
    return;
  }
  uint32_t thr, need_eq;
  threshold(v, k, thr, need_eq, wsum, s_bin);
  uint32_t gt_before, eq_before0;
  counts_before(v, thr, gt_before, eq_before0, wsum);
  const int lane = t & (kWave - 1), wave = t / kWave;
  uint32_t carry_eq = eq_before0;
  uint32_t carry_sel = gt_before + min(eq_before0, need_eq);
  const uint32_t* keys = v.keys;
  for (int base = v.seg0; base < v.seg1; base += kTile) {
    const int j0 = base + 4 * t;
    uint32_t kv[4];
    if (j0 + 4 <= v.seg1) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(keys + j0);
#pragma unroll
      for (int i = 0; i < 4; ++i) kv[i] = w[i];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) kv[i] = j0 + i < v.seg1 ? keys[j0 + i] : 0u;
    }
    uint32_t n_eq = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) n_eq += (j0 + i < v.seg1 && kv[i] == thr);
    const uint32_t eq_incl = wave_incl_scan(n_eq);
    if (lane == kWave - 1) s_weq[wave] = eq_incl;
    __syncthreads();
    uint32_t eq_rank = carry_eq, eq_tile = 0;
#pragma unroll
    for (int w = 0; w < kTopkWaves; ++w) {
      if (w < wave) eq_rank += s_weq[w];
      eq_tile += s_weq[w];
    }
    eq_rank += eq_incl - n_eq;
    bool sel[4];
    uint32_t n_sel = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool valid = j0 + i < v.seg1;
      const bool gt = valid && kv[i] > thr;
      const bool eqk = valid && kv[i] == thr;
      sel[i] = gt || (eqk && eq_rank < need_eq);
      eq_rank += eqk;
      n_sel += sel[i];
    }
    const uint32_t sel_incl = wave_incl_scan(n_sel);
    if (lane == kWave - 1) s_wsel[wave] = sel_incl;
    __syncthreads();
    uint32_t pos = carry_sel, sel_tile = 0;
#pragma unroll
    for (int w = 0; w < kTopkWaves; ++w) {
      if (w < wave) pos += s_wsel[w];
      sel_tile += s_wsel[w];
    }
    pos += sel_incl - n_sel;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (sel[i]) v.out[pos++] = j0 + i;
    carry_sel += sel_tile;
    carry_eq += eq_tile;
    __syncthreads();  // s_weq / s_wsel are rewritten by the next tile
  }
}

}  // namespace

hipError_t launch_topk(const TopkArgs& a, hipStream_t s) {
  const dim3 grid(kTopkParts, a.n_kv, a.B);
  hipLaunchKernelGGL(topk_hist_kernel<0>, grid, dim3(kTopkThreads), 0, s, a);
  hipLaunchKernelGGL(topk_hist_kernel<1>, grid, dim3(kTopkThreads), 0, s, a);
  hipLaunchKernelGGL(topk_compact_kernel, grid, dim3(kTopkThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace aoh
