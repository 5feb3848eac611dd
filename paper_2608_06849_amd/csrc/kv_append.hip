// KV-cache append (paper Sec. 5: retrieval heads retain every token; streaming
// heads evict all but the sink and the most recent tokens).
//
// One workgroup per (16-position page-aligned chunk, KV head, sequence).  The
// chunk is logical page start_pos/16 + blockIdx.x, clipped to the appended
// range [start, start + n_new), so the grid depends only on n_new and the
// start position is read on the device.
//   retrieval head -> paged cache: K rows copied as 16-byte vectors; V staged
//     in LDS and written dimension-major ([D][16] per page), only for the
//     positions of this append (a page may already hold earlier tokens), or,
//     for token-major V pages, copied like K.
//   streaming head -> ring: a position is written only if no later position of
//     the same append maps to its slot (p < n_sink or p >= end - window), so
//     the final state is independent of the order in which lanes write.
// All copies are bit-exact.
#include "aoh_device.h"
#include "aoh_internal.h"

namespace aoh {

template <int D, typename T>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  constexpr int kVec = 16 / sizeof(T);          // elements per 16-byte vector
  constexpr int kVecPerRow = D / kVec;
  __shared__ __align__(16) T vtile[kPage][D + kVec];

  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int start = (a.start_pos ? a.start_pos[b] : 0) + a.start_bias;
  if (start < 0) return;  // invalid start position: write nothing
  const int end = start + a.n_new;
  const int lp = start / kPage + (int)blockIdx.x;
  const int p_lo = max(lp * kPage, start);
  const int p_hi = min(lp * kPage + kPage, end);
  if (p_lo >= p_hi) return;
  const bool streaming = (a.streaming_mask >> g) & 1ull;
  const int rank = a.rank[g];

  const int tid = threadIdx.x;
  constexpr int kItems = kPage * kVecPerRow;    // 16-byte vectors per 16-position chunk
  const T* kn = reinterpret_cast<const T*>(a.k_new) + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh;
  const T* vn = reinterpret_cast<const T*>(a.v_new) + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh;

  if (!streaming) {
    // Positions beyond the block table, or unmapped/invalid pages, are skipped:
    // a write never leaves the cache.
    if (lp >= a.max_pages) return;
    const int page = a.block_table[(int64_t)b * a.max_pages + lp];
    if (page < 0 || page >= a.num_pages) return;
    const int64_t unit = (int64_t)page * a.n_ret + rank;
    T* pk = reinterpret_cast<T*>(a.pk) + unit * (kPage * D);
    T* pv = reinterpret_cast<T*>(a.pv) + unit * (kPage * D);
    for (int it = tid; it < kItems; it += blockDim.x) {
      const int row = it / kVecPerRow, cv = it % kVecPerRow;
      const int p = lp * kPage + row;
      if (p >= p_lo && p < p_hi) {
        const int t = p - start;
        st16(pk + (int64_t)row * D + cv * kVec, ld16(kn + (int64_t)t * a.k_st + cv * kVec));
        const u32x4 vv = ld16(vn + (int64_t)t * a.v_st + cv * kVec);
        if (a.v_token_major) st16(pv + (int64_t)row * D + cv * kVec, vv);
        else *reinterpret_cast<u32x4*>(&vtile[row][cv * kVec]) = vv;
      }
    }
    if (a.v_token_major) return;  // uniform across the workgroup
    __syncthreads();
    // Dimension-major V page: element (d, r) at pv[d * 16 + r].
    for (int e = tid; e < D * kPage; e += blockDim.x) {
      const int d = e / kPage, r = e % kPage;
      const int pp = lp * kPage + r;
      if (pp >= p_lo && pp < p_hi) pv[(int64_t)d * kPage + r] = vtile[r][d];
    }
  } else {
    for (int it = tid; it < kItems; it += blockDim.x) {
      const int row = it / kVecPerRow, cv = it % kVecPerRow;
      const int p = lp * kPage + row;
      if (p < p_lo || p >= p_hi) continue;
      if (!(p < a.n_sink || p >= end - a.window)) continue;  // overwritten later in this append
      const int t = p - start;
      const u32x4 kv = ld16(kn + (int64_t)t * a.k_st + cv * kVec);
      const u32x4 vv = ld16(vn + (int64_t)t * a.v_st + cv * kVec);
      const int slot = p < a.n_sink ? p : a.n_sink + (p - a.n_sink) % a.window;
      const int64_t unit = ((int64_t)b * a.n_str + rank) * a.ring_blocks + slot / kPage;
      const int r = slot % kPage;
      T* rk = reinterpret_cast<T*>(a.rk) + unit * (kPage * D);
      T* rv = reinterpret_cast<T*>(a.rv) + unit * (kPage * D);
      st16(rk + (int64_t)r * D + cv * kVec, kv);
      const T* ve = reinterpret_cast<const T*>(&vv);
#pragma unroll
      for (int e = 0; e < kVec; ++e) rv[(int64_t)(cv * kVec + e) * kPage + r] = ve[e];
    }
  }
}

template <int D, typename T>
static hipError_t launch(const AppendArgs& a, hipStream_t s) {
  dim3 grid(a.n_chunks, a.Hkv, a.B);
  hipLaunchKernelGGL((append_kernel<D, T>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, int dtype, int d, hipStream_t s) {
  if (dtype == 1) return d == 64 ? launch<64, float>(a, s) : launch<128, float>(a, s);
  return d == 64 ? launch<64, uint16_t>(a, s) : launch<128, uint16_t>(a, s);
}

}  // namespace aoh
