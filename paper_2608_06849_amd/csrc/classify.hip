// The effective-rank head classifier (paper Sec. 4, Eqs. 2-7 and Algorithm 1;
// group-level classification of the GQA appendix) on gfx950.
//
// For query head h of KV group g the method needs the singular values of
// M_h = W_K^g^T W_Q^h, obtained from the d_head x d_head proxy
// C_h = (W_Q W_Q^T)(W_K W_K^T) (Eq. 5): sigma_k^2 = lambda_k(C_h).  C_h is not
// symmetric, so instead of a general eigensolver this path uses the congruent
// symmetric matrix B_h = L_g^T (W_Q W_Q^T) L_g, where W_K W_K^T = L_g L_g^T
// (Cholesky): B_h = L^T QQ L is similar to QQ L L^T = C_h, so it has the same
// eigenvalues, and being symmetric positive semidefinite they are computed by
// Householder tridiagonalisation and Sturm-sequence bisection (Golub and Van
// Loan, Matrix Computations, Alg. 8.3.1 and Sec. 8.4.1).
//
// Kernels, in stream order:
//   gram_kernel      per (layer, head): G = W W^T over d_model, bf16 MFMA with
//                    fp32 accumulation, for the Hq query slices and Hkv key slices;
//   chol_kernel      per (layer, group): L_g from G_K in fp64 (LDS resident);
//   spectrum_kernel  per (layer, query head): B = L^T (QQ L) in fp64, tridiagonal
//                    form, all eigenvalues, sigma = sqrt(max(lambda, 0)) and
//                    eff_rank = exp(-sum p log p), p = sigma / sum sigma (Eq. 4);
//   select_kernel    per layer: group means and the k lowest groups as retrieval
//                    (stable: the lower group index wins a tie).
#include "aoh_device.h"
#include "aoh_internal.h"

namespace aoh {
namespace {

constexpr int kGramBK = 64;  // d_model columns per main-loop iteration

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

// G = W W^T for one d x d_model slice (W row-major, row stride rs elements).
// Wave w owns 32-row block w as the A operand and computes the 32x32 tiles
// (w, c) for c >= w; each tile is written with its transpose, so G is exactly
// symmetric.  The sum over d_model is order-free, so every lane loads 64
// contiguous bytes of its row per iteration and both operands use the same
// k mapping (k = k0 + 32 * half + 8 * s + j for MFMA step s, element j).
template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void gram_kernel(ClassifyArgs a) {
  constexpr int NRB = D / 32;
  const int n_heads = a.Hq + a.Hkv;
  const int u = blockIdx.x % n_heads;
  const int layer = blockIdx.x / n_heads;
  const bf16* w;
  int64_t rs;
  if (u < a.Hq) {
    w = static_cast<const bf16*>(a.wq) + layer * a.wq_sl + (int64_t)u * D * a.wq_sr;
    rs = a.wq_sr;
  } else {
    w = static_cast<const bf16*>(a.wk) + layer * a.wk_sl + (int64_t)(u - a.Hq) * D * a.wk_sr;
    rs = a.wk_sr;
  }
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;

  const bf16* rowa = w + (int64_t)(32 * wave + l32) * rs + 32 * half;
  const bf16* rowb[NRB];
#pragma unroll
  for (int c = 0; c < NRB; ++c) rowb[c] = w + (int64_t)(32 * c + l32) * rs + 32 * half;

  f32x16 acc[NRB];
#pragma unroll
  for (int c = 0; c < NRB; ++c) acc[c] = f32x16{};

  for (int k0 = 0; k0 < a.d_model; k0 += kGramBK) {
    u32x4 xa[4], xb[NRB][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) xa[s] = ld16(rowa + k0 + 8 * s);
#pragma unroll
    for (int c = 0; c < NRB; ++c)
      if (c >= wave)
#pragma unroll
        for (int s = 0; s < 4; ++s) xb[c][s] = ld16(rowb[c] + k0 + 8 * s);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int c = 0; c < NRB; ++c)
        if (c >= wave) acc[c] = mfma32(as_bf16x8(xa[s]), as_bf16x8(xb[c][s]), acc[c]);
  }

  float* g = a.gram + ((int64_t)layer * n_heads + u) * D * D;
#pragma unroll
  for (int c = 0; c < NRB; ++c) {
    if (c < wave) continue;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int m = 32 * wave + 8 * (i / 4) + 4 * half + (i % 4);
      const int n = 32 * c + l32;
      g[(int64_t)m * D + n] = acc[c][i];
      g[(int64_t)n * D + m] = acc[c][i];
    }
  }
}

constexpr int kEigThreads = 256;
constexpr int kEigWaves = kEigThreads / kWave;

// Right-looking Cholesky of G_K (fp64, in LDS).  A pivot <= 0 (W_K of lower
// rank than d_head, up to rounding) zeroes its column, which keeps L L^T equal
// to G_K on the range of W_K.
template <int D>
__global__ __launch_bounds__(kEigThreads) void chol_kernel(ClassifyArgs a) {
  __shared__ double A[D][D + 1];
  const int n_heads = a.Hq + a.Hkv;
  const int grp = blockIdx.x % a.Hkv;
  const int layer = blockIdx.x / a.Hkv;
  const float* g = a.gram + ((int64_t)layer * n_heads + a.Hq + grp) * D * D;
  const int t = threadIdx.x;
  for (int e = t; e < D * D; e += kEigThreads) A[e / D][e % D] = (double)g[e];
  __syncthreads();
  for (int k = 0; k < D; ++k) {
    const double dkk = A[k][k];
    const double lkk = dkk > 0.0 ? sqrt(dkk) : 0.0;
    const double inv = lkk > 0.0 ? 1.0 / lkk : 0.0;
    for (int i = k + 1 + t; i < D; i += kEigThreads) A[i][k] *= inv;
    __syncthreads();
    if (t == 0) A[k][k] = lkk;
    // trailing update of the lower triangle: rows i > k, columns k < j <= i
    const int wave = t >> 6, lane = t & 63;
    for (int i = k + 1 + wave; i < D; i += kEigWaves) {
      const double lik = A[i][k];
      for (int j = k + 1 + lane; j <= i; j += kWave) A[i][j] -= lik * A[j][k];
    }
    __syncthreads();
  }
  double* out = a.chol + ((int64_t)layer * a.Hkv + grp) * D * D;
  for (int e = t; e < D * D; e += kEigThreads) {
    const int i = e / D, j = e % D;
    out[e] = j <= i ? A[i][j] : 0.0;
  }
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

// Number of eigenvalues of the symmetric tridiagonal (d, e) below x (Sturm
// count from the LDL^T pivots; a pivot smaller than pivmin in magnitude is
// replaced by -pivmin).
template <int D>
__device__ __forceinline__ int sturm_count(const double* d, const double* e2, double x, double pivmin) {
  double q = d[0] - x;
  if (fabs(q) < pivmin) q = -pivmin;
  int c = q < 0.0;
  for (int i = 1; i < D; ++i) {
    q = (d[i] - x) - e2[i - 1] / q;
    if (fabs(q) < pivmin) q = -pivmin;
    c += q < 0.0;
  }
  return c;
}

template <int D>
__global__ __launch_bounds__(kEigThreads) void spectrum_kernel(ClassifyArgs a) {
  constexpr int R = D / 16;  // rows and columns per thread in the fp64 products
  __shared__ double A[D][D + 1];
  __shared__ double vv[D], pp[D], dd[D], ee[D];
  __shared__ double red[kEigWaves];

  const int n_heads = a.Hq + a.Hkv;
  const int h = blockIdx.x % a.Hq;
  const int layer = blockIdx.x / a.Hq;
  const int grp = h / a.gs;
  const float* qq = a.gram + ((int64_t)layer * n_heads + h) * D * D;
  const double* L = a.chol + ((int64_t)layer * a.Hkv + grp) * D * D;
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63;

  for (int e = t; e < D * D; e += kEigThreads) A[e / D][e % D] = (double)qq[e];
  __syncthreads();

  // T = QQ L  (thread tile: rows R*(t/16) + r, columns t%16 + 16c)
  const int r0 = R * (t / 16), c0 = t % 16;
  double acc[R][R];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < R; ++c) acc[r][c] = 0.0;
  for (int k = 0; k < D; ++k) {
    double lk[R], ar[R];
#pragma unroll
    for (int c = 0; c < R; ++c) lk[c] = L[(int64_t)k * D + c0 + 16 * c];
#pragma unroll
    for (int r = 0; r < R; ++r) ar[r] = A[r0 + r][k];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int c = 0; c < R; ++c) acc[r][c] = fma(ar[r], lk[c], acc[r][c]);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < R; ++c) A[r0 + r][c0 + 16 * c] = acc[r][c];
  __syncthreads();

  // B = L^T T
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < R; ++c) acc[r][c] = 0.0;
  for (int k = 0; k < D; ++k) {
    double lk[R], tc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) lk[r] = L[(int64_t)k * D + r0 + r];
#pragma unroll
    for (int c = 0; c < R; ++c) tc[c] = A[k][c0 + 16 * c];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int c = 0; c < R; ++c) acc[r][c] = fma(lk[r], tc[c], acc[r][c]);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < R; ++c) A[r0 + r][c0 + 16 * c] = acc[r][c];
  __syncthreads();
  // exact symmetry for the two-sided updates below
  for (int e = t; e < D * D; e += kEigThreads) {
    const int i = e / D, j = e % D;
    if (i < j) {
      const double s = 0.5 * (A[i][j] + A[j][i]);
      A[i][j] = s;
      A[j][i] = s;
    }
  }
  __syncthreads();

  // Householder tridiagonalisation: step k reflects rows/columns k+1..D-1 so
  // that column k has zeros below its subdiagonal.  Every wave computes the
  // column norm and the scalar K itself (same data, same order), so no extra
  // barrier is needed for them and all waves take the same branch.
  for (int k = 0; k < D - 2; ++k) {
    const int m = D - k - 1;
    const double x0 = A[k + 1][k];
    double part = 0.0;
    for (int i = 1 + lane; i < m; i += kWave) {
      const double x = A[k + 1 + i][k];
      part = fma(x, x, part);
    }
    const double xn2 = wave_sum_f64(part);
    if (xn2 == 0.0) {
      if (t == 0) { dd[k] = A[k][k]; ee[k] = x0; }
      continue;
    }
    const double nx = sqrt(fma(x0, x0, xn2));
    const double alpha = x0 > 0.0 ? -nx : nx;
    const double v0 = x0 - alpha;
    const double beta = 2.0 / fma(v0, v0, xn2);
    if (t == 0) { dd[k] = A[k][k]; ee[k] = alpha; }
    if (wave == 0)
      for (int i = lane; i < m; i += kWave) vv[i] = i == 0 ? v0 : A[k + 1 + i][k];
    __syncthreads();
    if (t < m) {
      double p = 0.0;
      for (int j = 0; j < m; ++j) p = fma(A[k + 1 + j][k + 1 + t], vv[j], p);
      pp[t] = beta * p;
    }
    __syncthreads();
    double pv = 0.0;
    for (int i = lane; i < m; i += kWave) pv = fma(pp[i], vv[i], pv);
    const double K = 0.5 * beta * wave_sum_f64(pv);
    for (int i = wave; i < m; i += kEigWaves) {
      const double vi = vv[i], wi = pp[i] - K * vi;
      for (int j = lane; j < m; j += kWave) {
        const double vj = vv[j], wj = pp[j] - K * vj;
        A[k + 1 + i][k + 1 + j] -= vi * wj + wi * vj;
      }
    }
    __syncthreads();
  }
  if (t == 0) {
    dd[D - 2] = A[D - 2][D - 2];
    dd[D - 1] = A[D - 1][D - 1];
    ee[D - 2] = A[D - 1][D - 2];
  }
  __syncthreads();
  double* e2 = pp;  // squared off-diagonal
  if (t < D - 1) e2[t] = ee[t] * ee[t];
  __syncthreads();

  // Gershgorin interval and the pivot floor (every thread, same order)
  double lo = dd[0] - fabs(ee[0]), hi = dd[0] + fabs(ee[0]), emax2 = 0.0;
  for (int i = 1; i < D; ++i) {
    const double r = fabs(ee[i - 1]) + (i < D - 1 ? fabs(ee[i]) : 0.0);
    lo = fmin(lo, dd[i] - r);
    hi = fmax(hi, dd[i] + r);
  }
  for (int i = 0; i < D - 1; ++i) emax2 = fmax(emax2, e2[i]);
  const double eps = 2.220446049250313e-16;
  const double pivmin = 2.2250738585072014e-308 * fmax(1.0, emax2);
  const double tnorm = fmax(fabs(lo), fabs(hi));
  const double atol = eps * tnorm;

  double sigma = 0.0;
  if (t < D) {
    // eigenvalue number t (ascending): count(a) <= t < count(b)
    double lo_t = lo - 2.0 * atol - pivmin, hi_t = hi + 2.0 * atol + pivmin;
    for (int it = 0; it < 160; ++it) {
      if (hi_t - lo_t <= 2.0 * eps * fmax(fabs(lo_t), fabs(hi_t)) + atol) break;
      const double mid = lo_t + 0.5 * (hi_t - lo_t);
      if (mid <= lo_t || mid >= hi_t) break;
      if (sturm_count<D>(dd, e2, mid, pivmin) > t) hi_t = mid; else lo_t = mid;
    }
    // eigenvalues at or below the rounding floor of the reduction are zero
    // (a rank-deficient W_Q or W_K leaves only such values), so they add no
    // term to the entropy; for the zero matrix every eigenvalue is zero
    const double lam = 0.5 * (lo_t + hi_t);
    sigma = (tnorm > 0.0 && lam > D * atol) ? sqrt(lam) : 0.0;
  }

  // eff_rank = exp(-sum p log p), p = sigma / sum sigma over sigma > 0
  double s = wave_sum_f64(sigma);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  double ssum = 0.0;
#pragma unroll
  for (int w = 0; w < kEigWaves; ++w) ssum += red[w];
  __syncthreads();
  double term = 0.0;
  if (sigma > 0.0 && ssum > 0.0) {
    const double p = sigma / ssum;
    term = p * log(p);
  }
  s = wave_sum_f64(term);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  if (t == 0) {
    double hsum = 0.0;
#pragma unroll
    for (int w = 0; w < kEigWaves; ++w) hsum += red[w];
    a.head_rank[(int64_t)layer * a.Hq + h] = exp(-hsum);
  }
}

// Group score = mean eff_rank of the group's query heads; the n_retrieval
// lowest scores are retrieval groups (0), the rest streaming (1).
__global__ __launch_bounds__(kWave) void select_kernel(ClassifyArgs a) {
  __shared__ double sc[kMaxKvHeads];
  const int layer = blockIdx.x;
  const int g = threadIdx.x;
  double s = 0.0;
  if (g < a.Hkv) {
    const double* hr = a.head_rank + (int64_t)layer * a.Hq + g * a.gs;
    for (int j = 0; j < a.gs; ++j) s += hr[j];
    s /= a.gs;
    sc[g] = s;
  }
  __syncthreads();
  if (g < a.Hkv) {
    int rank = 0;
    for (int o = 0; o < a.Hkv; ++o) rank += (sc[o] < s) || (sc[o] == s && o < g);
    a.group_score[(int64_t)layer * a.Hkv + g] = s;
    a.head_is_streaming[(int64_t)layer * a.Hkv + g] = rank >= a.n_retrieval ? 1 : 0;
  }
}

template <int D>
hipError_t launch_classify_d(const ClassifyArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(gram_kernel<D>, dim3(a.L * (a.Hq + a.Hkv)), dim3(64 * (D / 32)), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chol_kernel<D>, dim3(a.L * a.Hkv), dim3(kEigThreads), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(spectrum_kernel<D>, dim3(a.L * a.Hq), dim3(kEigThreads), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(select_kernel, dim3(a.L), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_classify(const ClassifyArgs& a, int d, hipStream_t s) {
  return d == 128 ? launch_classify_d<128>(a, s) : launch_classify_d<64>(a, s);
}

}  // namespace aoh
