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
// The slice is streamed through LDS 64 columns at a time: every thread loads
// 64 contiguous bytes of one row (two threads per row), one stage ahead of the
// MFMAs.  Wave w owns 32-row block w as the A operand and computes the 32x32
// tiles (w, c) for c >= w; each tile is written with its transpose, so G is
// exactly symmetric.  The sum over d_model is order-free, so both operands use
// the same k mapping (k = k0 + 32 * half + 8 * s + j for MFMA step s, element j).
constexpr int kGramRowPad = kGramBK + 8;  // bf16 per LDS row (bank spread)

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void gram_kernel(ClassifyArgs a) {
  constexpr int NRB = D / 32;
  __shared__ __align__(16) bf16 stage[2][D][kGramRowPad];
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
  const int t = threadIdx.x;
  const int wave = t >> 6;
  const int lane = t & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int lrow = t >> 1, lcol = (t & 1) * 32;  // this thread's part of a stage
  const bf16* src = w + (int64_t)lrow * rs + lcol;

  f32x16 acc[NRB];
#pragma unroll
  for (int c = 0; c < NRB; ++c) acc[c] = f32x16{};

  u32x4 ld[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int s = 0; s < 4; ++s) ld[s] = ld16(src + k0 + 8 * s);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int s = 0; s < 4; ++s) st16(&stage[buf][lrow][lcol + 8 * s], ld[s]);
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bf16x8 xa = as_bf16x8(*reinterpret_cast<const u32x4*>(&stage[buf][32 * wave + l32][32 * half + 8 * s]));
#pragma unroll
      for (int c = 0; c < NRB; ++c)
        if (c >= wave) {
          const bf16x8 xb = as_bf16x8(*reinterpret_cast<const u32x4*>(&stage[buf][32 * c + l32][32 * half + 8 * s]));
          acc[c] = mfma32(xa, xb, acc[c]);
        }
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();
  const int n_it = a.d_model / kGramBK;
  for (int it = 0; it < n_it; ++it) {
    const int cur = it & 1;
    const bool more = it + 1 < n_it;
    if (more) gload((it + 1) * kGramBK);
    compute(cur);
    if (more) lstore(cur ^ 1);
    __syncthreads();
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

// DPP move of a double (both 32-bit halves take the same lane pattern); lanes
// outside row_mask receive 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROW_MASK, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROW_MASK, 0xf, false);
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

// The fp64 D x D matrices of the two kernels below live in registers: row i
// belongs to the TPR = 256 / D adjacent threads t = TPR * i ... TPR * i + TPR - 1,
// each holding CPT = D / TPR consecutive columns.  By symmetry a row doubles
// as a column, so each elimination step publishes one row through LDS and
// every update is local to its owner.

// Right-looking Cholesky of G_K = L L^T.  Step k: the owners of row k publish
// it, every thread takes pivot and multiplier from it, writes its element of
// column k of L and updates its own row.  A pivot <= 0 (W_K of lower rank
// than d_head, up to rounding) zeroes its column, which keeps L L^T equal to
// G_K on the range of W_K.  The update runs over whole rows: left of the
// pivot the published row holds entries already eliminated to rounding level,
// which only touch columns that are not read again.
template <int D>
__global__ __launch_bounds__(kEigThreads) void chol_kernel(ClassifyArgs a) {
  constexpr int TPR = kEigThreads / D, CPT = D / TPR;
  __shared__ double rowbuf[2][D];
  const int n_heads = a.Hq + a.Hkv;
  const int grp = blockIdx.x % a.Hkv;
  const int layer = blockIdx.x / a.Hkv;
  const float* g = a.gram + ((int64_t)layer * n_heads + a.Hq + grp) * D * D;
  double* out = a.chol + ((int64_t)layer * a.Hkv + grp) * D * D;
  const int t = threadIdx.x;
  const int i = t / TPR, base = (t % TPR) * CPT;
  double r[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) r[c] = (double)g[(int64_t)i * D + base + c];
  for (int k = 0; k < D; ++k) {
    double* rb = rowbuf[k & 1];
    if (i == k)
#pragma unroll
      for (int c = 0; c < CPT; ++c) rb[base + c] = r[c];
    __syncthreads();
    const double piv = rb[k];
    const double aik = rb[i];
    const bool live = piv > 0.0 && i > k;
    const double lkk = piv > 0.0 ? sqrt(piv) : 0.0;
    if (t % TPR == 0) out[(int64_t)i * D + k] = live ? aik / lkk : (i == k ? lkk : 0.0);
    const double s = live ? aik / piv : 0.0;  // L[i][k] / L[k][k]
#pragma unroll
    for (int c = 0; c < CPT; ++c) r[c] = fma(-s, rb[base + c], r[c]);
  }
}

// Counts of eigenvalues of the symmetric tridiagonal (d, e2 = e^2) below x0
// and x1 (Sturm counts from the LDL^T pivots q, two independent chains).  A
// pivot smaller than pivmin in magnitude is replaced by -pivmin.  1/q is the
// hardware reciprocal refined by one Newton step; the count is backward
// stable, so its rounding only perturbs d and e by a few ulps.
template <int D>
__device__ __forceinline__ void sturm_count2(const double* d, const double* e2, double x0, double x1,
                                             double pivmin, int& c0, int& c1) {
  double q0 = d[0] - x0, q1 = d[0] - x1;
  q0 = fabs(q0) < pivmin ? -pivmin : q0;
  q1 = fabs(q1) < pivmin ? -pivmin : q1;
  int n0 = q0 < 0.0, n1 = q1 < 0.0;
  for (int i = 1; i < D; ++i) {
    const double di = d[i], ei = e2[i - 1];
    double r0 = __builtin_amdgcn_rcp(q0), r1 = __builtin_amdgcn_rcp(q1);
    r0 = fma(r0, fma(-q0, r0, 1.0), r0);
    r1 = fma(r1, fma(-q1, r1, 1.0), r1);
    q0 = fma(-ei, r0, di - x0);
    q1 = fma(-ei, r1, di - x1);
    q0 = fabs(q0) < pivmin ? -pivmin : q0;
    q1 = fabs(q1) < pivmin ? -pivmin : q1;
    n0 += q0 < 0.0;
    n1 += q1 < 0.0;
  }
  c0 = n0;
  c1 = n1;
}

template <int D>
__global__ __launch_bounds__(kEigThreads, 2) void spectrum_kernel(ClassifyArgs a) {
  constexpr int TPR = kEigThreads / D, CPT = D / TPR;
  constexpr int JC = 64;               // columns per chunk of the congruence products
  constexpr int NJ = D / JC;
  constexpr int RT = D / 16, CT = JC / 16;  // chunk tile per thread
  constexpr int SIDES = kEigThreads / D;    // threads per eigenvalue in the bisection
  constexpr int NPT = 2 * SIDES;            // points per bisection round
  __shared__ double buf[D][JC + 1];
  __shared__ double rowbuf[2][D], vbuf[2][D], pp[2][D];
  __shared__ double dd[D], ee[D];
  __shared__ double red[kEigWaves];

  const int n_heads = a.Hq + a.Hkv;
  const int h = blockIdx.x % a.Hq;
  const int layer = blockIdx.x / a.Hq;
  const int grp = h / a.gs;
  const float* qq = a.gram + ((int64_t)layer * n_heads + h) * D * D;
  const double* L = a.chol + ((int64_t)layer * a.Hkv + grp) * D * D;
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63;
  const int i = t / TPR, base = (t % TPR) * CPT;  // row owned in the register layout

  // B = L^T (QQ L), one chunk of JC columns at a time: T = QQ L[:, J] in
  // registers, through LDS, then B[:, J] = L^T T; the chunk of B goes to its
  // row owners' registers.  QQ is exactly symmetric, so row k of QQ serves as
  // its column k.
  double arow[CPT];
  const int rg = t / 16, c16 = t % 16;
#pragma unroll
  for (int J = 0; J < NJ; ++J) {
    double acc[RT][CT];
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int c = 0; c < CT; ++c) acc[r][c] = 0.0;
    for (int k = 0; k < D; ++k) {
      double qk[RT], lk[CT];
#pragma unroll
      for (int r = 0; r < RT; ++r) qk[r] = (double)qq[(int64_t)k * D + rg * RT + r];
#pragma unroll
      for (int c = 0; c < CT; ++c) lk[c] = L[(int64_t)k * D + J * JC + c16 + 16 * c];
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int c = 0; c < CT; ++c) acc[r][c] = fma(qk[r], lk[c], acc[r][c]);
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int c = 0; c < CT; ++c) buf[rg * RT + r][c16 + 16 * c] = acc[r][c];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int c = 0; c < CT; ++c) acc[r][c] = 0.0;
    for (int k = 0; k < D; ++k) {
      double lk[RT], tk[CT];
#pragma unroll
      for (int r = 0; r < RT; ++r) lk[r] = L[(int64_t)k * D + rg * RT + r];
#pragma unroll
      for (int c = 0; c < CT; ++c) tk[c] = buf[k][c16 + 16 * c];
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int c = 0; c < CT; ++c) acc[r][c] = fma(lk[r], tk[c], acc[r][c]);
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int c = 0; c < CT; ++c) buf[rg * RT + r][c16 + 16 * c] = acc[r][c];
    __syncthreads();
    if (base / JC == J)
#pragma unroll
      for (int c = 0; c < CPT; ++c) arow[c] = buf[i][base % JC + c];
  }

  // Householder tridiagonalisation (Golub and Van Loan, Alg. 8.3.1): step k
  // takes x = row k right of the diagonal (= column k below it), v = x - alpha
  // e_1 with |alpha| = |x|, p = beta A v, K = beta p.v / 2, and
  // A <- A - v p^T - (p - 2 K v) v^T on rows and columns k+1.. (v and p are
  // zero elsewhere, so the update runs over whole rows).  Every wave derives
  // alpha, beta and K from LDS itself, so all waves take the same branch.
  for (int k = 0; k < D - 2; ++k) {
    const int b = k & 1;
    double* rb = rowbuf[b];
    double* vb = vbuf[b];
    double* pb = pp[b];
    if (i == k)
#pragma unroll
      for (int c = 0; c < CPT; ++c) rb[base + c] = arow[c];
    __syncthreads();
    const double x0 = rb[k + 1];
    double part = 0.0;
    for (int j = k + 2 + lane; j < D; j += kWave) part = fma(rb[j], rb[j], part);
    const double xn2 = wave_sum_f64(part);
    if (t == 0) dd[k] = rb[k];
    if (xn2 == 0.0) {
      if (t == 0) ee[k] = x0;
      continue;
    }
    const double nx = sqrt(fma(x0, x0, xn2));
    const double alpha = x0 > 0.0 ? -nx : nx;
    const double v0 = x0 - alpha;
    const double beta = 2.0 / fma(v0, v0, xn2);
    if (t == 0) ee[k] = alpha;
    if (wave == 0)
      for (int j = lane; j < D; j += kWave) vb[j] = j <= k ? 0.0 : (j == k + 1 ? v0 : rb[j]);
    __syncthreads();
    double p0 = 0.0, p1 = 0.0;
#pragma unroll
    for (int c = 0; c < CPT; c += 2) {
      p0 = fma(arow[c], vb[base + c], p0);
      p1 = fma(arow[c + 1], vb[base + c + 1], p1);
    }
    double prow = p0 + p1;
    prow += dpp_f64<0xB1, 0xf>(prow);              // partner lane t ^ 1
    if (TPR == 4) prow += dpp_f64<0x4E, 0xf>(prow);  // lanes t ^ 2
    const double pi = i > k ? beta * prow : 0.0;
    if (t % TPR == 0) pb[i] = pi;
    __syncthreads();
    double pv = 0.0;
    for (int j = lane; j < D; j += kWave) pv = fma(pb[j], vb[j], pv);
    const double K = 0.5 * beta * wave_sum_f64(pv);
    const double vi = vb[i];
    const double ci = fma(-2.0 * K, vi, pi);
    // in groups of 16 columns, so that the LDS operands are not all held at once
#pragma unroll
    for (int c0 = 0; c0 < CPT; c0 += 16) {
#pragma unroll
      for (int c = c0; c < c0 + 16; ++c) arow[c] = fma(-vi, pb[base + c], fma(-ci, vb[base + c], arow[c]));
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();
  if (i == D - 2)
#pragma unroll
    for (int c = 0; c < CPT; ++c) rowbuf[0][base + c] = arow[c];
  if (i == D - 1)
#pragma unroll
    for (int c = 0; c < CPT; ++c) rowbuf[1][base + c] = arow[c];
  __syncthreads();
  if (t == 0) {
    dd[D - 2] = rowbuf[0][D - 2];
    ee[D - 2] = rowbuf[0][D - 1];
    dd[D - 1] = rowbuf[1][D - 1];
  }
  __syncthreads();
  double* e2 = pp[0];  // squared off-diagonal
  if (t < D - 1) e2[t] = ee[t] * ee[t];
  __syncthreads();

  // Gershgorin interval and the pivot floor (every thread, same order)
  double lo = dd[0] - fabs(ee[0]), hi = dd[0] + fabs(ee[0]), emax2 = 0.0;
  for (int j = 1; j < D; ++j) {
    const double r = fabs(ee[j - 1]) + (j < D - 1 ? fabs(ee[j]) : 0.0);
    lo = fmin(lo, dd[j] - r);
    hi = fmax(hi, dd[j] + r);
  }
  for (int j = 0; j < D - 1; ++j) emax2 = fmax(emax2, e2[j]);
  const double eps = 2.220446049250313e-16;
  const double pivmin = 2.2250738585072014e-308 * fmax(1.0, emax2);
  const double tnorm = fmax(fabs(lo), fabs(hi));
  const double atol = eps * tnorm;

  // Multisection: eigenvalue e (ascending) is bracketed by [blo, bhi] with
  // count(blo) <= e < count(bhi); each round the SIDES threads of e evaluate
  // NPT interior points (two chains each) and all of them keep the
  // sub-interval holding e.  Every eigenvalue runs the same number of rounds,
  // enough to shrink the Gershgorin width below atol.
  const int e = t % D, side = t / D;
  int* cnt = reinterpret_cast<int*>(&buf[0][0]);  // [2][NPT][D], free after the products
  double blo = lo - 2.0 * atol - pivmin, bhi = hi + 2.0 * atol + pivmin;
  int rounds = 0;
  {
    double w = bhi - blo;
    const double target = fmax(atol, 4.0 * pivmin);
    while (w > target && rounds < 64) {
      w /= (NPT + 1);
      ++rounds;
    }
  }
  for (int it = 0; it < rounds; ++it) {
    int* cb = cnt + (it & 1) * NPT * D;
    const double step = (bhi - blo) / (NPT + 1);
    const double xa = blo + step * (2 * side + 1), xb = blo + step * (2 * side + 2);
    int ca, cbn;
    sturm_count2<D>(dd, e2, xa, xb, pivmin, ca, cbn);
    cb[(2 * side) * D + e] = ca;
    cb[(2 * side + 1) * D + e] = cbn;
    __syncthreads();
    int m = 0;
    while (m < NPT && cb[m * D + e] <= e) ++m;
    const double nlo = m == 0 ? blo : blo + step * m;
    const double nhi = m == NPT ? bhi : blo + step * (m + 1);
    blo = nlo;
    bhi = nhi;
  }

  // eigenvalues at or below the rounding floor of the reduction are zero
  // (a rank-deficient W_Q or W_K leaves only such values), so they add no
  // term to the entropy; for the zero matrix every eigenvalue is zero
  double sigma = 0.0;
  if (side == 0) {
    const double lam = 0.5 * (blo + bhi);
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

// ---------------------------------------------------------------------------
// Cross-layer head similarity of H2Share (Eq. sim, by the trace identities of
// the trace-reduction appendix): for anchor layer l and reuse layer l',
//   <M_h, M_h'>_F = tr(W_Q^h W_Q'^h'^T . W_K'^g' W_K^g^T)
//                 = sum_ab (W_Q^h W_Q'^h'^T)[a][b] (W_K^g W_K'^g'^T)[a][b],
//   |M_h|_F^2     = sum_ab (W_Q W_Q^T)[a][b] (W_K W_K^T)[a][b]  (symmetric Grams).

// C = A B^T for a d x d_model slice A of one weight and a slice B of another
// (bf16 MFMA, fp32 accumulation), the slab of 64 columns of both staged in
// LDS.  Wave w computes the 32-row block w against all column blocks.
// STORE: C goes to kx[(g * Hkv + g') * D * D]; otherwise the tile is multiplied
// elementwise with kx of the heads' groups and summed into num[h][h'].
template <int D, bool STORE>
__global__ __launch_bounds__(64 * (D / 32)) void cross_kernel(SimilarityArgs a) {
  constexpr int NRB = D / 32;
  __shared__ __align__(16) bf16 stage[2][2][D][kGramRowPad];
  __shared__ double red[NRB];
  const int n = STORE ? a.Hkv : a.Hq;
  const int u = blockIdx.x / n, v = blockIdx.x % n;  // (anchor unit, reuse unit)
  const bf16* wa = STORE ? static_cast<const bf16*>(a.wk_a) + (int64_t)u * D * a.wk_a_sr
                         : static_cast<const bf16*>(a.wq_a) + (int64_t)u * D * a.wq_a_sr;
  const bf16* wb = STORE ? static_cast<const bf16*>(a.wk_r) + (int64_t)v * D * a.wk_r_sr
                         : static_cast<const bf16*>(a.wq_r) + (int64_t)v * D * a.wq_r_sr;
  const int64_t rsa = STORE ? a.wk_a_sr : a.wq_a_sr, rsb = STORE ? a.wk_r_sr : a.wq_r_sr;
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63, l32 = lane & 31, half = lane >> 5;
  const int lrow = t >> 1, lcol = (t & 1) * 32;
  const bf16* srca = wa + (int64_t)lrow * rsa + lcol;
  const bf16* srcb = wb + (int64_t)lrow * rsb + lcol;

  f32x16 acc[NRB];
#pragma unroll
  for (int c = 0; c < NRB; ++c) acc[c] = f32x16{};
  u32x4 la[4], lb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) {
      la[s2] = ld16(srca + k0 + 8 * s2);
      lb[s2] = ld16(srcb + k0 + 8 * s2);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) {
      st16(&stage[buf][0][lrow][lcol + 8 * s2], la[s2]);
      st16(&stage[buf][1][lrow][lcol + 8 * s2], lb[s2]);
    }
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) {
      const bf16x8 xa = as_bf16x8(*reinterpret_cast<const u32x4*>(&stage[buf][0][32 * wave + l32][32 * half + 8 * s2]));
#pragma unroll
      for (int c = 0; c < NRB; ++c) {
        const bf16x8 xb = as_bf16x8(*reinterpret_cast<const u32x4*>(&stage[buf][1][32 * c + l32][32 * half + 8 * s2]));
        acc[c] = mfma32(xa, xb, acc[c]);
      }
    }
  };
  gload(0);
  lstore(0);
  __syncthreads();
  const int n_it = a.d_model / kGramBK;
  for (int it = 0; it < n_it; ++it) {
    const int cur = it & 1;
    const bool more = it + 1 < n_it;
    if (more) gload((it + 1) * kGramBK);
    compute(cur);
    if (more) lstore(cur ^ 1);
    __syncthreads();
  }

  if (STORE) {
    float* out = a.kx + (int64_t)(u * a.Hkv + v) * D * D;
#pragma unroll
    for (int c = 0; c < NRB; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = 32 * wave + 8 * (i / 4) + 4 * half + (i % 4);
        out[(int64_t)m * D + 32 * c + l32] = acc[c][i];
      }
  } else {
    const float* kx = a.kx + (int64_t)((u / a.gs) * a.Hkv + v / a.gs) * D * D;
    double sum = 0.0;
#pragma unroll
    for (int c = 0; c < NRB; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = 32 * wave + 8 * (i / 4) + 4 * half + (i % 4);
        sum += (double)acc[c][i] * (double)kx[(int64_t)m * D + 32 * c + l32];
      }
    sum = wave_sum_f64(sum);
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    if (t == 0) {
      double tot = 0.0;
#pragma unroll
      for (int w = 0; w < NRB; ++w) tot += red[w];
      a.num[(int64_t)u * a.Hq + v] = tot;
    }
  }
}

// |M_h|_F^2 of every query head of both layers from the Grams:
// blockIdx.x = layer * Hq + h.
template <int D>
__global__ __launch_bounds__(kEigThreads) void norm_kernel(SimilarityArgs a) {
  __shared__ double red[kEigWaves];
  const int layer = blockIdx.x / a.Hq, h = blockIdx.x % a.Hq;
  const int n_heads = a.Hq + a.Hkv;
  const float* qq = a.gram + ((int64_t)layer * n_heads + h) * D * D;
  const float* kk = a.gram + ((int64_t)layer * n_heads + a.Hq + h / a.gs) * D * D;
  double sum = 0.0;
  for (int e = threadIdx.x; e < D * D; e += kEigThreads) sum += (double)qq[e] * (double)kk[e];
  sum = wave_sum_f64(sum);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
#pragma unroll
    for (int w = 0; w < kEigWaves; ++w) tot += red[w];
    a.n2[blockIdx.x] = tot;
  }
}

// Normalisation, group means and the mapping (one workgroup).
__global__ __launch_bounds__(kEigThreads) void mapping_kernel(SimilarityArgs a) {
  const int hq = a.Hq, hkv = a.Hkv, gs = a.gs;
  const double* n2 = a.n2;  // [2][Hq] squared norms
  for (int e = threadIdx.x; e < hq * hq; e += kEigThreads) {
    const int h = e / hq, h2 = e % hq;
    a.head_sim[e] = a.num[e] / (sqrt(n2[h]) * sqrt(n2[hq + h2]));
  }
  __syncthreads();
  for (int e = threadIdx.x; e < hkv * hkv; e += kEigThreads) {
    const int g = e / hkv, g2 = e % hkv;
    double sum = 0.0;
    for (int i = 0; i < gs; ++i)
      for (int j = 0; j < gs; ++j) sum += a.head_sim[(int64_t)(g * gs + i) * hq + g2 * gs + j];
    a.group_sim[e] = sum / (gs * gs);
  }
  __syncthreads();
  const int g2 = threadIdx.x;
  if (g2 < hkv) {
    int best = -1, rank = -1, r = 0;
    if (!((a.reuse_streaming >> g2) & 1ull)) {
      for (int g = 0; g < hkv; ++g) {
        if ((a.anchor_streaming >> g) & 1ull) continue;
        if (best < 0 || a.group_sim[g * hkv + g2] > a.group_sim[best * hkv + g2]) {
          best = g;
          rank = r;
        }
        ++r;
      }
    }
    a.mapping[g2] = rank;
  }
}

template <int D>
hipError_t launch_similarity_d(const SimilarityArgs& a, hipStream_t s) {
  // Grams of both layers (the classifier's kernel, one layer each)
  for (int layer = 0; layer < 2; ++layer) {
    ClassifyArgs c;
    __builtin_memset(&c, 0, sizeof(c));
    c.wq = layer ? a.wq_r : a.wq_a;
    c.wk = layer ? a.wk_r : a.wk_a;
    c.wq_sr = layer ? a.wq_r_sr : a.wq_a_sr;
    c.wk_sr = layer ? a.wk_r_sr : a.wk_a_sr;
    c.L = 1; c.Hq = a.Hq; c.Hkv = a.Hkv; c.gs = a.gs; c.d_model = a.d_model;
    c.gram = a.gram + (int64_t)layer * (a.Hq + a.Hkv) * D * D;
    hipLaunchKernelGGL(gram_kernel<D>, dim3(a.Hq + a.Hkv), dim3(64 * (D / 32)), 0, s, c);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((cross_kernel<D, true>), dim3(a.Hkv * a.Hkv), dim3(64 * (D / 32)), 0, s, a);
  hipLaunchKernelGGL((cross_kernel<D, false>), dim3(a.Hq * a.Hq), dim3(64 * (D / 32)), 0, s, a);
  hipLaunchKernelGGL(norm_kernel<D>, dim3(2 * a.Hq), dim3(kEigThreads), 0, s, a);
  hipLaunchKernelGGL(mapping_kernel, dim3(1), dim3(kEigThreads), 0, s, a);
  return hipGetLastError();
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

hipError_t launch_similarity(const SimilarityArgs& a, int d, hipStream_t s) {
  return d == 128 ? launch_similarity_d<128>(a, s) : launch_similarity_d<64>(a, s);
}

}  // namespace aoh
