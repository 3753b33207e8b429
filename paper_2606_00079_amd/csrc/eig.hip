// Shared basis on the GPU: the top-r eigenpairs of the symmetric M.
//
// The shared basis is the leading left singular vectors of the expert
// concatenation, i.e. the eigenvectors of M = sum_e W_e W_e^T of largest
// eigenvalue (App. B.1).  r is a large fraction of d (a half or a quarter
// here) and the spectrum of M is a few large values over a nearly flat bulk,
// so iterative subspace methods converge slowly; this is a direct solver:
//
//   1. Householder reduction to tridiagonal form, T = Q^T M Q, in panels of
//      NB columns (the blocked scheme of LAPACK's symmetric reduction, lower
//      form, stored by rows since M is symmetric).  Per column i of a panel:
//        trsymv_kernel  the reflector H_i = I - tau v v^T that zeroes row i
//                       right of its first off-diagonal entry (formed by
//                       every wave from row i, recorded by one), and
//                       y = A_t v over the trailing rows, and V^T v, W^T v
//                       over the panel's earlier reflectors V and vectors W,
//                       one wave per two rows;
//        trw_kernel     w = tau (y - V W^T v - W V^T v) - (tau/2)(w'^T v) v,
//                       row i of the work matrix overwritten by v (zeros up
//                       to i, 1 at i+1), and row i+1 brought up to date with
//                       the panel's rank-2 terms (it is the next column's
//                       row);
//      then trail_kernel applies A_t -= V W^T + W V^T to the trailing block
//      once per panel.
//   2. The selected eigenpairs of T on the device: eigenvalues n-r+1..n by
//      bisection on Sturm counts (bisect_kernel, a thread per eigenvalue),
//      eigenvectors by inverse iteration with a tridiagonal LU with partial
//      pivoting (inviter_kernel, a thread per eigenvector, three solves from
//      a hashed start vector).  Vectors of eigenvalues closer than 1e-7 ||T||
//      (a cluster) are made orthonormal by modified Gram-Schmidt
//      (mgs_kernel); others are orthogonal to about eps ||T|| / gap.
//   3. Back-transformation U = Q Z = H_0 H_1 ... H_{n-2} Z, one panel at a
//      time from the last, with the compact form H_j0 ... H_{j0+nb-1} =
//      I - V T V^T (T upper triangular from tau and V V^T).
//   4. Eigenvalues in descending order, each eigenvector signed so that its
//      entry of largest magnitude is positive (lowest index on ties), fp32.
//
// All arithmetic is fp64 with fixed reduction orders (deterministic).
#include <algorithm>
#include <chrono>
#include <cmath>
#include <string>
#include <vector>

#include "bitsmoe.h"
#include "common.hpp"
#include "internal.hpp"

namespace bitsmoe {
namespace {

constexpr int NB = 32;  // panel width

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over the workgroup in a fixed order (waves, then wave totals in wave
// order); every thread gets the result.  `red` holds one double per wave.
template <int THREADS>
__device__ double block_sum_f64(double v, double* red) {
  constexpr int W = THREADS / 64;
  v = wave_sum_f64(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();  // red may still be read by a previous call
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < W; ++w) s += red[w];
  return s;
}

// The last diagonal entry of T (row n-1 has no reflector).
__global__ void last_diag_kernel(const double* __restrict__ A, int64_t n, double* __restrict__ dvec) {
  if (threadIdx.x == 0) dvec[n - 1] = A[(n - 1) * n + n - 1];
}

// The reflector of row i, formed by every wave from the row as the previous
// kernels left it: x = A[i][i+1..n), alpha = x_0, sigma = sum_{j>=1} x_j^2,
// beta = -sign(alpha) sqrt(alpha^2 + sigma), tau = (beta - alpha) / beta,
// v = (1, x_1.. / (alpha - beta)); sigma = 0 gives tau = 0, beta = alpha.
// Then out[rr] = row_rr . v = row_rr[i+1] + (sum_{j>=1} row_rr[i+1+j] x_j)
// / (alpha - beta) over the rows rr < m: A[i+1+rr]; m <= rr < m+c:
// A[j0 + rr - m] (the panel's earlier reflectors); m+c <= rr < m+2c:
// Wp[rr - m - c].  Two rows per wave; sigma and the dot products come from
// the same pass over x (every wave sums sigma in the same order, so all
// agree).  Wave 0 of workgroup 0 records d[i] = A[i][i], e[i] = beta,
// tau[i] and v into vbuf[i+1..n); row i itself is rewritten by trw_kernel,
// after every wave here has read it.
__global__ __launch_bounds__(256) void trsymv_kernel(const double* __restrict__ A,
                                                     const double* __restrict__ Wp, int64_t n,
                                                     int64_t i, int64_t j0, int c,
                                                     double* __restrict__ out,
                                                     double* __restrict__ dvec,
                                                     double* __restrict__ evec,
                                                     double* __restrict__ tau,
                                                     double* __restrict__ vbuf) {
  const int lane = threadIdx.x & 63;
  const int64_t m = n - i - 1;
  const int64_t R = m + 2 * c;
  const int64_t rr0 = (static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6)) * 2;
  if (rr0 >= R) return;  // whole wave
  const double* x = A + i * n;
  const double* src[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int64_t rr = std::min<int64_t>(rr0 + q, R - 1);
    src[q] = rr < m ? A + (i + 1 + rr) * n
                    : (rr < m + c ? A + (j0 + rr - m) * n : Wp + (rr - m - c) * n);
  }
  double acc[2] = {0.0, 0.0}, sig = 0.0;
#pragma unroll 8
  for (int64_t col = i + 1 + lane; col < n; col += 64) {
    const double xx = col == i + 1 ? 0.0 : x[col];
    sig = fma(xx, xx, sig);
#pragma unroll
    for (int q = 0; q < 2; ++q) acc[q] = fma(src[q][col], xx, acc[q]);
  }
  const double sigma = wave_sum_f64(sig);
  const double alpha = x[i + 1];
  double beta = alpha, t = 0.0, sc = 0.0;
  if (sigma != 0.0) {
    beta = -copysign(sqrt(fma(alpha, alpha, sigma)), alpha);
    t = (beta - alpha) / beta;
    sc = 1.0 / (alpha - beta);
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const double s = wave_sum_f64(acc[q]);
    if (lane == 0 && rr0 + q < R) out[rr0 + q] = fma(s, sc, src[q][i + 1]);
  }
  if (blockIdx.x == 0 && threadIdx.x < 64) {
    if (lane == 0) {
      dvec[i] = x[i];
      evec[i] = beta;
      tau[i] = t;
      vbuf[i + 1] = 1.0;
    }
    for (int64_t j = i + 2 + lane; j < n; j += 64) vbuf[j] = x[j] * sc;
  }
}

// w for column c = i - j0 of the panel (rows j = i+1..n-1), stored in
// Wp[c], and, when do_row, the rank-2 terms of panel columns 0..c applied to
// row i+1 (entries j >= i+1); row i is overwritten by its reflector v (zeros
// up to i, then vbuf).  ybv = trsymv's output: y [m], V^T v [c], W^T v [c].
// Every workgroup forms y.v (and w_{i+1}) itself.  A workgroup covers 64
// entries j; its four waves take the panel columns c' = q mod 4 and their
// partial sums are added in wave order.  Every load is issued before the
// first barrier.
__global__ __launch_bounds__(256) void trw_kernel(double* __restrict__ A, double* __restrict__ Wp,
                                                  int64_t n, int64_t i, int64_t j0, int c,
                                                  const double* __restrict__ ybv,
                                                  const double* __restrict__ tau,
                                                  const double* __restrict__ vbuf, int do_row) {
  constexpr int KP = NB / 4;  // panel columns per wave
  __shared__ double red[4];
  __shared__ double s_vtv[NB], s_wtv[NB], s_vi1[NB], s_wi1[NB];
  __shared__ double part_w[4][64], part_r[4][64];
  const int64_t m = n - i - 1;
  const int jl = threadIdx.x & 63, sl = threadIdx.x >> 6;
  const int64_t j = i + 1 + static_cast<int64_t>(blockIdx.x) * 64 + jl;
  const bool jin = j < n;
  double part = 0.0;
  for (int64_t jj = threadIdx.x; jj < m; jj += 256) part = fma(ybv[jj], vbuf[i + 1 + jj], part);
  double vj[KP], wj[KP];
#pragma unroll
  for (int k = 0; k < KP; ++k) {
    const int cc = sl + 4 * k;
    vj[k] = wj[k] = 0.0;
    if (jin && cc < c) {
      vj[k] = A[(j0 + cc) * n + j];
      wj[k] = Wp[cc * n + j];
    }
  }
  if (threadIdx.x < c) {
    const int cc = threadIdx.x;
    s_vtv[cc] = ybv[m + cc];
    s_wtv[cc] = ybv[m + c + cc];
    s_vi1[cc] = A[(j0 + cc) * n + i + 1];  // V[i+1][c'] for c' < c
    s_wi1[cc] = Wp[cc * n + i + 1];        // W[i+1][c']
  }
  const double vjj = jin ? vbuf[j] : 0.0;
  const double t = tau[i];
  // nothing in this kernel reads row i
  if (sl == 0 && jin) A[i * n + j] = vjj;
  if (blockIdx.x == 0)
    for (int64_t jz = threadIdx.x; jz <= i; jz += 256) A[i * n + jz] = 0.0;
  const double yv = block_sum_f64<256>(part, red);  // its barriers publish s_*
  double q = 0.0;
  for (int cc = 0; cc < c; ++cc) q = fma(s_vtv[cc], s_wtv[cc], q);
  const double s = t * (yv - 2.0 * q);
  double pw = 0.0, pr = 0.0;
#pragma unroll
  for (int k = 0; k < KP; ++k) {
    const int cc = sl + 4 * k;
    if (cc < c) {
      pw = fma(vj[k], s_wtv[cc], fma(wj[k], s_vtv[cc], pw));
      pr = fma(vj[k], s_wi1[cc], fma(wj[k], s_vi1[cc], pr));
    }
  }
  part_w[sl][jl] = pw;
  part_r[sl][jl] = pr;
  __syncthreads();
  if (sl != 0 || !jin) return;
  const double acc = ybv[j - (i + 1)] - (((part_w[0][jl] + part_w[1][jl]) + part_w[2][jl]) + part_w[3][jl]);
  const double w = t * acc - 0.5 * t * s * vjj;
  Wp[static_cast<int64_t>(c) * n + j] = w;
  if (!do_row) return;
  // w_{i+1} (v_{i+1} = 1), formed the same way in every workgroup
  double acc1 = ybv[0];
  for (int cc = 0; cc < c; ++cc) acc1 -= s_vi1[cc] * s_wtv[cc] + s_wi1[cc] * s_vtv[cc];
  const double w1 = t * acc1 - 0.5 * t * s;
  // the current column: V[j][c] W[i+1][c] + W[j][c] V[i+1][c], then c' < c
  const double delta =
      vjj * w1 + w + (((part_r[0][jl] + part_r[1][jl]) + part_r[2][jl]) + part_r[3][jl]);
  A[(i + 1) * n + j] -= delta;
}

// A[r][q] -= sum_k Vp[k][r] Wp[k][q] + Wp[k][r] Vp[k][q] for r, q in [s, n),
// Vp = the panel's NB reflector rows.  64 x 64 tiles, 4 x 4 per thread.
__global__ __launch_bounds__(256) void trail_kernel(double* __restrict__ A,
                                                    const double* __restrict__ Vp,
                                                    const double* __restrict__ Wp, int64_t n,
                                                    int64_t s) {
  __shared__ double sVr[NB][64], sWr[NB][64], sVc[NB][64], sWc[NB][64];
  const int64_t r0 = s + static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t c0 = s + static_cast<int64_t>(blockIdx.x) * 64;
  for (int idx = threadIdx.x; idx < NB * 64; idx += 256) {
    const int k = idx / 64, l = idx % 64;
    const int64_t rr = r0 + l, cc = c0 + l;
    sVr[k][l] = rr < n ? Vp[k * n + rr] : 0.0;
    sWr[k][l] = rr < n ? Wp[k * n + rr] : 0.0;
    sVc[k][l] = cc < n ? Vp[k * n + cc] : 0.0;
    sWc[k][l] = cc < n ? Wp[k * n + cc] : 0.0;
  }
  __syncthreads();
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[4][4] = {};
#pragma unroll 4
  for (int k = 0; k < NB; ++k) {
    double av[4], aw[4], bv[4], bw[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      av[p] = sVr[k][ty + 16 * p];
      aw[p] = sWr[k][ty + 16 * p];
      bv[p] = sVc[k][tx + 16 * p];
      bw[p] = sWc[k][tx + 16 * p];
    }
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) acc[p][qq] = fma(av[p], bw[qq], fma(aw[p], bv[qq], acc[p][qq]));
  }
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int64_t rr = r0 + ty + 16 * p;
    if (rr >= n) continue;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int64_t cc = c0 + tx + 16 * qq;
      if (cc < n) A[rr * n + cc] -= acc[p][qq];
    }
  }
}

// out[k][c] = sum_{j >= jlo} P[k][j] Vp[c][j] for k < rows, c < nbp (rows
// of P with stride ldp, rows of Vp with stride n), rows 8 bx .. 8 bx + 7.
// Two rows per wave; the Vp columns of each 64-wide chunk are staged in LDS.
__device__ void rowdot_rows(const double* __restrict__ P, int64_t ldp, int64_t rows,
                            const double* __restrict__ Vp, int nbp, int64_t n, int64_t jlo,
                            double* __restrict__ out, int64_t bx) {
  __shared__ double sV[NB][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t k0 = (bx * 4 + wave) * 2;
  const bool ok0 = k0 < rows, ok1 = k0 + 1 < rows;
  double a0[NB], a1[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) a0[c] = a1[c] = 0.0;
  for (int64_t jc = jlo; jc < n; jc += 64) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < NB * 64; idx += 256) {
      const int c = idx / 64, l = idx % 64;
      const int64_t col = jc + l;
      sV[c][l] = (c < nbp && col < n) ? Vp[c * n + col] : 0.0;
    }
    __syncthreads();
    const int64_t col = jc + lane;
    const double p0 = (ok0 && col < n) ? P[k0 * ldp + col] : 0.0;
    const double p1 = (ok1 && col < n) ? P[(k0 + 1) * ldp + col] : 0.0;
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const double vv = sV[c][lane];
      a0[c] = fma(p0, vv, a0[c]);
      a1[c] = fma(p1, vv, a1[c]);
    }
  }
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const double s0 = wave_sum_f64(a0[c]);
    const double s1 = wave_sum_f64(a1[c]);
    if (lane == 0 && c < nbp) {
      if (ok0) out[k0 * NB + c] = s0;
      if (ok1) out[(k0 + 1) * NB + c] = s1;
    }
  }
}

__global__ __launch_bounds__(256) void rowdot_kernel(const double* __restrict__ P, int64_t ldp,
                                                     int64_t rows, const double* __restrict__ Vp,
                                                     int nbp, int64_t n, int64_t jlo,
                                                     double* __restrict__ out) {
  rowdot_rows(P, ldp, rows, Vp, nbp, n, jlo, out, blockIdx.x);
}

// G_p = Vp Vp^T of every panel p = blockIdx.y (Vp = the reflector rows
// 32 p .. 32 p + nbp - 1 of A), into G + p NB NB.
__global__ __launch_bounds__(256) void panel_gram_kernel(const double* __restrict__ A, int64_t n,
                                                         double* __restrict__ G) {
  const int64_t j0 = static_cast<int64_t>(blockIdx.y) * NB;
  const int nbp = static_cast<int>(std::min<int64_t>(NB, n - 1 - j0));
  const double* Vp = A + j0 * n;
  rowdot_rows(Vp, n, nbp, Vp, nbp, n, j0 + 1, G + blockIdx.y * NB * NB, blockIdx.x);
}

// Upper-triangular T of the panel's compact form (forward, by columns):
// T[c][c] = tau_c, T[0:c][c] = -tau_c T[0:c][0:c] G[0:c][c], G = Vp Vp^T.
// One workgroup per panel p = blockIdx.x (G, tau and T offset by p).
__global__ __launch_bounds__(64) void tfactor_kernel(const double* __restrict__ Gall,
                                                     const double* __restrict__ tau_all, int64_t n,
                                                     double* __restrict__ Tall) {
  __shared__ double sT[NB][NB], sG[NB][NB];
  const int64_t j0 = static_cast<int64_t>(blockIdx.x) * NB;
  const int nbp = static_cast<int>(std::min<int64_t>(NB, n - 1 - j0));
  const double* G = Gall + blockIdx.x * NB * NB;
  const double* tau = tau_all + j0;
  double* T = Tall + blockIdx.x * NB * NB;
  const int r = threadIdx.x;
  for (int idx = r; idx < NB * NB; idx += 64) {
    const int a = idx / NB, b = idx % NB;
    sT[a][b] = 0.0;
    sG[a][b] = (a < nbp && b < nbp) ? G[idx] : 0.0;
  }
  __syncthreads();
  for (int c = 0; c < nbp; ++c) {
    double v = 0.0;
    if (r < c) {
      for (int k = r; k < c; ++k) v = fma(sT[r][k], sG[k][c], v);
    }
    __syncthreads();
    if (r < c) sT[r][c] = -tau[c] * v;
    if (r == c) sT[c][c] = tau[c];
    __syncthreads();
  }
  if (r < NB)
    for (int c = 0; c < NB; ++c) T[r * NB + c] = sT[r][c];
}

// Zt[k][j] -= sum_c Y[k][c] Vp[c][j] for j >= jlo, Y = X T^T (the rows of X
// are Zt's products with the panel's reflectors).  One column j per thread,
// 32 rows k per workgroup.
__global__ __launch_bounds__(256) void zupdate_kernel(double* __restrict__ Zt, int64_t rows,
                                                      const double* __restrict__ X,
                                                      const double* __restrict__ T,
                                                      const double* __restrict__ Vp, int nbp,
                                                      int64_t n, int64_t jlo) {
  __shared__ double sT[NB][NB], sX[32][NB], sY[32][NB];
  const int64_t k0 = static_cast<int64_t>(blockIdx.y) * 32;
  for (int idx = threadIdx.x; idx < NB * NB; idx += 256) {
    sT[idx / NB][idx % NB] = T[idx];
    const int64_t k = k0 + idx / NB;
    sX[idx / NB][idx % NB] = k < rows ? X[k * NB + idx % NB] : 0.0;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * NB; idx += 256) {
    const int kk = idx / NB, c = idx % NB;
    double y = 0.0;
    for (int cp = c; cp < nbp; ++cp) y = fma(sX[kk][cp], sT[c][cp], y);  // T[c][c'] = 0 for c' < c
    sY[kk][c] = y;
  }
  __syncthreads();
  const int64_t j = jlo + static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j >= n) return;
  double vc[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) vc[c] = c < nbp ? Vp[c * n + j] : 0.0;
  for (int kk = 0; kk < 32; ++kk) {
    const int64_t k = k0 + kk;
    if (k >= rows) break;
    double dot = 0.0;
#pragma unroll
    for (int c = 0; c < NB; ++c) dot = fma(sY[kk][c], vc[c], dot);
    Zt[k * n + j] -= dot;
  }
}

// Number of eigenvalues of the tridiagonal (d, e) below x (the negative
// pivots of the LDL^T factorization of T - x I), pivots kept away from 0.
__device__ double sturm_below(const double* __restrict__ d, const double* __restrict__ e,
                              int64_t n, double x, double pivmin, int64_t* count) {
  double q = d[0] - x;
  int64_t c = q < 0.0;
  for (int64_t j = 1; j < n; ++j) {
    if (fabs(q) < pivmin) q = -pivmin;
    q = d[j] - x - e[j - 1] * e[j - 1] / q;
    c += q < 0.0;
  }
  *count = c;
  return q;
}

// w[k] = eigenvalue t0 + k (0-based, ascending): one wave per eigenvalue
// splits [lo, hi] at 64 interior points per step (lane l evaluates the
// Sturm count at lo + (hi - lo)(l + 1)/65); the counts grow with x, so the
// lanes whose count is <= t form a prefix and the new interval is the gap
// after it.  Stops when the interval is atol wide or the points no longer
// fall strictly inside.
__global__ __launch_bounds__(256) void bisect_kernel(const double* __restrict__ d,
                                                     const double* __restrict__ e, int64_t n,
                                                     int64_t r, int64_t t0, double lo0, double hi0,
                                                     double pivmin, double atol,
                                                     double* __restrict__ w) {
  const int lane = threadIdx.x & 63;
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (k >= r) return;  // whole wave
  const int64_t t = t0 + k;
  double lo = lo0, hi = hi0;
  for (int it = 0; it < 64 && hi - lo > atol; ++it) {
    const double x = lo + (hi - lo) * (static_cast<double>(lane + 1) / 65.0);
    const bool inside = x > lo && x < hi;
    if (__ballot(inside) != ~0ull) break;  // the interval is a few ulps wide
    int64_t cnt;
    sturm_below(d, e, n, x, pivmin, &cnt);
    const int p = __popcll(__ballot(cnt <= t));  // lanes 0..p-1 have count <= t
    const double xl = __shfl(x, p > 0 ? p - 1 : 0, 64);
    const double xh = __shfl(x, p < 64 ? p : 63, 64);
    lo = p > 0 ? xl : lo;
    hi = p < 64 ? xh : hi;
  }
  if (lane == 0) w[k] = 0.5 * (lo + hi);
}

// Start vector entry j of eigenvector k: a counter hash (splitmix64 of the
// pair) mapped to [-1, 1).
__device__ __forceinline__ double start_entry(int64_t k, int64_t j) {
  uint64_t z = static_cast<uint64_t>(k) * 0x9E3779B97F4A7C15ull + static_cast<uint64_t>(j) + 1;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  return static_cast<double>(z >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

// Eigenvector of eigenvalue w[k] by inverse iteration: three solves of
// (T - w I) x = b, b the previous x scaled to max |x| = 1, with T - w I
// factored by Gaussian elimination with partial pivoting (U has two
// superdiagonals; pivots below pivmin in magnitude are set to +-pivmin).
// Work arrays and Z are interleaved by thread (entry j of thread k at
// j r + k).  Z[j][k] = x_j / ||x||.
__global__ __launch_bounds__(64) void inviter_kernel(const double* __restrict__ d,
                                                     const double* __restrict__ e, int64_t n,
                                                     int64_t r, const double* __restrict__ w,
                                                     double pivmin, double* __restrict__ work,
                                                     double* __restrict__ Z) {
  const int64_t k = static_cast<int64_t>(blockIdx.x) * 64 + threadIdx.x;
  if (k >= r) return;
  const double lam = w[k];
  double* U0 = work;
  double* U1 = work + n * r;
  double* U2 = work + 2 * n * r;
  double* Y = work + 3 * n * r;
  auto at = [&](int64_t j) { return j * r + k; };
  auto guard = [&](double p) { return fabs(p) >= pivmin ? p : (p < 0.0 ? -pivmin : pivmin); };
  for (int64_t j = 0; j < n; ++j) Z[at(j)] = start_entry(k, j);
  for (int iter = 0; iter < 3; ++iter) {
    double p0 = d[0] - lam, p1 = n > 1 ? e[0] : 0.0, p2 = 0.0, y = Z[at(0)];
#pragma unroll 8
    for (int64_t j = 0; j + 1 < n; ++j) {
      const double ej = e[j], a1 = d[j + 1] - lam, c1 = j + 2 < n ? e[j + 1] : 0.0;
      const double bj1 = Z[at(j + 1)];
      if (fabs(p0) >= fabs(ej)) {
        const double piv = guard(p0);
        const double m = ej / piv;
        U0[at(j)] = piv;
        U1[at(j)] = p1;
        U2[at(j)] = p2;
        Y[at(j)] = y;
        p0 = a1 - m * p1;
        p1 = c1 - m * p2;
        p2 = 0.0;
        y = bj1 - m * y;
      } else {
        const double m = p0 / ej;
        U0[at(j)] = ej;
        U1[at(j)] = a1;
        U2[at(j)] = c1;
        Y[at(j)] = bj1;
        const double np0 = p1 - m * a1, np1 = p2 - m * c1;
        p0 = np0;
        p1 = np1;
        p2 = 0.0;
        y = y - m * bj1;
      }
    }
    U0[at(n - 1)] = guard(p0);
    Y[at(n - 1)] = y;
    double x1 = 0.0, x2 = 0.0, xmax = 0.0;
#pragma unroll 8
    for (int64_t j = n - 1; j >= 0; --j) {
      double sj = Y[at(j)];
      if (j + 1 < n) sj -= U1[at(j)] * x1;
      if (j + 2 < n) sj -= U2[at(j)] * x2;
      const double xj = sj / U0[at(j)];
      Z[at(j)] = xj;
      xmax = fmax(xmax, fabs(xj));
      x2 = x1;
      x1 = xj;
    }
    const double inv = xmax > 0.0 ? 1.0 / xmax : 1.0;
    double ss = 0.0;
#pragma unroll 8
    for (int64_t j = 0; j < n; ++j) {
      const double v = Z[at(j)] * inv;
      Z[at(j)] = v;
      ss = fma(v, v, ss);
    }
    if (iter == 2) {
      const double nrm = 1.0 / sqrt(ss);
      for (int64_t j = 0; j < n; ++j) Z[at(j)] *= nrm;
    }
  }
}

// Modified Gram-Schmidt, twice, over the vectors k0..k1-1 of each cluster
// (clusters[2q], clusters[2q+1]); one workgroup per cluster.
__global__ __launch_bounds__(256) void mgs_kernel(double* __restrict__ Z, int64_t n, int64_t r,
                                                  const int64_t* __restrict__ clusters) {
  __shared__ double red[4];
  const int64_t k0 = clusters[2 * blockIdx.x], k1 = clusters[2 * blockIdx.x + 1];
  for (int pass = 0; pass < 2; ++pass)
    for (int64_t a = k0; a < k1; ++a) {
      for (int64_t b = k0; b < a; ++b) {
        double part = 0.0;
        for (int64_t j = threadIdx.x; j < n; j += 256) part = fma(Z[j * r + a], Z[j * r + b], part);
        const double dot = block_sum_f64<256>(part, red);
        for (int64_t j = threadIdx.x; j < n; j += 256) Z[j * r + a] -= dot * Z[j * r + b];
        __syncthreads();
      }
      double part = 0.0;
      for (int64_t j = threadIdx.x; j < n; j += 256) part = fma(Z[j * r + a], Z[j * r + a], part);
      const double nrm = block_sum_f64<256>(part, red);
      const double inv = nrm > 0.0 ? 1.0 / sqrt(nrm) : 0.0;
      for (int64_t j = threadIdx.x; j < n; j += 256) Z[j * r + a] *= inv;
      __syncthreads();
    }
}

// Zt[k][j] = Z[j][k] (32 x 32 tiles through LDS).
__global__ __launch_bounds__(256) void transpose_kernel(const double* __restrict__ Z, int64_t n,
                                                        int64_t r, double* __restrict__ Zt) {
  __shared__ double tile[32][33];
  const int64_t j0 = static_cast<int64_t>(blockIdx.x) * 32, k0 = static_cast<int64_t>(blockIdx.y) * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int q = ty; q < 32; q += 8) {
    const int64_t j = j0 + q, k = k0 + tx;
    tile[q][tx] = (j < n && k < r) ? Z[j * r + k] : 0.0;
  }
  __syncthreads();
  for (int q = ty; q < 32; q += 8) {
    const int64_t k = k0 + q, j = j0 + tx;
    if (k < r && j < n) Zt[k * n + j] = tile[tx][q];
  }
}

// Ut[k] = sign * Zt[rows-1-k] in fp32, the sign making the entry of largest
// magnitude positive (lowest index on ties).  One workgroup per row.
__global__ __launch_bounds__(256) void finish_kernel(const double* __restrict__ Zt, int64_t rows,
                                                     int64_t n, float* __restrict__ Ut) {
  __shared__ double sv[256];
  __shared__ int64_t si[256];
  const int64_t k = blockIdx.x;
  const double* z = Zt + (rows - 1 - k) * n;
  double best = -1.0;
  int64_t bi = 0;
  for (int64_t j = threadIdx.x; j < n; j += 256) {
    const double a = fabs(z[j]);
    if (a > best) {
      best = a;
      bi = j;
    }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st) {
      const double o = sv[threadIdx.x + st];
      const int64_t oi = si[threadIdx.x + st];
      if (o > sv[threadIdx.x] || (o == sv[threadIdx.x] && oi < si[threadIdx.x])) {
        sv[threadIdx.x] = o;
        si[threadIdx.x] = oi;
      }
    }
    __syncthreads();
  }
  const double sg = z[si[0]] < 0.0 ? -1.0 : 1.0;
  for (int64_t j = threadIdx.x; j < n; j += 256) Ut[k * n + j] = static_cast<float>(sg * z[j]);
}

}  // namespace
}  // namespace bitsmoe

using namespace bitsmoe;

extern "C" bitsmoe_status bitsmoe_shared_basis_gpu(const double* M_dev, int64_t d_out, int64_t r,
                                                   float* Ut_dev, double* eigvals_host,
                                                   double* host_ms, void* stream) {
  auto t0 = std::chrono::steady_clock::now();
  if (!M_dev || !Ut_dev) return fail(BITSMOE_ERR_ARG, "shared_basis_gpu: null pointer");
  if (!aligned16({M_dev, Ut_dev}))
    return fail(BITSMOE_ERR_ARG, "shared_basis_gpu: device pointers must be 16-byte aligned");
  if (d_out <= 0 || r <= 0) return fail(BITSMOE_ERR_ARG, "shared_basis_gpu: non-positive size");
  if (r > d_out) return fail(BITSMOE_ERR_SHAPE, "shared_basis_gpu: r > d_out");
  if (d_out > 65536) return fail(BITSMOE_ERR_SHAPE, "shared_basis_gpu: d_out above 65536");
  const int64_t n = d_out;
  hipStream_t s = static_cast<hipStream_t>(stream);
  bitsmoe_status st;
  // work matrix (M, then the reflectors by rows), Z^T, and small buffers:
  // Wp [NB][n], trsymv output [n + 2 NB], d, e, tau, v [n], G and T [NB][NB],
  // X [r][NB], eigenvalues [r]
  double* A = static_cast<double*>(scratch(kScratchA, static_cast<size_t>(n * n) * 8, stream, &st));
  if (!A) return st;
  double* Zt = static_cast<double*>(scratch(kScratchB, static_cast<size_t>(r * n) * 8, stream, &st));
  if (!Zt) return st;
  const int64_t npan = (n - 1 + NB - 1) / NB;
  const size_t small = static_cast<size_t>(NB * n + (n + 2 * NB) + 4 * n +
                                           2 * std::max<int64_t>(npan, 1) * NB * NB + r * NB + r) *
                       8;
  double* Wp = static_cast<double*>(scratch(kScratchPart, small, stream, &st));
  if (!Wp) return st;
  double* ybv = Wp + NB * n;
  double* dvec = ybv + n + 2 * NB;
  double* evec = dvec + n;
  double* tau = evec + n;
  double* vbuf = tau + n;  // the current column's reflector
  double* G = vbuf + n;                                 // [npan][NB][NB]
  double* T = G + std::max<int64_t>(npan, 1) * NB * NB;  // [npan][NB][NB]
  double* X = T + std::max<int64_t>(npan, 1) * NB * NB;
  hipError_t he = hipMemcpyAsync(A, M_dev, static_cast<size_t>(n * n) * 8, hipMemcpyDeviceToDevice, s);
  if (he != hipSuccess) return device_error("shared_basis_gpu: copy of M", he);
  // 1. tridiagonal reduction
  {
    KernelTimer timer("eig_tridiag", stream);
    for (int64_t j0 = 0; j0 < n - 1; j0 += NB) {
      const int64_t pe = std::min<int64_t>(j0 + NB, n - 1);
      const bool full = j0 + NB <= n - 1;  // a trailing update follows the panel
      for (int64_t i = j0; i < pe; ++i) {
        const int c = static_cast<int>(i - j0);
        const int64_t m = n - i - 1;
        const int64_t R = m + 2 * c;
        hipLaunchKernelGGL(trsymv_kernel, dim3(static_cast<unsigned>((R + 7) / 8)), dim3(256), 0, s,
                           A, Wp, n, i, j0, c, ybv, dvec, evec, tau, vbuf);
        const int do_row = (full && c == NB - 1) ? 0 : 1;
        hipLaunchKernelGGL(trw_kernel, dim3(static_cast<unsigned>((m + 63) / 64)), dim3(256), 0, s,
                           A, Wp, n, i, j0, c, ybv, tau, vbuf, do_row);
      }
      if (full) {
        const int64_t sidx = j0 + NB;
        const unsigned tiles = static_cast<unsigned>((n - sidx + 63) / 64);
        hipLaunchKernelGGL(trail_kernel, dim3(tiles, tiles), dim3(256), 0, s, A, A + j0 * n, Wp, n,
                           sidx);
      }
    }
    hipLaunchKernelGGL(last_diag_kernel, dim3(1), dim3(64), 0, s, A, n, dvec);
  }
  BITSMOE_LAUNCH_CHECK("shared_basis_gpu: tridiagonal reduction");
  // 2. eigenpairs of T: bounds and clusters on the host, the rest on the device
  std::vector<double> dh, eh, w;
  try {
    dh.resize(static_cast<size_t>(n));
    eh.resize(static_cast<size_t>(n));
    w.resize(static_cast<size_t>(r));
  } catch (...) {
    return fail(BITSMOE_ERR_NOMEM, "shared_basis_gpu: host allocation failed");
  }
  he = hipMemcpyAsync(dh.data(), dvec, n * 8, hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipMemcpyAsync(eh.data(), evec, n * 8, hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) return device_error("shared_basis_gpu: copy of the tridiagonal", he);
  double lo = 0.0, hi = 0.0, tnorm = 0.0, emax2 = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    const double dj = dh[static_cast<size_t>(j)];
    const double el = j > 0 ? std::fabs(eh[static_cast<size_t>(j - 1)]) : 0.0;
    const double er = j + 1 < n ? std::fabs(eh[static_cast<size_t>(j)]) : 0.0;
    if (!std::isfinite(dj) || !std::isfinite(el) || !std::isfinite(er))
      return fail(BITSMOE_ERR_NUMERIC, "shared_basis_gpu: M is not finite");
    lo = j == 0 ? dj - el - er : std::min(lo, dj - el - er);  // Gershgorin
    hi = j == 0 ? dj + el + er : std::max(hi, dj + el + er);
    tnorm = std::max(tnorm, std::fabs(dj) + el + er);
    emax2 = std::max(emax2, er * er);
  }
  const double eps = 2.220446049250313e-16;
  const double pivmin = 2.2250738585072014e-308 * std::max(1.0, emax2);
  lo -= 2.0 * eps * tnorm + 2.0 * pivmin;
  hi += 2.0 * eps * tnorm + 2.0 * pivmin;
  double* Zn = static_cast<double*>(scratch(kScratchD, static_cast<size_t>(5 * r * n) * 8, stream, &st));
  if (!Zn) return st;
  double* work = Zn + r * n;
  double* wd = X + r * NB;  // eigenvalues, after X in the small buffer
  {
    KernelTimer timer("eig_tri_solve", stream);
    const unsigned g = static_cast<unsigned>((r + 63) / 64);
    hipLaunchKernelGGL(bisect_kernel, dim3(static_cast<unsigned>((r + 3) / 4)), dim3(256), 0, s, dvec,
                       evec, n, r, n - r, lo, hi, pivmin, 2.0 * eps * tnorm, wd);
    hipLaunchKernelGGL(inviter_kernel, dim3(g), dim3(64), 0, s, dvec, evec, n, r, wd, pivmin, work,
                       Zn);
  }
  BITSMOE_LAUNCH_CHECK("shared_basis_gpu: tridiagonal eigenpairs");
  he = hipMemcpyAsync(w.data(), wd, r * 8, hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) return device_error("shared_basis_gpu: copy of the eigenvalues", he);
  std::vector<int64_t> clusters;
  for (int64_t k = 0; k < r;) {
    int64_t k1 = k + 1;
    while (k1 < r && w[static_cast<size_t>(k1)] - w[static_cast<size_t>(k1 - 1)] < 1e-7 * tnorm) ++k1;
    if (k1 - k > 1) {
      clusters.push_back(k);
      clusters.push_back(k1);
    }
    k = k1;
  }
  if (!clusters.empty()) {
    int64_t* cd = reinterpret_cast<int64_t*>(
        scratch(kScratchMisc, clusters.size() * 8, stream, &st));
    if (!cd) return st;
    he = hipMemcpyAsync(cd, clusters.data(), clusters.size() * 8, hipMemcpyHostToDevice, s);
    if (he == hipSuccess) he = hipStreamSynchronize(s);  // clusters (host) may go away
    if (he != hipSuccess) return device_error("shared_basis_gpu: copy of the clusters", he);
    KernelTimer timer("eig_tri_solve", stream);
    hipLaunchKernelGGL(mgs_kernel, dim3(static_cast<unsigned>(clusters.size() / 2)), dim3(256), 0, s,
                       Zn, n, r, cd);
  }
  hipLaunchKernelGGL(transpose_kernel,
                     dim3(static_cast<unsigned>((n + 31) / 32), static_cast<unsigned>((r + 31) / 32)),
                     dim3(256), 0, s, Zn, n, r, Zt);
  BITSMOE_LAUNCH_CHECK("shared_basis_gpu: cluster orthogonalization");
  // 3. back-transformation, last panel first
  {
    KernelTimer timer("eig_backtransform", stream);
    if (npan > 0) {
      hipLaunchKernelGGL(panel_gram_kernel, dim3(NB / 8, static_cast<unsigned>(npan)), dim3(256), 0,
                         s, A, n, G);
      hipLaunchKernelGGL(tfactor_kernel, dim3(static_cast<unsigned>(npan)), dim3(64), 0, s, G, tau, n,
                         T);
    }
    for (int64_t p = npan - 1; p >= 0; --p) {
      const int64_t j0 = p * NB;
      const int nbp = static_cast<int>(std::min<int64_t>(j0 + NB, n - 1) - j0);
      const double* Vp = A + j0 * n;
      const int64_t jlo = j0 + 1;
      hipLaunchKernelGGL(rowdot_kernel, dim3(static_cast<unsigned>((r + 7) / 8)), dim3(256), 0, s,
                         Zt, n, r, Vp, nbp, n, jlo, X);
      hipLaunchKernelGGL(zupdate_kernel,
                         dim3(static_cast<unsigned>((n - jlo + 255) / 256),
                              static_cast<unsigned>((r + 31) / 32)),
                         dim3(256), 0, s, Zt, r, X, T + p * NB * NB, Vp, nbp, n, jlo);
    }
    // 4. order, sign, fp32
    hipLaunchKernelGGL(finish_kernel, dim3(static_cast<unsigned>(r)), dim3(256), 0, s, Zt, r, n, Ut_dev);
  }
  BITSMOE_LAUNCH_CHECK("shared_basis_gpu: back-transformation");
  he = hipStreamSynchronize(s);
  if (he != hipSuccess) return device_error("shared_basis_gpu: synchronize", he);
  if (eigvals_host)
    for (int64_t k = 0; k < r; ++k) eigvals_host[k] = w[static_cast<size_t>(r - 1 - k)];
  if (host_ms) {
    auto t1 = std::chrono::steady_clock::now();
    *host_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  }
  return ok();
}
