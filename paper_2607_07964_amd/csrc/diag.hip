// Diagnostics of the incoherence processing (Sec. 2.3 eq. incoherence_measure; Sec. 4.2 with
// Fig. 2; Prop. 2 eq. biip-bound and the optimality table of appendix A.3):
//  * matrix statistics: max |M_ij|, ||M||_F^2, mu(M), and the coefficients of variation of the
//    column and row norms, in three deterministic passes (tiles, lines, one final workgroup);
//  * the symmetric eigendecomposition behind mu(H), by cyclic two-sided Jacobi rotations in the
//    round-robin order (n/2 disjoint rotations per round, n - 1 rounds per sweep);
//  * the expected-loss factors of Prop. 2 and the optimality table.
// Sums are taken in fp64: every square of an fp32 value is exact there.
#include <cmath>

#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int ST_COLS = 2048;  // columns per tile (256 threads x 8)
constexpr int ST_ROWS = 32;    // rows per tile

__device__ __forceinline__ float ld_val(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_val(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}

// Tile (bx, by): columns [bx * 2048, +2048), rows [by * 32, +32). Writes the tile's column sums
// of squares col_part[by][c], row sums row_part[bx][r] and its largest magnitude mx[by][bx].
template <typename T>
__global__ __launch_bounds__(256) void stat_tiles(const T* __restrict__ M, int64_t rows,
                                                  int64_t cols, int64_t ld,
                                                  double* __restrict__ col_part,
                                                  double* __restrict__ row_part,
                                                  float* __restrict__ mx) {
  __shared__ double red[4][ST_ROWS];
  __shared__ float mred[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t c0 = int64_t(blockIdx.x) * ST_COLS + tid * 8;
  const int64_t r0 = int64_t(blockIdx.y) * ST_ROWS;
  const int nr = int(min(int64_t(ST_ROWS), rows - r0));
  double cs[8] = {0., 0., 0., 0., 0., 0., 0., 0.};
  float m = 0.f;
  for (int r = 0; r < ST_ROWS; ++r) {
    double rs = 0.;
    if (r < nr) {
      const T* row = M + (r0 + r) * ld;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (c0 + e < cols) {
          const float x = ld_val(row, c0 + e);
          const double v = double(x);
          cs[e] = fma(v, v, cs[e]);
          rs = fma(v, v, rs);
          m = fmaxf(m, fabsf(x));
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) rs += __shfl_xor(rs, o);
    if (lane == 0) red[wave][r] = rs;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if (lane == 0) mred[wave] = m;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (c0 + e < cols) col_part[int64_t(blockIdx.y) * cols + c0 + e] = cs[e];
  __syncthreads();
  if (tid < nr)
    row_part[int64_t(blockIdx.x) * rows + r0 + tid] =
        red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
  if (tid == 0)
    mx[int64_t(blockIdx.y) * gridDim.x + blockIdx.x] =
        fmaxf(fmaxf(mred[0], mred[1]), fmaxf(mred[2], mred[3]));
}

// colsq[c] = sum over row tiles, rowsq[r] = sum over column tiles (fixed order)
__global__ __launch_bounds__(256) void stat_lines(const double* __restrict__ col_part,
                                                  const double* __restrict__ row_part,
                                                  int64_t rows, int64_t cols, int64_t nby,
                                                  int64_t nbx, double* __restrict__ colsq,
                                                  double* __restrict__ rowsq) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i < cols) {
    double s = 0.;
    for (int64_t b = 0; b < nby; ++b) s += col_part[b * cols + i];
    colsq[i] = s;
  }
  if (i < rows) {
    double s = 0.;
    for (int64_t b = 0; b < nbx; ++b) s += row_part[b * rows + i];
    rowsq[i] = s;
  }
}

// block-wide sum of a double over 1024 threads (all threads get the result)
__device__ double block_sum(double v, double* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  double t = 0.;
  for (int w = 0; w < int(blockDim.x >> 6); ++w) t += sh[w];
  return t;
}

// population coefficient of variation of the norms sqrt(sq[i]), two passes
__device__ double norm_cv(const double* __restrict__ sq, int64_t n, double* sh) {
  double s = 0.;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) s += sqrt(sq[i]);
  const double mean = block_sum(s, sh) / double(n);
  double v = 0.;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    const double d = sqrt(sq[i]) - mean;
    v = fma(d, d, v);
  }
  const double var = block_sum(v, sh) / double(n);
  return mean > 0. ? sqrt(var) / mean : 0.;
}

// out = {max |M|, ||M||_F^2, mu(M), CV_in (columns), CV_out (rows)}
__global__ __launch_bounds__(1024) void stat_final(const double* __restrict__ colsq,
                                                   const double* __restrict__ rowsq,
                                                   const float* __restrict__ mx, int64_t nmx,
                                                   int64_t rows, int64_t cols,
                                                   double* __restrict__ out) {
  __shared__ double sh[16];
  __shared__ float shm[16];
  double s = 0.;
  for (int64_t i = threadIdx.x; i < cols; i += blockDim.x) s += colsq[i];
  const double fro2 = block_sum(s, sh);
  float m = 0.f;
  for (int64_t i = threadIdx.x; i < nmx; i += blockDim.x) m = fmaxf(m, mx[i]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) shm[threadIdx.x >> 6] = m;
  __syncthreads();
  float mm = 0.f;
  for (int w = 0; w < int(blockDim.x >> 6); ++w) mm = fmaxf(mm, shm[w]);
  const double cv_in = norm_cv(colsq, cols, sh);
  const double cv_out = norm_cv(rowsq, rows, sh);
  if (threadIdx.x == 0) {
    out[0] = double(mm);
    out[1] = fro2;
    out[2] = fro2 > 0. ? sqrt(double(rows) * double(cols)) * double(mm) / sqrt(fro2) : 0.;
    out[3] = cv_in;
    out[4] = cv_out;
  }
}

// ---- Jacobi eigensolver ----------------------------------------------------------------------
// Round r pairs the n (even) indices by the circle method: position 0 holds index 0, position
// k >= 1 holds 1 + (k - 1 + r) mod (n - 1), and pair j joins positions j and n - 1 - j. Every
// pair of indices meets once in n - 1 rounds.
__device__ __forceinline__ int64_t rr_index(int64_t k, int64_t r, int64_t n) {
  return k == 0 ? 0 : 1 + (k - 1 + r) % (n - 1);
}

struct Rot {
  int p, q;
  float c, s, t;
};

// The rotation of every pair of round r, from the current matrix: J = [[c, s], [-s, c]] on
// (p, q) with tau = (a_qq - a_pp) / (2 a_pq), t = sign(tau) / (|tau| + sqrt(1 + tau^2)),
// c = 1 / sqrt(1 + t^2), s = t c zeroes a_pq (the symmetric 2 x 2 Schur decomposition).
// Pairs with |a_pq| below 1e-7 sqrt(|a_pp a_qq|), or with the padding index d, are skipped.
__global__ __launch_bounds__(256) void jacobi_params(const float* __restrict__ A, int64_t lda,
                                                     int64_t d, int64_t n, int64_t r,
                                                     Rot* __restrict__ rot) {
  const int64_t j = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (j >= n / 2) return;
  const int64_t p = rr_index(j, r, n), q = rr_index(n - 1 - j, r, n);
  Rot o{int(p), int(q), 1.f, 0.f, 0.f};
  if (p < d && q < d) {
    const double app = A[p * lda + p], aqq = A[q * lda + q], apq = A[p * lda + q];
    if (apq != 0. && fabs(apq) > 1e-7 * sqrt(fabs(app * aqq))) {
      const double tau = (aqq - app) / (2. * apq);
      const double t = (tau >= 0. ? 1. : -1.) / (fabs(tau) + sqrt(1. + tau * tau));
      const double c = 1. / sqrt(1. + t * t);
      o.c = float(c);
      o.s = float(t * c);
      o.t = float(t);
    }
  }
  rot[j] = o;
}

// B = J^T A J for all pairs of the round and V <- V J. Thread (row pair k1, column pair k2)
// computes the 2 x 2 block of B on rows (p1, q1) and columns (p2, q2), and the entries of V on
// rows (p1, q1) and columns (p2, q2) (in place: no other thread touches them). The diagonal
// blocks take the exact form: b_pp = a_pp - t a_pq, b_qq = a_qq + t a_pq, b_pq = b_qp = 0.
__global__ __launch_bounds__(256) void jacobi_apply(const float* __restrict__ A, float* __restrict__ B,
                                                    int64_t lda, float* __restrict__ V,
                                                    int64_t ldv, int64_t d, int64_t np,
                                                    const Rot* __restrict__ rot) {
  __shared__ Rot rc[64], rr[4];
  const int tid = threadIdx.x;
  const int64_t k2 = int64_t(blockIdx.x) * 64 + (tid & 63);
  const int64_t k1 = int64_t(blockIdx.y) * 4 + (tid >> 6);
  if (tid < 64 && int64_t(blockIdx.x) * 64 + tid < np) rc[tid] = rot[blockIdx.x * 64 + tid];
  if (tid >= 64 && tid < 68 && int64_t(blockIdx.y) * 4 + tid - 64 < np)
    rr[tid - 64] = rot[blockIdx.y * 4 + tid - 64];
  __syncthreads();
  if (k1 >= np || k2 >= np) return;
  const Rot R1 = rr[tid >> 6], R2 = rc[tid & 63];
  const int64_t p1 = R1.p, q1 = R1.q, p2 = R2.p, q2 = R2.q;
  const bool hp1 = p1 < d, hq1 = q1 < d, hp2 = p2 < d, hq2 = q2 < d;
  if (k1 == k2) {
    if (hp1 && hq1) {
      const float app = A[p1 * lda + p1], aqq = A[q1 * lda + q1], apq = A[p1 * lda + q1];
      const float aqp = A[q1 * lda + p1];
      if (R1.t != 0.f) {
        B[p1 * lda + p1] = app - R1.t * apq;
        B[q1 * lda + q1] = aqq + R1.t * apq;
        B[p1 * lda + q1] = 0.f;
        B[q1 * lda + p1] = 0.f;
      } else {
        B[p1 * lda + p1] = app;
        B[q1 * lda + q1] = aqq;
        B[p1 * lda + q1] = apq;
        B[q1 * lda + p1] = aqp;
      }
    } else if (hp1) {
      B[p1 * lda + p1] = A[p1 * lda + p1];
    } else if (hq1) {
      B[q1 * lda + q1] = A[q1 * lda + q1];
    }
  } else {
    const float a = hp1 && hp2 ? A[p1 * lda + p2] : 0.f;
    const float b = hp1 && hq2 ? A[p1 * lda + q2] : 0.f;
    const float e = hq1 && hp2 ? A[q1 * lda + p2] : 0.f;
    const float f = hq1 && hq2 ? A[q1 * lda + q2] : 0.f;
    const float a1 = R2.c * a - R2.s * b, b1 = R2.s * a + R2.c * b;  // columns: A J2
    const float e1 = R2.c * e - R2.s * f, f1 = R2.s * e + R2.c * f;
    if (hp1 && hp2) B[p1 * lda + p2] = R1.c * a1 - R1.s * e1;  // rows: J1^T (A J2)
    if (hp1 && hq2) B[p1 * lda + q2] = R1.c * b1 - R1.s * f1;
    if (hq1 && hp2) B[q1 * lda + p2] = R1.s * a1 + R1.c * e1;
    if (hq1 && hq2) B[q1 * lda + q2] = R1.s * b1 + R1.c * f1;
  }
  // V <- V J2 on rows p1, q1
  if (hp2 && hq2) {
    if (hp1) {
      const float vp = V[p1 * ldv + p2], vq = V[p1 * ldv + q2];
      V[p1 * ldv + p2] = R2.c * vp - R2.s * vq;
      V[p1 * ldv + q2] = R2.s * vp + R2.c * vq;
    }
    if (hq1) {
      const float vp = V[q1 * ldv + p2], vq = V[q1 * ldv + q2];
      V[q1 * ldv + p2] = R2.c * vp - R2.s * vq;
      V[q1 * ldv + q2] = R2.s * vp + R2.c * vq;
    }
  }
}

// A = H (d x d, dense copy), V = I
__global__ __launch_bounds__(256) void jacobi_init(const float* __restrict__ H, int64_t ldh,
                                                   float* __restrict__ A, int64_t lda,
                                                   float* __restrict__ V, int64_t ldv, int64_t d) {
  const int64_t i = blockIdx.y, j = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (j >= d) return;
  A[i * lda + j] = H[i * ldh + j];
  V[i * ldv + j] = i == j ? 1.f : 0.f;
}

// per-row fp64 sums of squares of A (off-diagonal only when off != 0)
__global__ __launch_bounds__(256) void row_squares(const float* __restrict__ A, int64_t lda,
                                                   int64_t d, int off, double* __restrict__ out) {
  __shared__ double sh[4];
  const int64_t i = blockIdx.x;
  double s = 0.;
  for (int64_t j = threadIdx.x; j < d; j += 256)
    if (!off || j != i) {
      const double v = A[i * lda + j];
      s = fma(v, v, s);
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) out[i] = sh[0] + sh[1] + sh[2] + sh[3];
}

// evals[k] = A_kk; *off = sqrt(sum of off-diagonal squares of A / sum of squares of H)
__global__ __launch_bounds__(1024) void jacobi_finish(const float* __restrict__ A, int64_t lda,
                                                      int64_t d, const double* __restrict__ hsq,
                                                      const double* __restrict__ osq,
                                                      float* __restrict__ evals,
                                                      double* __restrict__ off) {
  __shared__ double sh[16];
  double h = 0., o = 0.;
  for (int64_t i = threadIdx.x; i < d; i += blockDim.x) {
    h += hsq[i];
    o += osq[i];
    evals[i] = A[i * lda + i];
  }
  const double hs = block_sum(h, sh);
  const double os = block_sum(o, sh);
  if (threadIdx.x == 0) *off = hs > 0. ? sqrt(os / hs) : 0.;
}

// ---- expected-loss factors (Prop. 2, optimality table) ---------------------------------------
struct Alphas {
  double v[KRONQ_MAX_ALPHAS];
};

// out = {nearest, gptq, kronq, rho, tr(D), tr(H~), F(alpha_k) tr(D) for k < n_alpha}, with
// h_i = [H_G]_ii, a_i the squared row norms, F(alpha) = (sum h/s^2)(sum s^2 a),
// s_i = (h_i / a_i)^alpha (1 where h_i a_i = 0), D_p = 1 / U_pp^2 (the pivots of the sweep).
__global__ __launch_bounds__(1024) void proxy_final(const float* __restrict__ HG, int64_t ldg,
                                                    const double* __restrict__ rowsq,
                                                    int64_t d_out, const float* __restrict__ Hd,
                                                    int64_t ldh, const float* __restrict__ U,
                                                    int64_t ldu, int64_t d_in, Alphas al,
                                                    int n_alpha, double* __restrict__ out) {
  __shared__ double sh[16];
  double sh_h = 0., sh_a = 0., sh_ha = 0.;
  for (int64_t i = threadIdx.x; i < d_out; i += blockDim.x) {
    const double h = HG[i * ldg + i], a = rowsq[i];
    sh_h += h;
    sh_a += a;
    sh_ha += sqrt(h * a);
  }
  double td = 0., th = 0.;
  for (int64_t p = threadIdx.x; p < d_in; p += blockDim.x) {
    const double u = U[p * ldu + p];
    td += 1. / (u * u);
    th += Hd[p * ldh + p];
  }
  const double sum_h = block_sum(sh_h, sh), sum_a = block_sum(sh_a, sh);
  const double sum_ha = block_sum(sh_ha, sh);
  const double trD = block_sum(td, sh), trH = block_sum(th, sh);
  if (threadIdx.x == 0) {
    out[0] = sum_h * sum_a * trH;
    out[1] = sum_h * sum_a * trD;
    out[2] = sum_ha * sum_ha * trD;
    out[3] = sum_ha * sum_ha / (sum_h * sum_a);
    out[4] = trD;
    out[5] = trH;
  }
  for (int k = 0; k < n_alpha; ++k) {
    double f1 = 0., f2 = 0.;
    for (int64_t i = threadIdx.x; i < d_out; i += blockDim.x) {
      const double h = HG[i * ldg + i], a = rowsq[i];
      const double s2 = (h > 0. && a > 0.) ? pow(h / a, 2. * al.v[k]) : 1.;
      f1 += h / s2;
      f2 += s2 * a;
    }
    const double F1 = block_sum(f1, sh), F2 = block_sum(f2, sh);
    if (threadIdx.x == 0) out[6 + k] = F1 * F2 * trD;
  }
}

struct StatPlan {
  int64_t nbx, nby;
};
StatPlan stat_plan(int64_t rows, int64_t cols) { return {cdiv(cols, ST_COLS), cdiv(rows, ST_ROWS)}; }

// column and row sums of squares of M into colsq / rowsq, tile maxima into mx
int stat_passes(const void* M, int dtype, int64_t rows, int64_t cols, int64_t ld, Carver& cv,
                double** colsq, double** rowsq, float** mx, hipStream_t s) {
  const StatPlan sp = stat_plan(rows, cols);
  double* col_part = cv.take<double>(size_t(sp.nby * cols));
  double* row_part = cv.take<double>(size_t(sp.nbx * rows));
  *mx = cv.take<float>(size_t(sp.nbx * sp.nby));
  *colsq = cv.take<double>(size_t(cols));
  *rowsq = cv.take<double>(size_t(rows));
  const dim3 grid(static_cast<unsigned>(sp.nbx), static_cast<unsigned>(sp.nby));
  if (dtype == KRONQ_BF16)
    KQ_TRY(launch("diag_stat_tiles", stat_tiles<uint16_t>, grid, dim3(256), 0, s,
                  static_cast<const uint16_t*>(M), rows, cols, ld, col_part, row_part, *mx));
  else
    KQ_TRY(launch("diag_stat_tiles", stat_tiles<float>, grid, dim3(256), 0, s,
                  static_cast<const float*>(M), rows, cols, ld, col_part, row_part, *mx));
  return launch("diag_stat_lines", stat_lines,
                dim3(static_cast<unsigned>(cdiv(rows > cols ? rows : cols, 256))), dim3(256), 0, s,
                static_cast<const double*>(col_part), static_cast<const double*>(row_part), rows,
                cols, sp.nby, sp.nbx, *colsq, *rowsq);
}

size_t stat_ws_bytes(int64_t rows, int64_t cols) {
  const StatPlan sp = stat_plan(rows, cols);
  return align256(size_t(sp.nby * cols) * 8) + align256(size_t(sp.nbx * rows) * 8) +
         align256(size_t(sp.nbx * sp.nby) * 4) + align256(size_t(cols) * 8) +
         align256(size_t(rows) * 8) + 256;
}

}  // namespace

size_t matrix_stats_ws_bytes(int64_t rows, int64_t cols) {
  if (rows <= 0 || cols <= 0) return 0;
  return stat_ws_bytes(rows, cols);
}

int matrix_stats_launch(const void* M, int dtype, int64_t rows, int64_t cols, int64_t ld,
                        double* out, void* ws, hipStream_t s) {
  Carver cv(ws);
  double *colsq, *rowsq;
  float* mx;
  KQ_TRY(stat_passes(M, dtype, rows, cols, ld, cv, &colsq, &rowsq, &mx, s));
  const StatPlan sp = stat_plan(rows, cols);
  return launch("diag_stat_final", stat_final, dim3(1), dim3(1024), 0, s,
                static_cast<const double*>(colsq), static_cast<const double*>(rowsq),
                static_cast<const float*>(mx), sp.nbx * sp.nby, rows, cols, out);
}

size_t eigh_ws_bytes(int64_t d) {
  if (d <= 0) return 0;
  const int64_t n = d + (d & 1);
  return 2 * align256(size_t(d) * size_t(d) * 4) + align256(size_t(n / 2) * sizeof(Rot)) +
         2 * align256(size_t(d) * 8) + 256;
}

int eigh_launch(const float* H, int64_t d, int64_t ldh, int sweeps, float* evals, float* Q,
                int64_t ldq, double* off, void* ws, hipStream_t s) {
  Carver cv(ws);
  const int64_t n = d + (d & 1), np = n / 2;
  float* A0 = cv.take<float>(size_t(d) * size_t(d));
  float* A1 = cv.take<float>(size_t(d) * size_t(d));
  Rot* rot = cv.take<Rot>(size_t(np));
  double* hsq = cv.take<double>(size_t(d));
  double* osq = cv.take<double>(size_t(d));
  KQ_TRY(launch("diag_jacobi_init", jacobi_init,
                dim3(static_cast<unsigned>(cdiv(d, 256)), static_cast<unsigned>(d)), dim3(256), 0,
                s, H, ldh, A0, d, Q, ldq, d));
  KQ_TRY(launch("diag_row_squares", row_squares, dim3(static_cast<unsigned>(d)), dim3(256), 0,
                s, static_cast<const float*>(A0), d, d, 0, hsq));
  const dim3 pgrid(static_cast<unsigned>(cdiv(np, 256)));
  const dim3 agrid(static_cast<unsigned>(cdiv(np, 64)), static_cast<unsigned>(cdiv(np, 4)));
  float* cur = A0;
  float* nxt = A1;
  for (int sw = 0; sw < sweeps; ++sw) {
    for (int64_t r = 0; r < n - 1; ++r) {
      KQ_TRY(launch("diag_jacobi_params", jacobi_params, pgrid, dim3(256), 0, s,
                    static_cast<const float*>(cur), d, d, n, r, rot));
      KQ_TRY(launch("diag_jacobi_apply", jacobi_apply, agrid, dim3(256), 0, s,
                    static_cast<const float*>(cur), nxt, d, Q, ldq, d, np,
                    static_cast<const Rot*>(rot)));
      float* t = cur;
      cur = nxt;
      nxt = t;
    }
  }
  KQ_TRY(launch("diag_row_squares", row_squares, dim3(static_cast<unsigned>(d)), dim3(256), 0,
                s, static_cast<const float*>(cur), d, d, 1, osq));
  return launch("diag_jacobi_finish", jacobi_finish, dim3(1), dim3(1024), 0, s,
                static_cast<const float*>(cur), d, d, static_cast<const double*>(hsq),
                static_cast<const double*>(osq), evals, off);
}

size_t proxy_ws_bytes(int64_t d_out, int64_t d_in) {
  if (d_out <= 0 || d_in <= 0) return 0;
  return stat_ws_bytes(d_out, d_in);
}

int proxy_launch(const float* HG, int64_t ldg, const void* W, int w_dtype, int64_t ldw,
                 int64_t d_out, int64_t d_in, const float* Hd, int64_t ldh, const float* U,
                 int64_t ldu, const double* alphas, int n_alpha, double* out, void* ws,
                 hipStream_t s) {
  Carver cv(ws);
  double *colsq, *rowsq;
  float* mx;
  KQ_TRY(stat_passes(W, w_dtype, d_out, d_in, ldw, cv, &colsq, &rowsq, &mx, s));
  Alphas al{};
  for (int k = 0; k < n_alpha; ++k) al.v[k] = alphas[k];
  return launch("diag_proxy_final", proxy_final, dim3(1), dim3(1024), 0, s, HG, ldg,
                static_cast<const double*>(rowsq), d_out, Hd, ldh, U, ldu, d_in, al, n_alpha, out);
}

}  // namespace kq
