// Diagnostics of the incoherence processing (Sec. 2.3 eq. incoherence_measure; Sec. 4.2 with
// Fig. 2; Prop. 2 eq. biip-bound and the optimality table of appendix A.3):
//  * matrix statistics: max |M_ij|, ||M||_F^2, mu(M), and the coefficients of variation of the
//    column and row norms, in three deterministic passes (tiles, lines, one final workgroup);
//  * the symmetric eigendecomposition behind mu(H), by block Jacobi: 64 x 64 subproblems of
//    block pairs solved in LDS by scalar Jacobi rotations, their rotations applied to the whole
//    matrix as 64 x 64 tile products, block pairs in round-robin order;
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

// ---- block Jacobi eigensolver ----------------------------------------------------------------
// The order-N matrix (N = d rounded up to a multiple of 64, zero padding) is split into nb = N/32
// blocks of 32 indices. Round r of a sweep pairs the blocks by the circle method (position 0
// holds block 0, position k >= 1 block 1 + (k - 1 + r) mod (nb - 1), pair j joins positions j
// and nb - 1 - j), so every pair of blocks meets once in nb - 1 rounds. For each pair (P, Q) the
// 64 x 64 principal submatrix S is diagonalised in LDS by cyclic scalar Jacobi rotations,
// S = Z diag Z^T; then A <- J^T A J and V <- V J with J the block-diagonal (permuted) product of
// the Z of all pairs of the round. Padding indices have zero rows and columns: their rotations
// are skipped, so they never mix with real indices.
constexpr int BJ = 32;  // block size
constexpr int BT = 64;  // two blocks: the subproblem order and the tile of the update
constexpr int TS = 68;  // padded LDS row of a tile
// inner sweeps per block-pair visit at most: the outer sweeps revisit every pair, so one suffices
// (measured: the same convergence per outer sweep as with two, at half the cost)
constexpr int kInnerSweeps = 1;

__device__ __forceinline__ int circle(int k, int r, int n) {
  return k == 0 ? 0 : 1 + (k - 1 + r) % (n - 1);
}
// global index of local index m < 64 of the block pair (P, Q)
__device__ __forceinline__ int64_t pair_index(int m, int P, int Q) {
  return int64_t(m < BJ ? P : Q) * BJ + (m & (BJ - 1));
}

// The rotation J = [[c, s], [-s, c]] on (p, q) that zeroes s_pq (the symmetric 2 x 2 Schur step:
// tau = (s_qq - s_pp) / (2 s_pq), t = sign(tau) / (|tau| + sqrt(1 + tau^2)), c = 1/sqrt(1+t^2),
// s = t c), in fp32 (its accuracy sets the convergence rate only: whatever angle results is
// applied as an orthogonal rotation); skipped (t = 0) when |s_pq| <= 1e-7 sqrt(|s_pp s_qq|). It
// is applied in Rutishauser's form, (x, y) -> (x - s (y + r x), y + s (x - r y)) with
// r = s / (1 + c): for small angles c rounds to 1 in fp32 and c x - s y would grow every norm by
// about s^2 / 2.
__device__ __forceinline__ void schur2(float spp, float sqq, float spq, float& sn, float& rr,
                                       float& t) {
  sn = 0.f, rr = 0.f, t = 0.f;
  if (spq != 0.f && fabsf(spq) > 1e-7f * sqrtf(fabsf(spp)) * sqrtf(fabsf(sqq))) {
    const float tau = (sqq - spp) / (2.f * spq);
    t = (tau >= 0.f ? 1.f : -1.f) / (fabsf(tau) + sqrtf(fmaf(tau, tau, 1.f)));
    const float c = 1.f / sqrtf(fmaf(t, t, 1.f));
    sn = t * c;
    rr = sn / (1.f + c);
  }
}
// (x, y) <- (c x - s y, s x + c y)
__device__ __forceinline__ void rot2(float& x, float& y, float sn, float rr) {
  const float x0 = x, y0 = y;
  x = x0 - sn * fmaf(rr, x0, y0);
  y = y0 + sn * fmaf(-rr, y0, x0);
}

// One workgroup per block pair of round r: diagonalise S (inner sweeps until a sweep rotates
// nothing, at most max_inner) and store its rotation Z (64 x 64, row-major) in zbuf[pair].
__global__ __launch_bounds__(256) void bjac_solve(const float* __restrict__ A, int64_t lda, int nb,
                                                  int r, int max_inner, float* __restrict__ zbuf) {
  __shared__ float S[BT][BT + 1], Z[BT][BT + 1];
  __shared__ float pr[BT / 2], ps[BT / 2], pt[BT / 2];
  __shared__ int pp[BT / 2], pq[BT / 2], any_rot;
  const int tid = threadIdx.x, j = blockIdx.x;
  const int P = circle(j, r, nb), Q = circle(nb - 1 - j, r, nb);
  for (int e = tid; e < BT * BT; e += 256) {
    const int i = e >> 6, c = e & 63;
    S[i][c] = A[pair_index(i, P, Q) * lda + pair_index(c, P, Q)];
    Z[i][c] = i == c ? 1.f : 0.f;
  }
  for (int sw = 0; sw < max_inner; ++sw) {
    if (tid == 0) any_rot = 0;
    __syncthreads();
    for (int rr = 0; rr < BT - 1; ++rr) {
      if (tid < BT / 2) {
        const int p = circle(tid, rr, BT), q = circle(BT - 1 - tid, rr, BT);
        float sn, rr2, t;
        schur2(S[p][p], S[q][q], S[p][q], sn, rr2, t);
        pp[tid] = p, pq[tid] = q, pr[tid] = rr2, ps[tid] = sn, pt[tid] = t;
        if (t != 0.f) any_rot = 1;
      }
      __syncthreads();
      // S <- J^T S J (the 2 x 2 block of row pair k1 and column pair k2) and Z <- Z J (row i,
      // column pair k2), in place: the entries of different work items are disjoint, so all
      // are read first, then rotated, then written (no load waits on an earlier store)
      int bp1[4], bq1[4], bp2[4], bq2[4], zi[8], zp2[8], zq2[8];
      float v[4][4], zv[8][2];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int bi = tid + 256 * u, k1 = bi >> 5, k2 = bi & 31;
        bp1[u] = pp[k1], bq1[u] = pq[k1], bp2[u] = pp[k2], bq2[u] = pq[k2];
        v[u][0] = S[bp1[u]][bp2[u]], v[u][1] = S[bp1[u]][bq2[u]];
        v[u][2] = S[bq1[u]][bp2[u]], v[u][3] = S[bq1[u]][bq2[u]];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = tid + 256 * u, k2 = e & 31;
        zi[u] = e >> 5, zp2[u] = pp[k2], zq2[u] = pq[k2];
        zv[u][0] = Z[zi[u]][zp2[u]], zv[u][1] = Z[zi[u]][zq2[u]];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int bi = tid + 256 * u, k1 = bi >> 5, k2 = bi & 31;
        if (k1 == k2) {  // diagonal block: the exact form
          const float t = pt[k1], apq = v[u][1];
          if (t != 0.f) {
            v[u][0] -= t * apq;
            v[u][3] += t * apq;
            v[u][1] = 0.f;
            v[u][2] = 0.f;
          }
        } else {
          rot2(v[u][0], v[u][1], ps[k2], pr[k2]);  // columns: S J2
          rot2(v[u][2], v[u][3], ps[k2], pr[k2]);
          rot2(v[u][0], v[u][2], ps[k1], pr[k1]);  // rows: J1^T (S J2)
          rot2(v[u][1], v[u][3], ps[k1], pr[k1]);
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k2 = (tid + 256 * u) & 31;
        rot2(zv[u][0], zv[u][1], ps[k2], pr[k2]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        S[bp1[u]][bp2[u]] = v[u][0], S[bp1[u]][bq2[u]] = v[u][1];
        S[bq1[u]][bp2[u]] = v[u][2], S[bq1[u]][bq2[u]] = v[u][3];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) Z[zi[u]][zp2[u]] = zv[u][0], Z[zi[u]][zq2[u]] = zv[u][1];
      __syncthreads();
    }
    const int rot = any_rot;
    __syncthreads();  // every thread has read the flag before the next sweep clears it
    if (!rot) break;
  }
  // unit columns: fp32 rotations leave each column's norm about 3e-8 too large on average, and
  // over the rounds of many sweeps that bias would scale V's columns and A's eigenvalues
  __shared__ float zs[BT];
  if (tid < BT) {
    double n2 = 0.;
    for (int i = 0; i < BT; ++i) n2 = fma(double(Z[i][tid]), double(Z[i][tid]), n2);
    zs[tid] = float(1. / sqrt(n2));
  }
  __syncthreads();
  float* zo = zbuf + int64_t(j) * BT * BT;
  for (int e = tid; e < BT * BT; e += 256) zo[e] = Z[e >> 6][e & 63] * zs[e & 63];
}

// out (64 x 64, 4 x 4 per thread) = X^T_or_not . Y from LDS tiles: trans selects X^T
__device__ __forceinline__ void tile_mm(const float (*X)[TS], const float (*Y)[TS], bool trans,
                                        int tid, float (&acc)[4][4]) {
  const int r0 = (tid >> 4) * 4, c0 = (tid & 15) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) acc[i][jj] = 0.f;
  for (int k = 0; k < BT; ++k) {
    float x[4];
    if (trans) {
      const float4 v = *reinterpret_cast<const float4*>(&X[k][r0]);
      x[0] = v.x, x[1] = v.y, x[2] = v.z, x[3] = v.w;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = X[r0 + i][k];
    }
    const float4 y = *reinterpret_cast<const float4*>(&Y[k][c0]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[i][0] = fmaf(x[i], y.x, acc[i][0]);
      acc[i][1] = fmaf(x[i], y.y, acc[i][1]);
      acc[i][2] = fmaf(x[i], y.z, acc[i][2]);
      acc[i][3] = fmaf(x[i], y.w, acc[i][3]);
    }
  }
}

// Tile (x, y) of the round's update: for y < np, B[rows of pair y][cols of pair x] =
// Z_y^T A[...][...] Z_x (from A, into the other buffer B); for y >= np, the 64 rows starting at
// 64 (y - np) of V times Z_x, in place (the workgroup holds its tile in LDS before writing it).
__global__ __launch_bounds__(256) void bjac_apply(const float* __restrict__ A, float* __restrict__ B,
                                                  float* __restrict__ V, int64_t lda, int nb, int r,
                                                  const float* __restrict__ zbuf) {
  __shared__ __attribute__((aligned(16))) float X[BT][TS], Zt[BT][TS], W[BT][TS];
  const int tid = threadIdx.x, np = nb / 2;
  const int kx = blockIdx.x, ky = blockIdx.y;
  const int P2 = circle(kx, r, nb), Q2 = circle(nb - 1 - kx, r, nb);
  const bool vt = ky >= np;
  int P1 = 0, Q1 = 0;
  if (!vt) P1 = circle(ky, r, nb), Q1 = circle(nb - 1 - ky, r, nb);
  const int64_t vrow0 = int64_t(ky - np) * BT;
  for (int e = tid; e < BT * BT; e += 256) {
    const int i = e >> 6, c = e & 63;
    const int64_t row = vt ? vrow0 + i : pair_index(i, P1, Q1);
    X[i][c] = (vt ? V : A)[row * lda + pair_index(c, P2, Q2)];
    Zt[i][c] = zbuf[int64_t(kx) * BT * BT + e];
  }
  __syncthreads();
  float acc[4][4];
  tile_mm(X, Zt, false, tid, acc);  // X Z_x
  const int r0 = (tid >> 4) * 4, c0 = (tid & 15) * 4;
  if (vt) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) V[(vrow0 + r0 + i) * lda + pair_index(c0 + jj, P2, Q2)] = acc[i][jj];
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) W[r0 + i][c0 + jj] = acc[i][jj];
  __syncthreads();  // W complete; Zt free
  for (int e = tid; e < BT * BT; e += 256) Zt[e >> 6][e & 63] = zbuf[int64_t(ky) * BT * BT + e];
  __syncthreads();
  tile_mm(Zt, W, true, tid, acc);  // Z_y^T (X Z_x)
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      B[pair_index(r0 + i, P1, Q1) * lda + pair_index(c0 + jj, P2, Q2)] = acc[i][jj];
}

// A = H padded with zeros to N x N, V = I (N x N)
__global__ __launch_bounds__(256) void bjac_init(const float* __restrict__ H, int64_t ldh, int64_t d,
                                                 float* __restrict__ A, float* __restrict__ V,
                                                 int64_t N) {
  const int64_t i = blockIdx.y, j = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (j >= N) return;
  A[i * N + j] = (i < d && j < d) ? H[i * ldh + j] : 0.f;
  V[i * N + j] = i == j ? 1.f : 0.f;
}

// Q = the leading d x d block of V
__global__ __launch_bounds__(256) void bjac_out(const float* __restrict__ V, int64_t N, int64_t d,
                                                float* __restrict__ Q, int64_t ldq) {
  const int64_t i = blockIdx.y, j = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (j < d) Q[i * ldq + j] = V[i * N + j];
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
  const int64_t N = cdiv(d, BT) * BT;
  return 3 * align256(size_t(N) * size_t(N) * 4) + align256(size_t(N / BT) * BT * BT * 4) +
         2 * align256(size_t(d) * 8) + 256;
}

int eigh_launch(const float* H, int64_t d, int64_t ldh, int sweeps, float* evals, float* Q,
                int64_t ldq, double* off, void* ws, hipStream_t s) {
  Carver cv(ws);
  const int64_t N = cdiv(d, BT) * BT;
  const int nb = int(N / BJ), np = nb / 2;
  float* A0 = cv.take<float>(size_t(N) * size_t(N));
  float* A1 = cv.take<float>(size_t(N) * size_t(N));
  float* V = cv.take<float>(size_t(N) * size_t(N));
  float* zbuf = cv.take<float>(size_t(np) * BT * BT);
  double* hsq = cv.take<double>(size_t(d));
  double* osq = cv.take<double>(size_t(d));
  KQ_TRY(launch("diag_bjac_init", bjac_init,
                dim3(static_cast<unsigned>(cdiv(N, 256)), static_cast<unsigned>(N)), dim3(256), 0,
                s, H, ldh, d, A0, V, N));
  KQ_TRY(launch("diag_row_squares", row_squares, dim3(static_cast<unsigned>(d)), dim3(256), 0,
                s, static_cast<const float*>(A0), N, d, 0, hsq));
  float* cur = A0;
  float* nxt = A1;
  for (int sw = 0; sw < sweeps; ++sw) {
    for (int r = 0; r < nb - 1; ++r) {
      KQ_TRY(launch("diag_bjac_solve", bjac_solve, dim3(static_cast<unsigned>(np)), dim3(256), 0,
                    s, static_cast<const float*>(cur), N, nb, r, kInnerSweeps, zbuf));
      KQ_TRY(launch("diag_bjac_apply", bjac_apply,
                    dim3(static_cast<unsigned>(np), static_cast<unsigned>(np + N / BT)),
                    dim3(256), 0, s, static_cast<const float*>(cur), nxt, V, N, nb, r,
                    static_cast<const float*>(zbuf)));
      float* t = cur;
      cur = nxt;
      nxt = t;
    }
  }
  KQ_TRY(launch("diag_bjac_out", bjac_out,
                dim3(static_cast<unsigned>(cdiv(d, 256)), static_cast<unsigned>(d)), dim3(256), 0,
                s, static_cast<const float*>(V), N, d, Q, ldq));
  KQ_TRY(launch("diag_row_squares", row_squares, dim3(static_cast<unsigned>(d)), dim3(256), 0,
                s, static_cast<const float*>(cur), N, d, 1, osq));
  return launch("diag_jacobi_finish", jacobi_finish, dim3(1), dim3(1024), 0, s,
                static_cast<const float*>(cur), N, d, static_cast<const double*>(hsq),
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
