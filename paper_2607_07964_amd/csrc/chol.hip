// Damping and the inverse-Cholesky factor (Alg. 2 first two lines; Prop. 1 uses rows of it).
//
// inv(H~) = U^T U with U upper. With J the index reversal, J H~ J = L L^T (ordinary lower
// Cholesky) gives H~ = (J L J)(J L J)^T, so U = (J L J)^-1 = J L^-1 J. Steps:
//   1. damping: H~ = H + damp * mean(diag H) * I (in place), M = J H~ J (workspace copy);
//   2. blocked right-looking Cholesky of M with 128-wide panels: the diagonal block is factored
//      and inverted in LDS by one workgroup; the panel solve is P <- P Linv_kk^T and the trailing
//      update M22 -= P P^T (lower tiles only), both on the fp32 MFMA GEMM;
//   3. X = L^-1 by right-looking blocked forward substitution on the identity:
//      X[k, :k] = Linv_kk Y[k, :k], X[k, k] = Linv_kk, Y[k+1:, :k+1] -= L[k+1:, k] X[k, :k+1];
//   4. U[i][j] = X[d-1-i][d-1-j] for i <= j, 0 below the diagonal.
// A non-positive pivot sets *info to its 1-based column in the original order (first failure).
#include <cmath>

#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int NB = 128;
constexpr int DLD = NB + 1;  // LDS leading dimension of the diagonal block

__global__ __launch_bounds__(256) void diag_shift(const float* __restrict__ H, int64_t d,
                                                  int64_t ldh, float damp, float* __restrict__ shift,
                                                  int* __restrict__ info) {
  __shared__ double red[256];
  const int tid = threadIdx.x;
  double s = 0.0;
  for (int64_t i = tid; i < d; i += 256) s += H[i * ldh + i];
  red[tid] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    *shift = float(double(damp) * (red[0] / double(d)));
    *info = 0;
  }
}

__global__ void add_diag(float* __restrict__ H, int64_t d, int64_t ldh,
                         const float* __restrict__ shift) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < d) H[i * ldh + i] += *shift;
}

// M[i][j] = H[d-1-i][d-1-j]; X = 0
__global__ void reverse_copy(const float* __restrict__ H, int64_t d, int64_t ldh,
                             float* __restrict__ M, float* __restrict__ X, int64_t ldm) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < d;
       j += int64_t(gridDim.x) * blockDim.x) {
    M[i * ldm + j] = H[(d - 1 - i) * ldh + (d - 1 - j)];
    X[i * ldm + j] = 0.f;
  }
}

// Factor the diagonal block M[kb:kb+bs, kb:kb+bs] (lower) and invert the factor, in one
// workgroup, in a single pass over the columns j = 0..bs-1. Thread (ty, tx) of a 16 x 16 grid
// keeps entries (ty + 16 p, tx + 16 q), p, q < 8, of two matrices in registers:
//   r: the trailing matrix of the right-looking factorisation (entries above the diagonal ride
//      along unused), updated by the rank-1 term of column j;
//   y: R = I - (already eliminated terms), turned into rows of Y = L^-1 by forward
//      substitution: at step j, Y[j, :] = R[j, :] / L_jj, then R[i, :] -= L_ij Y[j, :] for i > j.
// Column j of the trailing matrix and row j of Y are exchanged through LDS, two barriers per
// column. Writes L_kk to M (lower part), Linv_kk (exact zeros above the diagonal) to dinv and X.
__global__ __launch_bounds__(256) void potrf_diag(float* __restrict__ M, int64_t ldm, int64_t kb,
                                                  int bs, int64_t d, float* __restrict__ dinv,
                                                  float* __restrict__ X, int* __restrict__ info) {
  __shared__ float l[NB * DLD];   // the factor L
  __shared__ float col[2][NB];    // column j of the trailing matrix
  __shared__ float yrow[NB];      // row j of Y
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  float r[8][8], y[8][8];
#pragma unroll
  for (int p = 0; p < 8; ++p)
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = ty + 16 * p, j = tx + 16 * q;
      r[p][q] = (i < bs && j < bs) ? M[(kb + i) * ldm + kb + j] : 0.f;
      y[p][q] = (i == j) ? 1.f : 0.f;
    }
  if (tx == 0) {
#pragma unroll
    for (int p = 0; p < 8; ++p) col[0][ty + 16 * p] = r[p][0];
  }
  __syncthreads();
  for (int j = 0; j < bs; ++j) {
    const float* cj = col[j & 1];
    const float piv = cj[j];
    if (!(piv > 0.f) && tid == 0) atomicCAS(info, 0, int(d - (kb + j)));  // also catches NaN
    const float ljj = sqrtf(piv);
    const float rl = 1.f / ljj;
    if (tid >= j && tid < bs) l[tid * DLD + j] = (tid == j) ? ljj : cj[tid] * rl;
    // row j of Y from its owners
    if (ty == (j & 15)) {
#pragma unroll
      for (int p = 0; p < 8; ++p)
        if (p == (j >> 4)) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            y[p][q] *= rl;
            yrow[tx + 16 * q] = y[p][q];
          }
        }
    }
    __syncthreads();
    float lc[8], cc[8], yj[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      lc[p] = cj[ty + 16 * p] * rl;  // L[i][j] for this thread's rows
      cc[p] = cj[tx + 16 * p];
      yj[p] = yrow[tx + 16 * p];
    }
    // row blocks p < j / 16 hold only finished rows: skip them (a wave-uniform branch); the
    // block containing row j is masked per row, later blocks are updated unconditionally
    const int jb = j >> 4;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      if (p < jb) continue;
      const float f = -lc[p] * rl;
#pragma unroll
      for (int q = 0; q < 8; ++q) r[p][q] = fmaf(f, cc[q], r[p][q]);
      if (p > jb) {
#pragma unroll
        for (int q = 0; q < 8; ++q) y[p][q] = fmaf(-lc[p], yj[q], y[p][q]);
      } else if (ty > (j & 15)) {
#pragma unroll
        for (int q = 0; q < 8; ++q) y[p][q] = fmaf(-lc[p], yj[q], y[p][q]);
      }
    }
    const int jn = j + 1;
    if (jn < bs && tx == (jn & 15)) {
      float* cn = col[jn & 1];
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (q == (jn >> 4)) {
#pragma unroll
          for (int p = 0; p < 8; ++p) cn[ty + 16 * p] = r[p][q];
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int p = 0; p < 8; ++p)
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = ty + 16 * p, j = tx + 16 * q;
      if (i < bs && j < bs) {
        if (j <= i) M[(kb + i) * ldm + kb + j] = l[i * DLD + j];
        dinv[i * NB + j] = y[p][q];
        X[(kb + i) * ldm + kb + j] = y[p][q];
      }
    }
}

// U[i][j] = X[d-1-i][d-1-j] for i <= j, else 0
__global__ void reverse_out(const float* __restrict__ X, int64_t ldm, int64_t d,
                            float* __restrict__ U, int64_t ldu) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < d;
       j += int64_t(gridDim.x) * blockDim.x)
    U[i * ldu + j] = (j >= i) ? X[(d - 1 - i) * ldm + (d - 1 - j)] : 0.f;
}

int64_t ld_for(int64_t d) { return ((d + 63) / 64) * 64; }

}  // namespace

size_t chol_ws_bytes(int64_t d) {
  if (d <= 0) return 0;
  const int64_t ld = ld_for(d);
  const int64_t nblk = cdiv(d, NB);
  return 2 * align256(size_t(d) * ld * sizeof(float)) +
         align256(size_t(nblk) * NB * NB * sizeof(float)) + 256;
}

int chol_launch(float* H, int64_t d, int64_t ldh, float damp_rel, float* U, int64_t ldu,
                int* info, void* ws, hipStream_t s) {
  const int64_t ld = ld_for(d);
  const int64_t nblk = cdiv(d, NB);
  Carver cv(ws);
  float* M = cv.take<float>(size_t(d) * ld);
  float* X = cv.take<float>(size_t(d) * ld);
  float* dinv = cv.take<float>(size_t(nblk) * NB * NB);
  float* shift = cv.take<float>(1);

  KQ_TRY(launch("chol_diag_shift", diag_shift, dim3(1), dim3(256), 0, s,
                static_cast<const float*>(H), d, ldh, damp_rel, shift, info));
  KQ_TRY(launch("chol_add_diag", add_diag, dim3(unsigned(cdiv(d, 256))), dim3(256), 0, s, H, d,
                ldh, static_cast<const float*>(shift)));
  const unsigned gx = unsigned(cdiv(d, 256) < 64 ? cdiv(d, 256) : 64);
  KQ_TRY(launch("chol_reverse_copy", reverse_copy, dim3(gx, unsigned(d)), dim3(256), 0, s,
                static_cast<const float*>(H), d, ldh, M, X, ld));

  // Cholesky of M (lower)
  for (int64_t k = 0; k < nblk; ++k) {
    const int64_t kb = k * NB;
    const int bs = int(d - kb < NB ? d - kb : NB);
    float* dk = dinv + k * NB * NB;
    KQ_TRY(launch("chol_potrf_diag", potrf_diag, dim3(1), dim3(256), 0, s, M, ld, kb, bs, d, dk,
                  X, info));
    const int64_t rest = d - kb - bs;
    if (rest > 0) {
      float* P = M + (kb + bs) * ld + kb;
      // P <- P Linv_kk^T  (in place: each workgroup owns whole rows of P, N = bs <= 128)
      KQ_TRY(gemm_f32(GEMM_TB, rest, bs, bs, 1.f, P, ld, dk, NB, 0.f, P, ld, s, "chol_trsm"));
      // M22 -= P P^T (lower tiles)
      float* M22 = M + (kb + bs) * ld + kb + bs;
      KQ_TRY(gemm_f32(GEMM_TB | GEMM_LOWER_C, rest, rest, bs, -1.f, P, ld, P, ld, 1.f, M22, ld, s,
                      "chol_syrk"));
    }
  }
  // X = L^-1
  for (int64_t k = 0; k < nblk; ++k) {
    const int64_t kb = k * NB;
    const int bs = int(d - kb < NB ? d - kb : NB);
    const float* dk = dinv + k * NB * NB;
    if (kb > 0) {
      // X[k, :kb] = Linv_kk Y[k, :kb]   (in place: M = bs <= 128 rows, one row tile)
      float* Xk = X + kb * ld;
      KQ_TRY(gemm_f32(GEMM_A_LOWER, bs, kb, bs, 1.f, dk, NB, Xk, ld, 0.f, Xk, ld, s,
                      "trtri_row"));
    }
    const int64_t rest = d - kb - bs;
    if (rest > 0) {
      // Y[kb+bs:, :kb+bs] -= L[kb+bs:, kb:kb+bs] X[k, :kb+bs]
      KQ_TRY(gemm_f32(0, rest, kb + bs, bs, -1.f, M + (kb + bs) * ld + kb, ld, X + kb * ld, ld,
                      1.f, X + (kb + bs) * ld, ld, s, "trtri_update"));
    }
  }
  return launch("chol_reverse_out", reverse_out, dim3(gx, unsigned(d)), dim3(256), 0, s,
                static_cast<const float*>(X), ld, d, U, ldu);
}

}  // namespace kq
