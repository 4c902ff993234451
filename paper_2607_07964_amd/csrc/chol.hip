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

// Factor the diagonal block M[kb:kb+bs, kb:kb+bs] (lower) in LDS and invert it.
// Writes L_kk back to M (lower part) and Linv_kk (bs x bs, zero above the diagonal) to dinv.
__global__ __launch_bounds__(256) void potrf_diag(float* __restrict__ M, int64_t ldm, int64_t kb,
                                                  int bs, int64_t d, float* __restrict__ dinv,
                                                  int* __restrict__ info) {
  __shared__ float a[NB * DLD];
  __shared__ float x[NB * DLD];  // column c of the inverse lives in x[.][c]
  const int tid = threadIdx.x;
  for (int idx = tid; idx < bs * bs; idx += 256) {
    const int i = idx / bs, j = idx % bs;
    a[i * DLD + j] = M[(kb + i) * ldm + kb + j];
  }
  __syncthreads();
  for (int j = 0; j < bs; ++j) {
    const float piv = a[j * DLD + j];
    if (!(piv > 0.f) && tid == 0) atomicCAS(info, 0, int(d - (kb + j)));  // also catches NaN
    const float ljj = sqrtf(piv);
    __syncthreads();
    if (tid == 0) a[j * DLD + j] = ljj;
    for (int i = j + 1 + tid; i < bs; i += 256) a[i * DLD + j] /= ljj;
    __syncthreads();
    const int n = bs - j - 1;  // trailing order
    for (int idx = tid; idx < n * n; idx += 256) {
      const int i = j + 1 + idx / n, c = j + 1 + idx % n;
      if (c <= i) a[i * DLD + c] -= a[i * DLD + j] * a[c * DLD + j];
    }
    __syncthreads();
  }
  // inverse: thread c solves L x = e_c; rows in order, all threads read the same L entries
  if (tid < bs) {
    const int c = tid;
    for (int i = 0; i < bs; ++i) {
      float v;
      if (i < c) {
        v = 0.f;
      } else if (i == c) {
        v = 1.f / a[i * DLD + i];
      } else {
        float s = 0.f;
        for (int k = c; k < i; ++k) s = fmaf(a[i * DLD + k], x[k * DLD + c], s);
        v = -s / a[i * DLD + i];
      }
      x[i * DLD + c] = v;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < bs * bs; idx += 256) {
    const int i = idx / bs, j = idx % bs;
    if (j <= i) M[(kb + i) * ldm + kb + j] = a[i * DLD + j];
    dinv[i * NB + j] = x[i * DLD + j];
  }
}

// X[kb:kb+bs, kb:kb+bs] = Linv_kk (full block, zeros above the diagonal)
__global__ void put_diag(float* __restrict__ X, int64_t ldm, int64_t kb, int bs,
                         const float* __restrict__ dinv) {
  for (int idx = threadIdx.x; idx < bs * bs; idx += blockDim.x) {
    const int i = idx / bs, j = idx % bs;
    X[(kb + i) * ldm + kb + j] = dinv[i * NB + j];
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
                  info));
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
    KQ_TRY(launch("trtri_put_diag", put_diag, dim3(1), dim3(256), 0, s, X, ld, kb, bs, dk));
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
