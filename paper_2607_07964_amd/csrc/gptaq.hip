// Drift correction of the sweep (Prop. 1 eq. kronq_update; Alg. 2 third line):
// P = alpha ((D L) . M_U) L^T, where inv(H~) = L L^T with L the transpose of the upper factor U
// that kronq_cholesky_inv returns, and M_U keeps the strictly upper triangle. Row p of P is
// alpha D[p, p+1:] inv(H~[p+1:, p+1:]): the columns after p absorb column p's input drift.
// Two fp32 products on the fp32 matrix cores (gemm_f32.hip), each over half the tiles and a
// triangular K range:
//   T = D U^T      upper tiles only; k from the column-tile start (U^T is lower triangular);
//   T <- the strictly upper part of T;
//   P = alpha T U  upper tiles only; k from the row-tile start (T strictly upper) to the
//                  column-tile end (U upper);
// then everything on and below P's diagonal is cleared: those entries are zero by structure,
// and the tiles the product skips are never written. 2 d^3 / 3 flops in all.
#include "kq_common.hpp"

namespace kq {
namespace {

// M[i][j] = 0 for j <= i (row i = blockIdx.y)
__global__ __launch_bounds__(256) void clear_lower(float* __restrict__ M, int64_t d, int64_t ld) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j <= i && j < d;
       j += int64_t(gridDim.x) * blockDim.x)
    M[i * ld + j] = 0.f;
}

int64_t t_ld(int64_t d) { return cdiv(d, 64) * 64; }

}  // namespace

size_t gptaq_ws_bytes(int64_t d) {
  if (d <= 0) return 0;
  return align256(size_t(d) * size_t(t_ld(d)) * sizeof(float)) + 256;
}

int gptaq_launch(const float* D, int64_t d, int64_t ldd, const float* U, int64_t ldu, float alpha,
                 float* P, int64_t ldp, void* ws, hipStream_t s) {
  Carver cv(ws);
  const int64_t ldt = t_ld(d);
  float* T = cv.take<float>(size_t(d) * size_t(ldt));
  const dim3 mgrid(unsigned(cdiv(d, 256)), unsigned(d));
  KQ_TRY(gemm_f32(GEMM_TB | GEMM_B_LOWER | GEMM_UPPER_C, d, d, d, 1.f, D, ldd, U, ldu, 0.f, T,
                  ldt, s, "gptaq_d_ut"));
  KQ_TRY(launch("gptaq_mask", clear_lower, mgrid, dim3(256), 0, s, T, d, ldt));
  KQ_TRY(gemm_f32(GEMM_A_UPPER | GEMM_OPB_UPPER | GEMM_UPPER_C, d, d, d, alpha, T, ldt, U, ldu,
                  0.f, P, ldp, s, "gptaq_t_u"));
  return launch("gptaq_mask", clear_lower, mgrid, dim3(256), 0, s, P, d, ldp);
}

}  // namespace kq
