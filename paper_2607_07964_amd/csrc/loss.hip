// Traces (Sec. 4.3 eq. sensitivity) and the K-FAC layer loss (Sec. 4.1 eq. kron_obj).
//   traces: one workgroup sums both diagonals in float64.
//   loss:   dW = W - W_hat, A = H_G dW and B = dW H_X on the fp32 MFMA GEMM, then
//           sum_ij A_ij B_ij with float64 partial sums per workgroup and a final float64 sum.
#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int DOT_BLOCKS = 1024;

__global__ __launch_bounds__(256) void traces_kernel(const float* __restrict__ HX, int64_t d_in,
                                                     int64_t ldx, const float* __restrict__ HG,
                                                     int64_t d_out, int64_t ldg,
                                                     double* __restrict__ out3) {
  __shared__ double rx[256], rg[256];
  const int tid = threadIdx.x;
  double sx = 0.0, sg = 0.0;
  if (HX)
    for (int64_t i = tid; i < d_in; i += 256) sx += HX[i * ldx + i];
  if (HG)
    for (int64_t i = tid; i < d_out; i += 256) sg += HG[i * ldg + i];
  rx[tid] = sx;
  rg[tid] = sg;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) {
      rx[tid] += rx[tid + w];
      rg[tid] += rg[tid + w];
    }
    __syncthreads();
  }
  if (tid == 0) {
    const double tx = HX ? rx[0] : out3[0];
    const double tg = HG ? rg[0] : out3[1];
    out3[0] = tx;
    out3[1] = tg;
    out3[2] = tx * tg;
  }
}

template <typename T>
__device__ __forceinline__ float as_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float as_f32<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float as_f32<uint16_t>(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}

template <typename T>
__global__ void diff_kernel(const T* __restrict__ W, int64_t ldw, const float* __restrict__ Wh,
                            int64_t ldwh, int64_t d_out, int64_t d_in, float* __restrict__ D,
                            int64_t ldd) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < ldd;
       j += int64_t(gridDim.x) * blockDim.x) {
    float v = 0.f;
    if (j < d_in) {
      const float w = as_f32(W, i * ldw + j);
      v = Wh ? w - Wh[i * ldwh + j] : w;
    }
    D[i * ldd + j] = v;  // padding columns are zero so they add nothing to the dot product
  }
}

__global__ __launch_bounds__(256) void dot_partial(const float* __restrict__ A,
                                                   const float* __restrict__ B, int64_t rows,
                                                   int64_t cols, int64_t ld,
                                                   double* __restrict__ part) {
  __shared__ double red[256];
  const int tid = threadIdx.x;
  double s = 0.0;
  const int64_t n = rows * cols;
  for (int64_t i = int64_t(blockIdx.x) * 256 + tid; i < n; i += int64_t(gridDim.x) * 256) {
    const int64_t o = (i / cols) * ld + (i % cols);
    s += double(A[o]) * double(B[o]);
  }
  red[tid] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) part[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(256) void dot_final(const double* __restrict__ part, int n,
                                                 double* __restrict__ out) {
  __shared__ double red[256];
  const int tid = threadIdx.x;
  double s = 0.0;
  for (int i = tid; i < n; i += 256) s += part[i];
  red[tid] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) *out = red[0];
}

}  // namespace

int traces_launch(const float* HX, int64_t d_in, int64_t ldx, const float* HG, int64_t d_out,
                  int64_t ldg, double* out3, hipStream_t s) {
  return launch("traces", traces_kernel, dim3(1), dim3(256), 0, s, HX, d_in, ldx, HG, d_out, ldg,
                out3);
}

size_t loss_ws_bytes(int64_t d_out, int64_t d_in) {
  if (d_out <= 0 || d_in <= 0) return 0;
  const int64_t ldd = cdiv(d_in, 4) * 4;
  return 3 * align256(size_t(d_out) * ldd * sizeof(float)) +
         align256(DOT_BLOCKS * sizeof(double)) + 256;
}

int loss_launch(const void* W, int w_dtype, int64_t ldw, const float* W_hat, int64_t ldwh,
                int64_t d_out, int64_t d_in, const float* HX, int64_t ldx, const float* HG,
                int64_t ldg, double* loss, void* ws, hipStream_t s) {
  Carver cv(ws);
  const int64_t ldd = cdiv(d_in, 4) * 4;  // 16-byte rows for the GEMM's vector loads
  const size_t n = size_t(d_out) * ldd;
  float* D = cv.take<float>(n);
  float* A = cv.take<float>(n);
  float* B = cv.take<float>(n);
  double* part = cv.take<double>(DOT_BLOCKS);
  const dim3 g(unsigned(cdiv(d_in, 256) < 64 ? cdiv(d_in, 256) : 64), unsigned(d_out));
  if (w_dtype == KRONQ_BF16)
    KQ_TRY(launch("loss_diff", diff_kernel<uint16_t>, g, dim3(256), 0, s,
                  static_cast<const uint16_t*>(W), ldw, W_hat, ldwh, d_out, d_in, D, ldd));
  else
    KQ_TRY(launch("loss_diff", diff_kernel<float>, g, dim3(256), 0, s,
                  static_cast<const float*>(W), ldw, W_hat, ldwh, d_out, d_in, D, ldd));
  KQ_TRY(gemm_f32(0, d_out, d_in, d_out, 1.f, HG, ldg, D, ldd, 0.f, A, ldd, s, "loss_gemm"));
  KQ_TRY(gemm_f32(0, d_out, d_in, d_in, 1.f, D, ldd, HX, ldx, 0.f, B, ldd, s, "loss_gemm"));
  const int64_t nb = cdiv(int64_t(n), 256) < DOT_BLOCKS ? cdiv(int64_t(n), 256) : DOT_BLOCKS;
  KQ_TRY(launch("loss_dot", dot_partial, dim3(unsigned(nb)), dim3(256), 0, s,
                static_cast<const float*>(A), static_cast<const float*>(B), d_out, d_in, ldd, part));
  return launch("loss_final", dot_final, dim3(1), dim3(256), 0, s,
                static_cast<const double*>(part), int(nb), loss);
}

}  // namespace kq
