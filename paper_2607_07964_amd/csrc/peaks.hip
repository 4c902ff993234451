// Measured ceiling of the bf16 matrix cores on given data: a register-resident loop of
// v_mfma_f32_32x32x16_bf16 with no memory traffic inside the loop. The MI355X clock is
// power-limited under MFMA load and the limit depends on the operand values, so this gives the
// rate the covariance and trailing-update kernels can reach on the workload's data, next to the
// 2.5 PFLOP/s of the data sheet.
//   * Two workgroups of 4 waves per CU; each wave keeps 8 independent 32 x 32 accumulators and
//     cycles through 4 operand fragments read once from `data` (bf16 values of the caller's
//     choosing: zeros, N(0,1), the covariance's own inputs).
//   * Per iteration a wave issues 8 MFMAs of 32 x 32 x 16 (8 x 32768 flops).
//   * The accumulators are reduced to one float per workgroup in `out`, so nothing is elided.
#include "kq_common.hpp"

namespace kq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256, 2) void mfma_peak_loop(const uint16_t* __restrict__ data,
                                                         int iters, float* __restrict__ out) {
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // 4 fragments of 8 bf16 per lane, from distinct parts of the 4096-element buffer
  bf16x8_t f[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    f[i] = *reinterpret_cast<const bf16x8_t*>(data + ((i * 64 + lane) * 8 + wave * 16) % 4096);
  f32x16_t acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x16_t{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[i & 3], f[(i + 1 + (i >> 2)) & 3],
                                                        acc[i], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[i][r];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  if (tid == 0) out[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

}  // namespace

int mfma_peak_launch(const uint16_t* data, int iters, float* out, int* workgroups, hipStream_t s) {
  int dev = 0, cus = 0;
  KQ_HIP(hipGetDevice(&dev));
  KQ_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  const int wgs = 2 * cus;
  *workgroups = wgs;
  return launch("mfma_peak_loop", mfma_peak_loop, dim3(unsigned(wgs)), dim3(256), 0, s, data,
                iters, out);
}

}  // namespace kq
