// Butterflies of the fast Walsh-Hadamard transform in LDS, shared by the rotation passes and the
// online transforms (Sylvester order: entry (i, j) of H is (-1)^popcount(i & j)).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace kq {

template <int R>
__device__ __forceinline__ void hadamard_reg(float* x) {
#pragma unroll
  for (int s = 1; s < R; s <<= 1)
#pragma unroll
    for (int k = 0; k < R; ++k)
      if (!(k & s)) {
        const float a = x[k], b = x[k + s];
        x[k] = a + b;
        x[k + s] = a - b;
      }
}

// One group of up to 3 butterfly stages (strides h, 2h, 4h; h = 2^lgh) over a buffer of n
// floats in LDS (n <= 2^24, so 32-bit indices; shifts and masks instead of divisions).
template <int R>
__device__ __forceinline__ void fwht_stage_group(float* buf, int n, int lgh, int tid,
                                                 int nthreads) {
  const int groups = n / R, hm = (1 << lgh) - 1;
  for (int q = tid; q < groups; q += nthreads) {
    const int base = (q >> lgh) * (R << lgh) + (q & hm);
    float x[R];
#pragma unroll
    for (int k = 0; k < R; ++k) x[k] = buf[base + (k << lgh)];
    hadamard_reg<R>(x);
#pragma unroll
    for (int k = 0; k < R; ++k) buf[base + (k << lgh)] = x[k];
  }
}

// FWHT of every length-m segment (m a power of 2) of buf[0, n), from the stage of stride
// 2^lgh0 on
__device__ inline void fwht_lds(float* buf, int64_t n, int64_t m, int tid, int nthreads,
                                int lgh0 = 0) {
  int lgh = lgh0;  // stages of strides below 2^lgh0 already applied
  while ((int64_t(1) << lgh) < m) {
    const int64_t left = m >> lgh;
    if (left >= 8) {
      fwht_stage_group<8>(buf, int(n), lgh, tid, nthreads);
      lgh += 3;
    } else if (left == 4) {
      fwht_stage_group<4>(buf, int(n), lgh, tid, nthreads);
      lgh += 2;
    } else {
      fwht_stage_group<2>(buf, int(n), lgh, tid, nthreads);
      lgh += 1;
    }
    __syncthreads();
  }
}

}  // namespace kq
