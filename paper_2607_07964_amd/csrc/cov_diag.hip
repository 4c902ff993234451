// diag(A^T A) as column sums of squares (Sec. 4.1 eq. kfac; the diagonal that the rescaling of
// eq. rescale reads), for a caller that needs a side's S before that side's covariance exists.
#include <algorithm>
#include <mutex>

#include "kq_common.hpp"

// The chunk partials of kronq_cov_diag_noalloc: a fixed device array instead of a caller's
// workspace (16 MiB on each GPU the library runs on, held until the process ends). Host code
// never passes this name to a kernel: it stands for a host-side symbol, and each device's copy
// has its own address, taken with hipGetSymbolAddress (cov_diag_scratch below).
static __device__ __align__(256) double scratch[size_t(KRONQ_NOALLOC_SCRATCH_BYTES) / sizeof(double)];

namespace kq {
namespace {
// diag(A^T A) without the covariance: column sums of squares. A workgroup takes CSQ_COLS columns
// of one chunk of rows: thread t owns 16 of them (two runs of 8), so each row is read as one
// contiguous stretch of up to 8 KB (bf16) by the whole workgroup, with several rows in flight
// per thread. Squares are summed in fp64 (a bf16 input gives the exact sum up to fp64
// rounding); each chunk's sums go to the workspace and colsq_final adds the chunks in a fixed
// order and rounds once to fp32. No atomics: the result does not depend on scheduling.
constexpr int CSQ_COLS = 4096;        // 256 threads x 2 x 8 columns
constexpr int CSQ_TARGET_WGS = 512;   // two resident workgroups per CU

__device__ __forceinline__ void csq_load8(const uint16_t* p, int64_t n, float (&x)[8]) {
  if (n >= 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = e < n ? __uint_as_float(uint32_t(p[e]) << 16) : 0.f;
  }
}
__device__ __forceinline__ void csq_load8(const float* p, int64_t n, float (&x)[8]) {
  if (n >= 8) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x, x[1] = a.y, x[2] = a.z, x[3] = a.w, x[4] = b.x, x[5] = b.y, x[6] = b.z, x[7] = b.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = e < n ? p[e] : 0.f;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void colsq_partial(const T* __restrict__ A, int64_t n_rows,
                                                     int64_t d, int64_t lda, int64_t chunk_rows,
                                                     double* __restrict__ part) {
  // thread t owns columns c_lo + 0..7 and c_lo + 2048 + 0..7, so that each load instruction of
  // a wave reads 1 KB (bf16) without gaps
  const int64_t c_lo = int64_t(blockIdx.x) * CSQ_COLS + int64_t(threadIdx.x) * 8;
  const int64_t c_hi = c_lo + CSQ_COLS / 2;
  const int64_t r0 = int64_t(blockIdx.y) * chunk_rows;
  const int64_t r1 = min(n_rows, r0 + chunk_rows);
  if (c_lo >= d) return;
  const int64_t n_lo = d - c_lo, n_hi = d - c_hi;  // n_hi <= 0: no high half
  double acc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.0;
  constexpr int U = sizeof(T) == 2 ? 8 : 4;  // rows in flight per thread
  int64_t r = r0;
  // whole column blocks, or a block whose first half is whole and second half empty (tests
  // uniform over the workgroup): every load is a full 16-byte load, with no per-lane branch
  // between the loads and their use, so all U rows are in flight at once
  const int64_t b0 = int64_t(blockIdx.x) * CSQ_COLS;
  if (b0 + CSQ_COLS <= d) {
    for (; r + U <= r1; r += U) {
      float x[U][16];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float lo[8], hi[8];
        csq_load8(A + (r + u) * lda + c_lo, 8, lo);
        csq_load8(A + (r + u) * lda + c_hi, 8, hi);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[u][e] = lo[e], x[u][8 + e] = hi[e];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = fma(double(x[u][e]), double(x[u][e]), acc[e]);
    }
  } else if (b0 + CSQ_COLS / 2 == d) {
    for (; r + U <= r1; r += U) {
      float x[U][8];
#pragma unroll
      for (int u = 0; u < U; ++u) csq_load8(A + (r + u) * lda + c_lo, 8, x[u]);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fma(double(x[u][e]), double(x[u][e]), acc[e]);
    }
  }
  for (; r < r1; ++r) {
    float lo[8], hi[8];
    csq_load8(A + r * lda + c_lo, n_lo, lo);
    csq_load8(A + r * lda + c_hi, n_hi, hi);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[e] = fma(double(lo[e]), double(lo[e]), acc[e]);
      acc[8 + e] = fma(double(hi[e]), double(hi[e]), acc[8 + e]);
    }
  }
  double* out = part + int64_t(blockIdx.y) * d;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (e < n_lo) out[c_lo + e] = acc[e];
    if (e < n_hi) out[c_hi + e] = acc[8 + e];
  }
}

// hdiag[j] = sum of the chunks' partials of column j: a workgroup takes 64 columns, thread
// (g, c) adds the chunks g, g + 4, g + 8, ... of column c in order (eight loads in flight),
// and the four groups are added in order through LDS
__global__ __launch_bounds__(256) void colsq_final(const double* __restrict__ part, int n_chunks,
                                                   int64_t d, float* __restrict__ out) {
  __shared__ double red[4][64];
  const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int64_t j = int64_t(blockIdx.x) * 64 + c;
  double v = 0.0;
  if (j < d) {
    int k = g;
    for (; k + 28 < n_chunks; k += 32) {
      double t[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) t[q] = part[int64_t(k + 4 * q) * d + j];
#pragma unroll
      for (int q = 0; q < 8; ++q) v += t[q];
    }
    for (; k < n_chunks; k += 4) v += part[int64_t(k) * d + j];
  }
  red[g][c] = v;
  __syncthreads();
  if (g == 0 && j < d) out[j] = float(((red[0][c] + red[1][c]) + red[2][c]) + red[3][c]);
}

// row chunks of the column-square kernel: enough workgroups to fill the chip (or at most
// max_wgs of them, but never fewer than one chunk per column block), at least 64 rows each
int64_t colsq_chunk_rows(int64_t n_rows, int64_t d, int max_wgs = 0) {
  const int64_t col_blocks = cdiv(d, CSQ_COLS);
  const int64_t target = max_wgs > 0 ? std::min(max_wgs, CSQ_TARGET_WGS) : CSQ_TARGET_WGS;
  const int64_t want = std::max<int64_t>(1, target / col_blocks);
  return std::max<int64_t>(64, cdiv(n_rows, want));
}

}  // namespace

size_t cov_diag_ws_bytes(int64_t n_rows, int64_t d) {
  if (n_rows <= 0 || d <= 0) return 256;
  const int64_t chunks = cdiv(n_rows, colsq_chunk_rows(n_rows, d));
  return align256(size_t(chunks) * size_t(d) * sizeof(double));
}

size_t cov_diag_need_bytes(int64_t n_rows, int64_t d, int max_cus) {
  if (n_rows <= 0 || d <= 0) return 0;
  const int64_t rows = colsq_chunk_rows(n_rows, d, max_cus);
  return size_t(cdiv(n_rows, rows)) * size_t(d) * sizeof(double);
}

int cov_diag_scratch(hipStream_t s, void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* ptrs[kMaxDevices] = {};
  int dev = 0;
  if (s)
    KQ_HIP(hipStreamGetDevice(s, &dev));
  else
    KQ_HIP(hipGetDevice(&dev));
  KQ_REQUIRE(dev >= 0 && dev < kMaxDevices, KRONQ_ERR_HIP, "device ordinal %d out of range", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!ptrs[dev]) {  // once per device, with that device current
    int cur = 0;
    KQ_HIP(hipGetDevice(&cur));
    if (cur != dev) KQ_HIP(hipSetDevice(dev));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) {
      set_error("hipGetSymbolAddress of the cov_diag scratch array failed: %s",
                hipGetErrorString(e));
      return KRONQ_ERR_HIP;
    }
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return KRONQ_OK;
}

int cov_diag_launch(const void* A, int dtype, int64_t n_rows, int64_t d, int64_t lda,
                    float* hdiag, int max_cus, void* ws, hipStream_t s) {
  if (n_rows == 0)  // no chunks: the final kernel writes zeros
    return launch("cov_diag_final", colsq_final, dim3(unsigned(cdiv(d, 64))), dim3(256), 0, s,
                  static_cast<const double*>(nullptr), 0, d, hdiag);
  const int64_t rows = colsq_chunk_rows(n_rows, d, max_cus);
  const int64_t chunks = cdiv(n_rows, rows);
  double* part = static_cast<double*>(ws);
  const dim3 grid(unsigned(cdiv(d, CSQ_COLS)), unsigned(chunks));
  if (dtype == KRONQ_BF16)
    KQ_TRY(launch("cov_diag_partial", colsq_partial<uint16_t>, grid, dim3(256), 0, s,
                  static_cast<const uint16_t*>(A), n_rows, d, lda, rows, part));
  else
    KQ_TRY(launch("cov_diag_partial", colsq_partial<float>, grid, dim3(256), 0, s,
                  static_cast<const float*>(A), n_rows, d, lda, rows, part));
  return launch("cov_diag_final", colsq_final, dim3(unsigned(cdiv(d, 64))), dim3(256), 0, s,
                static_cast<const double*>(part), int(chunks), d, hdiag);
}

}  // namespace kq
