// Bidirectional incoherence processing (Sec. 4.2 eqs. rescale and biip; Alg. 1).
//
// The randomised Hadamard transform of a length-d vector is applied as sign flip, fast
// Walsh-Hadamard butterflies (O(d log d) adds) and, when d = 28 * 2^k, a dense 28-point mix of
// the slow index, instead of the dense d x d products the paper's implementation uses. All
// transforms are HBM-bound passes over fp32 matrices:
//   * norms:      one read of W_in -> squared row norms and per-block column partial sums (fp64);
//   * factors:    s = (diag H / norm^2)^(1/4) per side, and the per-index multipliers that the
//                 passes fold in (rescale x random sign);
//   * row pass:   one workgroup per row, the row staged in LDS; multipliers, radix-8/4/2
//                 butterflies in registers between LDS round trips, optional 28-point mix,
//                 1/sqrt(m) and output multipliers, written once;
//   * column pass: transform along the strided (row) axis for a strip of columns: L rows at a
//                 fixed row stride are staged in LDS and transformed there. An order-m transform
//                 is split into passes of length <= 512 (H_m = H_m1 (x) H_m2), plus a 28-point pass.
// Forward: W <- U S_G W S_X V^T; H_X <- V S_X^-1 H_X S_X^-1 V^T; H_G <- U S_G^-1 H_G S_G^-1 U^T.
// Inverse (W only): W <- S_G^-1 U^T W V S_X^-1 (column pass with Q28^T, then the row pass).
#include <cmath>

#include "kq_common.hpp"
#include "kq_fwht.hpp"

namespace kq {
namespace {

constexpr int RP_THREADS = 512;
constexpr int CP_THREADS = 256;
constexpr int CP_MAXL = 1024;
constexpr int NORM_ROWS = 16;

// ----------------------------------------------------------------------------- norms
template <typename T>
__device__ __forceinline__ float ld_as_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float ld_as_f32<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ld_as_f32<uint16_t>(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}

__device__ __forceinline__ void load8_f32(const uint16_t* p, int64_t n, float (&x)[8]) {
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
__device__ __forceinline__ void load8_f32(const float* p, int64_t n, float (&x)[8]) {
  if (n >= 8) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x, x[1] = a.y, x[2] = a.z, x[3] = a.w, x[4] = b.x, x[5] = b.y, x[6] = b.z, x[7] = b.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = e < n ? p[e] : 0.f;
  }
}

// Squared column norms (as per-block partials over NORM_ROWS rows) and squared row norms of W.
// Each thread loads 8 consecutive columns per row with one vector load and keeps the block's
// row sums and its 8 column sums in registers; row sums are reduced with wave shuffles.
// Squares of bf16 / fp32 values summed over at most NORM_ROWS rows (columns) or one row's
// share of a thread (rows) in fp32; the partials are stored and combined in fp64.
template <typename T>
__global__ __launch_bounds__(256) void w_norms(const T* __restrict__ W, int64_t d_out,
                                               int64_t d_in, int64_t ldw,
                                               double* __restrict__ col_part,
                                               double* __restrict__ rowsq) {
  __shared__ float red[4][NORM_ROWS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t r0 = int64_t(blockIdx.x) * NORM_ROWS;
  const int nr = int(min(int64_t(NORM_ROWS), d_out - r0));
  float rs[NORM_ROWS];
#pragma unroll
  for (int r = 0; r < NORM_ROWS; ++r) rs[r] = 0.f;
  // a block of NORM_ROWS whole rows of whole 8-column runs (tests uniform over the
  // workgroup) loads without bounds branches, all NORM_ROWS loads of a thread in flight
  // together; the sums are taken in the same order either way
  const bool whole = (d_in & 7) == 0 && nr == NORM_ROWS;
  for (int64_t c0 = int64_t(tid) * 8; c0 < d_in; c0 += 256 * 8) {
    float cs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (whole) {
      float x[NORM_ROWS][8];
#pragma unroll
      for (int r = 0; r < NORM_ROWS; ++r) load8_f32(W + (r0 + r) * ldw + c0, 8, x[r]);
#pragma unroll
      for (int r = 0; r < NORM_ROWS; ++r) {
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          cs[e] = fmaf(x[r][e], x[r][e], cs[e]);
          t = fmaf(x[r][e], x[r][e], t);
        }
        rs[r] += t;
      }
    } else {
#pragma unroll
      for (int r = 0; r < NORM_ROWS; ++r) {
        if (r < nr) {
          float x[8];
          load8_f32(W + (r0 + r) * ldw + c0, d_in - c0, x);
          float t = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            cs[e] = fmaf(x[e], x[e], cs[e]);
            t = fmaf(x[e], x[e], t);
          }
          rs[r] += t;
        }
      }
    }
    double* cp = col_part + int64_t(blockIdx.x) * d_in + c0;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (c0 + e < d_in) cp[e] = cs[e];
  }
#pragma unroll
  for (int r = 0; r < NORM_ROWS; ++r) {
    float v = rs[r];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if (lane == 0) red[wave][r] = v;
  }
  __syncthreads();
  if (tid < nr)
    rowsq[r0 + tid] = double(red[0][tid]) + double(red[1][tid]) + double(red[2][tid]) +
                      double(red[3][tid]);
}

// s = (h / a)^(1/4), 1 when either is zero (or the side is off). Also the multipliers used by
// the passes: mul_w = s * sign, mul_h = sign / s (sign = 1 when the side does not rotate).
__global__ void side_factors(int64_t n, const float* __restrict__ H, int64_t ldh,
                             const double* __restrict__ part, int64_t n_part,
                             const double* __restrict__ direct, const int8_t* __restrict__ sign,
                             int rescale, float* __restrict__ s_out, float* __restrict__ mul_w,
                             float* __restrict__ mul_h) {
  const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= n) return;
  float s = 1.f;
  if (rescale) {
    double a;
    if (direct) {
      a = direct[j];
    } else {
      // partials added in order; loaded eight at a time so that the loads overlap
      a = 0.0;
      int64_t p = 0;
      for (; p + 8 <= n_part; p += 8) {
        double t[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) t[q] = part[(p + q) * n + j];
#pragma unroll
        for (int q = 0; q < 8; ++q) a += t[q];
      }
      for (; p < n_part; ++p) a += part[p * n + j];
    }
    const double h = H[j * ldh + j];
    if (a > 0.0 && h > 0.0) s = float(sqrt(sqrt(h / a)));
  }
  const float sg = sign ? float(sign[j]) : 1.f;
  s_out[j] = s;
  mul_w[j] = s * sg;
  mul_h[j] = sg / s;
}

// multipliers from a given s: s * sign
__global__ void given_factors(int64_t n, const float* __restrict__ s, const int8_t* __restrict__ sign,
                              float* __restrict__ mul) {
  const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= n) return;
  mul[j] = s[j] * (sign ? float(sign[j]) : 1.f);
}

// inverse multipliers: sign / s (s == nullptr: 1)
__global__ void inv_factors(int64_t n, const float* __restrict__ s, const int8_t* __restrict__ sign,
                            float* __restrict__ mul) {
  const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= n) return;
  mul[j] = (sign ? float(sign[j]) : 1.f) / (s ? s[j] : 1.f);
}

// ----------------------------------------------------------------------------- row pass
// dst[r][c] = post_row[r] * post_col[c] * T(x)[c] with x[c] = pre_row[r] * pre_col[c] * src[r][c]
// and T = (Q (x) H_m) / sqrt(m) (Q = 28 x 28 or identity), or the identity when transform == 0.
template <typename T>
__global__ __launch_bounds__(RP_THREADS) void row_pass(
    const T* __restrict__ src, int64_t lds_, float* __restrict__ dst, int64_t ldd, int64_t rows,
    int64_t n, const float* __restrict__ pre_row, const float* __restrict__ pre_col,
    const float* __restrict__ post_row, const float* __restrict__ post_col, int transform,
    int64_t m, const float* __restrict__ q28, int q_trans, float norm) {
  extern __shared__ float smem[];
  float* buf = smem;       // n floats
  float* qs = smem + n;    // 28 x 28
  const int tid = threadIdx.x;
  if (transform && q28) {
    for (int i = tid; i < 28 * 28; i += RP_THREADS) {
      const int a = i / 28, b = i % 28;
      qs[i] = q_trans ? q28[b * 28 + a] : q28[i];
    }
  }
  for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
    const float pr = pre_row ? pre_row[r] : 1.f;
    const float po = (post_row ? post_row[r] : 1.f) * norm;
    const T* s = src + r * lds_;
    float* o = dst + r * ldd;
    if (!transform) {
      for (int64_t c = tid; c < n; c += RP_THREADS) {
        float x = ld_as_f32(s, c) * pr;
        if (pre_col) x *= pre_col[c];
        if (post_col) x *= post_col[c];
        o[c] = x * po;
      }
      continue;
    }
    __syncthreads();  // previous row finished with buf
    if (m >= 512) {
      // whole 512-element chunks (m is a power of two >= 512, n = L m): a wave takes a chunk,
      // 8 consecutive elements per lane, straight from global memory; the stages of strides
      // 1, 2, 4 run in registers and those of strides 8 ... 256 across lanes (lane xor 1 ...
      // 32), so the chunk reaches LDS with its first 9 stages done; the stages of strides
      // >= 512 follow in LDS
      const int wave = tid >> 6, lane = tid & 63;
      for (int64_t c0 = int64_t(wave) * 512 + lane * 8; c0 < n; c0 += int64_t(RP_THREADS) * 8) {
        float x[8];
        load8_f32(s + c0, 8, x);
        if (pre_col) {
          const float4 p0 = *reinterpret_cast<const float4*>(pre_col + c0);
          const float4 p1 = *reinterpret_cast<const float4*>(pre_col + c0 + 4);
          x[0] *= pr * p0.x, x[1] *= pr * p0.y, x[2] *= pr * p0.z, x[3] *= pr * p0.w;
          x[4] *= pr * p1.x, x[5] *= pr * p1.y, x[6] *= pr * p1.z, x[7] *= pr * p1.w;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] *= pr;
        }
        hadamard_reg<8>(x);
#pragma unroll
        for (int j = 0; j < 6; ++j) {
          const bool upper = (lane >> j) & 1;  // holds the second element of each pair
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float y = __shfl_xor(x[e], 1 << j);
            x[e] = upper ? y - x[e] : x[e] + y;
          }
        }
        *reinterpret_cast<float4*>(buf + c0) = make_float4(x[0], x[1], x[2], x[3]);
        *reinterpret_cast<float4*>(buf + c0 + 4) = make_float4(x[4], x[5], x[6], x[7]);
      }
      __syncthreads();
      fwht_lds(buf, n, m, tid, RP_THREADS, 9);
    } else if ((n & 7) == 0) {  // 16-byte rows (checked by the API): 8 values per vector load
      for (int64_t c0 = int64_t(tid) * 8; c0 < n; c0 += int64_t(RP_THREADS) * 8) {
        float x[8];
        load8_f32(s + c0, 8, x);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] *= pre_col ? pr * pre_col[c0 + e] : pr;
        *reinterpret_cast<float4*>(buf + c0) = make_float4(x[0], x[1], x[2], x[3]);
        *reinterpret_cast<float4*>(buf + c0 + 4) = make_float4(x[4], x[5], x[6], x[7]);
      }
    } else {
      for (int64_t c = tid; c < n; c += RP_THREADS) {
        float x = ld_as_f32(s, c) * pr;
        if (pre_col) x *= pre_col[c];
        buf[c] = x;
      }
    }
    if (m < 512) {
      __syncthreads();
      fwht_lds(buf, n, m, tid, RP_THREADS);
    }
    if (q28) {
      // output a * m + b = sum_k Q[a][k] buf[k * m + b]: one b per thread, its 28 inputs held in
      // registers, the rows of Q read as 16-byte broadcasts
      for (int64_t b = tid; b < m; b += RP_THREADS) {
        float x[28];
#pragma unroll
        for (int k = 0; k < 28; ++k) x[k] = buf[k * m + b];
        for (int a = 0; a < 28; ++a) {
          const float4* qa = reinterpret_cast<const float4*>(qs + a * 28);
          float acc = 0.f;
#pragma unroll
          for (int k4 = 0; k4 < 7; ++k4) {
            const float4 q = qa[k4];
            acc = fmaf(q.x, x[4 * k4], acc);
            acc = fmaf(q.y, x[4 * k4 + 1], acc);
            acc = fmaf(q.z, x[4 * k4 + 2], acc);
            acc = fmaf(q.w, x[4 * k4 + 3], acc);
          }
          const int64_t c = a * m + b;
          float y = acc * po;
          if (post_col) y *= post_col[c];
          o[c] = y;
        }
      }
    } else if ((n & 3) == 0) {
      for (int64_t c = int64_t(tid) * 4; c < n; c += int64_t(RP_THREADS) * 4) {
        float4 y = *reinterpret_cast<const float4*>(buf + c);
        const float4 pc = post_col ? *reinterpret_cast<const float4*>(post_col + c)
                                   : make_float4(1.f, 1.f, 1.f, 1.f);
        y.x *= po * pc.x, y.y *= po * pc.y, y.z *= po * pc.z, y.w *= po * pc.w;
        *reinterpret_cast<float4*>(o + c) = y;
      }
    } else {
      for (int64_t c = tid; c < n; c += RP_THREADS) {
        float y = buf[c] * po;
        if (post_col) y *= post_col[c];
        o[c] = y;
      }
    }
  }
}

// ----------------------------------------------------------------------------- column pass
// Transform along the row axis. Rows are indexed r = hi * (L * n_lo) + a * n_lo + lo; for each
// (hi, lo) and a strip of CW columns the L rows a = 0..L-1 are transformed:
//   kind 0: H_L / sqrt(L) (FWHT);  kind 1: the 28-point factor Q (or Q^T), L = 28.
template <int NT>
__global__ __launch_bounds__(NT) void col_pass(const float* __restrict__ src, int64_t lds_,
                                                       float* __restrict__ dst, int64_t ldd,
                                                       int64_t cols, int64_t L, int64_t n_lo,
                                                       int64_t n_groups, int CW, int kind,
                                                       const float* __restrict__ q28,
                                                       int q_trans, float norm) {
  extern __shared__ float smem[];
  const int CWP = CW + 4;
  float* tile = smem;                // L x CWP
  float* qs = smem + L * CWP;        // 28 x 28
  const int tid = threadIdx.x;
  const int64_t strips = cdiv(cols, CW);
  const int64_t g = blockIdx.x / strips;
  const int64_t c0 = (blockIdx.x % strips) * CW;
  if (g >= n_groups) return;
  const int64_t hi = g / n_lo, lo = g % n_lo;
  const int64_t row0 = hi * L * n_lo + lo;  // row of a = 0
  if (kind == 1) {
    for (int i = tid; i < 28 * 28; i += NT) {
      const int a = i / 28, b = i % 28;
      qs[i] = q_trans ? q28[b * 28 + a] : q28[i];
    }
  }
  const int cw4 = CW / 4;
  int lcw4 = 0;  // CW is a power of 2 (32, 64 or 256): shifts instead of divisions
  while ((1 << lcw4) < cw4) ++lcw4;
  // load the L x CW tile: 8 independent float4 loads in flight per thread before they are
  // stored (one workgroup per CU at L = 1024, so latency must be hidden within the thread)
  const int n_items = int(L) * cw4;
  for (int it0 = tid; it0 < n_items; it0 += 8 * NT) {
    float4 x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int it = it0 + u * NT;
      x[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (it < n_items) {
        const int64_t a = it >> lcw4;
        const int c = (it & (cw4 - 1)) * 4;
        const int64_t gr = row0 + a * n_lo;
        const int64_t gc = c0 + c;
        const float* p = src + gr * lds_;
        if (gc + 4 <= cols) {
          x[u] = *reinterpret_cast<const float4*>(p + gc);
        } else {
          x[u].x = gc + 0 < cols ? p[gc + 0] : 0.f;
          x[u].y = gc + 1 < cols ? p[gc + 1] : 0.f;
          x[u].z = gc + 2 < cols ? p[gc + 2] : 0.f;
          x[u].w = gc + 3 < cols ? p[gc + 3] : 0.f;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int it = it0 + u * NT;
      if (it < n_items)
        *reinterpret_cast<float4*>(tile + (it >> lcw4) * CWP + (it & (cw4 - 1)) * 4) = x[u];
    }
  }
  __syncthreads();
  if (kind == 0) {
    // butterflies along a, items (group q, column c)
    const int lcw = lcw4 + 2;
    int lgh = 0;
    while ((int64_t(1) << lgh) < L) {
      const int64_t left = L >> lgh;
      const int R = left >= 8 ? 8 : (left == 4 ? 4 : 2);
      const int h = 1 << lgh;
      const int items = int(L / R) * CW;
      for (int it = tid; it < items; it += NT) {
        const int q = it >> lcw;
        const int c = it & (CW - 1);
        const int base = (q >> lgh) * (R << lgh) + (q & (h - 1));
        float x[8];
        if (R == 8) {
#pragma unroll
          for (int k = 0; k < 8; ++k) x[k] = tile[(base + k * h) * CWP + c];
          hadamard_reg<8>(x);
#pragma unroll
          for (int k = 0; k < 8; ++k) tile[(base + k * h) * CWP + c] = x[k];
        } else if (R == 4) {
#pragma unroll
          for (int k = 0; k < 4; ++k) x[k] = tile[(base + k * h) * CWP + c];
          hadamard_reg<4>(x);
#pragma unroll
          for (int k = 0; k < 4; ++k) tile[(base + k * h) * CWP + c] = x[k];
        } else {
          x[0] = tile[base * CWP + c];
          x[1] = tile[(base + h) * CWP + c];
          tile[base * CWP + c] = x[0] + x[1];
          tile[(base + h) * CWP + c] = x[0] - x[1];
        }
      }
      lgh += R == 8 ? 3 : (R == 4 ? 2 : 1);
      __syncthreads();
    }
    for (int it = tid; it < n_items; it += NT) {
      const int64_t a = it >> lcw4;
      const int c = (it & (cw4 - 1)) * 4;
      const int64_t gr = row0 + a * n_lo;
      const int64_t gc = c0 + c;
      float4 x = *reinterpret_cast<const float4*>(tile + a * CWP + c);
      x.x *= norm;
      x.y *= norm;
      x.z *= norm;
      x.w *= norm;
      if (gc + 4 <= cols) {
        *reinterpret_cast<float4*>(dst + gr * ldd + gc) = x;
      } else {
        float* p = dst + gr * ldd;
        if (gc + 0 < cols) p[gc + 0] = x.x;
        if (gc + 1 < cols) p[gc + 1] = x.y;
        if (gc + 2 < cols) p[gc + 2] = x.z;
      }
    }
  } else {
    // 28-point mix: out[a][c] = sum_k Q[a][k] tile[k][c]; one column per thread, its 28 inputs
    // in registers, the rows of Q read as 16-byte broadcasts
    for (int c = tid; c < CW; c += NT) {
      const int64_t gc = c0 + c;
      float x[28];
#pragma unroll
      for (int k = 0; k < 28; ++k) x[k] = tile[k * CWP + c];
      for (int a = 0; a < 28; ++a) {
        const float4* qa = reinterpret_cast<const float4*>(qs + a * 28);
        float acc = 0.f;
#pragma unroll
        for (int k4 = 0; k4 < 7; ++k4) {
          const float4 q = qa[k4];
          acc = fmaf(q.x, x[4 * k4], acc);
          acc = fmaf(q.y, x[4 * k4 + 1], acc);
          acc = fmaf(q.z, x[4 * k4 + 2], acc);
          acc = fmaf(q.w, x[4 * k4 + 3], acc);
        }
        if (gc < cols) dst[(row0 + a * n_lo) * ldd + gc] = acc * norm;
      }
    }
  }
}

// ----------------------------------------------------------------------------- host helpers
int launch_row_pass(const void* src, int dtype, int64_t lds_, float* dst, int64_t ldd,
                    int64_t rows, int64_t n, const float* pre_row, const float* pre_col,
                    const float* post_row, const float* post_col, bool transform,
                    const RotDim& rd, const float* q28, bool q_trans, hipStream_t s,
                    const char* name) {
  const size_t shmem = transform ? (size_t(n) + 28 * 28) * sizeof(float) : 0;
  const unsigned grid = unsigned(rows < 4096 ? rows : 4096);
  const float norm = transform ? float(1.0 / std::sqrt(double(rd.m))) : 1.f;
  const float* q = (transform && rd.has28) ? q28 : nullptr;
  if (dtype == KRONQ_BF16)
    return launch(name, row_pass<uint16_t>, dim3(grid), dim3(RP_THREADS), shmem, s,
                  static_cast<const uint16_t*>(src), lds_, dst, ldd, rows, n, pre_row, pre_col,
                  post_row, post_col, int(transform), rd.m, q, int(q_trans), norm);
  return launch(name, row_pass<float>, dim3(grid), dim3(RP_THREADS), shmem, s,
                static_cast<const float*>(src), lds_, dst, ldd, rows, n, pre_row, pre_col,
                post_row, post_col, int(transform), rd.m, q, int(q_trans), norm);
}

int launch_col_step(const float* src, int64_t lds_, float* dst, int64_t ldd, int64_t rows,
                    int64_t cols, int64_t L, int64_t n_lo, int kind, const float* q28,
                    bool q_trans, hipStream_t s) {
  // strips of CW columns: 28-point mix 256 (one column per thread), FWHT 64 up to L = 256
  // and 32 beyond (L = 1024: 1024 x 36 floats + the 28 x 28 factor = 150 KB of LDS, one
  // workgroup per CU, so beyond L = 256 the workgroup has 1024 threads to keep enough loads in
  // flight)
  const int CW = kind == 1 ? 256 : (L <= 256 ? 64 : 32);
  const int64_t n_groups = rows / L;
  const int64_t strips = cdiv(cols, CW);
  const size_t shmem = (size_t(L) * (CW + 4) + 28 * 28) * sizeof(float);
  const float norm = kind == 0 ? float(1.0 / std::sqrt(double(L))) : 1.f;
  const char* name = kind == 0 ? "fwht_col" : "mix28_col";
  const dim3 grid(unsigned(n_groups * strips));
  if (kind == 0 && L > 256)
    return launch(name, col_pass<1024>, grid, dim3(1024), shmem, s, src, lds_, dst, ldd, cols, L,
                  n_lo, n_groups, CW, kind, q28, int(q_trans), norm);
  return launch(name, col_pass<CP_THREADS>, grid, dim3(CP_THREADS), shmem, s, src, lds_, dst, ldd,
                cols, L, n_lo, n_groups, CW, kind, q28, int(q_trans), norm);
}

// Full transform of every column (rows axis, length d): T = (Q (x) H_m) / sqrt(m).
int col_transform(const float* src, int64_t lds_, float* dst, int64_t ldd, int64_t d,
                  int64_t cols, const RotDim& rd, const float* q28, bool q_trans, hipStream_t s) {
  // Hadamard factors, fast index first: m = m1 * m2 * ..., each <= CP_MAXL, in as few passes
  // as possible and as even as possible (1024: one pass; 4096: 64 x 64; 8192: 128 x 64)
  int64_t n_lo = 1;
  int64_t left = rd.m;
  const float* cur = src;
  int64_t ldc = lds_;
  int lg = 0;
  while ((int64_t(1) << lg) < left) ++lg;
  int lgmax = 0;
  while ((int64_t(1) << (lgmax + 1)) <= CP_MAXL) ++lgmax;
  int passes = (lg + lgmax - 1) / (lgmax > 0 ? lgmax : 1);
  while (left > 1) {
    const int lgl = (lg + passes - 1) / passes;  // ceil: earlier passes take the larger share
    const int64_t L = int64_t(1) << lgl;
    lg -= lgl;
    --passes;
    KQ_TRY(launch_col_step(cur, ldc, dst, ldd, d, cols, L, n_lo, 0, nullptr, false, s));
    cur = dst;
    ldc = ldd;
    n_lo *= L;
    left /= L;
  }
  if (rd.has28) {
    KQ_TRY(launch_col_step(cur, ldc, dst, ldd, d, cols, 28, rd.m, 1, q28, q_trans, s));
  }
  return KRONQ_OK;
}

}  // namespace

// rows of src (B vectors of length n) -> diag(post_col) T diag(pre_col) x, with T the randomised
// Hadamard factor of order n (its transpose with q_trans) or the identity
int rotate_vectors(const void* src, int dtype, int64_t lds_, float* dst, int64_t ldd, int64_t rows,
                   int64_t n, const float* pre_col, const float* post_col, bool transform,
                   const float* q28, bool q_trans, hipStream_t s) {
  return launch_row_pass(src, dtype, lds_, dst, ldd, rows, n, nullptr, pre_col, nullptr, post_col,
                         transform, rot_dim(n), q28, q_trans, s, "online_rot_pass");
}

// mul = sign / s (sign == nullptr: 1)
int inverse_multipliers(const float* sv, const int8_t* sign, int64_t n, float* mul,
                        hipStream_t s) {
  return launch("online_factors", inv_factors, dim3(unsigned(cdiv(n, 256))), dim3(256), 0, s, n,
                sv, sign, mul);
}

size_t rotate_drift_ws_bytes(int64_t d) {
  if (d <= 0) return 0;
  return align256(size_t(d) * sizeof(float)) + 256;
}

// D <- V diag(1/sx) D diag(1/sx) V^T: the input-side transform of H_X applied to the (not
// symmetric) drift statistic, a row pass and a column pass like H_X's
int rotate_drift_launch(float* D, int64_t d, int64_t ldd, const float* sx, const int8_t* sign,
                        const float* q28, int flags, void* ws, hipStream_t s) {
  const bool rot = flags & KRONQ_ROT_IN;
  const RotDim r = rot_dim(d);
  Carver cv(ws);
  float* mh = cv.take<float>(d);
  KQ_TRY(launch("rot_inv_factors", inv_factors, dim3(unsigned(cdiv(d, 256))), dim3(256), 0, s, d,
                (flags & KRONQ_RESCALE_IN) ? sx : static_cast<const float*>(nullptr),
                rot ? sign : static_cast<const int8_t*>(nullptr), mh));
  KQ_TRY(launch_row_pass(D, KRONQ_FP32, ldd, D, ldd, d, d, mh, mh, nullptr, nullptr, rot, r, q28,
                         false, s, "rot_row_pass"));
  if (rot) KQ_TRY(col_transform(D, ldd, D, ldd, d, d, r, q28, false, s));
  return KRONQ_OK;
}

size_t rotate_ws_bytes(int64_t d_out, int64_t d_in) {
  if (d_out <= 0 || d_in <= 0) return 0;
  const int64_t nb = cdiv(d_out, NORM_ROWS);
  size_t b = 0;
  b += align256(size_t(nb) * d_in * sizeof(double));          // column partials
  b += align256(size_t(d_out) * sizeof(double));               // row sums
  b += 2 * align256(size_t(d_in) * sizeof(float));             // mul_w_in, mul_h_in
  b += 2 * align256(size_t(d_out) * sizeof(float));            // mul_w_out, mul_h_out
  return b + 256;
}

int rotate_launch(const void* W_in, int w_dtype, int64_t ldw_in, float* W, int64_t d_out,
                  int64_t d_in, int64_t ldw, float* HX, int64_t ldx, float* HG, int64_t ldg,
                  const int8_t* sign_in, const int8_t* sign_out, const float* q28_in,
                  const float* q28_out, float* sx, float* sg, int flags, void* ws,
                  hipStream_t s) {
  const bool rot_in = flags & KRONQ_ROT_IN, rot_out = flags & KRONQ_ROT_OUT;
  const RotDim ri = rot_dim(d_in), ro = rot_dim(d_out);
  Carver cv(ws);
  const int64_t nb = cdiv(d_out, NORM_ROWS);
  double* colp = cv.take<double>(size_t(nb) * d_in);
  double* rows = cv.take<double>(d_out);
  float* mw_in = cv.take<float>(d_in);
  float* mh_in = cv.take<float>(d_in);
  float* mw_out = cv.take<float>(d_out);
  float* mh_out = cv.take<float>(d_out);

  if (flags & KRONQ_INVERSE) {
    // W <- diag(sign_out / sg) (Q^T (x) H) W_in (...)  V-side: rows of the result get
    // diag(sign_in / sx) after the transposed row transform.
    KQ_TRY(launch("rot_inv_factors", inv_factors, dim3(unsigned(cdiv(d_in, 256))), dim3(256), 0,
                  s, d_in, static_cast<const float*>(sx), rot_in ? sign_in : nullptr, mw_in));
    KQ_TRY(launch("rot_inv_factors", inv_factors, dim3(unsigned(cdiv(d_out, 256))), dim3(256), 0,
                  s, d_out, static_cast<const float*>(sg), rot_out ? sign_out : nullptr, mw_out));
    const float* src = static_cast<const float*>(W_in);
    int64_t lsrc = ldw_in;
    if (rot_out) {
      KQ_TRY(col_transform(src, lsrc, W, ldw, d_out, d_in, ro, q28_out, true, s));
      src = W;
      lsrc = ldw;
    }
    return launch_row_pass(src, KRONQ_FP32, lsrc, W, ldw, d_out, d_in, nullptr, nullptr, mw_out,
                           mw_in, rot_in, ri, q28_in, true, s, "rot_row_pass");
  }

  // ---- forward (optionally split into the H_X half and the W / H_G half)
  const bool hx_only = flags & KRONQ_HX_ONLY, sx_given = flags & KRONQ_SX_GIVEN;
  const bool hg_diag = flags & KRONQ_HG_DIAG, sg_given = flags & KRONQ_SG_GIVEN;
  const bool do_w = !hx_only && !sg_given;  // W is transformed
  const bool need_norms = ((flags & KRONQ_RESCALE_IN) && !sx_given) ||
                          ((flags & KRONQ_RESCALE_OUT) && do_w);
  if (need_norms) {
    if (w_dtype == KRONQ_BF16)
      KQ_TRY(launch("rot_w_norms", w_norms<uint16_t>, dim3(unsigned(nb)), dim3(256), 0, s,
                    static_cast<const uint16_t*>(W_in), d_out, d_in, ldw_in, colp, rows));
    else
      KQ_TRY(launch("rot_w_norms", w_norms<float>, dim3(unsigned(nb)), dim3(256), 0, s,
                    static_cast<const float*>(W_in), d_out, d_in, ldw_in, colp, rows));
  }
  if (!sx_given)
    KQ_TRY(launch("rot_factors", side_factors, dim3(unsigned(cdiv(d_in, 256))), dim3(256), 0, s,
                  d_in, static_cast<const float*>(HX), ldx, static_cast<const double*>(colp), nb,
                  static_cast<const double*>(nullptr), rot_in ? sign_in : nullptr,
                  int((flags & KRONQ_RESCALE_IN) != 0), sx, mw_in, mh_in));
  else if (do_w)
    KQ_TRY(launch("rot_factors", given_factors, dim3(unsigned(cdiv(d_in, 256))), dim3(256), 0, s,
                  d_in, static_cast<const float*>(sx), rot_in ? sign_in : nullptr, mw_in));
  if (do_w) {
    // with KRONQ_HG_DIAG, HG is the diagonal itself: a zero stride reads H[j] as H[j][j]
    KQ_TRY(launch("rot_factors", side_factors, dim3(unsigned(cdiv(d_out, 256))), dim3(256), 0, s,
                  d_out, static_cast<const float*>(HG), hg_diag ? int64_t(0) : ldg,
                  static_cast<const double*>(nullptr), int64_t(0),
                  static_cast<const double*>(rows), rot_out ? sign_out : nullptr,
                  int((flags & KRONQ_RESCALE_OUT) != 0), sg, mw_out, mh_out));
    // W: rescale + signs + V side (row pass), then U side (column pass)
    KQ_TRY(launch_row_pass(W_in, w_dtype, ldw_in, W, ldw, d_out, d_in, mw_out, mw_in, nullptr,
                           nullptr, rot_in, ri, q28_in, false, s, "rot_row_pass"));
    if (rot_out) KQ_TRY(col_transform(W, ldw, W, ldw, d_out, d_in, ro, q28_out, false, s));
  }
  // H_X <- V S^-1 H_X S^-1 V^T
  if (!sx_given) {
    KQ_TRY(launch_row_pass(HX, KRONQ_FP32, ldx, HX, ldx, d_in, d_in, mh_in, mh_in, nullptr,
                           nullptr, rot_in, ri, q28_in, false, s, "rot_row_pass"));
    if (rot_in) KQ_TRY(col_transform(HX, ldx, HX, ldx, d_in, d_in, ri, q28_in, false, s));
  }
  // H_G <- U S^-1 H_G S^-1 U^T (with a given sg, the multipliers sign / s as side_factors
  // forms them)
  if (sg_given)
    KQ_TRY(launch("rot_factors", inv_factors, dim3(unsigned(cdiv(d_out, 256))), dim3(256), 0, s,
                  d_out, static_cast<const float*>(sg), rot_out ? sign_out : nullptr, mh_out));
  if (HG && !hx_only && !hg_diag) {
    KQ_TRY(launch_row_pass(HG, KRONQ_FP32, ldg, HG, ldg, d_out, d_out, mh_out, mh_out, nullptr,
                           nullptr, rot_out, ro, q28_out, false, s, "rot_row_pass"));
    if (rot_out) KQ_TRY(col_transform(HG, ldg, HG, ldg, d_out, d_out, ro, q28_out, false, s));
  }
  return KRONQ_OK;
}

}  // namespace kq
