// Inference with a quantised layer: the rotations are applied online, O(d log d) per layer
// (Sec. 3.2 and 4.2; Limitations), around a matvec on the packed low-bit codes, so that
// y = S_G^-1 U^T W_hat' V S_X^-1 x (the original-space layer of Alg. 2's last line) is never
// formed as a dense matrix. For B <= 4 activation vectors:
//   1. x' = V S_X^-1 x and 3. y = S_G^-1 U^T y' by seg_transform: a transform of order
//      d = L m (m = 2^k <= 1024) is A (x) H_m with A = Q28 (or Q28^T) when d = 28 m and A = H_L
//      otherwise (Sylvester: H_d = H_L (x) H_m). Segment a of the output is H_m applied to
//      sum_k A[a][k] x_k over the L input segments, so workgroup (a, vector) mixes the segments,
//      runs one FWHT of m points in LDS and applies the multipliers: L workgroups per vector
//      instead of one.
//   2. y' = W_hat' x': the packed-code GEMV, bound by the HBM reads of the codes.
// Packed format: each run of 32 consecutive codes of a row is one 32 * bits-bit little-endian
// string held in `bits` uint32 words.
// GEMV: a workgroup takes 4 * RPW rows, RPW per wave, and stages x' (B x d_in fp32, B <= 4 per
// launch) in LDS. Lane l
// takes steps of 32 * UPL columns (UPL = 2 at 2 bits, so every code load is 16 bytes) at a
// stride of 64 steps. A decode matvec moves little data per CU, so latency is the limit: a lane
// requests the codes of up to MAXU steps of its RPW rows at once, before x' is staged, and only
// then computes. For each step and row it adds s * (sum_j q_j x'_j - z * sum_j x'_j) with the
// row's group scale s and zero z (a group is a multiple of 128 columns, so a step lies in one
// group). Wave sums at the end.
#include <cmath>

#include "kq_common.hpp"

namespace kq {
namespace {

__device__ __forceinline__ float ld_f32(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_f32(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}

template <int BITS>
__device__ __forceinline__ void load_unit(const uint32_t* __restrict__ p, uint32_t (&w)[BITS]) {
  if constexpr (BITS == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    w[0] = v.x, w[1] = v.y;
  } else if constexpr (BITS == 4) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w;
  } else if constexpr (BITS == 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint4 u = *reinterpret_cast<const uint4*>(p + 4);
    w[0] = v.x, w[1] = v.y, w[2] = v.z, w[3] = v.w, w[4] = u.x, w[5] = u.y, w[6] = u.z,
    w[7] = u.w;
  } else {
#pragma unroll
    for (int k = 0; k < BITS; ++k) w[k] = p[k];
  }
}

// code j (compile-time after unrolling) of a unit
template <int BITS>
__device__ __forceinline__ uint32_t code_at(const uint32_t (&w)[BITS], int j) {
  constexpr uint32_t mask = (1u << BITS) - 1u;
  const int pos = j * BITS, wi = pos >> 5, off = pos & 31;
  if (off + BITS <= 32) return (w[wi] >> off) & mask;
  return ((w[wi] >> off) | (w[wi + 1] << (32 - off))) & mask;
}

// one thread per (row, unit of 32 codes)
template <int BITS>
__global__ __launch_bounds__(256) void pack_codes(const uint8_t* __restrict__ codes,
                                                  int64_t d_out, int64_t units, int64_t ldq,
                                                  uint32_t* __restrict__ packed, int64_t ldp) {
  const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (t >= d_out * units) return;
  const int64_t row = t / units, u = t % units;
  const uint8_t* c = codes + row * ldq + u * 32;
  uint32_t w[BITS];
#pragma unroll
  for (int k = 0; k < BITS; ++k) w[k] = 0u;
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const uint32_t q = uint32_t(c[j]) & ((1u << BITS) - 1u);
    const int pos = j * BITS, wi = pos >> 5, off = pos & 31;
    w[wi] |= q << off;
    if (off + BITS > 32) w[wi + 1] |= q >> (32 - off);
  }
  uint32_t* o = packed + row * ldp + u * BITS;
#pragma unroll
  for (int k = 0; k < BITS; ++k) o[k] = w[k];
}

template <int BITS, int NB, int RPW, int MAXU>
__global__ __launch_bounds__(256) void online_gemv(
    const uint32_t* __restrict__ packed, int64_t ldp, const float* __restrict__ scales,
    const float* __restrict__ zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
    const float* __restrict__ xr, int64_t ldxr, float* __restrict__ yr, int64_t ldyr) {
  constexpr int UPL = BITS == 2 ? 2 : 1;  // 32-code units per lane step
  constexpr int NW = BITS * UPL;          // code words per row per lane step
  constexpr int NC = 32 * UPL;            // columns per lane step
  extern __shared__ __attribute__((aligned(16))) float xs[];  // NB x d_in
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = (int64_t(blockIdx.x) * 4 + wave) * RPW;
  const int64_t steps = d_in / NC;  // d_in is a multiple of 128
  float acc[RPW][NB];
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = 0.f;
  // lane steps base + lane + 64 q (q < MAXU) per chunk; the codes of a chunk are all requested
  // before any is used, and the first chunk's before x' is staged
  for (int64_t base = 0; base < steps; base += 64 * MAXU) {
    uint32_t w[MAXU][RPW][NW];
#pragma unroll
    for (int q = 0; q < MAXU; ++q) {
      const int64_t st = base + lane + 64 * q;
      if (st < steps) {
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
          const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
          const uint32_t* p = packed + row * ldp + st * NW;
#pragma unroll
          for (int k = 0; k < UPL; ++k) {
            uint32_t t[BITS];
            load_unit<BITS>(p + k * BITS, t);
#pragma unroll
            for (int i = 0; i < BITS; ++i) w[q][r][k * BITS + i] = t[i];
          }
        }
      }
    }
    if (base == 0) {  // the same for every thread of the workgroup
#pragma unroll
      for (int b = 0; b < NB; ++b)
        for (int64_t c = int64_t(tid) * 4; c < d_in; c += 1024)
          *reinterpret_cast<float4*>(xs + b * d_in + c) =
              *reinterpret_cast<const float4*>(xr + b * ldxr + c);
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < MAXU; ++q) {
      const int64_t st = base + lane + 64 * q;
      if (st < steps) {
        const int64_t c0 = st * NC, g = c0 / group;
        float sc[RPW], ze[RPW];
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
          const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
          sc[r] = scales[row * ldsz + g];
          ze[r] = zeros[row * ldsz + g];
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          float xv[NC], xsum = 0.f;
#pragma unroll
          for (int k = 0; k < NC / 4; ++k) {
            const float4 v = *reinterpret_cast<const float4*>(xs + b * d_in + c0 + 4 * k);
            xv[4 * k] = v.x, xv[4 * k + 1] = v.y, xv[4 * k + 2] = v.z, xv[4 * k + 3] = v.w;
            xsum += (v.x + v.y) + (v.z + v.w);
          }
#pragma unroll
          for (int r = 0; r < RPW; ++r) {
            float dot = 0.f;
#pragma unroll
            for (int k = 0; k < UPL; ++k) {
              uint32_t t[BITS];
#pragma unroll
              for (int i = 0; i < BITS; ++i) t[i] = w[q][r][k * BITS + i];
#pragma unroll
              for (int j = 0; j < 32; ++j)
                dot = fmaf(float(code_at<BITS>(t, j)), xv[32 * k + j], dot);
            }
            acc[r][b] = fmaf(sc[r], fmaf(-ze[r], xsum, dot), acc[r][b]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float v = acc[r][b];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0 && row0 + r < d_out) yr[b * ldyr + row0 + r] = v;
    }
}

// rows per wave: 8 for one vector when that still gives 512 workgroups (two per CU), else 2
template <int BITS, int NB>
int gemv_launch(const uint32_t* packed, int64_t ldp, const float* scales, const float* zeros,
                int64_t ldsz, int group, int64_t d_out, int64_t d_in, const float* xr,
                float* yr, hipStream_t s) {
  const size_t lds = size_t(NB) * size_t(d_in) * sizeof(float);
  if constexpr (NB == 1) {
    if (cdiv(d_out, 32) >= 512)
      return launch("online_gemv", online_gemv<BITS, 1, 8, 2>,
                    dim3(static_cast<unsigned>(cdiv(d_out, 32))), dim3(256), lds, s, packed, ldp,
                    scales, zeros, ldsz, group, d_out, d_in, xr, d_in, yr, d_out);
  }
  return launch("online_gemv", online_gemv<BITS, NB, 2, 2>,
                dim3(static_cast<unsigned>(cdiv(d_out, 8))), dim3(256), lds, s, packed, ldp,
                scales, zeros, ldsz, group, d_out, d_in, xr, d_in, yr, d_out);
}

// the batch in chunks of 4, 2 and 1 vectors (each chunk reads the codes once)
template <int BITS>
int gemv_bits(int nb, const uint32_t* packed, int64_t ldp, const float* scales,
              const float* zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
              const float* xr, float* yr, hipStream_t s) {
  int b = 0;
  while (b < nb) {
    const float* x = xr + int64_t(b) * d_in;
    float* y = yr + int64_t(b) * d_out;
    if (nb - b >= 4) {
      KQ_TRY((gemv_launch<BITS, 4>(packed, ldp, scales, zeros, ldsz, group, d_out, d_in, x, y,
                                   s)));
      b += 4;
    } else if (nb - b >= 2) {
      KQ_TRY((gemv_launch<BITS, 2>(packed, ldp, scales, zeros, ldsz, group, d_out, d_in, x, y,
                                   s)));
      b += 2;
    } else {
      KQ_TRY((gemv_launch<BITS, 1>(packed, ldp, scales, zeros, ldsz, group, d_out, d_in, x, y,
                                   s)));
      b += 1;
    }
  }
  return KRONQ_OK;
}

// Transform of B vectors of order d = L m: out[b] = diag(post) (A (x) H_m) diag(pre) src[b] * norm
// (A = Q28 or Q28^T when has28, else the Sylvester H_L). Workgroup (a, b): segment a of vector b.
template <typename T>
__global__ __launch_bounds__(1024) void seg_transform(const T* __restrict__ src, int64_t lds_,
                                                      float* __restrict__ dst, int64_t ldd, int L,
                                                      int m, const float* __restrict__ pre,
                                                      const float* __restrict__ post,
                                                      const float* __restrict__ q28, int q_trans,
                                                      int has28, float norm) {
  __shared__ float t[1024];
  __shared__ float arow[32];
  const int a = blockIdx.x, tid = threadIdx.x;
  const T* x = src + int64_t(blockIdx.y) * lds_;
  if (tid < L)
    arow[tid] = has28 ? (q_trans ? q28[tid * 28 + a] : q28[a * 28 + tid])
                      : ((__popc(unsigned(a & tid)) & 1) ? -1.f : 1.f);
  __syncthreads();
  if (tid < m) {
    float acc = 0.f;
    for (int k = 0; k < L; ++k) {
      const int64_t idx = int64_t(k) * m + tid;
      float v = ld_f32(x, idx);
      if (pre) v *= pre[idx];
      acc = fmaf(arow[k], v, acc);
    }
    t[tid] = acc;
  }
  __syncthreads();
  for (int lh = 0; (1 << lh) < m; ++lh) {  // radix-2 FWHT of the segment, one butterfly/thread
    const int h = 1 << lh;
    if (tid < m / 2) {
      const int i = ((tid >> lh) << (lh + 1)) + (tid & (h - 1));
      const float u = t[i], v = t[i + h];
      t[i] = u + v;
      t[i + h] = u - v;
    }
    __syncthreads();
  }
  if (tid < m) {
    const int64_t idx = int64_t(a) * m + tid;
    float v = t[tid] * norm;
    if (post) v *= post[idx];
    dst[int64_t(blockIdx.y) * ldd + idx] = v;
  }
}

// launch seg_transform for B rows of order d (identity scaling when !rotate)
int seg_transform_launch(const void* src, int dtype, int64_t lds_, float* dst, int64_t ldd,
                         int64_t batch, int64_t d, const float* pre, const float* post,
                         bool rotate, const float* q28, bool q_trans, hipStream_t s) {
  int L, m, has28 = 0;
  float norm;
  const RotDim rd = rot_dim(d);
  if (rotate && rd.has28) {
    L = 28, m = int(rd.m), has28 = 1;
    norm = float(1.0 / std::sqrt(double(m)));
  } else if (rotate) {
    m = int(d < 1024 ? d : 1024), L = int(d / m);
    norm = float(1.0 / std::sqrt(double(d)));
  } else {  // no rotation: L = 1 segment of d <= 1024, or the identity as L x m with A = I
    return rotate_vectors(src, dtype, lds_, dst, ldd, batch, d, pre, post, false, nullptr, false,
                          s);
  }
  const dim3 grid(static_cast<unsigned>(L), static_cast<unsigned>(batch));
  if (dtype == KRONQ_BF16)
    return launch("online_transform", seg_transform<uint16_t>, grid, dim3(1024), 0, s,
                  static_cast<const uint16_t*>(src), lds_, dst, ldd, L, m, pre, post, q28,
                  int(q_trans), has28, norm);
  return launch("online_transform", seg_transform<float>, grid, dim3(1024), 0, s,
                static_cast<const float*>(src), lds_, dst, ldd, L, m, pre, post, q28,
                int(q_trans), has28, norm);
}

}  // namespace

int pack_codes_launch(const uint8_t* codes, int64_t d_out, int64_t d_in, int64_t ldq, int bits,
                      uint32_t* packed, int64_t ldp, hipStream_t s) {
  const int64_t units = d_in / 32;
  const dim3 grid(unsigned(cdiv(d_out * units, 256)));
  switch (bits) {
    case 2:
      return launch("pack_codes", pack_codes<2>, grid, dim3(256), 0, s, codes, d_out, units, ldq,
                    packed, ldp);
    case 3:
      return launch("pack_codes", pack_codes<3>, grid, dim3(256), 0, s, codes, d_out, units, ldq,
                    packed, ldp);
    case 4:
      return launch("pack_codes", pack_codes<4>, grid, dim3(256), 0, s, codes, d_out, units, ldq,
                    packed, ldp);
    default:
      return launch("pack_codes", pack_codes<8>, grid, dim3(256), 0, s, codes, d_out, units, ldq,
                    packed, ldp);
  }
}

size_t online_ws_bytes(int64_t d_out, int64_t d_in, int64_t batch) {
  if (d_out <= 0 || d_in <= 0 || batch <= 0) return 0;
  return align256(size_t(batch) * size_t(d_in) * sizeof(float)) +
         align256(size_t(batch) * size_t(d_out) * sizeof(float)) + 256;
}

int online_matvec_launch(const uint32_t* packed, int64_t ldp, const float* scales,
                         const float* zeros, int64_t ldsz, int bits, int group, int64_t d_out,
                         int64_t d_in, const float* mul_in, const float* mul_out,
                         const float* q28_in, const float* q28_out, int flags, const void* x,
                         int x_dtype, int64_t ldx, int64_t batch, float* y, int64_t ldy, void* ws,
                         hipStream_t s) {
  Carver cv(ws);
  float* xr = cv.take<float>(size_t(batch) * size_t(d_in));
  float* yr = cv.take<float>(size_t(batch) * size_t(d_out));
  const int nb = int(batch);
  // x' = V S_X^-1 x
  KQ_TRY(seg_transform_launch(x, x_dtype, ldx, xr, d_in, batch, d_in, mul_in, nullptr,
                              (flags & KRONQ_ROT_IN) != 0, q28_in, false, s));
  // y' = W_hat' x'
  switch (bits) {
    case 2:
      KQ_TRY(gemv_bits<2>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, xr, yr, s));
      break;
    case 3:
      KQ_TRY(gemv_bits<3>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, xr, yr, s));
      break;
    case 4:
      KQ_TRY(gemv_bits<4>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, xr, yr, s));
      break;
    default:
      KQ_TRY(gemv_bits<8>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, xr, yr, s));
  }
  // y = S_G^-1 U^T y'
  return seg_transform_launch(yr, KRONQ_FP32, d_out, y, ldy, batch, d_out, nullptr, mul_out,
                              (flags & KRONQ_ROT_OUT) != 0, q28_out, true, s);
}

}  // namespace kq
