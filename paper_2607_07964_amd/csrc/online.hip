// Inference with a quantised layer: the rotations are applied online, O(d log d) per layer
// (Sec. 3.2 and 4.2; Limitations), around a matvec on the packed low-bit codes, so that
// y = S_G^-1 U^T W_hat' V S_X^-1 x (the original-space layer of Alg. 2's last line) is never
// formed as a dense matrix. For B <= 4 activation vectors:
//   1. x' = V S_X^-1 x: one BiIP row pass per vector (multipliers sign / s_X, FWHT, 28-point mix);
//   2. y' = W_hat' x': the packed-code GEMV, bound by the HBM reads of the codes;
//   3. y = S_G^-1 U^T y': one row pass per vector with the transposed factor, then the
//      multipliers sign / s_G.
// Packed format: each run of 32 consecutive codes of a row is one 32 * bits-bit little-endian
// string held in `bits` uint32 words, so a lane's 32 codes are one 8-, 12-, 16- or 32-byte load.
// GEMV: a workgroup stages x' (B x d_in fp32) in LDS and takes 16 rows, 4 per wave. Lane l takes
// the 32-column units l, l + 64, ...: it reads the unit's x' once, then per row the unit's code
// words, and adds s * (sum_j q_j x'_j - z * sum_j x'_j) with the row's group scale s and zero z
// (a group is a multiple of 128 columns, so a unit lies in one group). Wave sums at the end.
#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int RPWAVE = 4;          // rows per wave
constexpr int RPWG = 4 * RPWAVE;   // rows per workgroup

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

template <int BITS, int NB>
__global__ __launch_bounds__(256) void online_gemv(
    const uint32_t* __restrict__ packed, int64_t ldp, const float* __restrict__ scales,
    const float* __restrict__ zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
    const float* __restrict__ xr, int64_t ldxr, float* __restrict__ yr, int64_t ldyr) {
  extern __shared__ __attribute__((aligned(16))) float xs[];  // NB x d_in
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll
  for (int b = 0; b < NB; ++b)
    for (int64_t c = int64_t(tid) * 4; c < d_in; c += 1024)
      *reinterpret_cast<float4*>(xs + b * d_in + c) =
          *reinterpret_cast<const float4*>(xr + b * ldxr + c);
  __syncthreads();
  const int64_t row0 = (int64_t(blockIdx.x) * 4 + wave) * RPWAVE;
  if (row0 >= d_out) return;  // whole waves; no barrier follows
  const int64_t units = d_in / 32;
  float acc[RPWAVE][NB];
#pragma unroll
  for (int r = 0; r < RPWAVE; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = 0.f;
  for (int64_t u = lane; u < units; u += 64) {
    const int64_t c0 = u * 32, g = c0 / group;
    uint32_t w[RPWAVE][BITS];
#pragma unroll
    for (int r = 0; r < RPWAVE; ++r) {
      const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
      load_unit<BITS>(packed + row * ldp + u * BITS, w[r]);
    }
    float xv[NB][32], xsum[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      xsum[b] = 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float4 v = *reinterpret_cast<const float4*>(xs + b * d_in + c0 + 4 * k);
        xv[b][4 * k] = v.x, xv[b][4 * k + 1] = v.y, xv[b][4 * k + 2] = v.z,
        xv[b][4 * k + 3] = v.w;
        xsum[b] += (v.x + v.y) + (v.z + v.w);
      }
    }
#pragma unroll
    for (int r = 0; r < RPWAVE; ++r) {
      const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
      const float s = scales[row * ldsz + g], z = zeros[row * ldsz + g];
      float dot[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) dot[b] = 0.f;
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        const float q = float(code_at<BITS>(w[r], j));
#pragma unroll
        for (int b = 0; b < NB; ++b) dot[b] = fmaf(q, xv[b][j], dot[b]);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[r][b] = fmaf(s, fmaf(-z, xsum[b], dot[b]), acc[r][b]);
    }
  }
#pragma unroll
  for (int r = 0; r < RPWAVE; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float v = acc[r][b];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0 && row0 + r < d_out) yr[b * ldyr + row0 + r] = v;
    }
}

template <int BITS>
int gemv_bits(int nb, const uint32_t* packed, int64_t ldp, const float* scales,
              const float* zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
              const float* xr, float* yr, hipStream_t s) {
  const dim3 grid(unsigned(cdiv(d_out, RPWG)));
  const size_t lds = size_t(nb) * size_t(d_in) * sizeof(float);
  switch (nb) {
    case 1:
      return launch("online_gemv", online_gemv<BITS, 1>, grid, dim3(256), lds, s, packed, ldp,
                    scales, zeros, ldsz, group, d_out, d_in, xr, d_in, yr, d_out);
    case 2:
      return launch("online_gemv", online_gemv<BITS, 2>, grid, dim3(256), lds, s, packed, ldp,
                    scales, zeros, ldsz, group, d_out, d_in, xr, d_in, yr, d_out);
    case 3:
      return launch("online_gemv", online_gemv<BITS, 3>, grid, dim3(256), lds, s, packed, ldp,
                    scales, zeros, ldsz, group, d_out, d_in, xr, d_in, yr, d_out);
    default:
      return launch("online_gemv", online_gemv<BITS, 4>, grid, dim3(256), lds, s, packed, ldp,
                    scales, zeros, ldsz, group, d_out, d_in, xr, d_in, yr, d_out);
  }
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
  KQ_TRY(rotate_vectors(x, x_dtype, ldx, xr, d_in, batch, d_in, mul_in, nullptr,
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
  return rotate_vectors(yr, KRONQ_FP32, d_out, y, ldy, batch, d_out, nullptr, mul_out,
                        (flags & KRONQ_ROT_OUT) != 0, q28_out, true, s);
}

}  // namespace kq
