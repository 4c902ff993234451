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
// GEMV with 2- and 4-bit codes (online_gemv_int): the input transform also writes x' as
// three byte digits per element, a 21-bit fixed point with one exponent per 32-column chunk
// (relative precision 2^-21 of the chunk's largest value), in the byte order in which the GEMV
// extracts codes from a packed word with one shift and one mask. Each code byte group then meets
// the digits in three integer dot4 products with exact sums, about 1.1 instructions per code
// against 3.5 for the fp32 dequantise-and-FMA, which made the GEMV ALU-bound.
// GEMV with 3- and 8-bit codes (online_gemv): a workgroup takes 4 * RPW rows, RPW per wave, and
// stages x' (B x d_in fp32, B <= 4 per launch) in LDS. Lane l
// takes steps of 32 * UPL columns (UPL = 2 at 2 bits, so every code load is 16 bytes) at a
// stride of 64 steps. A decode matvec moves little data per CU, so latency is the limit: a lane
// requests the codes of up to MAXU steps of its RPW rows at once, before x' is staged, and only
// then computes. For each step and row it adds s * (sum_j q_j x'_j - z * sum_j x'_j) with the
// row's group scale s and zero z (a group is a multiple of 128 columns, so a step lies in one
// group). Wave sums at the end.
#include <cmath>

#include "kq_common.hpp"
#include "kq_fwht.hpp"

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

// Digits of x' for the integer GEMV: per chunk of 32 columns, X_j = rint(x'_j 2^(21 - e)) with
// |x'_j| < 2^e over the chunk, split as X = d0 65536 + d1 256 + d2 (d0 = X >> 16 signed,
// d1, d2 unsigned bytes). The bytes are stored in the order the GEMV extracts codes from a packed
// word: digit dword (w, g) of a chunk holds the digits of the columns w * cpw + g + i * (8 / bits),
// i = 0..3 (cpw = 32 / bits codes per word), in bytes i; a chunk has 3 x 8 such dwords. Also the
// exponent e and the sum of the quantised chunk, sum_j X_j 2^(e - 21).
__device__ __forceinline__ void emit_digits(float v, int64_t col, int lane32, int bits,
                                            uint8_t* __restrict__ dig, int* __restrict__ dexp,
                                            float* __restrict__ dsum) {
  float mx = fabsf(v);
#pragma unroll
  for (int o = 1; o < 32; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 32));
  // |v| < 2^e from the exponent field (chunks below 2^-100 are taken as zero)
  const int e = max(int((__float_as_uint(mx) >> 23) & 0xFFu) - 126, -100);
  const float up = __uint_as_float(uint32_t(127 + 21 - e) << 23);  // 2^(21 - e)
  const int X = int(rintf(v * up));                                  // |X| <= 2^21
  int sx = X;
#pragma unroll
  for (int o = 1; o < 32; o <<= 1) sx += __shfl_xor(sx, o, 32);
  const int64_t c = col >> 5;
  const int j = int(col & 31), cpw = 32 / bits, per = 8 / bits;
  const int w = j / cpw, rem = j % cpw, g = rem % per, i = rem / per;
  uint8_t* base = dig + c * 96 + (w * per + g) * 4 + i;
  base[0] = uint8_t(X >> 16);   // d0, signed byte
  base[32] = uint8_t(X >> 8);   // d1
  base[64] = uint8_t(X);        // d2
  if (lane32 == 0) {
    dexp[c] = e;
    dsum[c] = float(sx) / up;  // |sx| <= 2^26: one rounding to fp32, then an exact scaling
  }
}

// 8 consecutive activations as loaded (16-byte loads), widened to fp32 later
template <typename T>
struct RawX;
template <>
struct RawX<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void widen(float* v) const {
    v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = b.x, v[5] = b.y, v[6] = b.z, v[7] = b.w;
  }
};
template <>
struct RawX<uint16_t> {
  uint4 a;
  __device__ __forceinline__ void load(const uint16_t* p) { a = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void widen(float* v) const {
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = __uint_as_float(w[k] << 16);
      v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
    }
  }
};

// Transform of B vectors of order d = L m: out[b] = diag(post) (A (x) H_m) diag(pre) src[b] * norm
// (A = Q28 or Q28^T when has28, else the Sylvester H_L). Workgroup (a, b): segment a of vector b.
// With dig != nullptr (and m a multiple of 32) it also writes the digits of the result.
template <typename T>
__global__ __launch_bounds__(1024) void seg_transform(
    const T* __restrict__ src, int64_t lds_, float* __restrict__ dst, int64_t ldd, int L, int m,
    const float* __restrict__ pre, const float* __restrict__ post, const float* __restrict__ q28,
    int q_trans, int has28, float norm, uint8_t* __restrict__ dig, int* __restrict__ dexp,
    float* __restrict__ dsum, int64_t ldc, int bits) {
  __shared__ float t[1024];
  __shared__ float arow[32];
  extern __shared__ __attribute__((aligned(16))) float xs[];  // L m floats: diag(pre) src[b]
  const int a = blockIdx.x, tid = threadIdx.x;
  const T* x = src + int64_t(blockIdx.y) * lds_;
  if (tid < L)
    arow[tid] = has28 ? (q_trans ? q28[tid * 28 + a] : q28[a * 28 + tid])
                      : ((__popc(unsigned(a & tid)) & 1) ? -1.f : 1.f);
  // the whole vector, scaled, into LDS with 16-byte loads (8 elements a thread and step), each
  // workgroup starting at its own offset: every workgroup reads all L segments, and in one
  // order, or with each thread's L loads in flight at once, their requests queued on the same
  // lines (a segment read straight from memory by each thread took about 10 us at 28 x 512)
  const int d = L * m;
  const bool vec = d % 8 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(pre) & 15) == 0;
  if (vec) {
    const int n8 = d / 8, rot = int((uint32_t(a) * 97u + uint32_t(blockIdx.y) * 31u) % uint32_t(n8));
    for (int i = tid; i < n8; i += 1024) {
      const int j = 8 * (i + rot < n8 ? i + rot : i + rot - n8);
      RawX<T> r;
      r.load(x + j);
      float v[8];
      r.widen(v);
      if (pre) {
        const float4 p0 = reinterpret_cast<const float4*>(pre + j)[0];
        const float4 p1 = reinterpret_cast<const float4*>(pre + j)[1];
        v[0] *= p0.x, v[1] *= p0.y, v[2] *= p0.z, v[3] *= p0.w;
        v[4] *= p1.x, v[5] *= p1.y, v[6] *= p1.z, v[7] *= p1.w;
      }
      float4* o = reinterpret_cast<float4*>(xs + j);
      o[0] = make_float4(v[0], v[1], v[2], v[3]);
      o[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
  } else {
    for (int i = tid; i < d; i += 1024) xs[i] = pre ? ld_f32(x, i) * pre[i] : ld_f32(x, i);
  }
  __syncthreads();
  if (tid < m) {
    float acc = 0.f;
    for (int k = 0; k < L; ++k) acc = fmaf(arow[k], xs[k * m + tid], acc);
    t[tid] = acc;
  }
  __syncthreads();
  fwht_lds(t, m, m, tid, 1024);  // radix-8 groups of stages; ends with a barrier
  if (tid < m) {
    const int64_t idx = int64_t(a) * m + tid;
    float v = t[tid] * norm;
    if (post) v *= post[idx];
    dst[int64_t(blockIdx.y) * ldd + idx] = v;
    if (dig) {
      const int64_t cb = int64_t(blockIdx.y) * ldc;  // chunks per vector
      emit_digits(v, idx, tid & 31, bits, dig + cb * 96, dexp + cb, dsum + cb);
    }
  }
}

// digits of B fp32 vectors of length d (a multiple of 32) that no transform produced
__global__ __launch_bounds__(256) void digitize(const float* __restrict__ src, int64_t d, int bits,
                                                uint8_t* __restrict__ dig, int* __restrict__ dexp,
                                                float* __restrict__ dsum, int64_t ldc) {
  const int64_t col = int64_t(blockIdx.x) * 256 + threadIdx.x;  // d % 32 == 0: whole chunks
  if (col - (threadIdx.x & 31) >= d) return;                     // uniform per 32 lanes
  const int64_t b = blockIdx.y, cb = b * ldc;
  emit_digits(src[b * d + col], col, int(threadIdx.x & 31), bits, dig + cb * 96, dexp + cb,
              dsum + cb);
}

// Packed-code GEMV with the activations as digits (2- and 4-bit codes): per chunk of 32 columns
// and row, the code bytes of each packed word (groups g: (word >> bits g) & byte mask) meet the
// digit dwords in three dot4 products (d0 signed, d1 and d2 unsigned), exact integer sums, and
// sum_j q_j x'_j = 2^(e - 21) (65536 I0 + 256 I1 + I2).
template <int BITS, int NB, int RPW>
__global__ __launch_bounds__(256) void online_gemv_int(
    const uint32_t* __restrict__ packed, int64_t ldp, const float* __restrict__ scales,
    const float* __restrict__ zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
    const uint32_t* __restrict__ dig, const int* __restrict__ dexp,
    const float* __restrict__ dsum, float* __restrict__ yr, int64_t ldyr) {
  constexpr int UPL = BITS == 2 ? 2 : 1;  // chunks per lane step (16-byte code loads)
  constexpr int PER = 8 / BITS;           // byte groups per code word
  constexpr uint32_t BM = BITS == 2 ? 0x03030303u : 0x0F0F0F0Fu;
  extern __shared__ __attribute__((aligned(16))) uint32_t sm[];
  const int64_t nch = d_in / 32;
  uint32_t* sd = sm;                                   // NB x nch x 24 digit dwords
  int* se = reinterpret_cast<int*>(sm + NB * nch * 24);  // NB x nch exponents
  float* ss = reinterpret_cast<float*>(se + NB * nch);  // NB x nch chunk sums
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = (int64_t(blockIdx.x) * 4 + wave) * RPW;
  const int64_t steps = nch / UPL;
  float acc[RPW][NB];
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = 0.f;
  for (int64_t base = 0; base < steps; base += 128) {  // 2 lane steps per chunk of work
    uint32_t w[2][RPW][4];  // 16 bytes of codes per row and lane step
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int64_t st = base + lane + 64 * q;
      if (st < steps) {
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
          const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
          const uint4 v = *reinterpret_cast<const uint4*>(packed + row * ldp + st * 4);
          w[q][r][0] = v.x, w[q][r][1] = v.y, w[q][r][2] = v.z, w[q][r][3] = v.w;
        }
      }
    }
    if (base == 0) {  // the same for every thread of the workgroup
      for (int64_t i = tid; i < NB * nch * 6; i += 256)
        reinterpret_cast<uint4*>(sd)[i] = reinterpret_cast<const uint4*>(dig)[i];
      for (int64_t i = tid; i < NB * nch; i += 256) {
        se[i] = dexp[i];
        ss[i] = dsum[i];
      }
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int64_t st = base + lane + 64 * q;
      if (st < steps) {
#pragma unroll
        for (int u = 0; u < UPL; ++u) {
          const int64_t c = st * UPL + u, g = (c * 32) / group;
          float sc[RPW], ze[RPW];
#pragma unroll
          for (int r = 0; r < RPW; ++r) {
            const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
            sc[r] = scales[row * ldsz + g];
            ze[r] = zeros[row * ldsz + g];
          }
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            const uint32_t* dd = sd + (b * nch + c) * 24;
            uint32_t d0[8], d1[8], d2[8];
#pragma unroll
            for (int k = 0; k < 8; k += 4) {
              const uint4 x0 = *reinterpret_cast<const uint4*>(dd + k);
              const uint4 x1 = *reinterpret_cast<const uint4*>(dd + 8 + k);
              const uint4 x2 = *reinterpret_cast<const uint4*>(dd + 16 + k);
              d0[k] = x0.x, d0[k + 1] = x0.y, d0[k + 2] = x0.z, d0[k + 3] = x0.w;
              d1[k] = x1.x, d1[k + 1] = x1.y, d1[k + 2] = x1.z, d1[k + 3] = x1.w;
              d2[k] = x2.x, d2[k + 1] = x2.y, d2[k + 2] = x2.z, d2[k + 3] = x2.w;
            }
            const float e = __uint_as_float(uint32_t(127 - 21 + se[b * nch + c]) << 23);
            const float xs = ss[b * nch + c];
#pragma unroll
            for (int r = 0; r < RPW; ++r) {
              int i0 = 0;
              uint32_t i1 = 0u, i2 = 0u;
#pragma unroll
              for (int wi = 0; wi < BITS; ++wi) {  // the chunk's code words
                const uint32_t word = w[q][r][u * BITS + wi];
#pragma unroll
                for (int gg = 0; gg < PER; ++gg) {
                  const uint32_t by = (word >> (BITS * gg)) & BM;
                  const int slot = wi * PER + gg;
                  i0 = __builtin_amdgcn_sdot4(int(by), int(d0[slot]), i0, false);
                  i1 = __builtin_amdgcn_udot4(by, d1[slot], i1, false);
                  i2 = __builtin_amdgcn_udot4(by, d2[slot], i2, false);
                }
              }
              const float dot =
                  e * fmaf(float(i0), 65536.f, fmaf(float(i1), 256.f, float(i2)));
              acc[r][b] = fmaf(sc[r], fmaf(-ze[r], xs, dot), acc[r][b]);
            }
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

// lane (lane ^ 1) and (lane ^ 2) of each quad (DPP quad_perm [1,0,3,2] and [2,3,0,1])
__device__ __forceinline__ int quad_xor1(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
}
__device__ __forceinline__ int quad_xor2(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
}

// The digits (as emit_digits) of 8 consecutive elements j0 .. j0 + 7 of x' held by one lane: the
// four lanes of a quad hold one 32-column chunk, so the chunk's largest magnitude and digit sum
// take two DPP steps each.
template <int BITS>
__device__ __forceinline__ void emit_digits8(const float (&v)[8], int j0, uint8_t* __restrict__ dig,
                                             int* __restrict__ dexp, float* __restrict__ dsum) {
  constexpr int CPW = 32 / BITS, PER = 8 / BITS;
  float mx = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) mx = fmaxf(mx, fabsf(v[k]));
  mx = fmaxf(mx, __int_as_float(quad_xor1(__float_as_int(mx))));
  mx = fmaxf(mx, __int_as_float(quad_xor2(__float_as_int(mx))));
  const int e = max(int((__float_as_uint(mx) >> 23) & 0xFFu) - 126, -100);
  const float up = __uint_as_float(uint32_t(127 + 21 - e) << 23);  // 2^(21 - e)
  const int c = j0 >> 5, jc = j0 & 31;
  int sx = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int X = int(rintf(v[k] * up));  // |X| <= 2^21
    sx += X;
    const int col = jc + k, w = col / CPW, rem = col % CPW, g = rem % PER, i = rem / PER;
    uint8_t* base = dig + c * 96 + (w * PER + g) * 4 + i;
    base[0] = uint8_t(X >> 16);
    base[32] = uint8_t(X >> 8);
    base[64] = uint8_t(X);
  }
  sx += quad_xor1(sx);
  sx += quad_xor2(sx);
  if (jc == 0) {
    dexp[c] = e;
    dsum[c] = float(sx) / up;
  }
}

// ---- one vector, 2- and 4-bit codes: the persistent GEMV -------------------------------------
// A workgroup requests the codes, scales and zeros of its first two tiles, puts the digits of x'
// in LDS, then walks its row blocks (4 * RPW rows each: blockIdx.x, + gridDim.x, ...) in tiles
// of 128 lane steps, two tile buffers in turn: a buffer is refilled with the tile two ahead as
// soon as its dot products are done. Every load is issued unconditionally (indices clamped into
// range), so the wait for a tile's loads counts exactly the other buffer's. With FUSE the
// workgroup computes x' itself: x and the multipliers are requested before the tiles' codes, so
// the transform (the Sylvester FWHT of a power-of-two d_in, or the scaling alone) runs while the
// codes are in flight; it is repeated by every workgroup, which costs less than a separate launch
// at these sizes.
template <int BITS, int RPW>
struct TileRegs {
  uint32_t w[2][RPW][4];
  float sc[2][RPW], ze[2][RPW];
};

// tile (k, b): row block blockIdx.x + k * gridDim.x, lane steps [128 b, 128 b + 128)
template <int BITS, int RPW>
__device__ __forceinline__ void load_tile(TileRegs<BITS, RPW>& T, int k, int b, int steps,
                                          int wave, int lane,
                                          const uint32_t* __restrict__ packed, int64_t ldp,
                                          const float* __restrict__ scales,
                                          const float* __restrict__ zeros, int64_t ldsz,
                                          unsigned spg, int64_t d_out) {
  const int64_t rb = blockIdx.x + int64_t(k) * gridDim.x;
  const int64_t row0 = (rb * 4 + wave) * RPW;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    int st = b * 128 + lane + 64 * q;
    st = st < steps ? st : steps - 1;
    const int64_t g = unsigned(st) / spg;  // spg lane steps per quantisation group
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int64_t row = row0 + r < d_out ? row0 + r : d_out - 1;
      const uint4 v = *reinterpret_cast<const uint4*>(packed + row * ldp + int64_t(st) * 4);
      T.w[q][r][0] = v.x, T.w[q][r][1] = v.y, T.w[q][r][2] = v.z, T.w[q][r][3] = v.w;
      T.sc[q][r] = scales[row * ldsz + g];
      T.ze[q][r] = zeros[row * ldsz + g];
    }
  }
}

template <int BITS, int RPW>
__device__ __forceinline__ void tile_dots(const TileRegs<BITS, RPW>& T, int b, int steps,
                                          int lane, const uint32_t* __restrict__ sd,
                                          const int* __restrict__ se,
                                          const float* __restrict__ ss, float (&acc)[RPW]) {
  constexpr int UPL = BITS == 2 ? 2 : 1, PER = 8 / BITS;
  constexpr uint32_t BM = BITS == 2 ? 0x03030303u : 0x0F0F0F0Fu;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int st = b * 128 + lane + 64 * q;
    if (st < steps) {
#pragma unroll
      for (int u = 0; u < UPL; ++u) {
        const int c = st * UPL + u;
        const uint32_t* dd = sd + c * 24;
        uint32_t d0[8], d1[8], d2[8];
#pragma unroll
        for (int k = 0; k < 8; k += 4) {
          const uint4 x0 = *reinterpret_cast<const uint4*>(dd + k);
          const uint4 x1 = *reinterpret_cast<const uint4*>(dd + 8 + k);
          const uint4 x2 = *reinterpret_cast<const uint4*>(dd + 16 + k);
          d0[k] = x0.x, d0[k + 1] = x0.y, d0[k + 2] = x0.z, d0[k + 3] = x0.w;
          d1[k] = x1.x, d1[k + 1] = x1.y, d1[k + 2] = x1.z, d1[k + 3] = x1.w;
          d2[k] = x2.x, d2[k + 1] = x2.y, d2[k + 2] = x2.z, d2[k + 3] = x2.w;
        }
        const float e = __uint_as_float(uint32_t(127 - 21 + se[c]) << 23);
        const float xs = ss[c];
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
          int i0 = 0;
          uint32_t i1 = 0u, i2 = 0u;
#pragma unroll
          for (int wi = 0; wi < BITS; ++wi) {
            const uint32_t word = T.w[q][r][u * BITS + wi];
#pragma unroll
            for (int gg = 0; gg < PER; ++gg) {
              const uint32_t by = (word >> (BITS * gg)) & BM;
              const int slot = wi * PER + gg;
              i0 = __builtin_amdgcn_sdot4(int(by), int(d0[slot]), i0, false);
              i1 = __builtin_amdgcn_udot4(by, d1[slot], i1, false);
              i2 = __builtin_amdgcn_udot4(by, d2[slot], i2, false);
            }
          }
          const float dot = e * fmaf(float(i0), 65536.f, fmaf(float(i1), 256.f, float(i2)));
          acc[r] = fmaf(T.sc[q][r], fmaf(-T.ze[q][r], xs, dot), acc[r]);
        }
      }
    }
  }
}

template <int RPW>
__device__ __forceinline__ void flush_rows(float (&acc)[RPW], int k, int wave, int lane,
                                           int64_t d_out, float* __restrict__ yr) {
  const int64_t rb = blockIdx.x + int64_t(k) * gridDim.x;
  const int64_t row0 = (rb * 4 + wave) * RPW;
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    float v = acc[r];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if (lane == 0 && row0 + r < d_out) yr[row0 + r] = v;
    acc[r] = 0.f;
  }
}

constexpr int FUSE_MAX_DIN = 8192;

// LDS slot of element j of the staged x': 4 floats of padding after every 128, so that the
// strided butterfly passes below hit distinct banks (a stride of 256 moves 8 banks)
__device__ __forceinline__ int xslot(int j) { return j + ((j >> 7) << 2); }

// stages [lo, lo + LB) of the FWHT of d = 256 * 2^LB staged elements: thread tid holds the 2^LB
// elements whose other index bits spell tid, all in registers for the LB stages
template <int LB>
__device__ __forceinline__ void fwht_pass(float* xt, int lo, int tid) {
  constexpr int E = 1 << LB;
  const int base = (tid & ((1 << lo) - 1)) | ((tid >> lo) << (lo + LB));
  float v[E];
#pragma unroll
  for (int i = 0; i < E; ++i) v[i] = xt[xslot(base + (i << lo))];
  hadamard_reg<E>(v);
#pragma unroll
  for (int i = 0; i < E; ++i) xt[xslot(base + (i << lo))] = v[i];
}

// the stages of strides 8 .. d/2 of the FWHT of d = 2^k staged elements (those of strides 1, 2, 4
// are applied in registers while staging), in groups of up to three stages per LDS round trip
template <int R>
__device__ __forceinline__ void stage_group_x(float* xt, int d, int lgh, int tid) {
  const int hm = (1 << lgh) - 1;
  for (int q = tid; q < d / R; q += 256) {
    const int base = ((q >> lgh) * (R << lgh)) + (q & hm);
    float v[R];
#pragma unroll
    for (int i = 0; i < R; ++i) v[i] = xt[xslot(base + (i << lgh))];
    hadamard_reg<R>(v);
#pragma unroll
    for (int i = 0; i < R; ++i) xt[xslot(base + (i << lgh))] = v[i];
  }
}
__device__ __forceinline__ void fwht_x(float* xt, int d, int tid) {
  if (d == 8192) {  // stages 3-7 and 8-12, 32 elements per thread
    fwht_pass<5>(xt, 3, tid);
    __syncthreads();
    fwht_pass<5>(xt, 8, tid);
    __syncthreads();
    return;
  }
  if (d == 4096) {  // stages 3-6, 7-10, then 11
    fwht_pass<4>(xt, 3, tid);
    __syncthreads();
    fwht_pass<4>(xt, 7, tid);
    __syncthreads();
    stage_group_x<2>(xt, d, 11, tid);
    __syncthreads();
    return;
  }
  for (int lgh = 3; (1 << lgh) < d;) {
    const int left = d >> lgh;
    if (left >= 8) {
      stage_group_x<8>(xt, d, lgh, tid);
      lgh += 3;
    } else if (left == 4) {
      stage_group_x<4>(xt, d, lgh, tid);
      lgh += 2;
    } else {
      stage_group_x<2>(xt, d, lgh, tid);
      lgh += 1;
    }
    __syncthreads();
  }
}  // x and its multipliers held in registers: 32 per thread

template <int BITS, int RPW, int FUSE, typename TX>
__global__ __launch_bounds__(256) void online_gemv_p(
    const uint32_t* __restrict__ packed, int64_t ldp, const float* __restrict__ scales,
    const float* __restrict__ zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
    const uint32_t* __restrict__ dig, const int* __restrict__ dexp,
    const float* __restrict__ dsum, const TX* __restrict__ x, const float* __restrict__ mul,
    int rotate, float norm, float* __restrict__ yr) {
  extern __shared__ __attribute__((aligned(16))) uint32_t sm[];
  constexpr int UPL = BITS == 2 ? 2 : 1;
  const int nch = int(d_in / 32);
  uint32_t* sd = sm;                                  // nch x 24 digit dwords
  int* se = reinterpret_cast<int*>(sm + nch * 24);    // nch exponents
  float* ss = reinterpret_cast<float*>(se + nch);     // nch chunk sums
  float* xt = ss + nch;  // FUSE: d_in + d_in / 32 floats (slots xslot(j)), 16-byte aligned
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int steps = nch / UPL, nbase = (steps + 127) / 128;
  const unsigned spg = unsigned(group / (32 * UPL));
  const int64_t nblk = cdiv(d_out, 4 * RPW);
  const int nrb = int((nblk - 1 - blockIdx.x) / gridDim.x + 1);  // row blocks (grid <= nblk)
  // FUSE: x and the multipliers, 8 consecutive elements per thread and step, requested
  // unconditionally (indices clamped; a missing mul reads x's first bytes and is not used) and
  // widened only after the first tile's loads are out
  RawX<TX> xr[FUSE ? 4 : 1];
  float4 mr[FUSE ? 8 : 1];
  if constexpr (FUSE) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int j0 = 8 * (tid + 256 * k), j = j0 < d_in ? j0 : 0;
      xr[k].load(x + j);
      const float4* mp = reinterpret_cast<const float4*>(mul ? mul + j : reinterpret_cast<const float*>(x));
      mr[2 * k] = mp[0];
      mr[2 * k + 1] = mp[1];
    }
  }
  // tiles in (row block k, base b) order; next() steps to the following tile, clamped to the
  // last one (a clamped tile is loaded again and never used)
  auto next = [&](int& kk, int& bb) {
    if (++bb == nbase) bb = 0, ++kk;
    if (kk == nrb) kk = nrb - 1, bb = nbase - 1;
  };
  // the first two tiles are requested before the prologue, so that their codes stream in while
  // x' is formed (the prologue is a few microseconds; one tile alone left HBM idle meanwhile)
  int k = 0, b = 0, k1 = 0, b1 = 0;
  next(k1, b1);
  TileRegs<BITS, RPW> A, B;
  load_tile(A, k, b, steps, wave, lane, packed, ldp, scales, zeros, ldsz, spg, d_out);
  load_tile(B, k1, b1, steps, wave, lane, packed, ldp, scales, zeros, ldsz, spg, d_out);
  if constexpr (FUSE) {
    // the butterflies of strides 1, 2, 4 on each thread's 8 consecutive values, in registers;
    // the other stages in LDS; then the digits, a quad of lanes per 32-column chunk
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int j = 8 * (tid + 256 * k);
      if (j < d_in) {
        float v[8];
        xr[k].widen(v);
        const float m[8] = {mr[2 * k].x, mr[2 * k].y, mr[2 * k].z, mr[2 * k].w,
                            mr[2 * k + 1].x, mr[2 * k + 1].y, mr[2 * k + 1].z, mr[2 * k + 1].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = mul ? v[e] * m[e] : v[e];
        if (rotate) hadamard_reg<8>(v);
        float4* dst = reinterpret_cast<float4*>(xt + xslot(j));  // 8 slots, no padding inside
        dst[0] = make_float4(v[0], v[1], v[2], v[3]);
        dst[1] = make_float4(v[4], v[5], v[6], v[7]);
      }
    }
    __syncthreads();
    if (rotate) fwht_x(xt, int(d_in), tid);  // each group ends with a barrier
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int j = 8 * (tid + 256 * k);
      if (j < d_in) {  // uniform over each quad (d_in % 32 == 0)
        const float4 a = reinterpret_cast<const float4*>(xt + xslot(j))[0];
        const float4 b = reinterpret_cast<const float4*>(xt + xslot(j))[1];
        const float v[8] = {a.x * norm, a.y * norm, a.z * norm, a.w * norm,
                            b.x * norm, b.y * norm, b.z * norm, b.w * norm};
        emit_digits8<BITS>(v, j, reinterpret_cast<uint8_t*>(sd), se, ss);
      }
    }
  } else {
    // every workgroup copies the same digits: each starts at its own offset, so that their
    // requests spread over the L2 channels instead of queueing on one line at a time
    const int n16 = nch * 6, r16 = int((uint32_t(blockIdx.x) * 97u) % uint32_t(n16));
    for (int i = tid; i < n16; i += 256) {
      const int ii = i + r16 < n16 ? i + r16 : i + r16 - n16;
      reinterpret_cast<uint4*>(sd)[ii] = reinterpret_cast<const uint4*>(dig)[ii];
    }
    for (int i = tid; i < nch; i += 256) {
      se[i] = dexp[i];
      ss[i] = dsum[i];
    }
  }
  __syncthreads();
  float acc[RPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r) acc[r] = 0.f;
  // A holds tile (k, b), B the tile after it, (k1, b1); a buffer is refilled with the tile two
  // ahead as soon as its dot products are done
  for (;;) {
    tile_dots(A, b, steps, lane, sd, se, ss, acc);
    if (b == nbase - 1) flush_rows(acc, k, wave, lane, d_out, yr);
    if (k == nrb - 1 && b == nbase - 1) break;
    int k2 = k1, b2 = b1;
    next(k2, b2);
    load_tile(A, k2, b2, steps, wave, lane, packed, ldp, scales, zeros, ldsz, spg, d_out);
    tile_dots(B, b1, steps, lane, sd, se, ss, acc);
    if (b1 == nbase - 1) flush_rows(acc, k1, wave, lane, d_out, yr);
    if (k1 == nrb - 1 && b1 == nbase - 1) break;
    k = k2, b = b2, k1 = k2, b1 = b2;
    next(k1, b1);
    load_tile(B, k1, b1, steps, wave, lane, packed, ldp, scales, zeros, ldsz, spg, d_out);
  }
}

// the persistent GEMV for one vector: row blocks of 4 * RPW rows dealt to two workgroups per
// CU (one where the LDS holds less)
template <int BITS>
int gemv_pers(bool fuse, const uint32_t* packed, int64_t ldp, const float* scales,
              const float* zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
              const uint8_t* dig, const int* dexp, const float* dsum, const void* x, int x_dtype,
              const float* mul, bool rotate, float* yr, hipStream_t s) {
  constexpr int RPW = 4;
  const int64_t nch = d_in / 32;
  const size_t lds = size_t(nch) * (96 + 8) + (fuse ? size_t(d_in + d_in / 32) * 4 : 0);
  const int64_t per_cu = lds <= 64 * 1024 ? 2 : 1;
  const int64_t nblk = cdiv(d_out, 4 * RPW);
  // one workgroup per slot: workgroup w takes row blocks w, w + grid, ..., so the two that share
  // a CU (w and w + CUs, dispatched in the second round) hold together an equal share; a grid
  // of nblk / 4 workgroups left a quarter of the CUs with one workgroup and the rest with two,
  // whose later end set the kernel's time
  const int64_t slots = int64_t(device_cus()) * per_cu;
  const dim3 grid(static_cast<unsigned>(nblk < slots ? nblk : slots));
  const float norm = rotate ? float(1.0 / std::sqrt(double(d_in))) : 1.f;
  const uint32_t* dg = reinterpret_cast<const uint32_t*>(dig);
  if (!fuse)
    return launch("online_gemv", online_gemv_p<BITS, RPW, 0, float>, grid, dim3(256), lds, s,
                  packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dg, dexp, dsum,
                  static_cast<const float*>(nullptr), mul, 0, norm, yr);
  if (x_dtype == KRONQ_BF16)
    return launch("online_gemv", online_gemv_p<BITS, RPW, 1, uint16_t>, grid, dim3(256), lds, s,
                  packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dg, dexp, dsum,
                  static_cast<const uint16_t*>(x), mul, int(rotate), norm, yr);
  return launch("online_gemv", online_gemv_p<BITS, RPW, 1, float>, grid, dim3(256), lds, s,
                packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dg, dexp, dsum,
                static_cast<const float*>(x), mul, int(rotate), norm, yr);
}

// launch seg_transform for B rows of order d (identity scaling when !rotate); with dig, also the
// digits of the result (for chunk-aligned segments, else by a separate pass)
int seg_transform_launch(const void* src, int dtype, int64_t lds_, float* dst, int64_t ldd,
                         int64_t batch, int64_t d, const float* pre, const float* post,
                         bool rotate, const float* q28, bool q_trans, hipStream_t s,
                         uint8_t* dig = nullptr, int* dexp = nullptr, float* dsum = nullptr,
                         int bits = 0) {
  int L = 0, m = 0, has28 = 0;
  float norm = 1.f;
  const RotDim rd = rot_dim(d);
  if (rotate && rd.has28) {
    L = 28, m = int(rd.m), has28 = 1;
    norm = float(1.0 / std::sqrt(double(m)));
  } else if (rotate) {
    m = int(d < 1024 ? d : 1024), L = int(d / m);
    norm = float(1.0 / std::sqrt(double(d)));
  }
  const int64_t nch = d / 32;
  const bool fused = dig && rotate && m % 32 == 0;
  if (!rotate) {
    KQ_TRY(rotate_vectors(src, dtype, lds_, dst, ldd, batch, d, pre, post, false, nullptr, false,
                          s));
  } else {
    const dim3 grid(static_cast<unsigned>(L), static_cast<unsigned>(batch));
    const size_t xs_bytes = size_t(L) * size_t(m) * sizeof(float);  // the staged vector
    uint8_t* dg = fused ? dig : nullptr;
    if (dtype == KRONQ_BF16)
      KQ_TRY(launch("online_transform", seg_transform<uint16_t>, grid, dim3(1024), xs_bytes, s,
                    static_cast<const uint16_t*>(src), lds_, dst, ldd, L, m, pre, post, q28,
                    int(q_trans), has28, norm, dg, dexp, dsum, nch, bits));
    else
      KQ_TRY(launch("online_transform", seg_transform<float>, grid, dim3(1024), xs_bytes, s,
                    static_cast<const float*>(src), lds_, dst, ldd, L, m, pre, post, q28,
                    int(q_trans), has28, norm, dg, dexp, dsum, nch, bits));
  }
  if (dig && !fused)
    KQ_TRY(launch("online_digitize", digitize,
                  dim3(static_cast<unsigned>(cdiv(d, 256)), static_cast<unsigned>(batch)),
                  dim3(256), 0, s, static_cast<const float*>(dst), d, bits, dig, dexp, dsum,
                  nch));
  return KRONQ_OK;
}

// the integer GEMV over the batch in chunks of 4, 2 and 1 vectors
template <int BITS>
int gemv_int(int nb, const uint32_t* packed, int64_t ldp, const float* scales,
             const float* zeros, int64_t ldsz, int group, int64_t d_out, int64_t d_in,
             const uint8_t* dig, const int* dexp, const float* dsum, float* yr, hipStream_t s) {
  const int64_t nch = d_in / 32;
  int b = 0;
  while (b < nb) {
    const int k = nb - b >= 4 ? 4 : (nb - b >= 2 ? 2 : 1);
    const uint32_t* dg = reinterpret_cast<const uint32_t*>(dig + int64_t(b) * nch * 96);
    const int* de = dexp + int64_t(b) * nch;
    const float* ds = dsum + int64_t(b) * nch;
    float* y = yr + int64_t(b) * d_out;
    const size_t lds = size_t(k) * size_t(nch) * (96 + 8);
    // rows per wave (measured on the 70B up_proj shape): 4 for one vector of 2-bit codes when
    // that still gives 512 workgroups, else 2
    const bool four = BITS == 2 && k == 1 && cdiv(d_out, 16) >= 512;
    const dim3 grid(static_cast<unsigned>(cdiv(d_out, four ? 16 : 8)));
#define KQ_GEMV_INT(NB_, RPW_)                                                                 \
  launch("online_gemv", online_gemv_int<BITS, NB_, RPW_>, grid, dim3(256), lds, s, packed, ldp, \
         scales, zeros, ldsz, group, d_out, d_in, dg, de, ds, y, d_out)
    if (k == 4)
      KQ_TRY(KQ_GEMV_INT(4, 2));
    else if (k == 2)
      KQ_TRY(KQ_GEMV_INT(2, 2));
    else if (four)
      KQ_TRY(KQ_GEMV_INT(1, 4));
    else
      KQ_TRY(KQ_GEMV_INT(1, 2));
#undef KQ_GEMV_INT
    b += k;
  }
  return KRONQ_OK;
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
  const size_t nch = size_t(batch) * size_t(d_in / 32);
  return align256(size_t(batch) * size_t(d_in) * sizeof(float)) +
         align256(size_t(batch) * size_t(d_out) * sizeof(float)) + align256(nch * 96) +
         2 * align256(nch * 4) + 256;
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
  const size_t nch = size_t(batch) * size_t(d_in / 32);
  uint8_t* dig = cv.take<uint8_t>(nch * 96);
  int* dexp = cv.take<int>(nch);
  float* dsum = cv.take<float>(nch);
  const int nb = int(batch);
  const bool integer = bits == 2 || bits == 4;  // codes that fill whole bytes of a word
  const bool rot_in = (flags & KRONQ_ROT_IN) != 0;
  if (integer && nb == 1) {  // decode: the persistent GEMV, with the input transform inside
    const bool pow2 = (d_in & (d_in - 1)) == 0;
    const bool fuse = d_in <= FUSE_MAX_DIN && (!rot_in || pow2);
    if (!fuse)
      KQ_TRY(seg_transform_launch(x, x_dtype, ldx, xr, d_in, batch, d_in, mul_in, nullptr, rot_in,
                                  q28_in, false, s, dig, dexp, dsum, bits));
    if (bits == 2)
      KQ_TRY(gemv_pers<2>(fuse, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dig, dexp,
                          dsum, x, x_dtype, mul_in, rot_in, yr, s));
    else
      KQ_TRY(gemv_pers<4>(fuse, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dig, dexp,
                          dsum, x, x_dtype, mul_in, rot_in, yr, s));
    return seg_transform_launch(yr, KRONQ_FP32, d_out, y, ldy, batch, d_out, nullptr, mul_out,
                                (flags & KRONQ_ROT_OUT) != 0, q28_out, true, s);
  }
  // x' = V S_X^-1 x (and its digits for the integer GEMV)
  KQ_TRY(seg_transform_launch(x, x_dtype, ldx, xr, d_in, batch, d_in, mul_in, nullptr,
                              (flags & KRONQ_ROT_IN) != 0, q28_in, false, s,
                              integer ? dig : nullptr, dexp, dsum, bits));
  // y' = W_hat' x'
  switch (bits) {
    case 2:
      KQ_TRY(gemv_int<2>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dig, dexp,
                         dsum, yr, s));
      break;
    case 3:
      KQ_TRY(gemv_bits<3>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, xr, yr, s));
      break;
    case 4:
      KQ_TRY(gemv_int<4>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, dig, dexp,
                         dsum, yr, s));
      break;
    default:
      KQ_TRY(gemv_bits<8>(nb, packed, ldp, scales, zeros, ldsz, group, d_out, d_in, xr, yr, s));
  }
  // y = S_G^-1 U^T y'
  return seg_transform_launch(yr, KRONQ_FP32, d_out, y, ldy, batch, d_out, nullptr, mul_out,
                              (flags & KRONQ_ROT_OUT) != 0, q28_out, true, s);
}

}  // namespace kq
