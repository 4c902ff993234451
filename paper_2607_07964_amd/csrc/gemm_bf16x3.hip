// C -= A B with fp32 operands on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16), fp32-accurate
// through a three-term split: x = x_hi + x_lo with x_hi = bf16(x), x_lo = bf16(x - x_hi), and
// A B ~ A_hi B_hi + A_hi B_lo + A_lo B_hi (the dropped A_lo B_lo term and the parts of x below
// x_lo are ~2^-16 of each product). Used for the OBS trailing updates W[:, rest] -= E U[blk, rest]
// (and, with the drift correction, the second product -W_blk P[blk, rest] in the same pass),
// where A = E (fp32, k contiguous) is split as it is staged and B = U rows comes pre-split and
// transposed (Ut_hi / Ut_lo, [n][k] bf16) by split_transpose, once per layer.
//   * TM x TM output tile per workgroup (TM = 128 or 64), 4 waves in a 2 x 2 grid, each wave
//     (TM/2) x (TM/2) = up to 2 x 2 MFMA blocks of 32 x 32 with fp32 accumulators.
//   * K advances 32 at a time through one LDS stage: A_hi, A_lo [m][k] and B_hi, B_lo [n][k],
//     first over the K of the first pair, then over the K2 of the second;
//     rows padded to 80 bytes so that the 16-byte operand reads of 8 consecutive lanes hit
//     distinct banks; the next stage is fetched into registers during the MFMAs.
#include <type_traits>

#include "kq_common.hpp"

namespace kq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int BK = 32;      // K per stage
constexpr int RS = 40;      // LDS row stride in bf16 (32 + 8 pad = 80 bytes)

// round-to-nearest-even fp32 -> bf16 bits (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

template <int TM>
__global__ __launch_bounds__(256) void gemm_bf16x3_sub(
    int64_t M, int64_t N, int64_t K, const float* __restrict__ A, int64_t lda,
    const uint16_t* __restrict__ Bh, const uint16_t* __restrict__ Bl, int64_t ldb, int64_t K2,
    const float* __restrict__ A2, int64_t lda2, const uint16_t* __restrict__ B2h,
    const uint16_t* __restrict__ B2l, int64_t ldb2, float* __restrict__ C, int64_t ldc) {
  constexpr int NB = TM / 64;                  // 32 x 32 blocks per wave edge (1 or 2)
  constexpr int AV = TM * BK / 4 / 256;        // float4 of A per thread per stage
  constexpr int BV = TM * BK / 8 / 256;        // 16-byte chunks of each B half per thread
  __shared__ __attribute__((aligned(16))) uint16_t sAh[TM * RS], sAl[TM * RS];
  __shared__ __attribute__((aligned(16))) uint16_t sBh[TM * RS], sBl[TM * RS];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1, l32 = lane & 31, lhi = lane >> 5;
  const int64_t m0 = int64_t(blockIdx.y) * TM, n0 = int64_t(blockIdx.x) * TM;

  float4 ra[AV];
  uint4 rbh[BV], rbl[BV];
  auto fetch = [&](int64_t kk) {
    // stage kk of the concatenated K: the first pair for kk < K, else the second
    const bool first = kk < K;
    const float* a = first ? A : A2;
    const uint16_t* bh = first ? Bh : B2h;
    const uint16_t* bl = first ? Bl : B2l;
    const int64_t la = first ? lda : lda2, lb = first ? ldb : ldb2, k0 = first ? kk : kk - K;
#pragma unroll
    for (int v = 0; v < AV; ++v) {
      const int e = tid + 256 * v, m = e / (BK / 4), kq = (e % (BK / 4)) * 4;
      ra[v] = (m0 + m < M) ? *reinterpret_cast<const float4*>(a + (m0 + m) * la + k0 + kq)
                           : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int v = 0; v < BV; ++v) {
      const int e = tid + 256 * v, n = e / (BK / 8), kc = (e % (BK / 8)) * 8;
      const bool ok = n0 + n < N;
      rbh[v] = ok ? *reinterpret_cast<const uint4*>(bh + (n0 + n) * lb + k0 + kc)
                  : make_uint4(0u, 0u, 0u, 0u);
      rbl[v] = ok ? *reinterpret_cast<const uint4*>(bl + (n0 + n) * lb + k0 + kc)
                  : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int v = 0; v < AV; ++v) {
      const int e = tid + 256 * v, m = e / (BK / 4), kq = (e % (BK / 4)) * 4;
      const float x[4] = {ra[v].x, ra[v].y, ra[v].z, ra[v].w};
      uint32_t h[4], l[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        h[c] = bf16_rne(x[c]);
        l[c] = bf16_rne(x[c] - bf16_to_f32(h[c]));
      }
      *reinterpret_cast<uint2*>(sAh + m * RS + kq) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
      *reinterpret_cast<uint2*>(sAl + m * RS + kq) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
    }
#pragma unroll
    for (int v = 0; v < BV; ++v) {
      const int e = tid + 256 * v, n = e / (BK / 8), kc = (e % (BK / 8)) * 8;
      *reinterpret_cast<uint4*>(sBh + n * RS + kc) = rbh[v];
      *reinterpret_cast<uint4*>(sBl + n * RS + kc) = rbl[v];
    }
  };

  f32x16_t acc[NB][NB];
#pragma unroll
  for (int a = 0; a < NB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = f32x16_t{};
  const int64_t KT = K + K2;
  if (KT > 0) fetch(0);
  for (int64_t k0 = 0; k0 < KT; k0 += BK) {
    __syncthreads();
    stash();
    __syncthreads();
    if (k0 + BK < KT) fetch(k0 + BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int kc = ks * 16 + 8 * lhi;  // this lane's 8 k of the 16
      bf16x8_t ah[NB], al[NB], bh[NB], bl[NB];
#pragma unroll
      for (int bi = 0; bi < NB; ++bi) {
        const int m = wm * (TM / 2) + bi * 32 + l32;
        ah[bi] = *reinterpret_cast<const bf16x8_t*>(sAh + m * RS + kc);
        al[bi] = *reinterpret_cast<const bf16x8_t*>(sAl + m * RS + kc);
      }
#pragma unroll
      for (int bj = 0; bj < NB; ++bj) {
        const int n = wn * (TM / 2) + bj * 32 + l32;
        bh[bj] = *reinterpret_cast<const bf16x8_t*>(sBh + n * RS + kc);
        bl[bj] = *reinterpret_cast<const bf16x8_t*>(sBl + n * RS + kc);
      }
#pragma unroll
      for (int bi = 0; bi < NB; ++bi)
#pragma unroll
        for (int bj = 0; bj < NB; ++bj) {
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[bi], bh[bj], acc[bi][bj], 0, 0, 0);
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[bi], bl[bj], acc[bi][bj], 0, 0, 0);
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[bi], bh[bj], acc[bi][bj], 0, 0, 0);
        }
    }
  }
#pragma unroll
  for (int bi = 0; bi < NB; ++bi)
#pragma unroll
    for (int bj = 0; bj < NB; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t gm = m0 + wm * (TM / 2) + bi * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        const int64_t gn = n0 + wn * (TM / 2) + bj * 32 + l32;
        if (gm < M && gn < N) C[gm * ldc + gn] -= acc[bi][bj][r];
      }
}

// C -= (Ah + Al)(Bh + Bl)^T ~ Al Bh^T + Ah Bl^T + Ah Bh^T with both operands split beforehand
// into bf16 high and low parts and stored [row][k] (k contiguous): the OBS trailing update of
// the P = 0 path, whose error block the sweep writes already split. The tiling of
// gemm_bf16x3_sub (TM x TM per workgroup, 2 x 2 waves), with two LDS stages instead of one (one
// barrier per stage) and every operand loaded as 16-byte chunks of bf16: the next stage is
// fetched into registers during the current stage's MFMAs and written to the other buffer.
template <int TM>
__global__ __launch_bounds__(256, 2) void gemm3_presplit_sub(
    int64_t M, int64_t N, int64_t K, const uint16_t* __restrict__ Ah,
    const uint16_t* __restrict__ Al, int64_t lda, const uint16_t* __restrict__ Bh,
    const uint16_t* __restrict__ Bl, int64_t ldb, float* __restrict__ C, int64_t ldc) {
  constexpr int NB = TM / 64;               // 32 x 32 blocks per wave edge (1 or 2)
  constexpr int V = TM * BK / 8 / 256;      // 16-byte chunks of each array per thread per stage
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][2][TM * RS], sB[2][2][TM * RS];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1, l32 = lane & 31, lhi = lane >> 5;
  const int64_t m0 = int64_t(blockIdx.y) * TM, n0 = int64_t(blockIdx.x) * TM;
  // this thread's 16-byte chunks: row r_v of the tile, k offset kc_v within the stage
  int64_t oa[V], ob[V];
  int so[V];
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int e = tid + 256 * v, r = e / (BK / 8), kc = (e % (BK / 8)) * 8;
    const int64_t ra = m0 + r < M ? m0 + r : M - 1, rb = n0 + r < N ? n0 + r : N - 1;
    oa[v] = ra * lda + kc;
    ob[v] = rb * ldb + kc;
    so[v] = r * RS + kc;
  }
  u32x4_t rah[V], ral[V], rbh[V], rbl[V];
  f32x16_t acc[NB][NB];
#pragma unroll
  for (int a = 0; a < NB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = f32x16_t{};
  // this lane's elements of the C tile (in the accumulator layout), requested first so that
  // their latency hides behind the whole K loop instead of ending the tile
  float cin[NB][NB][16];
#pragma unroll
  for (int bi = 0; bi < NB; ++bi)
#pragma unroll
    for (int bj = 0; bj < NB; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t gm = m0 + wm * (TM / 2) + bi * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        const int64_t gn = n0 + wn * (TM / 2) + bj * 32 + l32;
        cin[bi][bj][r] = (gm < M && gn < N) ? C[gm * ldc + gn] : 0.f;
      }
  const int nst = int(K / BK);  // even: K is a multiple of 64
#define KQ_FETCH(k0)                                                         \
  _Pragma("unroll") for (int v = 0; v < V; ++v) {                            \
    rah[v] = *reinterpret_cast<const u32x4_t*>(Ah + oa[v] + (k0));             \
    ral[v] = *reinterpret_cast<const u32x4_t*>(Al + oa[v] + (k0));             \
    rbh[v] = *reinterpret_cast<const u32x4_t*>(Bh + ob[v] + (k0));             \
    rbl[v] = *reinterpret_cast<const u32x4_t*>(Bl + ob[v] + (k0));             \
  }
#define KQ_STASH(b)                                                          \
  _Pragma("unroll") for (int v = 0; v < V; ++v) {                            \
    *reinterpret_cast<u32x4_t*>(&sA[b][0][so[v]]) = rah[v];                    \
    *reinterpret_cast<u32x4_t*>(&sA[b][1][so[v]]) = ral[v];                    \
    *reinterpret_cast<u32x4_t*>(&sB[b][0][so[v]]) = rbh[v];                    \
    *reinterpret_cast<u32x4_t*>(&sB[b][1][so[v]]) = rbl[v];                    \
  }
  // one stage from buffer B (compile-time), while the next stage (clamped to the last one at
  // the end: a harmless reload) is fetched into registers and then written to the other buffer
  auto stage = [&](auto bc, int st) {
    constexpr int B = decltype(bc)::value;
    __syncthreads();  // stage st is in LDS; the other buffer is free
    const int64_t kn = int64_t(st + 1 < nst ? st + 1 : st) * BK;
    KQ_FETCH(kn)
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int kc = ks * 16 + 8 * lhi;  // this lane's 8 k of the 16
      bf16x8_t ah[NB], al[NB], bh[NB], bl[NB];
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int m = wm * (TM / 2) + i * 32 + l32, n = wn * (TM / 2) + i * 32 + l32;
        ah[i] = *reinterpret_cast<const bf16x8_t*>(&sA[B][0][m * RS + kc]);
        al[i] = *reinterpret_cast<const bf16x8_t*>(&sA[B][1][m * RS + kc]);
        bh[i] = *reinterpret_cast<const bf16x8_t*>(&sB[B][0][n * RS + kc]);
        bl[i] = *reinterpret_cast<const bf16x8_t*>(&sB[B][1][n * RS + kc]);
      }
#pragma unroll
      for (int bi = 0; bi < NB; ++bi)
#pragma unroll
        for (int bj = 0; bj < NB; ++bj) {
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[bi], bh[bj], acc[bi][bj], 0, 0, 0);
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[bi], bl[bj], acc[bi][bj], 0, 0, 0);
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[bi], bh[bj], acc[bi][bj], 0, 0, 0);
        }
    }
    KQ_STASH(1 - B)
  };
  KQ_FETCH(0)
  KQ_STASH(0)
  for (int st = 0; st < nst; st += 2) {
    stage(std::integral_constant<int, 0>{}, st);
    stage(std::integral_constant<int, 1>{}, st + 1);
  }
#undef KQ_FETCH
#undef KQ_STASH
#pragma unroll
  for (int bi = 0; bi < NB; ++bi)
#pragma unroll
    for (int bj = 0; bj < NB; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t gm = m0 + wm * (TM / 2) + bi * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        const int64_t gn = n0 + wn * (TM / 2) + bj * 32 + l32;
        if (gm < M && gn < N) C[gm * ldc + gn] = cin[bi][bj][r] - acc[bi][bj][r];
      }
}

// Ut_hi[n][k] + Ut_lo[n][k] = sgn U[k][n] (the three-term split of +-U^T), 64 x 64 tiles
// through LDS: 16-byte loads of U rows, 8-byte stores of four bf16 of a Ut row. U is upper
// triangular (strictly, for P) and the sweep's products read Ut[n][k] only for k < n, so tiles
// wholly below that (k0 >= n0 + 64) are not written. With Fh / Fl (d a multiple of 64) the same
// values also go to a copy in MFMA-fragment order, the operand layout of the sweep's in-kernel
// updates.
__global__ __launch_bounds__(256) void split_transpose(const float* __restrict__ U, int64_t ldu,
                                                       int64_t d, uint16_t* __restrict__ Th,
                                                       uint16_t* __restrict__ Tl, int64_t ldt,
                                                       float sgn, uint16_t* __restrict__ Fh,
                                                       uint16_t* __restrict__ Fl) {
  __shared__ float t[64][65];
  const int64_t k0 = int64_t(blockIdx.y) * 64, n0 = int64_t(blockIdx.x) * 64;
  if (k0 >= n0 + 64) return;
  const int tid = threadIdx.x, q = (tid & 15) * 4, r = tid >> 4;  // 16 x 16
  const bool whole = k0 + 64 <= d && n0 + 64 <= d;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int kk = r + 16 * i;
    const int64_t k = k0 + kk, n = n0 + q;
    float4 v;
    if (whole) {
      v = *reinterpret_cast<const float4*>(U + k * ldu + n);
    } else {
      v.x = (k < d && n < d) ? U[k * ldu + n] : 0.f;
      v.y = (k < d && n + 1 < d) ? U[k * ldu + n + 1] : 0.f;
      v.z = (k < d && n + 2 < d) ? U[k * ldu + n + 2] : 0.f;
      v.w = (k < d && n + 3 < d) ? U[k * ldu + n + 3] : 0.f;
    }
    t[kk][q] = sgn * v.x, t[kk][q + 1] = sgn * v.y, t[kk][q + 2] = sgn * v.z;
    t[kk][q + 3] = sgn * v.w;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int nn = r + 16 * i;
    const int64_t n = n0 + nn, k = k0 + q;
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = t[q + e][nn];
      hi[e] = bf16_rne(x);
      lo[e] = bf16_rne(x - bf16_to_f32(hi[e]));
    }
    if (whole) {
      const uint2 h2 = make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
      const uint2 l2 = make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
      *reinterpret_cast<uint2*>(Th + n * ldt + k) = h2;
      *reinterpret_cast<uint2*>(Tl + n * ldt + k) = l2;
      if (Fh) {  // the MFMA-fragment copy (see split_frag_index)
        const int64_t f = split_frag_index(n, k, d / 16);
        *reinterpret_cast<uint2*>(Fh + f) = h2;
        *reinterpret_cast<uint2*>(Fl + f) = l2;
      }
    } else if (n < d) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (k + e < d) {
          Th[n * ldt + k + e] = uint16_t(hi[e]);
          Tl[n * ldt + k + e] = uint16_t(lo[e]);
        }
    }
  }
}

}  // namespace

int split_transpose_launch(const float* U, int64_t ldu, int64_t d, uint16_t* Th, uint16_t* Tl,
                           int64_t ldt, hipStream_t s, bool neg, uint16_t* Fh, uint16_t* Fl) {
  KQ_REQUIRE(!Fh || (Fl && d % 64 == 0), KRONQ_ERR_INVALID_ARG,
             "split_transpose: the fragment copy needs both planes and d %% 64 == 0");
  const dim3 grid(unsigned(cdiv(d, 64)), unsigned(cdiv(d, 64)));
  return launch(neg ? "obs_split_p" : "obs_split_u", split_transpose, grid, dim3(256), 0, s, U,
                ldu, d, Th, Tl, ldt, neg ? -1.f : 1.f, Fh, Fl);
}

int gemm_bf16x3_presplit_sub(int64_t M, int64_t N, int64_t K, const uint16_t* Ah,
                             const uint16_t* Al, int64_t lda, const uint16_t* Bh,
                             const uint16_t* Bl, int64_t ldb, float* C, int64_t ldc,
                             hipStream_t s, const char* name) {
  if (M <= 0 || N <= 0 || K <= 0) return KRONQ_OK;
  KQ_REQUIRE(K % (2 * BK) == 0 && lda % 8 == 0 && ldb % 8 == 0 && aligned(Ah, 16) &&
                 aligned(Al, 16) && aligned(Bh, 16) && aligned(Bl, 16),
             KRONQ_ERR_INVALID_ARG,
             "gemm_bf16x3_presplit_sub: K %% 64, lda %% 8, ldb %% 8 and 16-byte operands needed");
  if (cdiv(M, 128) * cdiv(N, 128) >= 192) {
    const dim3 grid(unsigned(cdiv(N, 128)), unsigned(cdiv(M, 128)));
    return launch(name, gemm3_presplit_sub<128>, grid, dim3(256), 0, s, M, N, K, Ah, Al, lda, Bh,
                  Bl, ldb, C, ldc);
  }
  const dim3 grid(unsigned(cdiv(N, 64)), unsigned(cdiv(M, 64)));
  return launch(name, gemm3_presplit_sub<64>, grid, dim3(256), 0, s, M, N, K, Ah, Al, lda, Bh,
                Bl, ldb, C, ldc);
}

int gemm_bf16x3_sub(int64_t M, int64_t N, const Bf16x3Pair& p1, const Bf16x3Pair& p2, float* C,
                    int64_t ldc, hipStream_t s, const char* name) {
  if (M <= 0 || N <= 0 || p1.K + p2.K <= 0) return KRONQ_OK;
  KQ_REQUIRE(p1.K % BK == 0 && p1.lda % 4 == 0 && p1.ldb % 8 == 0 && p2.K % BK == 0 &&
                 (p2.K == 0 || (p2.lda % 4 == 0 && p2.ldb % 8 == 0)),
             KRONQ_ERR_INVALID_ARG, "gemm_bf16x3_sub: K %% 32, lda %% 4 and ldb %% 8 must be 0");
  if (cdiv(M, 128) * cdiv(N, 128) >= 192) {
    const dim3 grid(unsigned(cdiv(N, 128)), unsigned(cdiv(M, 128)));
    return launch(name, gemm_bf16x3_sub<128>, grid, dim3(256), 0, s, M, N, p1.K, p1.A, p1.lda,
                  p1.Bh, p1.Bl, p1.ldb, p2.K, p2.A, p2.lda, p2.Bh, p2.Bl, p2.ldb, C, ldc);
  }
  const dim3 grid(unsigned(cdiv(N, 64)), unsigned(cdiv(M, 64)));
  return launch(name, gemm_bf16x3_sub<64>, grid, dim3(256), 0, s, M, N, p1.K, p1.A, p1.lda, p1.Bh,
                p1.Bl, p1.ldb, p2.K, p2.A, p2.lda, p2.Bh, p2.Bl, p2.ldb, C, ldc);
}

}  // namespace kq
