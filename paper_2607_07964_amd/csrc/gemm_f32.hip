// fp32 GEMM on the fp32 matrix cores (v_mfma_f32_32x32x2f32): C = alpha op(A) op(B) + beta C.
//
// Used where the path needs fp32-accurate dense products: the trailing updates of the
// Cholesky factorisation and of the triangular inverse, the lazy-block OBS update, and the
// two products of the K-FAC loss.
//   * 128 x 128 output tile per workgroup, 4 waves in a 2 x 2 grid, each wave 64 x 64 =
//     2 x 2 MFMA blocks (64 fp32 accumulators per lane).
//   * K advances 16 at a time through LDS stored k-major ([k][m], [k][n]) so that every MFMA
//     operand is one 4-byte LDS read by 32 consecutive lanes; the row stride of 160 floats puts
//     the two k rows a wave reads at once in disjoint bank halves.
//   * The next K chunk is fetched into registers while the current one is multiplied.
//   * Triangular flags skip tiles or K ranges that are known to be zero or unused.
#include "kq_common.hpp"

namespace kq {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int GT = 128;    // tile edge
constexpr int GK = 16;     // K per stage
constexpr int GLD = 160;   // LDS row stride (floats)

struct Frag {
  float v[8];
};

// Fetch an operand chunk: 16 (k) x 128 (m) elements of op(X), 8 per thread.
// trans == false: X[m][k] (k contiguous); trans == true: X[k][m] (m contiguous).
__device__ __forceinline__ void fetch(Frag& f, const float* X, int64_t ldx,
                                      bool kcontig, int64_t m0, int64_t k0, int64_t M, int64_t K,
                                      int tid) {
  if (kcontig) {
    const int m = tid >> 1, kb = (tid & 1) * 8;
    const int64_t gm = m0 + m;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t gk = k0 + kb + h * 4;
      if (gm < M && gk + 4 <= K) {
        const float4 x = *reinterpret_cast<const float4*>(X + gm * ldx + gk);
        f.v[h * 4 + 0] = x.x;
        f.v[h * 4 + 1] = x.y;
        f.v[h * 4 + 2] = x.z;
        f.v[h * 4 + 3] = x.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          f.v[h * 4 + e] = (gm < M && gk + e < K) ? X[gm * ldx + gk + e] : 0.f;
      }
    }
  } else {
    const int k = tid >> 4, mb = (tid & 15) * 8;
    const int64_t gk = k0 + k;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t gm = m0 + mb + h * 4;
      if (gk < K && gm + 4 <= M) {
        const float4 x = *reinterpret_cast<const float4*>(X + gk * ldx + gm);
        f.v[h * 4 + 0] = x.x;
        f.v[h * 4 + 1] = x.y;
        f.v[h * 4 + 2] = x.z;
        f.v[h * 4 + 3] = x.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          f.v[h * 4 + e] = (gk < K && gm + e < M) ? X[gk * ldx + gm + e] : 0.f;
      }
    }
  }
}

// Store the fetched chunk k-major into LDS: s[k][m].
__device__ __forceinline__ void stash(float* __restrict__ s, const Frag& f, bool kcontig,
                                      int tid) {
  if (kcontig) {
    const int m = tid >> 1, kb = (tid & 1) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) s[(kb + e) * GLD + m] = f.v[e];
  } else {
    const int k = tid >> 4, mb = (tid & 15) * 8;
    *reinterpret_cast<float4*>(s + k * GLD + mb) = make_float4(f.v[0], f.v[1], f.v[2], f.v[3]);
    *reinterpret_cast<float4*>(s + k * GLD + mb + 4) = make_float4(f.v[4], f.v[5], f.v[6], f.v[7]);
  }
}

__global__ __launch_bounds__(256, 2) void gemm_f32_mfma(int flags, int64_t M, int64_t N,
                                                        int64_t K, float alpha,
                                                        const float* A, int64_t lda,
                                                        const float* B, int64_t ldb,
                                                        float beta, float* C,
                                                        int64_t ldc) {
  // A, B and C may overlap (in-place panel solves): all loads of A and B precede the stores,
  // and each workgroup reads only the rows/columns it writes.
  __shared__ float sA[GK * GLD];
  __shared__ float sB[GK * GLD];
  const int tid = threadIdx.x;
  const int64_t m0 = int64_t(blockIdx.y) * GT, n0 = int64_t(blockIdx.x) * GT;
  if ((flags & GEMM_LOWER_C) && m0 + GT <= n0) return;  // tile strictly above the diagonal

  int64_t kbeg = 0, kend = K;
  if (flags & GEMM_B_LOWER) kbeg = (n0 / GK) * GK;  // B[k][n] = 0 for k < n
  if ((flags & GEMM_A_LOWER) && m0 + GT < kend) kend = m0 + GT;  // A[m][k] = 0 for k > m
  if ((flags & GEMM_OPB_UPPER) && n0 + GT < kend) kend = n0 + GT;  // op(B)[k][n] = 0, k > n

  const bool a_kc = !(flags & GEMM_TA);  // A[m][k] row-major: k contiguous
  const bool b_kc = (flags & GEMM_TB);   // B^T stored [n][k]: k contiguous
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, lhi = lane >> 5;

  f32x16_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16_t{};

  Frag fa, fb;
  if (kbeg < kend) {
    fetch(fa, A, lda, a_kc, m0, kbeg, M, kend, tid);
    fetch(fb, B, ldb, b_kc, n0, kbeg, N, kend, tid);
  }
  for (int64_t k0 = kbeg; k0 < kend; k0 += GK) {
    __syncthreads();
    stash(sA, fa, a_kc, tid);
    stash(sB, fb, b_kc, tid);
    __syncthreads();
    if (k0 + GK < kend) {
      fetch(fa, A, lda, a_kc, m0, k0 + GK, M, kend, tid);
      fetch(fb, B, ldb, b_kc, n0, k0 + GK, N, kend, tid);
    }
#pragma unroll
    for (int kk = 0; kk < GK / 2; ++kk) {
      const int kr = 2 * kk + lhi;
      float av[2], bv[2];
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) av[bi] = sA[kr * GLD + wm * 64 + bi * 32 + l32];
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) bv[bj] = sB[kr * GLD + wn * 64 + bj * 32 + l32];
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[bi], bv[bj], acc[bi][bj], 0, 0, 0);
    }
  }

#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t gm = m0 + wm * 64 + bi * 32 + (r >> 2) * 8 + lhi * 4 + (r & 3);
        const int64_t gn = n0 + wn * 64 + bj * 32 + l32;
        if (gm < M && gn < N) {
          float* c = C + gm * ldc + gn;
          const float x = alpha * acc[bi][bj][r];
          *c = beta == 0.f ? x : x + beta * *c;
        }
      }
}

}  // namespace

int gemm_f32(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
             int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
             hipStream_t s, const char* name) {
  if (M <= 0 || N <= 0) return KRONQ_OK;
  const dim3 grid(unsigned(cdiv(N, GT)), unsigned(cdiv(M, GT)));
  return launch(name, gemm_f32_mfma, grid, dim3(256), 0, s, flags, M, N, K, alpha, A, lda, B,
                ldb, beta, C, ldc);
}

}  // namespace kq
