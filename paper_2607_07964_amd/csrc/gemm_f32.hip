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
// Problems too small to give the 128 x 128 kernel enough workgroups (the short products of the
// recursive Cholesky) use gemm_f32_small: a 32 x 32 or 64 x 64 tile per workgroup, K staged 64
// at a time through LDS, and for 32 x 32 tiles each stage's K split over the four waves (the
// partial blocks are summed through LDS at the end). The dispatcher takes the largest tile that
// still gives at least 128 workgroups.
#include <algorithm>

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
  if ((flags & GEMM_UPPER_C) && n0 + GT <= m0) return;  // tile strictly below the diagonal

  int64_t kbeg = 0, kend = K;
  if (flags & GEMM_B_LOWER) kbeg = (n0 / GK) * GK;  // B[k][n] = 0 for k < n
  if ((flags & GEMM_A_UPPER) && m0 > kbeg) kbeg = (m0 / GK) * GK;  // A[m][k] = 0 for k < m
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


// Small-tile variant (see the file comment). A, B and C must not overlap.
template <int TM>
__global__ __launch_bounds__(256) void gemm_f32_small(int flags, int64_t M, int64_t N, int64_t K,
                                                      float alpha, const float* __restrict__ A,
                                                      int64_t lda, const float* __restrict__ B,
                                                      int64_t ldb, float beta,
                                                      float* __restrict__ C, int64_t ldc) {
  constexpr int KC = 64;                      // K per stage
  constexpr int NB32 = TM / 32;               // 32 x 32 blocks per tile edge
  constexpr int SK = 4 / (NB32 * NB32);       // waves per block (split of each stage's K)
  constexpr int KW = KC / SK;                 // K per wave per stage
  constexpr int AS = KC + 1;                  // LDS row stride of the A tile, [m][k]
  constexpr int BS = TM == 32 ? 32 : 96;      // LDS row stride of the B tile, [k][n]
  constexpr int NV = TM * KC / 1024;          // float4 per thread per operand per stage
  __shared__ float sA[TM * AS];
  __shared__ float sB[KC * BS];
  __shared__ float red[(SK - 1) * 1024 + 1];
  const int tid = threadIdx.x;
  const int64_t m0 = int64_t(blockIdx.y) * TM, n0 = int64_t(blockIdx.x) * TM;
  if ((flags & GEMM_LOWER_C) && m0 + TM <= n0) return;
  if ((flags & GEMM_UPPER_C) && n0 + TM <= m0) return;
  int64_t kbeg = 0, kend = K;
  if (flags & GEMM_B_LOWER) kbeg = n0;
  if ((flags & GEMM_A_UPPER) && m0 > kbeg) kbeg = m0;
  if ((flags & GEMM_A_LOWER) && m0 + TM < kend) kend = m0 + TM;
  if ((flags & GEMM_OPB_UPPER) && n0 + TM < kend) kend = n0 + TM;
  const bool a_kc = !(flags & GEMM_TA), b_kc = (flags & GEMM_TB);
  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, lhi = lane >> 5;
  const int blk = wave % (NB32 * NB32), part = wave / (NB32 * NB32);
  const int bm = (blk / NB32) * 32, bn = (blk % NB32) * 32;

  float4 ra[NV], rb[NV];
  // load 4 consecutive elements X[r][c..c+3] (row stride ldx) with bounds rows < R, cols < Cn
  auto ld4 = [](const float* X, int64_t ldx, int64_t r, int64_t c, int64_t R, int64_t Cn) {
    if (r < R && c + 4 <= Cn) return *reinterpret_cast<const float4*>(X + r * ldx + c);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < R) {
      if (c < Cn) v.x = X[r * ldx + c];
      if (c + 1 < Cn) v.y = X[r * ldx + c + 1];
      if (c + 2 < Cn) v.z = X[r * ldx + c + 2];
      if (c + 3 < Cn) v.w = X[r * ldx + c + 3];
    }
    return v;
  };
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int e = tid + 256 * v;
      if (a_kc) {  // A[m][k]
        const int m = e / (KC / 4), k4 = (e % (KC / 4)) * 4;
        ra[v] = ld4(A, lda, m0 + m, k0 + k4, M, kend);
      } else {     // A stored [k][m]
        const int k = e / (TM / 4), m4 = (e % (TM / 4)) * 4;
        ra[v] = (k0 + k < kend) ? ld4(A, lda, k0 + k, m0 + m4, K, M) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      if (b_kc) {  // B stored [n][k]
        const int n = e / (KC / 4), k4 = (e % (KC / 4)) * 4;
        rb[v] = ld4(B, ldb, n0 + n, k0 + k4, N, kend);
      } else {     // B[k][n]
        const int k = e / (TM / 4), n4 = (e % (TM / 4)) * 4;
        rb[v] = (k0 + k < kend) ? ld4(B, ldb, k0 + k, n0 + n4, K, N) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int e = tid + 256 * v;
      const float x[4] = {ra[v].x, ra[v].y, ra[v].z, ra[v].w};
      const float z[4] = {rb[v].x, rb[v].y, rb[v].z, rb[v].w};
      if (a_kc) {
        const int m = e / (KC / 4), k4 = (e % (KC / 4)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) sA[m * AS + k4 + c] = x[c];
      } else {
        const int k = e / (TM / 4), m4 = (e % (TM / 4)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) sA[(m4 + c) * AS + k] = x[c];
      }
      if (b_kc) {
        const int n = e / (KC / 4), k4 = (e % (KC / 4)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) sB[(k4 + c) * BS + n] = z[c];
      } else {
        const int k = e / (TM / 4), n4 = (e % (TM / 4)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) sB[k * BS + n4 + c] = z[c];
      }
    }
  };

  f32x16_t acc = f32x16_t{};
  if (kbeg < kend) fetch(kbeg);
  for (int64_t k0 = kbeg; k0 < kend; k0 += KC) {
    __syncthreads();
    stash();
    __syncthreads();
    if (k0 + KC < kend) fetch(k0 + KC);
#pragma unroll
    for (int s2 = 0; s2 < KW / 2; ++s2) {
      const int kk = part * KW + 2 * s2 + lhi;
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sA[(bm + l32) * AS + kk], sB[kk * BS + bn + l32],
                                                 acc, 0, 0, 0);
    }
  }
  if (SK > 1) {
    if (part > 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(part - 1) * 1024 + r * 64 + lane] = acc[r];
    }
    __syncthreads();
    if (part > 0) return;
#pragma unroll
    for (int p = 0; p < SK - 1; ++p)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] += red[p * 1024 + r * 64 + lane];
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t gm = m0 + bm + 8 * (r >> 2) + 4 * lhi + (r & 3), gn = n0 + bn + l32;
    if (gm < M && gn < N) {
      float* c = C + gm * ldc + gn;
      const float x = alpha * acc[r];
      *c = beta == 0.f ? x : x + beta * *c;
    }
  }
}

}  // namespace

int gemm_f32(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
             int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
             hipStream_t s, const char* name) {
  if (M <= 0 || N <= 0) return KRONQ_OK;
  // workgroups that do work for a tile edge t (LOWER_C drops the tiles above the diagonal,
  // UPPER_C those below it)
  auto work = [&](int64_t t) {
    const int64_t tm = cdiv(M, t), tn = cdiv(N, t);
    if (!(flags & (GEMM_LOWER_C | GEMM_UPPER_C))) return tm * tn;
    int64_t c = 0;
    for (int64_t i = 0; i < tm; ++i)
      c += (flags & GEMM_LOWER_C) ? std::min(tn, i + 1) : std::max<int64_t>(0, tn - i);
    return c;
  };
  if (work(GT) >= 128) {
    const dim3 grid(unsigned(cdiv(N, GT)), unsigned(cdiv(M, GT)));
    return launch(name, gemm_f32_mfma, grid, dim3(256), 0, s, flags, M, N, K, alpha, A, lda, B,
                  ldb, beta, C, ldc);
  }
  if (work(64) >= 128) {
    const dim3 grid(unsigned(cdiv(N, 64)), unsigned(cdiv(M, 64)));
    return launch(name, gemm_f32_small<64>, grid, dim3(256), 0, s, flags, M, N, K, alpha, A, lda,
                  B, ldb, beta, C, ldc);
  }
  const dim3 grid(unsigned(cdiv(N, 32)), unsigned(cdiv(M, 32)));
  return launch(name, gemm_f32_small<32>, grid, dim3(256), 0, s, flags, M, N, K, alpha, A, lda, B,
                ldb, beta, C, ldc);
}

}  // namespace kq
