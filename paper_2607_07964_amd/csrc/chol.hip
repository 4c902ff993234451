// Damping and the inverse-Cholesky factor (Alg. 2 first two lines; Prop. 1 uses rows of it).
//
// inv(H~) = U^T U with U upper. With J the index reversal, J H~ J = L L^T (ordinary lower
// Cholesky) gives H~ = (J L J)(J L J)^T, so U = (J L J)^-1 = J L^-1 J. Steps:
//   1. damping: H~ = H + damp * mean(diag H) * I (in place), M = J H~ J (workspace copy);
//   2. L and X = L^-1 together, recursively on [[M11, .], [M21, M22]] split at a multiple of 128:
//        factor and invert M11 (X11 = L11^-1);
//        L21 = M21 X11^T                  (written to the X21 slot, which is still free);
//        M22 -= L21 L21^T                 (lower tiles only) and T = L21 X11 (scratch kept
//                                          until the last step), both in one launch;
//        factor and invert M22 (X22);
//        X21 = -X22 T                     (over L21).
//      Leaves of at most 128 columns are factored and inverted in LDS by one workgroup; every
//      other step is a fp32 MFMA GEMM, so the large updates have a long K. Three dependent
//      launches per split: the chain of small ones, not the flops, sets the time at d = 4096;
//   3. U[i][j] = X[d-1-i][d-1-j] for i <= j, 0 below the diagonal.
// A non-positive pivot sets *info to its 1-based column in the original order (first failure).
#include <algorithm>
#include <cmath>

#include "kq_common.hpp"

namespace kq {
namespace {

constexpr int NB = 128;
constexpr int DLD = NB + 1;  // LDS leading dimension of the diagonal block

__global__ __launch_bounds__(256) void diag_shift(const float* __restrict__ H, int64_t d,
                                                  int64_t ldh, float damp, float* __restrict__ shift,
                                                  int* __restrict__ info) {
  __shared__ double red[256];
  const int tid = threadIdx.x;
  double s = 0.0;
  for (int64_t i = tid; i < d; i += 256) s += H[i * ldh + i];
  red[tid] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    *shift = float(double(damp) * (red[0] / double(d)));
    *info = 0;
  }
}

__global__ void add_diag(float* __restrict__ H, int64_t d, int64_t ldh,
                         const float* __restrict__ shift) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < d) H[i * ldh + i] += *shift;
}

// M[i][j] = H[d-1-i][d-1-j]
__global__ void reverse_copy(const float* __restrict__ H, int64_t d, int64_t ldh,
                             float* __restrict__ M, int64_t ldm) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < d;
       j += int64_t(gridDim.x) * blockDim.x)
    M[i * ldm + j] = H[(d - 1 - i) * ldh + (d - 1 - j)];
}

// the same with four columns per thread (d divisible by 4; rows 16-byte aligned)
__global__ void reverse_copy4(const float* __restrict__ H, int64_t d, int64_t ldh,
                              float* __restrict__ M, int64_t ldm) {
  const int64_t i = blockIdx.y;
  for (int64_t j = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) * 4; j < d;
       j += int64_t(gridDim.x) * blockDim.x * 4) {
    const float4 h = *reinterpret_cast<const float4*>(H + (d - 1 - i) * ldh + (d - 4 - j));
    *reinterpret_cast<float4*>(M + i * ldm + j) = make_float4(h.w, h.z, h.y, h.x);
  }
}

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// One 32 x 32 block C = alpha * A op(B) + beta * C on LDS arrays, by one wave on the fp32
// matrix cores (v_mfma_f32_32x32x2f32, two k per instruction). A is 32 x k (row stride lda);
// op(B) is k x 32: B[k][n] at B[k * ldb + n], or with bt, B^T with (k, n) at B[n * ldb + k].
// k is even. The caller orders the LDS traffic (a wave's LDS accesses complete in order).
__device__ __forceinline__ void mfma_block(float* C, int ldc, const float* A, int lda,
                                           const float* B, int ldb, bool bt, int k, float alpha,
                                           float beta, int lane) {
  const int l32 = lane & 31, lhi = lane >> 5;
  f32x16_t acc = {};
  for (int k0 = 0; k0 < k; k0 += 2) {
    const float av = A[l32 * lda + k0 + lhi];
    const float bv = bt ? B[l32 * ldb + k0 + lhi] : B[(k0 + lhi) * ldb + l32];
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float* c = C + (8 * (r >> 2) + 4 * lhi + (r & 3)) * ldc + l32;
    *c = beta == 0.f ? alpha * acc[r] : alpha * acc[r] + beta * *c;
  }
}

// One 32-column panel of the diagonal-block factorisation (see potrf_diag), by one wave.
template <int c0>
__device__ __forceinline__ void panel_factor(float* a, float* colbuf, float* dummy, int64_t kb,
                                             int64_t d, int* info, int lane) {
  {
    const int r0 = c0 + lane, r1 = c0 + 64 + lane;
    const bool ok0 = r0 < NB, ok1 = r1 < NB;  // r1 < NB only for c0 < 64
    float v0[32], v1[32];
    int first_bad = 32;  // first column of the panel with a non-positive pivot
    // lanes past the last row work on a copy of row NB - 1 (never stored): no divergent loads
    const int q0 = ok0 ? r0 : NB - 1, q1 = ok1 ? r1 : NB - 1;
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      v0[k] = a[q0 * DLD + c0 + k];
      v1[k] = c0 < 64 ? a[q1 * DLD + c0 + k] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      colbuf[lane] = v0[j];  // every lane stores (no branch); entries 0..31 are read
      float raw[32];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float4 t = reinterpret_cast<const float4*>(colbuf)[q];
        raw[4 * q] = t.x, raw[4 * q + 1] = t.y, raw[4 * q + 2] = t.z, raw[4 * q + 3] = t.w;
      }
      const float piv = raw[j];
      if (!(piv > 0.f) && first_bad == 32) first_bad = j;  // also catches NaN; a select
      const float rl = __builtin_amdgcn_rsqf(piv);  // pivots are normal or the factor fails
      const float ljj = piv * rl;
      const float l0 = v0[j] * rl, l1 = v1[j] * rl;
      // A[i][k] -= L[i][j] L[k][j] = (l_i rl) raw_k
      const float g0 = l0 * rl, g1 = l1 * rl;
#pragma unroll
      for (int k = j + 1; k < 32; ++k) {
        v0[k] = fmaf(-g0, raw[k], v0[k]);
        if (c0 < 64) v1[k] = fmaf(-g1, raw[k], v1[k]);
      }
      v0[j] = lane > j ? l0 : (lane == j ? ljj : 0.f);
      v1[j] = l1;
    }
    // unconditional stores (a divergent branch here would make the compiler sink the row
    // updates into it): rows past the end go to a dummy area of the idle product scratch
    const int dummy_off = int(dummy - a) + lane * 33;  // same LDS array: an index select
    float* d0 = a + (ok0 ? r0 * DLD + c0 : dummy_off);
    float* d1 = a + (ok1 ? r1 * DLD + c0 : dummy_off);
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      d0[k] = v0[k];
      if (c0 < 64) d1[k] = v1[k];
    }
    if (lane == 0 && first_bad < 32 && kb + c0 + first_bad < d)
      atomicCAS(info, 0, int(d - (kb + c0 + first_bad)));
  }
}

// A[bi][bj] -= L[bi][p] L[bj][p]^T for 32 x 32 blocks of the diagonal block, one wave
__device__ __forceinline__ void upd_block(float* a, int bi, int bj, int p, int lane) {
  mfma_block(a + 32 * bi * DLD + 32 * bj, DLD, a + 32 * bi * DLD + 32 * p, DLD,
             a + 32 * bj * DLD + 32 * p, DLD, true, 32, -1.f, 1.f, lane);
}

// Y_pp = L_pp^-1 for the 32 x 32 diagonal block p, one wave: lane c solves column c by forward
// substitution (a multiplication by the reciprocal of L_ii, not a division)
__device__ __forceinline__ void inv_block(const float* a, float* y, int p,
                                          int lane) {
  const int b0 = 32 * p;
  if (lane < 32) {
    float x[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      float s = (i == lane) ? 1.f : 0.f;
#pragma unroll
      for (int k = 0; k < i; ++k) s = fmaf(-a[(b0 + i) * DLD + b0 + k], x[k], s);
      x[i] = s * __builtin_amdgcn_rcpf(a[(b0 + i) * DLD + b0 + i]);
      __builtin_amdgcn_sched_barrier(0);  // read one row of L at a time
    }
#pragma unroll
    for (int i = 0; i < 32; ++i) y[(b0 + i) * DLD + b0 + lane] = x[i];
  }
}

// Factor the diagonal block M[kb:kb+bs, kb:kb+bs] (lower) and invert the factor, one workgroup.
// The block is padded to 128 x 128 with the identity, so a partial block needs no special case.
// Factorisation, in four 32-column panels:
//   * panel: wave 0 factors the panel for every row at or below it; lane l keeps rows c0 + l
//     and c0 + 64 + l (32 panel entries each) in registers. Column j of the panel's diagonal
//     rows is published once through a 64-float LDS buffer and read back as broadcasts, and the
//     1 / L_jj scaling is folded into the per-row coefficient, so each column costs one LDS
//     round trip and one FMA per remaining entry;
//   * rank-32 updates of the lower 32 x 32 blocks right of the panel (MFMA), the next panel's
//     block column first; the rest, and the inverse of the panel's diagonal block, run on the
//     other waves while wave 0 factors the next panel.
// Inverse Y = L^-1 by recursive doubling, inv([[A, 0], [B, C]]) = [[A^-1, 0], [-C^-1 B A^-1, C^-1]]:
//   32 x 32 diagonal blocks (one wave each, columns by forward substitution), then 64, then 128.
// Writes Linv_kk, with exact zeros above the diagonal, to X (M itself is left as read).
__global__ __launch_bounds__(256) void potrf_diag(const float* __restrict__ M, int64_t ldm,
                                                  int64_t kb, int bs, int64_t d,
                                                  float* __restrict__ X, int* __restrict__ info) {
  __shared__ __attribute__((aligned(16))) float lds[2 * NB * DLD + 64 * 68];
  float* const a = lds;                 // the block, becomes L (lower part meaningful)
  float* const y = lds + NB * DLD;      // Y = L^-1
  float* const tb = lds + 2 * NB * DLD; // product scratch (a dummy store target in the panels)
  __shared__ __attribute__((aligned(16))) float colbuf[64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: per-wave branches
  const bool full = bs == NB;
  if (full) {
    float4 q[NB * NB / 1024];
#pragma unroll
    for (int it = 0; it < NB * NB / 1024; ++it) {
      const int e = tid + 256 * it, i = e >> 5, j = (e & 31) * 4;
      q[it] = *reinterpret_cast<const float4*>(M + (kb + i) * ldm + kb + j);
    }
#pragma unroll
    for (int it = 0; it < NB * NB / 1024; ++it) {
      const int e = tid + 256 * it, i = e >> 5, j = (e & 31) * 4;
      a[i * DLD + j] = q[it].x, a[i * DLD + j + 1] = q[it].y;
      a[i * DLD + j + 2] = q[it].z, a[i * DLD + j + 3] = q[it].w;
    }
  } else {
    for (int e = tid; e < NB * NB; e += 256) {
      const int i = e >> 7, j = e & 127;
      a[i * DLD + j] = (i < bs && j < bs) ? M[(kb + i) * ldm + kb + j] : (i == j ? 1.f : 0.f);
    }
  }
  // upper 32-blocks of Y that the doubling reads as operands: (0, 1) and (2, 3)
  for (int e = tid; e < 2 * 32 * 32; e += 256) {
    const int o = (e >> 10) * 64, i = (e >> 5) & 31, j = e & 31;
    y[(o + i) * DLD + o + 32 + j] = 0.f;
  }
  __syncthreads();
  // Panels with a one-block lookahead: before panel p + 1 its block column gets panel p's
  // update from all waves; then wave 0 factors panel p + 1 while the other waves apply panel
  // p's update to the blocks further right and invert the diagonal block of panel p.
  if (wave == 0) panel_factor<0>(a, colbuf, tb, kb, d, info, lane);
  __syncthreads();
  if (wave < 3) upd_block(a, 1 + wave, 1, 0, lane);  // block column 1 from panel 0
  __syncthreads();
  if (wave == 0) {
    panel_factor<32>(a, colbuf, tb, kb, d, info, lane);
  } else if (wave == 1) {
    inv_block(a, y, 0, lane);
  } else if (wave == 2) {
    upd_block(a, 2, 2, 0, lane);
    upd_block(a, 3, 3, 0, lane);
  } else {
    upd_block(a, 3, 2, 0, lane);
  }
  __syncthreads();
  if (wave < 2) upd_block(a, 2 + wave, 2, 1, lane);  // block column 2 from panel 1
  __syncthreads();
  if (wave == 0) {
    panel_factor<64>(a, colbuf, tb, kb, d, info, lane);
  } else if (wave == 1) {
    inv_block(a, y, 1, lane);
  } else if (wave == 2) {
    upd_block(a, 3, 3, 1, lane);
  }
  __syncthreads();
  if (wave == 0) upd_block(a, 3, 3, 2, lane);  // block column 3 from panel 2
  __syncthreads();
  if (wave == 0) {
    panel_factor<96>(a, colbuf, tb, kb, d, info, lane);
  } else if (wave == 1) {
    inv_block(a, y, 2, lane);
  }
  __syncthreads();
  if (wave == 0) inv_block(a, y, 3, lane);
  __syncthreads();
  // 64: Y10 = -Y11 (L10 Y00) for the block pairs at 0 and 64, one wave each
  if (wave < 2) {
    const int o = wave * 64;
    float* T = tb + wave * 32 * 33;
    mfma_block(T, 33, a + (o + 32) * DLD + o, DLD, y + o * DLD + o, DLD, false, 32, 1.f, 0.f,
               lane);
    mfma_block(y + (o + 32) * DLD + o, DLD, y + (o + 32) * DLD + o + 32, DLD, T, 33, false, 32,
               -1.f, 0.f, lane);
  }
  __syncthreads();
  // 128: Y[64:, :64] = -Y[64:, 64:] (L[64:, :64] Y[:64, :64]), one 32-block per wave
  {
    const int bi = wave >> 1, bj = wave & 1;
    mfma_block(tb + 32 * bi * 68 + 32 * bj, 68, a + (64 + 32 * bi) * DLD, DLD, y + 32 * bj, DLD,
               false, 64, 1.f, 0.f, lane);
    __syncthreads();
    mfma_block(y + (64 + 32 * bi) * DLD + 32 * bj, DLD, y + (64 + 32 * bi) * DLD + 64, DLD,
               tb + 32 * bj, 68, false, 64, -1.f, 0.f, lane);
  }
  __syncthreads();
  if (full) {
#pragma unroll 4
    for (int it = 0; it < NB * NB / 1024; ++it) {
      const int e = tid + 256 * it, i = e >> 5, j = (e & 31) * 4;
      float v[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) v[c] = (j + c <= i) ? y[i * DLD + j + c] : 0.f;
      *reinterpret_cast<float4*>(X + (kb + i) * ldm + kb + j) = make_float4(v[0], v[1], v[2], v[3]);
    }
  } else {
    for (int e = tid; e < bs * NB; e += 256) {
      const int i = e >> 7, j = e & 127;
      if (j < bs) X[(kb + i) * ldm + kb + j] = (j <= i) ? y[i * DLD + j] : 0.f;
    }
  }
}

// U[i][j] = X[d-1-i][d-1-j] for i <= j, else 0
__global__ void reverse_out(const float* __restrict__ X, int64_t ldm, int64_t d,
                            float* __restrict__ U, int64_t ldu) {
  const int64_t i = blockIdx.y;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < d;
       j += int64_t(gridDim.x) * blockDim.x)
    U[i * ldu + j] = (j >= i) ? X[(d - 1 - i) * ldm + (d - 1 - j)] : 0.f;
}

// the same with four columns per thread (d divisible by 4; rows 16-byte aligned)
__global__ void reverse_out4(const float* __restrict__ X, int64_t ldm, int64_t d,
                             float* __restrict__ U, int64_t ldu) {
  const int64_t i = blockIdx.y;
  for (int64_t j = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) * 4; j < d;
       j += int64_t(gridDim.x) * blockDim.x * 4) {
    const float4 x = *reinterpret_cast<const float4*>(X + (d - 1 - i) * ldm + (d - 4 - j));
    *reinterpret_cast<float4*>(U + i * ldu + j) =
        make_float4(j >= i ? x.w : 0.f, j + 1 >= i ? x.z : 0.f, j + 2 >= i ? x.y : 0.f,
                    j + 3 >= i ? x.x : 0.f);
  }
}

int64_t ld_for(int64_t d) { return ((d + 63) / 64) * 64; }

// split of an n-column block: the first h columns, a multiple of NB, about half
int64_t split_at(int64_t n) { return (cdiv(n, NB) / 2) * NB; }

// Scratch floats the recursion below needs for an n-column block: a node keeps its product
// T (r x h) until its last step, while the second child's recursion runs after it.
int64_t chol_scratch(int64_t n) {
  if (n <= NB) return 0;
  const int64_t h = split_at(n), r = n - h;
  return std::max(chol_scratch(h), r * h + chol_scratch(r));
}

// Products of at least this many multiply-adds run on the bf16 matrix cores with the six-term
// split (gemm_f32_split6, as accurate as fp32): the 3584-order and larger products of the top
// levels of an 8192 or larger factorisation. Below that (2048-order products and smaller, too
// few 256 x 128 tiles to fill the chip) the fp32 kernels are faster.
constexpr double SPLIT6_MIN = 3000.0 * 3000.0 * 3000.0;

bool use_split6(int flags, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                const float* B, int64_t ldb) {
  return double(M) * double(N) * double(K) >= SPLIT6_MIN &&
         gemm_split6_supports(flags, M, N, K, A, lda, B, ldb);
}

// one product of the recursion: the split path when it is large enough, else the fp32 kernels
int chol_gemm(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
              int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
              hipStream_t s, const char* name) {
  if (use_split6(flags, M, N, K, A, lda, B, ldb))
    return gemm_f32_split6(flags, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, s, name);
  return gemm_f32(flags, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, s, name);
}

// L and L^-1 of the block [n0, n0 + n) of M; the lower part of the same block of X receives
// L^-1 (zeros on the upper part of the diagonal leaves). T is scratch of tcap floats (at least
// chol_scratch(n)).
int chol_rec(float* M, float* X, float* T, int64_t tcap, int64_t ld, int64_t n0, int64_t n,
             int64_t d, int* info, hipStream_t s) {
  if (n <= NB)
    return launch("chol_potrf_diag", potrf_diag, dim3(1), dim3(256), 0, s,
                  static_cast<const float*>(M), ld, n0, int(n), d, X, info);
  const int64_t h = split_at(n), r = n - h;
  KQ_REQUIRE(r * h <= tcap, KRONQ_ERR_WORKSPACE, "chol_rec: scratch too small");
  KQ_TRY(chol_rec(M, X, T, tcap, ld, n0, h, d, info, s));
  const float* M21 = M + (n0 + h) * ld + n0;
  const float* X11 = X + n0 * ld + n0;
  float* X21 = X + (n0 + h) * ld + n0;
  float* X22 = X + (n0 + h) * ld + n0 + h;
  float* M22 = M + (n0 + h) * ld + n0 + h;
  // L21 = M21 X11^T (op(B) = X11^T is upper triangular)
  KQ_TRY(chol_gemm(GEMM_TB | GEMM_OPB_UPPER, r, h, h, 1.f, M21, ld, X11, ld, 0.f, X21, ld, s,
                   "chol_trsm"));
  // M22 -= L21 L21^T (lower tiles only) and T = L21 X11 (X11 lower triangular), in one launch
  // (both need only L21 and X11)
  const GemmProb syrk{GEMM_TB | GEMM_LOWER_C, r, r, h, -1.f, X21, ld, X21, ld, 1.f, M22, ld};
  const GemmProb row{GEMM_B_LOWER, r, h, h, 1.f, X21, ld, X11, ld, 0.f, T, h};
  if (use_split6(syrk.flags, r, r, h, X21, ld, X21, ld) &&
      use_split6(row.flags, r, h, h, X21, ld, X11, ld)) {
    // the syrk's tiles (all of full K) first, the row product's (K ranges of every length)
    // after them, filling the last round of workgroups
    KQ_TRY(gemm_f32_split6_dual(syrk, row, s, "chol_syrk_trtri_row"));
  } else {
    KQ_TRY(gemm_f32_dual(syrk, row, s, "chol_syrk_trtri_row"));
  }
  KQ_TRY(chol_rec(M, X, T + r * h, tcap - r * h, ld, n0 + h, r, d, info, s));
  // X21 = -X22 T
  return chol_gemm(GEMM_A_LOWER, r, h, r, -1.f, X22, ld, T, h, 0.f, X21, ld, s, "trtri_update");
}

}  // namespace

size_t chol_ws_bytes(int64_t d) {
  if (d <= 0) return 0;
  const int64_t ld = ld_for(d);
  return 2 * align256(size_t(d) * ld * sizeof(float)) +
         align256(size_t(std::max<int64_t>(1, chol_scratch(d))) * sizeof(float)) + 256;
}

int chol_launch(float* H, int64_t d, int64_t ldh, float damp_rel, float* U, int64_t ldu,
                int* info, void* ws, hipStream_t s) {
  const int64_t ld = ld_for(d);
  Carver cv(ws);
  float* M = cv.take<float>(size_t(d) * ld);
  float* X = cv.take<float>(size_t(d) * ld);
  const int64_t tcap = std::max<int64_t>(1, chol_scratch(d));
  float* T = cv.take<float>(size_t(tcap));
  float* shift = cv.take<float>(1);

  KQ_TRY(launch("chol_diag_shift", diag_shift, dim3(1), dim3(256), 0, s,
                static_cast<const float*>(H), d, ldh, damp_rel, shift, info));
  KQ_TRY(launch("chol_add_diag", add_diag, dim3(unsigned(cdiv(d, 256))), dim3(256), 0, s, H, d,
                ldh, static_cast<const float*>(shift)));
  const unsigned gx = unsigned(cdiv(d, 256) < 64 ? cdiv(d, 256) : 64);
  const bool v4 = d % 4 == 0 && ldh % 4 == 0 && ldu % 4 == 0 && aligned(H, 16) && aligned(U, 16);
  const unsigned gx4 = unsigned(cdiv(d, 1024) < 64 ? cdiv(d, 1024) : 64);
  if (v4)
    KQ_TRY(launch("chol_reverse_copy", reverse_copy4, dim3(gx4, unsigned(d)), dim3(256), 0, s,
                  static_cast<const float*>(H), d, ldh, M, ld));
  else
    KQ_TRY(launch("chol_reverse_copy", reverse_copy, dim3(gx, unsigned(d)), dim3(256), 0, s,
                  static_cast<const float*>(H), d, ldh, M, ld));
  KQ_TRY(chol_rec(M, X, T, tcap, ld, 0, d, d, info, s));
  if (v4)
    return launch("chol_reverse_out", reverse_out4, dim3(gx4, unsigned(d)), dim3(256), 0, s,
                  static_cast<const float*>(X), ld, d, U, ldu);
  return launch("chol_reverse_out", reverse_out, dim3(gx, unsigned(d)), dim3(256), 0, s,
                static_cast<const float*>(X), ld, d, U, ldu);
}

}  // namespace kq
