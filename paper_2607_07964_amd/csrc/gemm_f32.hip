// fp32 GEMM on the fp32 matrix cores (v_mfma_f32_32x32x2f32): C = alpha op(A) op(B) + beta C.
//
// Used where the path needs fp32-accurate dense products: the trailing updates of the
// Cholesky factorisation and of the triangular inverse, the lazy-block OBS update, and the
// two products of the K-FAC loss.
//   * 128 x 128 output tile per workgroup, 4 waves in a 2 x 2 grid, each wave 64 x 64 =
//     2 x 2 MFMA blocks (64 fp32 accumulators per lane).
//   * K advances 32 at a time through two LDS buffers: the next stage is fetched into
//     registers before the current stage's products and stored into the other buffer after
//     them, one barrier per stage. An operand read with k contiguous stays [m][k] in LDS (row
//     stride 36 floats, so 16-byte stores and at most 2-way conflicts on the MFMA reads); one
//     read with m contiguous is stored [k][m] (row stride 160 floats: the two k rows a wave
//     reads at once fall in disjoint bank halves).
//   * Triangular flags skip tiles or K ranges that are known to be zero or unused.
// The recursive Cholesky's products, most of them with a triangular operand, use
// gemm_f32_small: a 32 x 32 or 64 x 64 tile per workgroup, K staged 64 at a time through LDS,
// and for 32 x 32 tiles each stage's K split over the four waves (the partial blocks are summed
// through LDS at the end). With a triangular operand the tiles' K ranges are unequal; the
// 64 x 64 tiles are then dealt longest range first, which balances the chip far better than
// 128 x 128 tiles, whose longest tile sets the time (the 2048-order products of a 4096
// factorisation: 210 -> 110-125 us, the lower-triangle update 210 -> 186 us). Otherwise the
// dispatcher takes the largest tile that still gives at least 128 workgroups.
#include <algorithm>

#include "kq_common.hpp"

namespace kq {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int GT = 128;    // tile edge
constexpr int GK = 32;     // K per stage
constexpr int GLD = 160;   // LDS row stride (floats)

constexpr int SKC = GK + 4;  // LDS row stride of a k-contiguous operand stored [m][k]

struct Frag {
  float v[GK / 2];
};

// Fetch an operand chunk: GK (k) x 128 (m) elements of op(X), GK / 2 per thread in float4s.
// KC: X[m][k] (k contiguous), two threads per row m; else X[k][m] (m contiguous).
template <bool KC>
__device__ __forceinline__ void fetch(Frag& f, const float* X, int64_t ldx, int64_t m0,
                                      int64_t k0, int64_t M, int64_t K, int tid) {
  constexpr int NQ = GK / 8;  // float4 per thread
#pragma unroll
  for (int h = 0; h < NQ; ++h) {
    int64_t r, c;  // element (r, c) of X starts the float4; c is the contiguous index
    bool full, in_r;
    if (KC) {
      r = m0 + (tid >> 1);
      c = k0 + (tid & 1) * (GK / 2) + h * 4;
      in_r = r < M;
      full = in_r && c + 4 <= K;
    } else {
      r = k0 + tid / (256 / GK);
      c = m0 + (tid % (256 / GK)) * (GK / 2) + h * 4;
      in_r = r < K;
      full = in_r && c + 4 <= M;
    }
    if (full) {
      const float4 x = *reinterpret_cast<const float4*>(X + r * ldx + c);
      f.v[h * 4 + 0] = x.x;
      f.v[h * 4 + 1] = x.y;
      f.v[h * 4 + 2] = x.z;
      f.v[h * 4 + 3] = x.w;
    } else {
      const int64_t lim = KC ? K : M;
#pragma unroll
      for (int e = 0; e < 4; ++e) f.v[h * 4 + e] = (in_r && c + e < lim) ? X[r * ldx + c + e] : 0.f;
    }
  }
}

// Store a fetched chunk in LDS: KC as [m][k] (row stride SKC), else as [k][m] (row stride GLD);
// both with 16-byte writes.
template <bool KC>
__device__ __forceinline__ void stash(float* __restrict__ s, const Frag& f, int tid) {
#pragma unroll
  for (int h = 0; h < GK / 8; ++h) {
    float* p = KC ? s + (tid >> 1) * SKC + (tid & 1) * (GK / 2) + 4 * h
                  : s + (tid / (256 / GK)) * GLD + (tid % (256 / GK)) * (GK / 2) + 4 * h;
    *reinterpret_cast<float4*>(p) =
        make_float4(f.v[4 * h], f.v[4 * h + 1], f.v[4 * h + 2], f.v[4 * h + 3]);
  }
}

// operand value (m, k) of a stage held in LDS
template <bool KC>
__device__ __forceinline__ float opnd(const float* s, int m, int k) {
  return KC ? s[m * SKC + k] : s[k * GLD + m];
}

// Double-buffered LDS: stage s + 1 is fetched into registers before the products of stage s
// and stored into the other buffer after them, so one barrier per stage suffices and the
// global loads' latency hides behind the products. AKC / BKC: op(A) / op(B) is read with k
// contiguous (the layout in LDS follows, so every store is 16 bytes wide).
template <bool AKC, bool BKC>
__global__ __launch_bounds__(256, 2) void gemm_f32_mfma(int flags, int64_t M, int64_t N,
                                                        int64_t K, float alpha,
                                                        const float* A, int64_t lda,
                                                        const float* B, int64_t ldb,
                                                        float beta, float* C,
                                                        int64_t ldc) {
  // A, B and C may overlap (in-place panel solves): all loads of A and B precede the stores,
  // and each workgroup reads only the rows/columns it writes.
  __shared__ __attribute__((aligned(16))) float lds[2][2][GK * GLD];  // [buffer][A, B]
  const int tid = threadIdx.x;
  const int64_t m0 = int64_t(blockIdx.y) * GT, n0 = int64_t(blockIdx.x) * GT;
  if ((flags & GEMM_LOWER_C) && m0 + GT <= n0) return;  // tile strictly above the diagonal
  if ((flags & GEMM_UPPER_C) && n0 + GT <= m0) return;  // tile strictly below the diagonal

  int64_t kbeg = 0, kend = K;
  if (flags & GEMM_B_LOWER) kbeg = (n0 / GK) * GK;  // B[k][n] = 0 for k < n
  if ((flags & GEMM_A_UPPER) && m0 > kbeg) kbeg = (m0 / GK) * GK;  // A[m][k] = 0 for k < m
  if ((flags & GEMM_A_LOWER) && m0 + GT < kend) kend = m0 + GT;  // A[m][k] = 0 for k > m
  if ((flags & GEMM_OPB_UPPER) && n0 + GT < kend) kend = n0 + GT;  // op(B)[k][n] = 0, k > n
  const int nst = kbeg < kend ? int(cdiv(kend - kbeg, GK)) : 0;

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int l32 = lane & 31, lhi = lane >> 5;

  f32x16_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16_t{};

  Frag fa, fb;
  if (nst > 0) {
    fetch<AKC>(fa, A, lda, m0, kbeg, M, kend, tid);
    fetch<BKC>(fb, B, ldb, n0, kbeg, N, kend, tid);
    stash<AKC>(lds[0][0], fa, tid);
    stash<BKC>(lds[0][1], fb, tid);
  }
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) {
      const int64_t k1 = kbeg + int64_t(st + 1) * GK;
      fetch<AKC>(fa, A, lda, m0, k1, M, kend, tid);
      fetch<BKC>(fb, B, ldb, n0, k1, N, kend, tid);
    }
    const float* sa = lds[st & 1][0];
    const float* sb = lds[st & 1][1];
#pragma unroll
    for (int kk = 0; kk < GK / 2; ++kk) {
      const int kr = 2 * kk + lhi;
      float av[2], bv[2];
#pragma unroll
      for (int bi = 0; bi < 2; ++bi) av[bi] = opnd<AKC>(sa, wm * 64 + bi * 32 + l32, kr);
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) bv[bj] = opnd<BKC>(sb, wn * 64 + bj * 32 + l32, kr);
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[bi], bv[bj], acc[bi][bj], 0, 0, 0);
    }
    if (more) {
      stash<AKC>(lds[(st + 1) & 1][0], fa, tid);
      stash<BKC>(lds[(st + 1) & 1][1], fb, tid);
    }
    __syncthreads();
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


// Tiles of a product on a tm-edge grid (gx x gy tiles): with LOWER_C / UPPER_C on a square grid
// only the tiles that touch that triangle are enumerated.
__host__ __device__ inline int64_t tile_count(int flags, int64_t gx, int64_t gy) {
  if ((flags & (GEMM_LOWER_C | GEMM_UPPER_C)) && gx == gy) return gx * (gx + 1) / 2;
  return gx * gy;
}

// Tile number lin of a product -> its corner. Triangular outputs are enumerated row by row
// (LOWER_C) or column by column (UPPER_C). Otherwise, with a triangular operand the K range of a
// tile depends on its row (A_LOWER, A_UPPER) or column (B_LOWER, OPB_UPPER) index, and
// workgroups are dispatched in order, so the tiles are dealt with that index running slowest,
// from the longest range to the shortest (the short ones then fill in at the end).
__device__ __forceinline__ void tile_from(int flags, int64_t lin, int64_t gx, int64_t gy,
                                          int tm, int64_t& m0, int64_t& n0) {
  int64_t bm = lin / gx, bn = lin % gx;
  if ((flags & (GEMM_LOWER_C | GEMM_UPPER_C)) && gx == gy) {
    // lin = i (i + 1) / 2 + j with j <= i
    int64_t i = int64_t((sqrt(8.0 * double(lin) + 1.0) - 1.0) * 0.5);
    while (i * (i + 1) / 2 > lin) --i;
    while ((i + 1) * (i + 2) / 2 <= lin) ++i;
    const int64_t j = lin - i * (i + 1) / 2;
    bm = (flags & GEMM_LOWER_C) ? i : j;
    bn = (flags & GEMM_LOWER_C) ? j : i;
  } else if (flags & (GEMM_B_LOWER | GEMM_OPB_UPPER)) {  // K set by the column
    const int64_t c = lin / gy;
    bm = lin % gy;
    bn = (flags & GEMM_OPB_UPPER) ? gx - 1 - c : c;
  } else if (flags & (GEMM_A_LOWER | GEMM_A_UPPER)) {  // K set by the row
    const int64_t r = lin / gx;
    bn = lin % gx;
    bm = (flags & GEMM_A_LOWER) ? gy - 1 - r : r;
  }
  m0 = bm * tm;
  n0 = bn * tm;
}

template <int TM>
struct SmallLds {
  static constexpr int KC = 64, AS = KC + 1, BS = TM == 32 ? 32 : 96;
  static constexpr int SK = 4 / ((TM / 32) * (TM / 32));
  static constexpr int A = TM * AS;
  static constexpr int B = TM * AS > KC * BS ? TM * AS : KC * BS;  // either B layout
  static constexpr int R = (SK - 1) * 1024 + 1;
};

// One tile of the small-tile product (see the file comment). A, B and C must not overlap.
// BKC: op(B) is read with k contiguous (B^T stored [n][k]); B then stays [n][k] in LDS (row
// stride AS, like A) so that both the transposing store and the MFMA reads are free of bank
// conflicts.
template <int TM, bool BKC>
__device__ __forceinline__ void small_tile(const GemmProb& p, int64_t m0, int64_t n0,
                                           float* __restrict__ sA, float* __restrict__ sB,
                                           float* __restrict__ red) {
  constexpr int KC = 64;                      // K per stage
  constexpr int NB32 = TM / 32;               // 32 x 32 blocks per tile edge
  constexpr int SK = 4 / (NB32 * NB32);       // waves per block (split of each stage's K)
  constexpr int KW = KC / SK;                 // K per wave per stage
  constexpr int AS = KC + 1;                  // LDS row stride of the A tile, [m][k]
  constexpr int BS = TM == 32 ? 32 : 96;      // LDS row stride of the B tile, [k][n]
  constexpr int NV = TM * KC / 1024;          // float4 per thread per operand per stage
  constexpr int SB = (BKC ? TM * AS : KC * BS);
  (void)SB;
  const int flags = p.flags;
  const int64_t M = p.M, N = p.N, K = p.K, lda = p.lda, ldb = p.ldb, ldc = p.ldc;
  const float alpha = p.alpha, beta = p.beta;
  const float* __restrict__ A = p.A;
  const float* __restrict__ B = p.B;
  float* __restrict__ C = p.C;
  const int tid = threadIdx.x;
  if ((flags & GEMM_LOWER_C) && m0 + TM <= n0) return;
  if ((flags & GEMM_UPPER_C) && n0 + TM <= m0) return;
  int64_t kbeg = 0, kend = K;
  if (flags & GEMM_B_LOWER) kbeg = n0;
  if ((flags & GEMM_A_UPPER) && m0 > kbeg) kbeg = m0;
  if ((flags & GEMM_A_LOWER) && m0 + TM < kend) kend = m0 + TM;
  if ((flags & GEMM_OPB_UPPER) && n0 + TM < kend) kend = n0 + TM;
  const bool a_kc = !(flags & GEMM_TA);
  constexpr bool b_kc = BKC;
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
        for (int c = 0; c < 4; ++c) sB[n * AS + k4 + c] = z[c];
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
      const float bv = BKC ? sB[(bn + l32) * AS + kk] : sB[kk * BS + bn + l32];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sA[(bm + l32) * AS + kk], bv, acc, 0, 0, 0);
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


template <int TM, bool BKC>
__global__ __launch_bounds__(256) void gemm_f32_small(GemmProb p, int64_t gx, int64_t gy) {
  __shared__ float sA[SmallLds<TM>::A];
  __shared__ float sB[SmallLds<TM>::B];
  __shared__ float red[SmallLds<TM>::R];
  int64_t m0, n0;
  tile_from(p.flags, blockIdx.x, gx, gy, TM, m0, n0);
  small_tile<TM, BKC>(p, m0, n0, sA, sB, red);
}

// Two independent products in one launch (the first problem's tiles first): one dependent
// launch fewer where the recursion has two products with the same inputs ready.
template <int TM, bool BKC1, bool BKC2>
__global__ __launch_bounds__(256) void gemm_f32_dual(GemmProb p1, int64_t gx1, int64_t gy1,
                                                     int64_t n1, GemmProb p2, int64_t gx2,
                                                     int64_t gy2) {
  __shared__ float sA[SmallLds<TM>::A];
  __shared__ float sB[SmallLds<TM>::B];
  __shared__ float red[SmallLds<TM>::R];
  int64_t m0, n0;
  const int64_t lin = blockIdx.x;
  if (lin < n1) {
    tile_from(p1.flags, lin, gx1, gy1, TM, m0, n0);
    small_tile<TM, BKC1>(p1, m0, n0, sA, sB, red);
  } else {
    tile_from(p2.flags, lin - n1, gx2, gy2, TM, m0, n0);
    small_tile<TM, BKC2>(p2, m0, n0, sA, sB, red);
  }
}

}  // namespace

namespace {

// workgroups that do work for a tile edge t
int64_t work(int flags, int64_t M, int64_t N, int64_t t) {
  const int64_t tm = cdiv(M, t), tn = cdiv(N, t);
  if (!(flags & (GEMM_LOWER_C | GEMM_UPPER_C))) return tm * tn;
  int64_t c = 0;
  for (int64_t i = 0; i < tm; ++i)
    c += (flags & GEMM_LOWER_C) ? std::min(tn, i + 1) : std::max<int64_t>(0, tn - i);
  return c;
}

// tile edge of the small-tile kernel for a product: 64 when that still gives enough workgroups
int small_edge(int flags, int64_t M, int64_t N) { return work(flags, M, N, 64) >= 128 ? 64 : 32; }

}  // namespace

int gemm_f32(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
             int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
             hipStream_t s, const char* name) {
  if (M <= 0 || N <= 0) return KRONQ_OK;
  // a triangular operand or output makes the tiles' work unequal: 64 x 64 tiles, longest
  // first, balance them better than 128 x 128 tiles, whose longest tile sets the time
  const bool tri = flags & (GEMM_B_LOWER | GEMM_OPB_UPPER | GEMM_A_LOWER | GEMM_A_UPPER |
                            GEMM_LOWER_C | GEMM_UPPER_C);
  if (work(flags, M, N, GT) >= 128 && !(tri && work(flags, M, N, 64) >= 256)) {
    const dim3 grid(unsigned(cdiv(N, GT)), unsigned(cdiv(M, GT)));
    const bool akc = !(flags & GEMM_TA), bkc = flags & GEMM_TB;
    auto kern = akc ? (bkc ? gemm_f32_mfma<true, true> : gemm_f32_mfma<true, false>)
                    : (bkc ? gemm_f32_mfma<false, true> : gemm_f32_mfma<false, false>);
    return launch(name, kern, grid, dim3(256), 0, s, flags, M, N, K, alpha, A, lda, B, ldb, beta,
                  C, ldc);
  }
  const GemmProb p{flags, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc};
  const int t = small_edge(flags, M, N);
  const int64_t gx = cdiv(N, t), gy = cdiv(M, t);
  const dim3 grid(unsigned(tile_count(flags, gx, gy)));
  const bool bkc = flags & GEMM_TB;
  if (t == 64)
    return launch(name, bkc ? gemm_f32_small<64, true> : gemm_f32_small<64, false>, grid,
                  dim3(256), 0, s, p, gx, gy);
  return launch(name, bkc ? gemm_f32_small<32, true> : gemm_f32_small<32, false>, grid, dim3(256),
                0, s, p, gx, gy);
}

int gemm_f32_dual(const GemmProb& p1, const GemmProb& p2, hipStream_t s, const char* name) {
  if (p1.M <= 0 || p1.N <= 0) return gemm_f32(p2.flags, p2.M, p2.N, p2.K, p2.alpha, p2.A, p2.lda,
                                              p2.B, p2.ldb, p2.beta, p2.C, p2.ldc, s, name);
  if (p2.M <= 0 || p2.N <= 0) return gemm_f32(p1.flags, p1.M, p1.N, p1.K, p1.alpha, p1.A, p1.lda,
                                              p1.B, p1.ldb, p1.beta, p1.C, p1.ldc, s, name);
  // one tile edge for both: 64 when the two together give enough workgroups
  const int64_t w64 = work(p1.flags, p1.M, p1.N, 64) + work(p2.flags, p2.M, p2.N, 64);
  const int t = w64 >= 128 ? 64 : 32;
  const int64_t gx1 = cdiv(p1.N, t), gy1 = cdiv(p1.M, t), gx2 = cdiv(p2.N, t),
                gy2 = cdiv(p2.M, t);
  const int64_t n1 = tile_count(p1.flags, gx1, gy1), n2 = tile_count(p2.flags, gx2, gy2);
  const dim3 grid(unsigned(n1 + n2));
  const bool b1 = p1.flags & GEMM_TB, b2 = p2.flags & GEMM_TB;
  if (t == 64) {
    auto kern = b1 ? (b2 ? gemm_f32_dual<64, true, true> : gemm_f32_dual<64, true, false>)
                   : (b2 ? gemm_f32_dual<64, false, true> : gemm_f32_dual<64, false, false>);
    return launch(name, kern, grid, dim3(256), 0, s, p1, gx1, gy1, n1, p2, gx2, gy2);
  }
  auto kern = b1 ? (b2 ? gemm_f32_dual<32, true, true> : gemm_f32_dual<32, true, false>)
                 : (b2 ? gemm_f32_dual<32, false, true> : gemm_f32_dual<32, false, false>);
  return launch(name, kern, grid, dim3(256), 0, s, p1, gx1, gy1, n1, p2, gx2, gy2);
}

}  // namespace kq
