// fp32 GEMM on the bf16 matrix cores with fp32 accuracy, for the large products of the
// inverse-Cholesky factorisation (Alg. 2, first two lines): C = alpha op(A) op(B) + beta C.
//   * Six-term split: x = x_h + x_m + x_l with x_h = bf16(x), x_m = bf16(x - x_h),
//     x_l = bf16(x - x_h - x_m) (24 significant bits, the whole fp32 significand), and
//     A B ~ A_h B_h + A_h B_m + A_m B_h + A_h B_l + A_l B_h + A_m B_m: the dropped terms are
//     ~2^-24 of each product and every kept product of two bf16 is exact in fp32, so the result
//     is as accurate as an fp32 GEMM, on matrix cores with 16 times the fp32 rate (6 products:
//     2.7 times the fp32 MFMA peak).
//   * The operands stay fp32 in memory (4 bytes an element instead of the 6 of three planes):
//     each workgroup reads its fp32 tiles into registers, splits them (v_cvt_pk_bf16_f32 and two
//     subtractions per pair) and writes the three bf16 planes to LDS. The structural zeros of a
//     triangular operand are zeroed there, so that K ranges can be rounded out to whole stages.
//   * 256 x 128 output tile per workgroup, 8 waves of 64 x 64 (2 x 2 MFMA blocks of 32 x 32),
//     K advancing 32 at a time through two LDS stages of 72 KB (all six planes); the next
//     stage's fp32 tiles are fetched into registers during the current stage's 48 MFMAs a wave.
//     LDS rows of 64 bytes (m- or n-major planes) are read with ds_read_b128 under an XOR
//     swizzle of their 16-byte chunks; a k-major op(B) (B stored [K][N]) is kept k-major in LDS
//     and read with the transposing ds_read_b64_tr_b16.
//   * Tile order: row-major, or whole tile columns per XCD in a paired order that balances
//     triangular work over the 8 XCDs, whichever leaves the busiest XCD the least work.
//   * Triangular structure limits each tile's K range (GEMM_B_LOWER, GEMM_OPB_UPPER,
//     GEMM_A_LOWER) or skips the tile (GEMM_LOWER_C), as in the fp32 kernels.
#include <algorithm>
#include <type_traits>

#include "kq_common.hpp"

namespace kq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short v4s_t __attribute__((ext_vector_type(4)));

constexpr int TM = 256;  // output tile rows
constexpr int TN = 128;  // output tile columns
constexpr int BK = 32;   // K per stage
constexpr int PA = TM * BK;              // bf16 per A plane per stage
constexpr int PB = TN * BK;              // bf16 per B plane per stage
constexpr int STAGE = 3 * (PA + PB);     // bf16 per stage (73,728 bytes)
constexpr int NT = 512;                  // threads: 8 waves, two per SIMD
constexpr int NWM = 4, NWN = 2;          // waves along M and N
constexpr int WTM = TM / NWM, WTN = TN / NWN;  // wave tile: 64 x 64
constexpr int BI = WTM / 32, BJ = WTN / 32;    // 32 x 32 MFMA blocks per wave: 2 x 2
constexpr int FA = TM * BK / 4 / NT;     // float4 of A per thread per stage
constexpr int FB = TN * BK / 4 / NT;     // float4 of B per thread per stage
constexpr int RSTEP = NT / 8;            // m- / n-major rows per float4 step (8 float4 a row)
constexpr int KSTEP = NT / 32;           // k-major rows per float4 step (32 float4 a row)

// bf16 (round to nearest even) of two floats packed in one word; a, b become their values
__device__ __forceinline__ uint32_t pk_bf16(float& a, float& b) {
  const bf16x2_t v = __builtin_convertvector(f32x2_t{a, b}, bf16x2_t);
  uint32_t u;
  __builtin_memcpy(&u, &v, 4);
  a = __uint_as_float(u << 16);
  b = __uint_as_float(u & 0xFFFF0000u);
  return u;
}

// three-plane split of four floats (4 bf16 per plane)
__device__ __forceinline__ void split4(float4 x, uint2& h, uint2& m, uint2& l) {
  float a0 = x.x, a1 = x.y, a2 = x.z, a3 = x.w;
  h.x = pk_bf16(a0, a1);
  h.y = pk_bf16(a2, a3);
  float r0 = x.x - a0, r1 = x.y - a1, r2 = x.z - a2, r3 = x.w - a3;
  float b0 = r0, b1 = r1, b2 = r2, b3 = r3;
  m.x = pk_bf16(b0, b1);
  m.y = pk_bf16(b2, b3);
  r0 -= b0;
  r1 -= b1;
  r2 -= b2;
  r3 -= b3;
  l.x = pk_bf16(r0, r1);
  l.y = pk_bf16(r2, r3);
}

// chunk swizzle of a 64-byte LDS row (four 16-byte chunks): the 16-byte reads of 16
// consecutive rows at one logical chunk land on distinct banks
__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }

// keep elements lo .. hi of a float4, zero the others
__device__ __forceinline__ float4 keep4(float4 x, int lo, int hi) {
  x.x = (0 >= lo && 0 <= hi) ? x.x : 0.f;
  x.y = (1 >= lo && 1 <= hi) ? x.y : 0.f;
  x.z = (2 >= lo && 2 <= hi) ? x.z : 0.f;
  x.w = (3 >= lo && 3 <= hi) ? x.w : 0.f;
  return x;
}
__device__ __forceinline__ int clamp_idx(int64_t v) {
  return int(v < -1 ? -1 : (v > 4 ? 4 : v));
}

template <int V>
using ic = std::integral_constant<int, V>;

// one product as the kernel sees it, with its tile grid
struct Job {
  int flags;
  int64_t M, N, K;
  float alpha;
  const float* A;
  int64_t lda;
  const float* B;
  int64_t ldb;
  float beta;
  float* C;
  int64_t ldc;
  int nt_m, nt_n;  // tiles along M and N
  int vc;          // column order: virtual tile columns per XCD (0: row-major tile order)
  int blocks;      // workgroups of the launch
};

// tile b of product J (all workgroup-uniform but the thread index)
template <bool KMAJ>  // op(B) stored [K][N] (k-major) rather than [N][K]
__device__ __forceinline__ void gemm6_tile(const Job& J, int b, uint16_t* lds) {
  const int flags = J.flags;
  const int64_t M = J.M, N = J.N, K = J.K, lda = J.lda, ldb = J.ldb, ldc = J.ldc;
  const float* __restrict__ A = J.A;
  const float* __restrict__ B = J.B;
  float* __restrict__ C = J.C;
  const float alpha = J.alpha, beta = J.beta;
  const int nt_m = J.nt_m, nt_n = J.nt_n, vc = J.vc;
  const int tid = threadIdx.x;
  int tm, tn;
  if (vc > 0) {  // column order: XCD x = b % 8 owns columns x, 15 - x, 16 + x, 31 - x, ...
    const int x = b & 7, s = b >> 3, j = s % vc;
    tm = s / vc;
    tn = 16 * (j >> 1) + ((j & 1) ? 15 - x : x);
  } else {
    tm = b / nt_n;
    tn = b % nt_n;
  }
  if (tm >= nt_m || tn >= nt_n) return;
  const int64_t m0 = int64_t(tm) * TM, n0 = int64_t(tn) * TN;
  if ((flags & GEMM_LOWER_C) && m0 + TM <= n0) return;  // tile strictly above the diagonal
  int64_t kbeg = 0, kend = K;
  if ((flags & GEMM_B_LOWER) && n0 > kbeg) kbeg = n0;                // op(B)[k][n] = 0, k < n
  if ((flags & GEMM_A_LOWER) && m0 + TM < kend) kend = m0 + TM;      // A[m][k] = 0, k > m
  if ((flags & GEMM_OPB_UPPER) && n0 + TN < kend) kend = n0 + TN;    // op(B)[k][n] = 0, k > n
  const int nst = kend > kbeg ? int((kend - kbeg + BK - 1) / BK) : 0;
  const bool alow = flags & GEMM_A_LOWER;
  const bool blow = flags & GEMM_B_LOWER, bup = flags & GEMM_OPB_UPPER;
  const bool edge = m0 + TM > M || n0 + TN > N;
  // a stage needs the checked path when it reaches past kend or M / N, or crosses the diagonal
  // of a triangular operand
  auto checked = [&](int st) {
    const int64_t k0 = kbeg + int64_t(st) * BK;
    return edge || k0 + BK > kend || (alow && k0 + BK - 1 > m0) ||
           (bup && k0 + BK - 1 > n0) || (blow && k0 < n0 + TN);
  };

  // fetch: A 256 rows x 8 float4 (4 per thread); B 128 rows x 8 float4, or k-major 32 rows of
  // k x 32 float4 (2 per thread); two register sets, so that a stage's tiles are fetched two
  // stages ahead of their use and split one stage ahead
  // The lambdas below derive their lane indices from t, a copy of the thread index that the
  // compiler cannot see through: they are then formed inside each stage rather than hoisted out
  // of the loop into registers that the stage needs.
  float4 ra[2][FA], rb[2][FB];
  // Uniform bases plus 32-bit per-lane byte offsets (a 256-row tile spans well under 4 GB),
  // so that the loads take the scalar-base addressing form. Checked: every index clamped into
  // the matrices relative to the tile's own origin (so that no offset goes negative); the
  // elements so fetched are zeroed when split.
  const int ra_lim = int(M - 1 - m0), rb_lim = int(N - 1 - n0);  // >= 0: m0 < M, n0 < N
  auto ld4 = [](const float* base, uint32_t byte_off) {
    return *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(base) + byte_off);
  };
  auto fetch = [&](auto chk, auto set, int64_t k0, int t) {
    constexpr bool CHK = decltype(chk)::value;
    constexpr int S = decltype(set)::value;
    const int ar = t >> 3, ak = 4 * (t & 7), bkr = t >> 5, bn = 4 * (t & 31);
    const int klim = int(K - 4 - k0);  // >= 0: k0 < K, both multiples of 4
#pragma unroll
    for (int v = 0; v < FA; ++v) {
      if (CHK) {
        const int r = min(ar + RSTEP * v, ra_lim), k = min(ak, klim);
        ra[S][v] = ld4(A + m0 * lda + k0, 4u * (uint32_t(r) * uint32_t(lda) + uint32_t(k)));
      } else {
        ra[S][v] = ld4(A + (m0 + RSTEP * v) * lda + k0,
                       4u * (uint32_t(ar) * uint32_t(lda) + uint32_t(ak)));
      }
    }
#pragma unroll
    for (int v = 0; v < FB; ++v) {
      if (KMAJ) {
        if (CHK) {
          const int k = min(bkr + KSTEP * v, int(K - 1 - k0)), n = min(bn, int(N - 4 - n0));
          rb[S][v] = ld4(B + k0 * ldb + n0, 4u * (uint32_t(k) * uint32_t(ldb) + uint32_t(n)));
        } else {
          rb[S][v] = ld4(B + (k0 + KSTEP * v) * ldb + n0,
                         4u * (uint32_t(bkr) * uint32_t(ldb) + uint32_t(bn)));
        }
      } else {
        if (CHK) {
          const int r = min(ar + RSTEP * v, rb_lim), k = min(ak, klim);
          rb[S][v] = ld4(B + n0 * ldb + k0, 4u * (uint32_t(r) * uint32_t(ldb) + uint32_t(k)));
        } else {
          rb[S][v] = ld4(B + (n0 + RSTEP * v) * ldb + k0,
                         4u * (uint32_t(ar) * uint32_t(ldb) + uint32_t(ak)));
        }
      }
    }
  };
  // split register set S (the tiles of stage k0) into the three planes of LDS buffer BUF;
  // checked: zero what lies outside the matrices, past kend or across a triangle's diagonal
  auto stash = [&](auto chk, auto set, auto bufc, int64_t k0, int t) {
    constexpr bool CHK = decltype(chk)::value;
    constexpr int S = decltype(set)::value, BUF = decltype(bufc)::value;
    const int ar = t >> 3, ak = 4 * (t & 7), bkr = t >> 5, bn = 4 * (t & 31);
    uint16_t* sa = lds + BUF * STAGE;
    uint16_t* sb = sa + 3 * PA;
#pragma unroll
    for (int v = 0; v < FA; ++v) {
      const int r = ar + RSTEP * v;
      float4 x = ra[S][v];
      if (CHK) {  // element (m, k + i): k + i < kend, m < M; lower A: k + i <= m
        const int64_t m = m0 + r, k = k0 + ak;
        int hi = (m < M && k < kend) ? 3 : -1;
        if (alow) hi = min(hi, clamp_idx(m - k));
        x = keep4(x, 0, hi);
      }
      uint2 h, md, l;
      split4(x, h, md, l);
      const int off = r * BK + (((ak >> 3) ^ swz(r)) << 3) + (ak & 4);
      *reinterpret_cast<uint2*>(sa + off) = h;
      *reinterpret_cast<uint2*>(sa + PA + off) = md;
      *reinterpret_cast<uint2*>(sa + 2 * PA + off) = l;
    }
#pragma unroll
    for (int v = 0; v < FB; ++v) {
      float4 x = rb[S][v];
      int off;
      if (KMAJ) {  // element (k, n + i) of op(B): lower: n + i <= k; upper: n + i >= k
        const int kr = bkr + KSTEP * v;
        if (CHK) {
          const int64_t k = k0 + kr, n = n0 + bn;
          int lo = 0, hi = (k < kend && n < N) ? 3 : -1;
          if (blow) hi = min(hi, clamp_idx(k - n));
          if (bup) lo = max(lo, clamp_idx(k - n));
          x = keep4(x, lo, hi);
        }
        off = kr * TN + (((bn >> 3) ^ (4 * (kr & 3))) << 3) + (bn & 4);
      } else {  // element (k + i, n) of op(B): lower: k + i >= n; upper: k + i <= n
        const int r = ar + RSTEP * v;
        if (CHK) {
          const int64_t n = n0 + r, k = k0 + ak;
          int lo = 0, hi = (n < N && k < kend) ? 3 : -1;
          if (bup) hi = min(hi, clamp_idx(n - k));
          if (blow) lo = max(lo, clamp_idx(n - k));
          x = keep4(x, lo, hi);
        }
        off = r * BK + (((ak >> 3) ^ swz(r)) << 3) + (ak & 4);
      }
      uint2 h, md, l;
      split4(x, h, md, l);
      *reinterpret_cast<uint2*>(sb + off) = h;
      *reinterpret_cast<uint2*>(sb + PB + off) = md;
      *reinterpret_cast<uint2*>(sb + 2 * PB + off) = l;
    }
  };

  f32x16_t acc[BI][BJ];
#pragma unroll
  for (int a = 0; a < BI; ++a)
#pragma unroll
    for (int b = 0; b < BJ; ++b) acc[a][b] = f32x16_t{};
  // the 48 MFMAs of one stage from LDS buffer BUF
  auto compute = [&](auto bufc, int t) {
    constexpr int BUF = decltype(bufc)::value;
    const int wave = t >> 6, lane = t & 63;
    const int wm = wave % NWM, wn = wave / NWM, l32 = lane & 31, lhi = lane >> 5;
    const uint16_t* sa = lds + BUF * STAGE;
    const uint16_t* sb = sa + 3 * PA;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8_t fa[3][BI], fb[3][BJ];
#pragma unroll
      for (int i = 0; i < BI; ++i) {
        const int m = wm * WTM + i * 32 + l32, c = 2 * ks + lhi;
        const int off = m * BK + ((c ^ swz(m)) << 3);
#pragma unroll
        for (int p = 0; p < 3; ++p)
          fa[p][i] = *reinterpret_cast<const bf16x8_t*>(sa + p * PA + off);
      }
#pragma unroll
      for (int j = 0; j < BJ; ++j) {
        if (KMAJ) {
          // within a group of 16 lanes, lane L names k row t = kt + L / 4 at columns
          // nb + 4 (L % 4) .. +3 and gets back column nb + L at rows kt .. kt + 3
          const int L = lane & 15, g = (lane >> 4) & 1;
          const int c8 = (wn * WTN + j * 32 + g * 16 + 4 * (L & 3)) >> 3;
#pragma unroll
          for (int p = 0; p < 3; ++p) {
            v4s_t r[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int t = ks * 16 + lhi * 8 + h * 4 + (L >> 2);
              const int off = t * TN + ((c8 ^ (4 * (t & 3))) << 3) + 4 * (L & 1);
              r[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                  (__attribute__((address_space(3))) v4s_t*)(sb + p * PB + off));
            }
            __builtin_memcpy(&fb[p][j], r, 16);
          }
        } else {
          const int n = wn * WTN + j * 32 + l32, c = 2 * ks + lhi;
          const int off = n * BK + ((c ^ swz(n)) << 3);
#pragma unroll
          for (int p = 0; p < 3; ++p)
            fb[p][j] = *reinterpret_cast<const bf16x8_t*>(sb + p * PB + off);
        }
      }
      // grouped by A plane, so that one A plane at a time is live: (h, h), (h, m), (h, l),
      // (m, h), (m, m), (l, h)
      constexpr int ta[6] = {0, 0, 0, 1, 1, 2}, tb[6] = {0, 1, 2, 0, 1, 0};
#pragma unroll
      for (int t = 0; t < 6; ++t)
#pragma unroll
        for (int bi = 0; bi < BI; ++bi)
#pragma unroll
          for (int bj = 0; bj < BJ; ++bj)
            acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ta[t]][bi], fb[tb[t]][bj],
                                                                  acc[bi][bj], 0, 0, 0);
    }
  };
  // stage st (in buffer P = st % 2): fetch stage st + 2 into register set P (clamped to the last
  // stage: a harmless reload), run stage st's MFMAs and split stage st + 1 (set 1 - P, fetched
  // one stage ago) into buffer 1 - P (past the last stage: a buffer nobody reads). One
  // straight-line block per variant, so that the split's arithmetic can fill the MFMA slots.
  auto body = [&](auto par, int st) {
    constexpr int P = decltype(par)::value;
    int t = tid;
    asm volatile("" : "+v"(t));
    __syncthreads();  // stage st is in LDS; every wave is done with buffer 1 - P
    const int nxt = st + 2 < nst ? st + 2 : nst - 1;
    const int64_t kn = kbeg + int64_t(nxt) * BK, ks1 = kbeg + int64_t(st + 1) * BK;
    if (checked(nxt) || (st + 1 < nst && checked(st + 1))) {
      fetch(std::true_type{}, ic<P>{}, kn, t);
      compute(ic<P>{}, t);
      stash(std::true_type{}, ic<1 - P>{}, ic<1 - P>{}, ks1, t);
    } else {
      fetch(std::false_type{}, ic<P>{}, kn, t);
      compute(ic<P>{}, t);
      stash(std::false_type{}, ic<1 - P>{}, ic<1 - P>{}, ks1, t);
    }
  };

  if (nst > 0) {
    const int s1 = nst > 1 ? 1 : 0;
    if (checked(0)) {
      fetch(std::true_type{}, ic<0>{}, kbeg, tid);
      stash(std::true_type{}, ic<0>{}, ic<0>{}, kbeg, tid);
    } else {
      fetch(std::false_type{}, ic<0>{}, kbeg, tid);
      stash(std::false_type{}, ic<0>{}, ic<0>{}, kbeg, tid);
    }
    if (checked(s1))
      fetch(std::true_type{}, ic<1>{}, kbeg + int64_t(s1) * BK, tid);
    else
      fetch(std::false_type{}, ic<1>{}, kbeg + int64_t(s1) * BK, tid);
  }
  for (int st = 0; st < nst; st += 2) {
    body(ic<0>{}, st);
    if (st + 1 < nst) body(ic<1>{}, st + 1);
  }
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave % NWM, wn = wave / NWM, l32 = lane & 31, lhi = lane >> 5;
#pragma unroll
  for (int bi = 0; bi < BI; ++bi)
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t gm = m0 + wm * WTM + bi * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        const int64_t gn = n0 + wn * WTN + bj * 32 + l32;
        if (gm < M && gn < N) {
          float* c = C + gm * ldc + gn;
          const float x = alpha * acc[bi][bj][r];
          *c = beta == 0.f ? x : x + beta * *c;
        }
      }
}

template <bool KMAJ>
__global__ __launch_bounds__(NT) void gemm6(Job J) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];
  gemm6_tile<KMAJ>(J, int(blockIdx.x), lds);
}

// two independent products in one launch: the first product's workgroups come first
template <bool KMAJ0, bool KMAJ1>
__global__ __launch_bounds__(NT) void gemm6_dual(Job J0, Job J1) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];
  const int b = int(blockIdx.x);
  if (b < J0.blocks)
    gemm6_tile<KMAJ0>(J0, b, lds);
  else
    gemm6_tile<KMAJ1>(J1, b - J0.blocks, lds);
}

// K stages of tile (tm, tn), as the kernel bounds them (-1: tile skipped)
int tile_stages(const GemmProb& p, int tm, int tn) {
  const int64_t m0 = int64_t(tm) * TM, n0 = int64_t(tn) * TN;
  if ((p.flags & GEMM_LOWER_C) && m0 + TM <= n0) return -1;
  int64_t kbeg = 0, kend = p.K;
  if ((p.flags & GEMM_B_LOWER) && n0 > kbeg) kbeg = n0;
  if ((p.flags & GEMM_A_LOWER) && m0 + TM < kend) kend = m0 + TM;
  if ((p.flags & GEMM_OPB_UPPER) && n0 + TN < kend) kend = n0 + TN;
  return kend > kbeg ? int((kend - kbeg + BK - 1) / BK) : 0;
}

// Tile order. Workgroups go to the 8 XCDs round-robin, one at a time per CU here (the LDS
// stages fill it). Row-major order gives XCD x every 8th tile; the column order gives XCD x
// whole tile columns x, 15 - x, 16 + x, ... walked row by row, so that the 32 tiles an XCD runs
// together share a few A row blocks and its B column blocks in its L2, and, pairing column
// c with 15 - c, evens out work that grows or shrinks along N (triangular K ranges, the lower
// triangle of GEMM_LOWER_C). The launch takes the order whose busiest XCD has the least work
// (in K stages, plus a few a tile for its prologue and epilogue).
Job make_job(const GemmProb& p) {
  Job j{p.flags, p.M, p.N, p.K, p.alpha, p.A, p.lda, p.B, p.ldb, p.beta, p.C, p.ldc,
        int(cdiv(p.M, TM)), int(cdiv(p.N, TN)), 0, 0};
  constexpr int64_t TILE_COST = 4;
  int64_t row_major[8] = {}, col_order[8] = {};
  const int vc = int(cdiv(j.nt_n, 8));
  for (int tm = 0; tm < j.nt_m; ++tm)
    for (int tn = 0; tn < j.nt_n; ++tn) {
      const int st = tile_stages(p, tm, tn);
      if (st < 0) continue;
      row_major[(int64_t(tm) * j.nt_n + tn) % 8] += st + TILE_COST;
      // column tn belongs to XCD tn % 16 (< 8) or 15 - tn % 16
      const int c16 = tn % 16;
      col_order[c16 < 8 ? c16 : 15 - c16] += st + TILE_COST;
    }
  const int64_t rm = *std::max_element(row_major, row_major + 8);
  const int64_t co = *std::max_element(col_order, col_order + 8);
  j.blocks = j.nt_m * j.nt_n;
  if (co < rm) {
    j.vc = vc;
    j.blocks = 8 * j.nt_m * vc;
  }
  return j;
}

}  // namespace

bool gemm_split6_supports(int flags, int64_t M, int64_t N, int64_t K, const float* A,
                          int64_t lda, const float* B, int64_t ldb) {
  if (flags & (GEMM_TA | GEMM_UPPER_C | GEMM_A_UPPER)) return false;
  if (M <= 0 || N <= 0 || K <= 0) return false;
  if (cdiv(M, TM) * cdiv(N, TN) >= (int64_t(1) << 30)) return false;
  // whole float4 loads: 16-byte aligned rows and no float4 straddling the end of a row
  if (K % 4 || lda % 4 || ldb % 4 ||
      ((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(B)) & 15))
    return false;
  return (flags & GEMM_TB) || N % 4 == 0;
}

bool split6_ok(const GemmProb& p) {
  return gemm_split6_supports(p.flags, p.M, p.N, p.K, p.A, p.lda, p.B, p.ldb);
}

int gemm_f32_split6(int flags, int64_t M, int64_t N, int64_t K, float alpha, const float* A,
                    int64_t lda, const float* B, int64_t ldb, float beta, float* C, int64_t ldc,
                    hipStream_t s, const char* name) {
  if (M <= 0 || N <= 0) return KRONQ_OK;
  const GemmProb p{flags, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc};
  KQ_REQUIRE(split6_ok(p), KRONQ_ERR_UNSUPPORTED,
             "gemm_f32_split6: flags %d, shape %lld x %lld x %lld or alignment not supported",
             flags, (long long)M, (long long)N, (long long)K);
  const Job j = make_job(p);
  if (flags & GEMM_TB)
    return launch(name, gemm6<false>, dim3(unsigned(j.blocks)), dim3(NT), 0, s, j);
  return launch(name, gemm6<true>, dim3(unsigned(j.blocks)), dim3(NT), 0, s, j);
}

int gemm_f32_split6_dual(const GemmProb& p0, const GemmProb& p1, hipStream_t s,
                         const char* name) {
  KQ_REQUIRE(p0.M > 0 && p0.N > 0 && p1.M > 0 && p1.N > 0 && split6_ok(p0) && split6_ok(p1),
             KRONQ_ERR_UNSUPPORTED, "gemm_f32_split6_dual: products not supported");
  Job j0 = make_job(p0);
  const Job j1 = make_job(p1);
  // the second product's XCD assignment assumes its first workgroup lands on XCD 0
  if (j1.vc > 0) j0.blocks = int(cdiv(j0.blocks, 8)) * 8;
  const dim3 grid(unsigned(j0.blocks + j1.blocks));
  const bool t0 = p0.flags & GEMM_TB, t1 = p1.flags & GEMM_TB;
  if (t0 && t1) return launch(name, gemm6_dual<false, false>, grid, dim3(NT), 0, s, j0, j1);
  if (t0) return launch(name, gemm6_dual<false, true>, grid, dim3(NT), 0, s, j0, j1);
  if (t1) return launch(name, gemm6_dual<true, false>, grid, dim3(NT), 0, s, j0, j1);
  return launch(name, gemm6_dual<true, true>, grid, dim3(NT), 0, s, j0, j1);
}

}  // namespace kq
